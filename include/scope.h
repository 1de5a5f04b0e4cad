/*
 * scope.h -- C ABI of the SCOPE sparse self-attention layer for video DiTs,
 * for AMD Instinct MI355X (gfx950).
 *
 * The layer (one attention head at a fixed layer and denoising step; heads
 * are independent and batched) takes post-3D-RoPE queries and keys Q, K and
 * values V, each N x d, and computes
 *   1. a k-means clustering of the queries in the full d-dim space   (Sec. 3.2, Eq. 2)
 *   2. a k-means clustering of each RoPE key subspace T, H, W and the
 *      composite code of every key                                   (Sec. 3.3, Eq. 3-4)
 *   3. score tables P_m = Qbar^m (U^m)^T and lookup-and-sum proxy
 *      logits for every (query cluster, key)                         (Eq. 5-6, Alg. 2)
 *   4. hybrid Top-p / fixed Top-k counts, the online per-head Top-k
 *      and each cluster's final key set                              (Eq. 7-10, Alg. 3)
 *   5. exact attention of each query cluster over its key set        (Eq. 11, Alg. 1)
 * Calls 1-5 below map one-to-one onto these stages.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller.  Scalars
 *    and the shape/size structs are host values.  The library allocates and
 *    frees nothing.  Its only global state belongs to the no-allocation
 *    attention call (5n): a fixed device array per GPU and a host table of
 *    their addresses.
 *  - Every call is asynchronous: it validates its arguments on the host,
 *    enqueues its kernels on `stream` (a hipStream_t; NULL = the default
 *    stream) and returns.  No call synchronises or copies to the host.
 *  - Layout: Q, K, V, O are [heads][n][d], d contiguous, in the dtype of the
 *    shape (fp32 or bf16).  All other arrays are dense, row-major, with the
 *    shapes given per argument, heads outermost.
 *  - Workspace: calls that need scratch take `workspace` (256-byte aligned)
 *    of at least scope_workspace_size() bytes.  One workspace serves every
 *    call, but two calls that may run concurrently need two workspaces.
 *  - Errors: argument checks run before any GPU work and return
 *    SCOPE_ERR_INVALID_ARGUMENT (bad value), SCOPE_ERR_UNSUPPORTED (valid but
 *    outside what the kernels implement) or SCOPE_ERR_WORKSPACE; nothing is
 *    enqueued then.  A failed kernel launch returns SCOPE_ERR_HIP.  Faults
 *    that depend on data are OR-ed into the optional device word
 *    `dev_status` (bit 0: non-finite input; bit 1: |x| >= 2^e with
 *    e = min(22, 39 - ceil(log2 n)), outside the range in which the int64
 *    fixed-point sums of the k-means means are exact (2^22 for n <= 2^17,
 *    2^15 at n = 2^24), also set for non-finite input; bit 2: an initial
 *    row index out of range, replaced by the default row).  The inputs are
 *    checked in the first update pass of calls 1 and 2.  Nothing aborts or
 *    prints.
 *  - Determinism: every output is bitwise reproducible run to run and
 *    independent of launch geometry; calls 1-4 are bit-exact with respect to
 *    the canonical arithmetic defined under each call.
 */
#ifndef SCOPE_H
#define SCOPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SCOPE_ABI_VERSION 2

typedef enum {
  SCOPE_OK = 0,
  SCOPE_ERR_INVALID_ARGUMENT = 1,
  SCOPE_ERR_UNSUPPORTED = 2,
  SCOPE_ERR_WORKSPACE = 3,
  SCOPE_ERR_HIP = 4,
  SCOPE_ERR_SCRATCH_LIMIT = 5 /* beyond the no-allocation entry point's list */
} scope_status;

typedef enum { SCOPE_F32 = 0, SCOPE_BF16 = 1 } scope_dtype;

/* Selection policies (call 4b): the online per-head Top-k of Eq. 9-10, and
 * the two variants it is compared with in Fig. 6. */
typedef enum {
  SCOPE_POLICY_ONLINE = 0, /* r_c = max(b_c, k_head)              (Eq. 10) */
  SCOPE_POLICY_FIXED = 1,  /* r_c = b_c = max(t_c, k_fix), no top-up      */
  SCOPE_POLICY_TOPP = 2    /* r_c = t_c, pure Top-p                       */
} scope_policy;

/* Problem shape.  The three RoPE channel ranges I_T, I_H, I_W (Sec. 3.3;
 * App. A: disjoint, covering all d channels) are given as (offset, length)
 * in T, H, W order.  Supported: 1 <= heads <= 65535, 1 <= n <= 2^24, 2 <= d <= 128
 * for clustering/scoring/selection, d in {64, 128} for attention.         */
typedef struct {
  int32_t heads;
  int32_t n;
  int32_t d;
  int32_t dtype; /* scope_dtype of Q, K, V and O */
  int32_t range_off[3];
  int32_t range_len[3];
} scope_shape;

/* A general key partition (App. B; the partition ablation of Table 3): the
 * d channels split into M disjoint sets I_1 .. I_M that together cover all
 * of them, subspace m clustered into c[m] centroids.  `channels` lists I_1,
 * then I_2, ... (len[0] + ... + len[M-1] = d entries), each set in strictly
 * ascending channel order; entries past d are ignored.  The three RoPE
 * ranges in T, H, W order give exactly the results of calls 2-4.
 * Supported: 1 <= M <= 8, 1 <= c[m] <= min(n, 1024), c[0] + ... + c[M-1]
 * <= 3072 (one table row of a cluster is staged on chip during selection). */
#define SCOPE_MAX_SUBSPACES 8
#define SCOPE_MAX_D 128
typedef struct {
  int32_t m;
  int32_t c[SCOPE_MAX_SUBSPACES];
  int32_t len[SCOPE_MAX_SUBSPACES];
  int32_t channels[SCOPE_MAX_D];
} scope_partition;

int32_t scope_abi_version(void);
const char *scope_status_string(int32_t status);

/* Workspace bytes that suffice for every call below with these sizes.     */
int32_t scope_workspace_size(const scope_shape *shape, int32_t c_q,
                             const int32_t c_m[3], size_t *bytes);

/* 1. Query clustering (Sec. 3.2, Eq. 2; Alg. 1 first step).
 * Lloyd k-means of each head's n query rows into c_q clusters, `iters`
 * iterations of (assign, update), starting from rows init_idx[h][0..c_q)
 * (distinct rows in [0, n); NULL selects row floor((2r+1) n / (2 c_q))).
 * Canonical arithmetic: assign = argmin_r fl(||u_r||^2 - 2<x,u_r>) with
 * every dot product an fp32 fma chain in ascending channel order and ties
 * to the lowest r; update = exact int64 sums of rint(x * 2^24) over the
 * members, one fp64 division by count * 2^24, rounded to fp32; an empty
 * cluster keeps its centroid.  The iteration ends on an update, so each
 * returned centroid is the mean of its returned members (Eq. 2).
 * Outputs: q_centroids [heads][c_q][d] fp32; assign g [heads][n];
 * counts n_c [heads][c_q]; offsets [heads][c_q+1] (exclusive prefix sum of
 * counts); perm [heads][n] = the members of each cluster in ascending token
 * order, cluster after cluster (the query permutation of Alg. 1).
 * Requires 1 <= c_q <= min(n, 1024), 1 <= iters.                           */
int32_t scope_cluster_queries(const scope_shape *shape, const void *q,
                              int32_t c_q, int32_t iters,
                              const int32_t *init_idx, float *q_centroids,
                              int32_t *assign, int32_t *counts,
                              int32_t *offsets, int32_t *perm,
                              void *workspace, size_t ws_bytes,
                              int32_t *dev_status, void *stream);

/* 2. Key subspace clustering (Sec. 3.3, Eq. 3-4; Alg. 2 k-means step).
 * For m = T, H, W: k-means of K[:, I_m] into c_m[m] centroids with the same
 * canonical arithmetic as call 1, from rows init_idx[h][m][0..c_m[m])
 * (row stride init_stride >= max c_m; NULL = default rows), `iters`
 * iterations followed by one more assignment, so every code is the exact
 * argmin against the returned codebook (Eq. 3).
 * Outputs: k_centroids [heads][sum_m c_m*len_m] fp32, per head U^T, U^H,
 * U^W back to back, each [c_m][len_m]; codes [heads][n] composite code
 * z_T | z_H << 10 | z_W << 20 (Eq. 4).  Requires 1 <= c_m <= min(n, 1024). */
int32_t scope_cluster_key_subspaces(const scope_shape *shape, const void *k,
                                    const int32_t c_m[3], int32_t iters,
                                    const int32_t *init_idx,
                                    int32_t init_stride, float *k_centroids,
                                    uint32_t *codes, void *workspace,
                                    size_t ws_bytes, int32_t *dev_status,
                                    void *stream);

/* 1w, 2w. Warm starts across denoising steps (Sec. 4 setup: SCOPE runs at
 * every step after a dense prefix, and the query and key distributions of
 * one head change little from step to step).  As calls 1 and 2, but Lloyd's
 * iterations start from the centroids already in q_centroids (call 1w) or
 * k_centroids (call 2w), e.g. the previous step's results, instead of the
 * rows init_idx; those buffers are read, then overwritten with the result.
 * Arguments, layouts, outputs and errors otherwise as calls 1 and 2 (no
 * init_idx; the starting centroids must be finite).  With the centroids a
 * call returned, iters more iterations from them give exactly what a
 * single call with the total iteration count gives.                      */
int32_t scope_cluster_queries_warm(const scope_shape *shape, const void *q,
                                   int32_t c_q, int32_t iters,
                                   float *q_centroids, int32_t *assign,
                                   int32_t *counts, int32_t *offsets,
                                   int32_t *perm, void *workspace,
                                   size_t ws_bytes, int32_t *dev_status,
                                   void *stream);
int32_t scope_cluster_key_subspaces_warm(const scope_shape *shape,
                                         const void *k, const int32_t c_m[3],
                                         int32_t iters, float *k_centroids,
                                         uint32_t *codes, void *workspace,
                                         size_t ws_bytes, int32_t *dev_status,
                                         void *stream);

/* 3. Score tables and proxy logits (Eq. 5-6; Alg. 2 scoring steps).
 * tables [heads][c_q][C_T+C_H+C_W]: P_m[c][r] = <qbar_c[I_m], u_r^m> as an
 * fp32 fma chain over the subspace channels in ascending order, columns
 * T then H then W.  If `scores` is not NULL it receives the proxy logits
 * [heads][c_q][n]: s_cj = fl(fl(fl(P_T[c][zT] + P_H[c][zH]) + P_W[c][zW])
 * * fl32(1/sqrt(d))) + 0.0 (the + 0 maps -0 to +0).  scope_select computes
 * the same logits on the fly, so `scores` is only needed for inspection.   */
int32_t scope_proxy_scores(const scope_shape *shape, const float *q_centroids,
                           int32_t c_q, const float *k_centroids,
                           const int32_t c_m[3], const uint32_t *codes,
                           float *tables, float *scores, void *stream);

/* 4. Key selection (Eq. 7-10; Alg. 3).
 * Logits come from `scores` if not NULL, else from (tables, codes) exactly
 * as in call 3.  For each cluster c, with pi_c = keys by logit descending,
 * ties by ascending key index:
 *   t_c   = the shortest prefix of pi_c whose softmax mass reaches rho
 *           (Eq. 7), rho >= 1 keeps all n; the softmax mass of key j is
 *           E_j = fixexp(s_cj - max_j s_cj), an integer in units of 2^-32
 *           (z = y*fl32(log2 e); 0 below z = -40; 2^frac(z) by a degree-7
 *           Taylor polynomial in fp32), and the prefix must reach
 *           ceil(rho * sum_j E_j) computed exactly;
 *   b_c   = max(t_c, k_fix)                                         (Eq. 8)
 *   k_head= ceil(sum_c n_c b_c / sum_c n_c), exact integers         (Eq. 9)
 *   r_c   = max(b_c, k_head), S_c = the first r_c keys of pi_c      (Eq. 10)
 * Outputs: base_counts b [heads][c_q]; topp_counts t [heads][c_q] (may be
 * NULL); k_head [heads]; sel_counts r [heads][c_q]; sel_idx
 * [heads][c_q][n]: S_c in ascending key order in the first r_c entries
 * (the rest are left untouched).  counts are the n_c of call 1.
 * Requires 0 < rho <= 1 (finite) and 1 <= k_fix <= n.                      */
int32_t scope_select(const scope_shape *shape, int32_t c_q,
                     const int32_t c_m[3], const float *scores,
                     const float *tables, const uint32_t *codes,
                     const int32_t *counts, float rho, int32_t k_fix,
                     int32_t *base_counts, int32_t *topp_counts,
                     int32_t *k_head, int32_t *sel_counts, int32_t *sel_idx,
                     void *workspace, size_t ws_bytes, void *stream);

/* 4b. Selection under a named policy (the ablation of Fig. 6).  Arguments,
 * layouts, outputs and errors as call 4, plus `policy` (a scope_policy):
 * ONLINE is call 4; FIXED keeps b_c keys per cluster (Eq. 8) and TOPP the
 * t_c keys of Eq. 7, with no top-up to k_head.  k_head (Eq. 9) is written
 * for every policy.  An unknown policy is SCOPE_ERR_INVALID_ARGUMENT.     */
int32_t scope_select_policy(const scope_shape *shape, int32_t c_q,
                            const int32_t c_m[3], const float *scores,
                            const float *tables, const uint32_t *codes,
                            const int32_t *counts, float rho, int32_t k_fix,
                            int32_t *base_counts, int32_t *topp_counts,
                            int32_t *k_head, int32_t *sel_counts,
                            int32_t *sel_idx, void *workspace, size_t ws_bytes,
                            int32_t policy, void *stream);

/* 2p-4p. Calls 2-4 for a general key partition (App. B; Table 3).  The
 * shape's range fields are ignored (checked only by calls 2-4); `part`
 * (host memory) gives the sets and codebook sizes.  Errors as calls 2-4, and
 * SCOPE_ERR_INVALID_ARGUMENT for sets that are not a partition of the d
 * channels or not ascending, SCOPE_ERR_UNSUPPORTED beyond the limits above.
 *
 * Workspace bytes that suffice for the three partition calls and for calls 1
 * and 5 with these sizes.  When the sets are not the contiguous ranges
 * [0, len[0]), [len[0], len[0] + len[1]), ... this includes a channel-
 * reordered copy of K (heads * n * d elements).                            */
int32_t scope_partition_workspace_size(const scope_shape *shape, int32_t c_q,
                                       const scope_partition *part,
                                       size_t *bytes);

/* Key subspace clustering over the sets of `part`: for each m, k-means of
 * K[:, I_m] (the channels of I_m in ascending order) into c[m] centroids,
 * exactly as call 2 (same arithmetic, iterations plus one last assignment).
 * init_idx[(h * M + m) * init_stride + r] are the starting rows (NULL =
 * default rows), init_stride >= max c[m].
 * Outputs: k_centroids [heads][sum_m c[m] * len[m]] fp32, per head U^1 ..
 * U^M back to back, each [c[m]][len[m]] with column k on channel I_m[k];
 * codes [heads][M][n] uint16, z^m of key j at codes[(h * M + m) * n + j].  */
int32_t scope_cluster_key_partition(const scope_shape *shape, const void *k,
                                    const scope_partition *part, int32_t iters,
                                    const int32_t *init_idx,
                                    int32_t init_stride, float *k_centroids,
                                    uint16_t *codes, void *workspace,
                                    size_t ws_bytes, int32_t *dev_status,
                                    void *stream);

/* Tables and proxy logits over the sets of `part` (Eq. 5-6): tables
 * [heads][c_q][c[0] + ... + c[M-1]], P_m[c][r] = <qbar_c[I_m], u_r^m> as an
 * fp32 fma chain over I_m in ascending channel order; if `scores` is not
 * NULL, s_cj = fl(fl(...fl(P_1[z^1] + P_2[z^2]) ... + P_M[z^M]) *
 * fl32(1/sqrt(d))) + 0.0, summed left to right (M = 1: no addition).
 * Uses the workspace when the sets are not contiguous ranges in order.    */
int32_t scope_proxy_scores_partition(const scope_shape *shape,
                                     const float *q_centroids, int32_t c_q,
                                     const float *k_centroids,
                                     const scope_partition *part,
                                     const uint16_t *codes, float *tables,
                                     float *scores, void *workspace,
                                     size_t ws_bytes, void *stream);

/* Selection (call 4b) with the logits of `part`: from `scores` if not
 * NULL, else from (tables, codes) exactly as scope_proxy_scores_partition
 * computes them.  Arguments, outputs and errors otherwise as call 4b.      */
int32_t scope_select_partition(const scope_shape *shape, int32_t c_q,
                               const scope_partition *part,
                               const float *scores, const float *tables,
                               const uint16_t *codes, const int32_t *counts,
                               float rho, int32_t k_fix, int32_t *base_counts,
                               int32_t *topp_counts, int32_t *k_head,
                               int32_t *sel_counts, int32_t *sel_idx,
                               void *workspace, size_t ws_bytes, int32_t policy,
                               void *stream);

/* 5. Sparse attention over the selected keys (Eq. 11; Alg. 1 last step).
 * For every cluster c and every query i in perm[offsets[c] .. offsets[c+1]):
 *   O[i] = softmax(q_i K[S_c]^T * scale) V[S_c],  S_c = sel_idx[c][0..r_c),
 * with the original Q, K, V rows (scale <= 0 selects 1/sqrt(d)).  Products
 * run on bf16 matrix cores with fp32 accumulation and an fp32 online
 * softmax; fp32 inputs are rounded to bf16 on load; O is written in the
 * input dtype, in original token order.  A cluster with r_c = 0 writes 0.
 * Dense attention (Eq. 1) is the special case of one cluster holding all
 * queries (c_q = 1, offsets = {0, n}, perm = identity) and all keys.
 * Bad indices cannot fault: index arrays are clamped to their valid
 * ranges on the device, or read through range-checked loads that return
 * 0 (the selected-key gather of bf16 inputs).  Requires d in {64, 128},
 * 16-byte aligned q, k, v, o, and for bf16 inputs n * d * 2 < 2^32
 * (n < 2^24 at d = 128), else SCOPE_ERR_UNSUPPORTED.                     */
int32_t scope_sparse_attention(const scope_shape *shape, const void *q,
                               const void *k, const void *v, int32_t c_q,
                               const int32_t *offsets, const int32_t *perm,
                               const int32_t *sel_counts,
                               const int32_t *sel_idx, float scale, void *o,
                               void *workspace, size_t ws_bytes, void *stream);

/* 5n. Sparse attention without allocation or workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * and harnesses that forbid it).  Arguments, outputs, layout and errors as
 * call 5 without `workspace`/`ws_bytes`: the call's work list (heads *
 * (ceil(n / 256) + c_q) slots of two 16-byte entries) lives in a fixed
 * device array of SCOPE_NOALLOC_MAX_WORK_ITEMS entries (1 MiB), one per GPU, held until
 * the process ends; larger problems return SCOPE_ERR_SCRATCH_LIMIT before
 * anything is enqueued.  The array's device address is looked up on the
 * first call on each device (the current device).  No call allocates or
 * frees memory.  Every call on a GPU shares that GPU's array and rewrites
 * the entries it reads, so calls that overlap on one GPU (two streams, or
 * two host threads) race; serialise them.                                 */
#define SCOPE_NOALLOC_MAX_WORK_ITEMS 65536
int32_t scope_sparse_attention_noalloc(const scope_shape *shape,
                                       const void *q, const void *k,
                                       const void *v, int32_t c_q,
                                       const int32_t *offsets,
                                       const int32_t *perm,
                                       const int32_t *sel_counts,
                                       const int32_t *sel_idx, float scale,
                                       void *o, void *stream);

/* Diagnostics: the measured peaks that roofline fractions are also quoted
 * against.  scope_debug_copy copies `bytes` (a multiple of 16; src and dst
 * 16-byte aligned, not overlapping) with a plain vector copy kernel, so its
 * time gives the achievable HBM bandwidth (2 * bytes moved).
 * scope_debug_mfma_loop launches `blocks` blocks of 256 threads whose waves
 * each issue iters * 8 independent bf16 32x32x16 matrix products from
 * registers (8 * 32768 * iters flops per wave) and write one float per
 * thread to out[blocks * 256]: the achievable bf16 MFMA rate.              */
int32_t scope_debug_copy(const void *src, void *dst, size_t bytes, void *stream);
int32_t scope_debug_mfma_loop(float *out, int32_t blocks, int32_t iters,
                              void *stream);

/* Diagnostic: the selection's fixed-point exponential (call 4) applied to
 * y[0..count) (y <= 0), results in out[0..count).                          */
int32_t scope_debug_fixexp(const float *y, uint64_t *out, int64_t count,
                           void *stream);

/* Diagnostic: the work list of call 5 for `heads` heads, as the sparse
 * attention builds it.  offsets [heads][c_q + 1] and sel_counts
 * [heads][c_q] (device) are as for scope_sparse_attention.  *items_per_head
 * (host) receives S, the slots per head; items (device, 16-byte aligned,
 * `capacity` int32 values, at least heads * S * 8) receives
 * [heads][S][2][4] int32: each slot holds two entries (cluster, first row,
 * rows, selected keys) run by one block, the second with rows = 0 when the
 * block runs one chunk, and slots with both entries empty after the used
 * ones.  pair != 0 lets two remainder chunks share a slot, as the bf16,
 * d = 128 kernel does.  Returns SCOPE_ERR_INVALID_ARGUMENT on bad sizes or
 * pointers, before any launch.                                              */
int32_t scope_debug_attention_items(int32_t heads, int32_t n, int32_t c_q,
                                    int32_t pair, const int32_t *offsets,
                                    const int32_t *sel_counts, int32_t *items,
                                    int64_t capacity, int32_t *items_per_head,
                                    void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SCOPE_H */
