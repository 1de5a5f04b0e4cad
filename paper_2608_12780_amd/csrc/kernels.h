// Host-side launchers of the SCOPE kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/scope.h"

namespace scope {

// One batch of k-means problems, one problem per head: the rows of
// X[h] (row stride ld elements, channels col0 .. col0+dx) clustered into C
// centroids U[h] ([C][dx] fp32).
struct KmProblem {
  const void *x;          // element type given by bf16 flag
  bool bf16;
  size_t x_head_stride;   // elements between heads
  int ld, col0, dx, n, C;
  float *u;               // centroids of head 0 (this subspace)
  size_t u_head_stride;   // floats between heads
  int32_t *assign;        // [heads][n] (a_head_stride apart)
  size_t a_head_stride;
  int32_t *counts;        // [heads][C]
  int32_t *offsets;       // [heads][C+1]
  int32_t *perm;          // [heads][n]
  int32_t *chunk_hist;    // [heads][nchunks][C]
  int32_t *chunk_rel;     // [heads][nchunks][C]
  int heads;
  // matrix-core assignment (bf16 inputs): bf16 copy of the centroids,
  // their squared norms and the error-bound constants, refreshed per pass
  bool mfma;
  int cpad, dxp;          // centroids padded to 32, channels padded to 16
  uint16_t *ubf;          // [heads][cpad][2 * dxp]: bf16 hi then lo terms
  float *nu;              // [heads][cpad]
  float *bnd;             // [heads][cpad][2]: per-row bound parts
  // codebooks beyond the LDS: per chunk and point the four smallest packed
  // scores ([parts][heads][n][4]) and the point's norm bound ([heads][n])
  float *part, *pnx;
};

// Whether the matrix-core assignment applies: bf16 rows at even offsets and
// at most 1024 centroids (codebooks beyond the LDS are streamed in chunks).
bool km_mfma_ok(bool bf16, int ld, int col0, int dx, int C);
int km_parts(int C, int dx);
// floats of KmProblem::part and ::pnx together (0 when the codebook fits)
size_t km_split_floats(int C, int dx, int heads, int n);
int km_cpad(int C);
int km_dxp(int dx);

constexpr int kAssignBlock = 256;  // points per assign block == grouping chunk

inline int km_nchunks(int n) { return (n + kAssignBlock - 1) / kAssignBlock; }

hipError_t km_init(const KmProblem &p, const int32_t *init, int init_stride,
                   int32_t *status, hipStream_t s);
hipError_t km_assign(const KmProblem &p, bool with_hist, hipStream_t s);
hipError_t km_group(const KmProblem &p, hipStream_t s);
// The three key subspaces' assignments in one pass over the rows (matrix
// cores; codebooks side by side in LDS): applies when km_assign3_ok.
bool km_assign3_ok(const KmProblem (&p)[3]);
// scratch: km_assign3_scratch_bytes() of device memory (its arguments)
size_t km_assign3_scratch_bytes();
// store_args: write the launch arguments to the scratch (once per call; the
// later passes of the call reuse them)
hipError_t km_assign3(const KmProblem (&p)[3], void *scratch, bool store_args,
                      hipStream_t s);

// Centroid update by one streaming pass over the rows.  Up to kMaxSub
// subspaces of the same rows (channels col0[m] .. col0[m]+dx[m], C[m]
// clusters, centroids [C[m]][dx[m]] at float offset ucol[m] of a head) are
// updated together; their channels are cut into windows whose int64 sums
// fit one block's LDS.
constexpr int kAccLds = 19200;           // int64 sums per block (150 KB of LDS)
constexpr int kAccCnt = 1024;            // int32 cluster counts per block
constexpr int kAccMaxPieces = 4;
constexpr int kAccMaxWindows = 16;
constexpr int kMaxSub = 8;               // subspaces of a key partition
constexpr int kAccTargetBlocks = 256;    // blocks per launch, about one per CU
struct AccPiece {
  int m, sub0, width;   // channels sub0 .. sub0+width of subspace m
  int lds;              // first int64 LDS sum of the piece ([C][width])
  int cnt;              // first LDS count of subspace m, or -1 if not counted here
};
struct AccWindow {
  int npieces, lanes, elems, cnt_elems;
  AccPiece piece[kAccMaxPieces];
};
struct AccPlan {
  int nsub;
  int C[kMaxSub], dx[kMaxSub], col0[kMaxSub], ucol[kMaxSub], ccol[kMaxSub];
  int S, SC;            // centroid elements and clusters of one head
  int nwin, blocks;     // windows; blocks per (head, window)
  AccWindow win[kAccMaxWindows];
};
bool km_accum_plan(int nsub, const int *col0, const int *dx, const int *C,
                   int heads, int n, AccPlan *plan);
size_t km_accum_slab_bytes(const AccPlan &p, int heads);
size_t km_accum_cslab_bytes(const AccPlan &p, int heads);
// assign of subspace m, head h at assign[h * a_hs + m * a_ss]; with a
// status word, the visited inputs are also checked for |x| >= 2^22 and
// non-finite values.
hipError_t km_accum(const AccPlan &plan, const void *x, bool bf16, size_t x_hs,
                    int ld, int n, int heads, const int32_t *assign,
                    size_t a_hs, size_t a_ss, long long *slab, int32_t *cslab,
                    float *U, size_t u_hs, int32_t *status, hipStream_t s);
hipError_t km_pack_codes(const int32_t *a3, size_t a_head_stride,
                         size_t a_sub_stride, int n, int heads,
                         uint32_t *codes, hipStream_t s);
// Per-subspace codes of a general partition: z[h][m][j] = assign as uint16.
hipError_t km_codes16(const int32_t *assign, size_t count, uint16_t *codes,
                      hipStream_t s);
// dst[r][t] = src[r][chan[t]] for rows r < rows (each of d elements of
// elem_bytes = 2 or 4 bytes): the channels of a partition's sets, in order.
struct ChannelMap {
  int chan[128];
};
hipError_t gather_channels(const void *src, void *dst, size_t rows, int d,
                           int elem_bytes, const ChannelMap &map, hipStream_t s);

// Codebooks of the key subspaces: M sets, sizes c[0..M).  The logits read
// codes packed as zT | zH << 10 | zW << 20 (M = 3, codes32) or one uint16
// plane per subspace, [heads][M][n] (codes16).
struct Subspaces {
  int M;
  int c[kMaxSub];
};

// Tables over the M channel ranges (off[m], len[m]) of the query centroids
// (row stride d), one per subspace.
hipError_t score_tables(int heads, int d, const int *off, const int *len,
                        int c_q, const Subspaces &sub, const float *qc,
                        const float *kc, float *tables, hipStream_t s);
hipError_t score_logits(int heads, int n, int d, int c_q, const Subspaces &sub,
                        const float *tables, const uint32_t *codes32,
                        const uint16_t *codes16, float *scores, hipStream_t s);

constexpr int kSelMaxTable = 3072;    // LUT floats of one cluster row in LDS
hipError_t select_run(int heads, int n, int c_q, const Subspaces &sub, int d,
                      const float *scores, const float *tables,
                      const uint32_t *codes32, const uint16_t *codes16,
                      const int32_t *counts, float rho,
                      int k_fix, int32_t *base, int32_t *topp, int32_t *k_head,
                      int32_t *sel_counts, int32_t *sel_idx, float *row_max,
                      uint32_t *row_state, uint32_t *coarse_hist, uint32_t *dedup,
                      int policy, hipStream_t s);
// 32-bit words of the distinct-code scratch of select_run
size_t select_dedup_words(int heads, int n);
constexpr int kSelCoarseBins = 2048;  // coarse histogram bins per cluster row
// Measured-peak microbenchmarks (diagnostics).
hipError_t peak_copy(const void *src, void *dst, size_t bytes, hipStream_t s);
hipError_t peak_mfma(float *out, int blocks, int iters, hipStream_t s);

hipError_t debug_fixexp(const float *y, uint64_t *out, int64_t count,
                        hipStream_t s);

int attn_items_per_head(int n, int c_q);
// 16-byte work-list entries of the no-allocation attention entry point
// (1 MiB; two per work slot).
constexpr size_t kAttnScratchItems = SCOPE_NOALLOC_MAX_WORK_ITEMS;
// Device address of that work list on the current device (looked up once
// per device).
hipError_t attention_scratch(int4 **items);
// The work list alone (as attention_run builds it), for diagnostics.
hipError_t attention_items(int heads, int n, int c_q, bool pair, const int32_t *offsets,
                           const int32_t *sel_counts, int4 *items, hipStream_t s);
hipError_t attention_run(int heads, int n, int d, bool bf16, const void *q,
                         const void *k, const void *v, void *o, int c_q,
                         const int32_t *offsets, const int32_t *perm,
                         const int32_t *sel_counts, const int32_t *sel_idx,
                         float scale, int4 *items, hipStream_t s);

}  // namespace scope
