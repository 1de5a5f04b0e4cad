/*
 * SCOPE attention layer -- CPU ORACLE.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously-correct
 * reference that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no source, header, table or helper with the GPU library: every constant and
 * every step below is written here from the method's definition.
 *
 * What it computes, per attention head (Sec. 3, Alg. 1-3):
 *   1. query k-means over full d-dim post-RoPE queries          (Sec. 3.2, Eq. 2)
 *   2. k-means of each RoPE key subspace T/H/W, composite code  (Sec. 3.3, Eq. 3-4)
 *   3. score tables P_m = Qbar^m (U^m)^T                         (Eq. 5)
 *   4. lookup-and-sum proxy logits                               (Eq. 6, Alg. 2)
 *   5. softmax + Top-p count, fixed floor, online per-head k,
 *      top-up and final key sets                                 (Eq. 7-10, Alg. 3)
 *   6. exact attention of each query cluster over its key set    (Eq. 11; Eq. 1)
 *   7. general M-way key partitions (any disjoint channel sets,
 *      M <= 8) for the partition ablation                       (App. B; Table 3)
 *
 * Arithmetic.  The method is stated over the reals.  Steps 1-5 decide
 * integers (assignments, counts, index sets), so both this oracle and the GPU
 * library fix one canonical finite-precision evaluation and must agree on it
 * bit for bit:
 *   - every dot product: fp32, ascending channel order, one fmaf per channel;
 *   - k-means distance: ||u||^2 - 2<x,u>, argmin ties -> lowest centroid;
 *   - k-means means: exact int64 sums of rint(x * 2^24), one fp64 divide,
 *     one rounding to fp32; an empty cluster keeps its previous centroid;
 *   - proxy logit: ((P_T + P_H) + P_W) * fl32(1/sqrt(d)), then + 0.0f;
 *   - softmax mass: a self-defined exp2-based fixed-point exponential
 *     (fixexp below) in uint64 units of 2^-32, exact integer sums, and the
 *     Top-p target ceil(rho * total) evaluated exactly in integers;
 *   - ranking pi_c: logit descending, key index ascending on ties.
 * Step 6 is the plain definition of attention evaluated in fp64.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fopenmp -mfma -shared -fPIC.
 * No fast-math: rounding must be IEEE round-to-nearest-even throughout.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_OK 0
#define OR_ERR_ARG 1
#define OR_ERR_RANGE 2
#define OR_ERR_MEM 3

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Canonical dot product: fp32, sequential in ascending channel order.       */
static float cdot(const float *a, const float *b, int len) {
  float acc = 0.0f;
  for (int c = 0; c < len; ++c) acc = fmaf(a[c], b[c], acc);
  return acc;
}

/* ------------------------------------------------------------------------ */
/* K-means (Lloyd), Sec. 3.2 (queries, squared-L2 as for keys) and Eq. 3.
 * X: n rows, row stride ldx floats, dx channels.  U: C x dx centroids.
 * Starting centroids are the rows init[0..C).  Each iteration assigns every
 * row to its nearest centroid and then replaces each non-empty centroid by
 * the mean of its members (Eq. 2).  With final_assign, one more assignment
 * follows the last update, so the returned labels are exact argmins w.r.t.
 * the returned centroids (Eq. 3); without it, the returned centroids are
 * exact means of the returned clusters (Eq. 2).                            */

static void km_assign(const float *X, long ldx, int n, int dx, const float *U,
                      int C, int *a) {
  float *nu = (float *)malloc(sizeof(float) * (size_t)C);
  for (int r = 0; r < C; ++r) nu[r] = cdot(U + (size_t)r * dx, U + (size_t)r * dx, dx);
#pragma omp parallel for schedule(static)
  for (int i = 0; i < n; ++i) {
    const float *x = X + (size_t)i * ldx;
    float best = INFINITY;
    int arg = 0;
    for (int r = 0; r < C; ++r) {
      float s = fmaf(-2.0f, cdot(x, U + (size_t)r * dx, dx), nu[r]);
      if (s < best) { best = s; arg = r; } /* strict: lowest index wins ties */
    }
    a[i] = arg;
  }
  free(nu);
}

/* Largest magnitude the fixed-point sums of n rows hold exactly: every
 * |rint(x 2^24)| is below 2^(e+24) for |x| < 2^e, and n <= 2^L such terms sum
 * below 2^63 when e <= 39 - L; e is capped at 22 (2^22 for n <= 2^17).    */
static float range_limit(int n) {
  int L = 0;
  while (L < 31 && (1L << L) < n) ++L;
  return ldexpf(1.0f, 39 - L < 22 ? 39 - L : 22);
}

/* rint(x * 2^24) as a two's complement 64-bit pattern.  Within the range
 * the value is exact; outside it (flagged by the caller) a finite value
 * still gives a defined pattern and a non-finite one gives 0.             */
static uint64_t fixed24(float x) {
  const double t = rint((double)x * 16777216.0);
  if (!(fabs(t) < 9.0e18)) return 0;
  return (uint64_t)(int64_t)t;
}

/* returns OR_ERR_RANGE if some |x| >= range_limit(n) or is not finite.  The
 * sums wrap modulo 2^64 (unsigned), so out-of-range input yields some
 * value, never undefined arithmetic; within the range no sum wraps.     */
static int km_update(const float *X, long ldx, int n, int dx, const int *a,
                     int C, float *U, int *cnt) {
  uint64_t *S = (uint64_t *)calloc((size_t)C * dx, sizeof(uint64_t));
  if (!S) return OR_ERR_MEM;
  int status = OR_OK;
  const float lim = range_limit(n);
  for (int r = 0; r < C; ++r) cnt[r] = 0;
  for (int i = 0; i < n; ++i) {
    const float *x = X + (size_t)i * ldx;
    int r = a[i];
    cnt[r] += 1;
    for (int c = 0; c < dx; ++c) {
      if (!(fabsf(x[c]) < lim)) status = OR_ERR_RANGE;
      S[(size_t)r * dx + c] += fixed24(x[c]);
    }
  }
  for (int r = 0; r < C; ++r) {
    if (cnt[r] == 0) continue; /* empty cluster: keep previous centroid */
    double den = (double)cnt[r] * 16777216.0;
    for (int c = 0; c < dx; ++c)
      U[(size_t)r * dx + c] = (float)((double)(int64_t)S[(size_t)r * dx + c] / den);
  }
  free(S);
  return status;
}

/* Lloyd's iterations from the centroids in U (in/out). */
int oracle_kmeans_from(const float *X, long ldx, int n, int dx, int C, int iters,
                       int final_assign, float *U, int *assign, int *counts) {
  if (n < 1 || dx < 1 || C < 1 || C > n || iters < 0) return OR_ERR_ARG;
  int status = OR_OK;
  for (int r = 0; r < C; ++r) counts[r] = 0;
  for (int it = 0; it < iters; ++it) {
    km_assign(X, ldx, n, dx, U, C, assign);
    int s = km_update(X, ldx, n, dx, assign, C, U, counts);
    if (s == OR_ERR_MEM) return s;
    if (s != OR_OK) status = s;
  }
  if (final_assign || iters == 0) {
    km_assign(X, ldx, n, dx, U, C, assign);
    for (int r = 0; r < C; ++r) counts[r] = 0;
    for (int i = 0; i < n; ++i) counts[assign[i]] += 1;
  }
  return status;
}

/* Lloyd's k-means from the rows init[0..C) of X. */
int oracle_kmeans(const float *X, long ldx, int n, int dx, int C, int iters,
                  const int *init, int final_assign, float *U, int *assign,
                  int *counts) {
  if (n < 1 || dx < 1 || C < 1 || C > n || iters < 0) return OR_ERR_ARG;
  for (int r = 0; r < C; ++r) {
    if (init[r] < 0 || init[r] >= n) return OR_ERR_ARG;
    memcpy(U + (size_t)r * dx, X + (size_t)init[r] * ldx, sizeof(float) * (size_t)dx);
  }
  return oracle_kmeans_from(X, ldx, n, dx, C, iters, final_assign, U, assign, counts);
}

/* Grouping of queries by cluster (the cluster-based query permutation of
 * Alg. 1's index sets Q_c): offsets = exclusive prefix sum of the sizes,
 * perm lists the members of each cluster in ascending token order.         */
int oracle_group(const int *assign, int n, int C, int *counts, int *offsets,
                 int *perm) {
  for (int r = 0; r < C; ++r) counts[r] = 0;
  for (int i = 0; i < n; ++i) {
    if (assign[i] < 0 || assign[i] >= C) return OR_ERR_ARG;
    counts[assign[i]] += 1;
  }
  offsets[0] = 0;
  for (int r = 0; r < C; ++r) offsets[r + 1] = offsets[r] + counts[r];
  int *fill = (int *)malloc(sizeof(int) * (size_t)C);
  memcpy(fill, offsets, sizeof(int) * (size_t)C);
  for (int i = 0; i < n; ++i) perm[fill[assign[i]]++] = i;
  free(fill);
  return OR_OK;
}

/* Alg. 1, first steps: (Qbar, g) <- KMeans(Q, C_q); Q_c, n_c.               */
/* init == NULL: warm start from the centroids already in `centroids` */
static int cluster_queries(int heads, int n, int d, const float *q, int c_q,
                           int iters, const int *init, float *centroids,
                           int *assign, int *counts, int *offsets, int *perm) {
  int status = OR_OK;
  for (int h = 0; h < heads; ++h) {
    float *U = centroids + (size_t)h * c_q * d;
    int s = init ? oracle_kmeans(q + (size_t)h * n * d, d, n, d, c_q, iters,
                                 init + (size_t)h * c_q, 0, U,
                                 assign + (size_t)h * n, counts + (size_t)h * c_q)
                 : oracle_kmeans_from(q + (size_t)h * n * d, d, n, d, c_q, iters, 0, U,
                                      assign + (size_t)h * n, counts + (size_t)h * c_q);
    if (s == OR_ERR_ARG || s == OR_ERR_MEM) return s;
    if (s != OR_OK) status = s;
    s = oracle_group(assign + (size_t)h * n, n, c_q, counts + (size_t)h * c_q,
                     offsets + (size_t)h * (c_q + 1), perm + (size_t)h * n);
    if (s != OR_OK) return s;
  }
  return status;
}

/* Alg. 2, k-means of each key subspace K^m = K[:, I_m] (Eq. 3), m = T, H, W,
 * and the composite code z_j = (z_j^T, z_j^H, z_j^W) of Eq. 4, packed as
 * zT | zH << 10 | zW << 20.  Centroids per head: U^T, U^H, U^W back to back,
 * each [C_m][d_m].  init: [heads][3][init_stride].                          */
int oracle_cluster_queries(int heads, int n, int d, const float *q, int c_q,
                           int iters, const int *init, float *centroids,
                           int *assign, int *counts, int *offsets, int *perm) {
  if (!init) return OR_ERR_ARG;
  return cluster_queries(heads, n, d, q, c_q, iters, init, centroids, assign, counts,
                         offsets, perm);
}

/* Query clustering from the centroids in `centroids` (in/out): a warm
 * start, e.g. from the previous denoising step's result. */
int oracle_cluster_queries_from(int heads, int n, int d, const float *q, int c_q,
                                int iters, float *centroids, int *assign, int *counts,
                                int *offsets, int *perm) {
  return cluster_queries(heads, n, d, q, c_q, iters, NULL, centroids, assign, counts,
                         offsets, perm);
}

/* init == NULL: warm start from the codebooks already in `centroids` */
static int cluster_key_subspaces(int heads, int n, int d, const int *off,
                                 const int *len, const float *k,
                                 const int *c_m, int iters, const int *init,
                                 int init_stride, float *centroids,
                                 uint32_t *codes, int *assign3) {
  int per_head = 0;
  for (int m = 0; m < 3; ++m) {
    if (c_m[m] < 1 || c_m[m] > 1024 || off[m] < 0 || len[m] < 1 || off[m] + len[m] > d)
      return OR_ERR_ARG;
    per_head += c_m[m] * len[m];
  }
  int status = OR_OK;
  int *cnt = (int *)malloc(sizeof(int) * 1024);
  for (int h = 0; h < heads; ++h) {
    float *U = centroids + (size_t)h * per_head;
    for (int m = 0; m < 3; ++m) {
      int *a = assign3 + ((size_t)h * 3 + m) * n;
      const float *X = k + (size_t)h * n * d + off[m];
      int s = init ? oracle_kmeans(X, d, n, len[m], c_m[m], iters,
                                   init + ((size_t)h * 3 + m) * init_stride, 1, U, a, cnt)
                   : oracle_kmeans_from(X, d, n, len[m], c_m[m], iters, 1, U, a, cnt);
      if (s == OR_ERR_ARG || s == OR_ERR_MEM) { free(cnt); return s; }
      if (s != OR_OK) status = s;
      U += (size_t)c_m[m] * len[m];
    }
    const int *aT = assign3 + ((size_t)h * 3 + 0) * n;
    const int *aH = assign3 + ((size_t)h * 3 + 1) * n;
    const int *aW = assign3 + ((size_t)h * 3 + 2) * n;
    for (int j = 0; j < n; ++j)
      codes[(size_t)h * n + j] = (uint32_t)aT[j] | ((uint32_t)aH[j] << 10) |
                                 ((uint32_t)aW[j] << 20);
  }
  free(cnt);
  return status;
}

int oracle_cluster_key_subspaces(int heads, int n, int d, const int *off,
                                 const int *len, const float *k,
                                 const int *c_m, int iters, const int *init,
                                 int init_stride, float *centroids,
                                 uint32_t *codes, int *assign3) {
  if (!init) return OR_ERR_ARG;
  return cluster_key_subspaces(heads, n, d, off, len, k, c_m, iters, init, init_stride,
                               centroids, codes, assign3);
}

/* Key subspace clustering from the codebooks in `centroids` (in/out). */
int oracle_cluster_key_subspaces_from(int heads, int n, int d, const int *off,
                                      const int *len, const float *k, const int *c_m,
                                      int iters, float *centroids, uint32_t *codes,
                                      int *assign3) {
  return cluster_key_subspaces(heads, n, d, off, len, k, c_m, iters, NULL, 0, centroids,
                               codes, assign3);
}

/* Eq. 5: P_m[c, r] = <qbar_c^m, u_r^m>, the query-centroid slice on I_m
 * against subspace centroid r.  Tables per head: [c_q][C_T + C_H + C_W].   */
int oracle_tables(int heads, int d, const int *off, const int *len, int c_q,
                  const int *c_m, const float *qc, const float *kc,
                  float *tables) {
  int cs = c_m[0] + c_m[1] + c_m[2];
  int per_head = c_m[0] * len[0] + c_m[1] * len[1] + c_m[2] * len[2];
  for (int h = 0; h < heads; ++h) {
    const float *Q = qc + (size_t)h * c_q * d;
    float *P = tables + (size_t)h * c_q * cs;
    const float *U = kc + (size_t)h * per_head;
    int col = 0;
    for (int m = 0; m < 3; ++m) {
      for (int c = 0; c < c_q; ++c)
        for (int r = 0; r < c_m[m]; ++r)
          P[(size_t)c * cs + col + r] =
              cdot(Q + (size_t)c * d + off[m], U + (size_t)r * len[m], len[m]);
      U += (size_t)c_m[m] * len[m];
      col += c_m[m];
    }
  }
  return OR_OK;
}

/* Eq. 6 / Alg. 2: s_cj = (1/sqrt d) * sum_m P_m[c, z_j^m], summed in T, H, W
 * order, then scaled; + 0.0f turns a -0 into +0.                            */
static inline float proxy_logit(const float *Prow, const int *c_m, uint32_t code,
                                float sigma) {
  uint32_t zT = code & 1023u, zH = (code >> 10) & 1023u, zW = (code >> 20) & 1023u;
  float s = Prow[zT] + Prow[c_m[0] + zH];
  s = s + Prow[c_m[0] + c_m[1] + zW];
  s = s * sigma;
  return s + 0.0f;
}

float oracle_sigma(int d) { return (float)(1.0 / sqrt((double)d)); }

int oracle_proxy_scores(int heads, int n, int d, int c_q, const int *c_m,
                        const float *tables, const uint32_t *codes,
                        float *scores) {
  int cs = c_m[0] + c_m[1] + c_m[2];
  float sigma = oracle_sigma(d);
  for (int h = 0; h < heads; ++h)
#pragma omp parallel for schedule(static)
    for (int c = 0; c < c_q; ++c) {
      const float *P = tables + ((size_t)h * c_q + c) * cs;
      float *S = scores + ((size_t)h * c_q + c) * n;
      for (int j = 0; j < n; ++j)
        S[j] = proxy_logit(P, c_m, codes[(size_t)h * n + j], sigma);
    }
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* General M-way key partitions (App. B; the partition ablation of Table 3).
 * The d channels are split into M disjoint sets I_1 .. I_M that cover all of
 * them; chan lists I_1, then I_2, ... (d entries), each set in ascending
 * channel order, and len[m] = d_m = |I_m|.  Subspace m is the key matrix
 * restricted to I_m, K^m = K[:, I_m], clustered exactly like a T/H/W
 * subspace above (Eq. 3).  Codes stay per subspace: z[h][m][j] (Eq. 4 with
 * M entries).  Centroids per head: U^1 .. U^M back to back, each
 * [C_m][d_m], column k of U^m belonging to channel I_m[k].  With the three
 * RoPE ranges as the sets, everything equals the T/H/W functions above.   */
#define OR_MAX_SUB 8

static int check_partition(int n, int d, int M, const int *chan,
                           const int *len, const int *c_m) {
  if (M < 1 || M > OR_MAX_SUB || d < 1) return OR_ERR_ARG;
  unsigned char seen[1024];
  if (d > 1024) return OR_ERR_ARG;
  memset(seen, 0, sizeof seen);
  int o = 0;
  for (int m = 0; m < M; ++m) {
    if (len[m] < 1 || o + len[m] > d) return OR_ERR_ARG;
    if (c_m && (c_m[m] < 1 || c_m[m] > 1024 || c_m[m] > n)) return OR_ERR_ARG;
    for (int k = 0; k < len[m]; ++k) {
      int ch = chan[o + k];
      if (ch < 0 || ch >= d || seen[ch]) return OR_ERR_ARG;
      if (k > 0 && ch <= chan[o + k - 1]) return OR_ERR_ARG;
      seen[ch] = 1;
    }
    o += len[m];
  }
  return o == d ? OR_OK : OR_ERR_ARG;
}

int oracle_cluster_key_partition(int heads, int n, int d, int M,
                                 const int *chan, const int *len,
                                 const float *k, const int *c_m, int iters,
                                 const int *init, int init_stride,
                                 float *centroids, uint16_t *codes,
                                 int *assign) {
  if (check_partition(n, d, M, chan, len, c_m) != OR_OK) return OR_ERR_ARG;
  int per_head = 0;
  for (int m = 0; m < M; ++m) per_head += c_m[m] * len[m];
  int status = OR_OK;
  int *cnt = (int *)malloc(sizeof(int) * 1024);
  float *X = (float *)malloc(sizeof(float) * (size_t)n * d);
  if (!cnt || !X) { free(cnt); free(X); return OR_ERR_MEM; }
  for (int h = 0; h < heads; ++h) {
    const float *Kh = k + (size_t)h * n * d;
    float *U = centroids + (size_t)h * per_head;
    int o = 0;
    for (int m = 0; m < M; ++m) {
      /* K^m = K[:, I_m] as a dense [n][d_m] matrix */
      for (int j = 0; j < n; ++j)
        for (int kk = 0; kk < len[m]; ++kk)
          X[(size_t)j * len[m] + kk] = Kh[(size_t)j * d + chan[o + kk]];
      int *a = assign + ((size_t)h * M + m) * n;
      int s = oracle_kmeans(X, len[m], n, len[m], c_m[m], iters,
                            init + ((size_t)h * M + m) * init_stride, 1, U, a, cnt);
      if (s == OR_ERR_ARG || s == OR_ERR_MEM) { free(cnt); free(X); return s; }
      if (s != OR_OK) status = s;
      for (int j = 0; j < n; ++j) codes[((size_t)h * M + m) * n + j] = (uint16_t)a[j];
      U += (size_t)c_m[m] * len[m];
      o += len[m];
    }
  }
  free(cnt);
  free(X);
  return status;
}

/* Eq. 5 for M subspaces: P_m[c, r] = <qbar_c[I_m], u_r^m>, the centroid's
 * channels of I_m taken in the listed (ascending) order.  Tables per head:
 * [c_q][C_1 + ... + C_M].                                                   */
int oracle_tables_partition(int heads, int d, int M, const int *chan,
                            const int *len, int c_q, const int *c_m,
                            const float *qc, const float *kc, float *tables) {
  if (check_partition(1 << 30, d, M, chan, len, c_m) != OR_OK) return OR_ERR_ARG;
  int cs = 0, per_head = 0;
  for (int m = 0; m < M; ++m) {
    cs += c_m[m];
    per_head += c_m[m] * len[m];
  }
  float qs[1024];
  for (int h = 0; h < heads; ++h) {
    const float *Q = qc + (size_t)h * c_q * d;
    float *P = tables + (size_t)h * c_q * cs;
    const float *U = kc + (size_t)h * per_head;
    int col = 0, o = 0;
    for (int m = 0; m < M; ++m) {
      for (int c = 0; c < c_q; ++c) {
        for (int kk = 0; kk < len[m]; ++kk) qs[kk] = Q[(size_t)c * d + chan[o + kk]];
        for (int r = 0; r < c_m[m]; ++r)
          P[(size_t)c * cs + col + r] = cdot(qs, U + (size_t)r * len[m], len[m]);
      }
      U += (size_t)c_m[m] * len[m];
      col += c_m[m];
      o += len[m];
    }
  }
  return OR_OK;
}

/* Eq. 6 for M subspaces: s_cj = (1/sqrt d) * sum_m P_m[c, z_j^m], the sum
 * taken left to right in subspace order, then scaled; + 0.0f as above.     */
int oracle_proxy_scores_partition(int heads, int n, int d, int M, int c_q,
                                  const int *c_m, const float *tables,
                                  const uint16_t *codes, float *scores) {
  if (M < 1 || M > OR_MAX_SUB) return OR_ERR_ARG;
  int col[OR_MAX_SUB], cs = 0;
  for (int m = 0; m < M; ++m) {
    col[m] = cs;
    cs += c_m[m];
  }
  float sigma = oracle_sigma(d);
  for (int h = 0; h < heads; ++h)
#pragma omp parallel for schedule(static)
    for (int c = 0; c < c_q; ++c) {
      const float *P = tables + ((size_t)h * c_q + c) * cs;
      float *S = scores + ((size_t)h * c_q + c) * n;
      for (int j = 0; j < n; ++j) {
        float s = P[col[0] + codes[((size_t)h * M + 0) * n + j]];
        for (int m = 1; m < M; ++m) s = s + P[col[m] + codes[((size_t)h * M + m) * n + j]];
        s = s * sigma;
        S[j] = s + 0.0f;
      }
    }
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Fixed-point exponential used for the proxy softmax of Eq. 7.
 * For y <= 0 returns round(e^y * 2^32) up to the approximation error:
 *   z = fl32(y * fl32(log2 e)); below z = -40 the mass is 0;
 *   z = n + f with n = rint(z), |f| <= 1/2 (exact);
 *   2^f by its degree-7 Taylor series in f (coefficients (ln 2)^k / k!
 *   rounded to fp32), Horner with fmaf;
 *   result = rint(2^(n+32) * p) as an integer.                              */
static const float FX_L2E = 0x1.715476p+0f;
static const float FX_C[8] = {0x1p+0f,        0x1.62e43p-1f,  0x1.ebfbep-3f,
                              0x1.c6b08ep-5f, 0x1.3b2ab6p-7f, 0x1.5d87fep-10f,
                              0x1.430912p-13f, 0x1.ffcbfcp-17f};

uint64_t oracle_fixexp(float y) {
  float z = y * FX_L2E;
  if (!(z >= -40.0f)) return 0;
  float nr = rintf(z);
  float f = z - nr;
  float p = FX_C[7];
  for (int k = 6; k >= 0; --k) p = fmaf(p, f, FX_C[k]);
  double e = ldexp((double)p, (int)nr + 32);
  return (uint64_t)rint(e);
}

void oracle_fixexp_batch(const float *y, uint64_t *out, long count) {
#pragma omp parallel for schedule(static)
  for (long i = 0; i < count; ++i) out[i] = oracle_fixexp(y[i]);
}

/* Exact ceil(rho * tot) for finite rho in (0, 1) and tot < 2^63.            */
uint64_t oracle_mass_target(float rho, uint64_t tot) {
  int e;
  float fr = frexpf(rho, &e);                  /* rho = fr * 2^e, fr in [.5,1) */
  uint64_t m = (uint64_t)ldexpf(fr, 24);       /* 24-bit integer significand  */
  int sh = 24 - e;                             /* rho = m / 2^sh, sh >= 24    */
  if (sh >= 100) return tot ? 1 : 0;           /* m*tot < 2^88: ceil is 1     */
  unsigned __int128 prod = (unsigned __int128)m * tot;
  unsigned __int128 one = (unsigned __int128)1 << sh;
  return (uint64_t)((prod + one - 1) >> sh);
}

/* Alg. 3 for one head.  scores: [c_q][n]; counts: n_c.                      */
typedef struct { float s; int j; } keyed;

static int cmp_rank(const void *pa, const void *pb) {
  const keyed *a = (const keyed *)pa, *b = (const keyed *)pb;
  if (a->s > b->s) return -1;       /* larger logit first */
  if (a->s < b->s) return 1;
  return (a->j > b->j) - (a->j < b->j); /* ties: smaller key index first */
}

static int cmp_int(const void *pa, const void *pb) {
  int a = *(const int *)pa, b = *(const int *)pb;
  return (a > b) - (a < b);
}

/* policy: 0 = online (Eq. 10, r_c = max(b_c, k_head)); 1 = fixed floor
 * without top-up (r_c = b_c = max(t_c, k_fix)); 2 = pure Top-p (r_c = t_c).
 * The last two are the selection-policy ablation of Fig. 6.                */
int oracle_select(int heads, int n, int c_q, const float *scores,
                  const int *counts, float rho, int k_fix, int policy, int *base,
                  int *k_head, int *sel_counts, int *sel_idx, int *topp) {
  if (!(rho > 0.0f && rho <= 1.0f) || k_fix < 1 || k_fix > n) return OR_ERR_ARG;
  if (policy < 0 || policy > 2) return OR_ERR_ARG;
  for (int h = 0; h < heads; ++h) {
    const float *S = scores + (size_t)h * c_q * n;
    int *b = base + (size_t)h * c_q;
    /* Eq. 7-8 for every query cluster; the rankings are kept for Eq. 10. */
    keyed *order = (keyed *)malloc(sizeof(keyed) * (size_t)c_q * n);
    int *tcs = (int *)malloc(sizeof(int) * (size_t)c_q);
    if (!order || !tcs) { free(order); free(tcs); return OR_ERR_MEM; }
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < c_q; ++c) {
      keyed *pi = order + (size_t)c * n;
      const float *s = S + (size_t)c * n;
      for (int j = 0; j < n; ++j) { pi[j].s = s[j]; pi[j].j = j; }
      qsort(pi, (size_t)n, sizeof(keyed), cmp_rank);       /* pi_c */
      float M = pi[0].s;                                   /* max logit */
      uint64_t tot = 0;
      for (int j = 0; j < n; ++j) tot += oracle_fixexp(s[j] - M);
      int t;
      if (rho >= 1.0f) {
        t = n;   /* every real softmax weight is positive: the whole row */
      } else {
        uint64_t T = oracle_mass_target(rho, tot);
        uint64_t acc = 0;
        t = n;
        for (int l = 0; l < n; ++l) {
          acc += oracle_fixexp(pi[l].s - M);
          if (acc >= T) { t = l + 1; break; }
        }
      }
      tcs[c] = t;
      if (topp) topp[(size_t)h * c_q + c] = t;
      b[c] = t > k_fix ? t : k_fix;                        /* Eq. 8 */
    }
    /* Eq. 9: query-size-weighted mean of b_c, rounded up, exact in integers */
    uint64_t num = 0, den = 0;
    for (int c = 0; c < c_q; ++c) {
      num += (uint64_t)counts[(size_t)h * c_q + c] * (uint64_t)b[c];
      den += (uint64_t)counts[(size_t)h * c_q + c];
    }
    if (den == 0) { free(order); free(tcs); return OR_ERR_ARG; }
    int kh = (int)((num + den - 1) / den);
    k_head[h] = kh;
    /* Eq. 10: r_c = max(b_c, k_head) (or the policy's count); S_c = first r_c
     * keys of pi_c, emitted in ascending key index.                         */
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < c_q; ++c) {
      int r = policy == 0 ? (b[c] > kh ? b[c] : kh) : policy == 1 ? b[c] : tcs[c];
      sel_counts[(size_t)h * c_q + c] = r;
      int *out = sel_idx + ((size_t)h * c_q + c) * n;
      keyed *pi = order + (size_t)c * n;
      for (int l = 0; l < r; ++l) out[l] = pi[l].j;
      qsort(out, (size_t)r, sizeof(int), cmp_int);
    }
    free(order);
    free(tcs);
  }
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Eq. 11 (and Eq. 1 when every key set is [0, n)): each query of cluster c
 * attends over the keys S_c with softmax(q k^T * scale) v, evaluated in fp64.
 * Queries are visited through perm/offsets; rows with row_mask[i] == 0 are
 * skipped (row_mask may be NULL), so a caller can check sampled rows.       */
int oracle_attention(int heads, int n, int d, const float *q, const float *k,
                     const float *v, int c_q, const int *offsets,
                     const int *perm, const int *sel_counts, const int *sel_idx,
                     double scale, const unsigned char *row_mask, float *out) {
  for (int h = 0; h < heads; ++h) {
    const float *Q = q + (size_t)h * n * d;
    const float *K = k + (size_t)h * n * d;
    const float *V = v + (size_t)h * n * d;
    float *O = out + (size_t)h * n * d;
    const int *off = offsets + (size_t)h * (c_q + 1);
    const int *pm = perm + (size_t)h * n;
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < c_q; ++c) {
      int r = sel_counts[(size_t)h * c_q + c];
      const int *S = sel_idx + ((size_t)h * c_q + c) * n;
      double *logit = (double *)malloc(sizeof(double) * (size_t)(r > 0 ? r : 1));
      double *acc = (double *)malloc(sizeof(double) * (size_t)d);
      for (int p = off[c]; p < off[c + 1]; ++p) {
        int i = pm[p];
        if (row_mask && !row_mask[(size_t)h * n + i]) continue;
        const float *qi = Q + (size_t)i * d;
        double mx = -INFINITY;
        for (int l = 0; l < r; ++l) {
          const float *kj = K + (size_t)S[l] * d;
          double dot = 0.0;
          for (int ch = 0; ch < d; ++ch) dot += (double)qi[ch] * (double)kj[ch];
          logit[l] = dot * scale;
          if (logit[l] > mx) mx = logit[l];
        }
        double den = 0.0;
        for (int ch = 0; ch < d; ++ch) acc[ch] = 0.0;
        for (int l = 0; l < r; ++l) {
          double w = exp(logit[l] - mx);
          den += w;
          const float *vj = V + (size_t)S[l] * d;
          for (int ch = 0; ch < d; ++ch) acc[ch] += w * (double)vj[ch];
        }
        for (int ch = 0; ch < d; ++ch)
          O[(size_t)i * d + ch] = r > 0 ? (float)(acc[ch] / den) : 0.0f;
      }
      free(logit);
      free(acc);
    }
  }
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Single steps of the k-means above, exposed so that properties of a full-
 * size clustering can be checked one row or one cluster at a time.         */
int oracle_assign_rows(const float *X, long ldx, int n, int dx, const float *U,
                       int C, int *assign) {
  if (n < 0 || dx < 1 || C < 1) return OR_ERR_ARG;
  km_assign(X, ldx, n, dx, U, C, assign);
  return OR_OK;
}

int oracle_mean_rows(const float *X, long ldx, int n, int dx, const int *assign,
                     int C, float *U, int *counts) {
  if (n < 0 || dx < 1 || C < 1) return OR_ERR_ARG;
  for (int i = 0; i < n; ++i)
    if (assign[i] < 0 || assign[i] >= C) return OR_ERR_ARG;
  return km_update(X, ldx, n, dx, assign, C, U, counts);
}

/* ------------------------------------------------------------------------
 * Proxy comparison measurements (App. C, Fig. 9: matched oracle recall;
 * Fig. 2: attention recall against density).  They compare key-side
 * proxies of the exact scores and are not part of the layer.  A proxy row
 * scores every key for one query; keys are ranked by proxy descending, ties
 * by ascending key index.                                                  */

/* Block-wise proxy: the keys cut into blocks of `block` consecutive tokens
 * (the last block may be shorter), each represented by the mean of its keys
 * (fp64 sums divided by the block's size).  Row r scores key j by
 * <qrep_r, mean of j's block> * scale, in fp64, stored as fp32.           */
int oracle_block_proxy(int rows, int n, int d, const float *qrep, const float *k,
                       int block, double scale, float *proxy) {
  if (rows < 0 || n < 1 || d < 1 || block < 1) return OR_ERR_ARG;
  const int nb = (n + block - 1) / block;
  double *kbar = (double *)malloc(sizeof(double) * (size_t)nb * d);
  if (!kbar) return OR_ERR_MEM;
  for (int b = 0; b < nb; ++b) {
    const int j0 = b * block, j1 = j0 + block < n ? j0 + block : n;
    for (int c = 0; c < d; ++c) {
      double s = 0.0;
      for (int j = j0; j < j1; ++j) s += (double)k[(size_t)j * d + c];
      kbar[(size_t)b * d + c] = s / (double)(j1 - j0);
    }
  }
#pragma omp parallel for schedule(static)
  for (int r = 0; r < rows; ++r) {
    for (int b = 0; b < nb; ++b) {
      double s = 0.0;
      for (int c = 0; c < d; ++c) s += (double)qrep[(size_t)r * d + c] * kbar[(size_t)b * d + c];
      const float v = (float)(s * scale);
      const int j0 = b * block, j1 = j0 + block < n ? j0 + block : n;
      for (int j = j0; j < j1; ++j) proxy[(size_t)r * n + j] = v;
    }
  }
  free(kbar);
  return OR_OK;
}

typedef struct {
  float v;
  int j;
} ranked_t;

static int cmp_ranked(const void *pa, const void *pb) {
  const ranked_t *a = (const ranked_t *)pa, *b = (const ranked_t *)pb;
  if (a->v > b->v) return -1;
  if (a->v < b->v) return 1;
  return (a->j > b->j) - (a->j < b->j);
}

/* keys of one row in ranked order: value descending, index ascending */
static void rank_row(const float *row, int n, ranked_t *out) {
  for (int j = 0; j < n; ++j) {
    out[j].v = row[j] + 0.0f; /* -0 ranks with +0 */
    out[j].j = j;
  }
  qsort(out, (size_t)n, sizeof(ranked_t), cmp_ranked);
}

/* Matched oracle recall, per row: the oracle set O is the first kt keys of
 * the exact ranking; keys are taken in proxy order until `need` keys of O
 * are held, and then every key whose proxy equals the last one taken (a
 * block or a centroid is kept whole).  retention[r] = kept / n and
 * recall[r] = |kept and O| / kt.                                          */
int oracle_matched_retention(int rows, int n, const float *exact, const float *proxy,
                             int kt, int need, double *retention, double *recall) {
  if (rows < 0 || n < 1 || kt < 1 || kt > n || need < 1 || need > kt) return OR_ERR_ARG;
  int status = OR_OK;
#pragma omp parallel
  {
    ranked_t *re = (ranked_t *)malloc(sizeof(ranked_t) * (size_t)n);
    ranked_t *rp = (ranked_t *)malloc(sizeof(ranked_t) * (size_t)n);
    char *in_o = (char *)malloc((size_t)n);
    if (!re || !rp || !in_o) {
#pragma omp atomic write
      status = OR_ERR_MEM;
    } else {
#pragma omp for schedule(dynamic)
      for (int r = 0; r < rows; ++r) {
        rank_row(exact + (size_t)r * n, n, re);
        memset(in_o, 0, (size_t)n);
        for (int i = 0; i < kt; ++i) in_o[re[i].j] = 1;
        rank_row(proxy + (size_t)r * n, n, rp);
        int hits = 0, pos = 0;
        for (; pos < n; ++pos) {
          hits += in_o[rp[pos].j];
          if (hits >= need) break;
        }
        const float s_star = rp[pos].v;
        long kept = 0, kept_o = 0;
        for (int j = 0; j < n; ++j) {
          if (proxy[(size_t)r * n + j] + 0.0f >= s_star) {
            ++kept;
            kept_o += in_o[j];
          }
        }
        retention[r] = (double)kept / (double)n;
        recall[r] = (double)kept_o / (double)kt;
      }
    }
    free(re);
    free(rp);
    free(in_o);
  }
  return status;
}

/* Attention recall at a density: per row, the sum (fp64) of the exact
 * attention weights p of the first `count` keys in proxy order.          */
int oracle_recall_at_density(int rows, int n, const double *p, const float *proxy,
                             int count, double *mass) {
  if (rows < 0 || n < 1 || count < 1 || count > n) return OR_ERR_ARG;
  int status = OR_OK;
#pragma omp parallel
  {
    ranked_t *rp = (ranked_t *)malloc(sizeof(ranked_t) * (size_t)n);
    if (!rp) {
#pragma omp atomic write
      status = OR_ERR_MEM;
    } else {
#pragma omp for schedule(dynamic)
      for (int r = 0; r < rows; ++r) {
        rank_row(proxy + (size_t)r * n, n, rp);
        double s = 0.0;
        for (int i = 0; i < count; ++i) s += p[(size_t)r * n + rp[i].j];
        mass[r] = s;
      }
    }
    free(rp);
  }
  return status;
}
