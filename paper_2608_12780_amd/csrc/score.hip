// Score tables (Eq. 5) and lookup-and-sum proxy logits (Eq. 6, Alg. 2).
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

static_assert(kCodeMaxSub == kMaxSub, "one bound on the number of subspaces");

namespace {

struct TableGeom {
  int M;
  int off[kMaxSub], len[kMaxSub];
  int col[kMaxSub + 1];  // first table column of subspace m; col[M] = row length
  int ucol[kMaxSub];     // float offset of U^m within a head's centroids
};

// P[h][c][col] = <qbar_c[I_m], u_r^m>, fp32 fma chain in channel order.
// A block takes kTabC clusters of one head: their centroid rows are staged
// in LDS, and each thread runs the kTabC independent chains of one table
// column (one codebook row read once for all of them).
constexpr int kTabC = 8;
constexpr int kTabMaxD = 128;
__global__ __launch_bounds__(256) void tables_kernel(int d, int c_q, int per_head, TableGeom g,
                                                     const float *__restrict__ qc,
                                                     const float *__restrict__ kc, float *tables) {
  __shared__ float qs[kTabC][kTabMaxD];
  const int c0 = blockIdx.x * kTabC, h = blockIdx.y;
  const int cs = g.col[g.M];
  const int nc = c_q - c0 < kTabC ? c_q - c0 : kTabC;
  for (int e = threadIdx.x; e < kTabC * d; e += blockDim.x) {
    const int k = e / d, ch = e % d;
    qs[k][ch] = k < nc ? qc[(static_cast<size_t>(h) * c_q + c0 + k) * d + ch] : 0.0f;
  }
  __syncthreads();
  for (int col = threadIdx.x; col < cs; col += blockDim.x) {
    int m = 0;
    while (m + 1 < g.M && col >= g.col[m + 1]) ++m;
    const int r = col - g.col[m], len = g.len[m], off = g.off[m];
    const float *u = kc + static_cast<size_t>(h) * per_head + g.ucol[m] +
                     static_cast<size_t>(r) * len;
    float acc[kTabC];
#pragma unroll
    for (int k = 0; k < kTabC; ++k) acc[k] = 0.0f;
    for (int ch = 0; ch < len; ++ch) {
      const float uv = u[ch];
#pragma unroll
      for (int k = 0; k < kTabC; ++k) acc[k] = fmaf(qs[k][off + ch], uv, acc[k]);
    }
#pragma unroll
    for (int k = 0; k < kTabC; ++k)
      if (k < nc) tables[(static_cast<size_t>(h) * c_q + c0 + k) * cs + col] = acc[k];
  }
}

__global__ void logits_kernel(int n, int c_q, int cs, int cT, int cTH,
                              float sigma, const float *__restrict__ tables,
                              const uint32_t *__restrict__ codes,
                              float *scores) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int c = blockIdx.y, h = blockIdx.z;
  if (j >= n) return;
  const float *P = tables + (static_cast<size_t>(h) * c_q + c) * cs;
  scores[(static_cast<size_t>(h) * c_q + c) * n + j] =
      proxy_logit(P, cT, cTH, cs, codes[static_cast<size_t>(h) * n + j], sigma);
}

__global__ void logits_planes_kernel(int n, int c_q, CodePlanes cp, float sigma,
                                     const float *__restrict__ tables,
                                     const uint16_t *__restrict__ codes,
                                     float *scores) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int c = blockIdx.y, h = blockIdx.z;
  if (j >= n) return;
  const int cs = cp.col[cp.M];
  const float *P = tables + (static_cast<size_t>(h) * c_q + c) * cs;
  const uint16_t *planes = codes + static_cast<size_t>(h) * cp.M * n;
  scores[(static_cast<size_t>(h) * c_q + c) * n + j] =
      proxy_logit_planes(P, cp, planes, static_cast<size_t>(n), j, sigma);
}

}  // namespace

hipError_t score_tables(int heads, int d, const int *off, const int *len,
                        int c_q, const Subspaces &sub, const float *qc,
                        const float *kc, float *tables, hipStream_t s) {
  TableGeom g{};
  g.M = sub.M;
  int col = 0, ucol = 0;
  for (int m = 0; m < sub.M; ++m) {
    g.off[m] = off[m];
    g.len[m] = len[m];
    g.col[m] = col;
    g.ucol[m] = ucol;
    col += sub.c[m];
    ucol += sub.c[m] * len[m];
  }
  g.col[sub.M] = col;
  if (d > kTabMaxD) return hipErrorInvalidValue;
  hipLaunchKernelGGL(tables_kernel, dim3((c_q + kTabC - 1) / kTabC, heads),
                     dim3(256), 0, s, d, c_q, ucol, g, qc, kc, tables);
  return hipGetLastError();
}

hipError_t score_logits(int heads, int n, int d, int c_q, const Subspaces &sub,
                        const float *tables, const uint32_t *codes32,
                        const uint16_t *codes16, float *scores, hipStream_t s) {
  const float sigma = static_cast<float>(1.0 / sqrt(static_cast<double>(d)));
  const dim3 grid((n + 255) / 256, c_q, heads);
  if (codes16) {
    CodePlanes cp{};
    cp.M = sub.M;
    for (int m = 0; m < sub.M; ++m) cp.col[m + 1] = cp.col[m] + sub.c[m];
    hipLaunchKernelGGL(logits_planes_kernel, grid, dim3(256), 0, s, n, c_q, cp,
                       sigma, tables, codes16, scores);
  } else {
    const int cs = sub.c[0] + sub.c[1] + sub.c[2];
    hipLaunchKernelGGL(logits_kernel, grid, dim3(256), 0, s, n, c_q, cs, sub.c[0],
                       sub.c[0] + sub.c[1], sigma, tables, codes32, scores);
  }
  return hipGetLastError();
}

}  // namespace scope
