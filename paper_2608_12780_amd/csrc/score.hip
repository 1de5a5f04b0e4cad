// Score tables (Eq. 5) and lookup-and-sum proxy logits (Eq. 6, Alg. 2).
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

struct TableGeom {
  int off[3], len[3], cm[3], col[3], ucol[3];  // ucol: float offset of U^m
};

// P[h][c][col] = <qbar_c[I_m], u_r^m>, fp32 fma chain in channel order.
__global__ void tables_kernel(int d, int c_q, int cs, int per_head, TableGeom g,
                              const float *__restrict__ qc,
                              const float *__restrict__ kc, float *tables) {
  const int col = blockIdx.x * blockDim.x + threadIdx.x;
  const int c = blockIdx.y, h = blockIdx.z;
  if (col >= cs) return;
  const int m = col < g.col[1] ? 0 : (col < g.col[2] ? 1 : 2);
  const int r = col - g.col[m];
  const float *q = qc + (static_cast<size_t>(h) * c_q + c) * d + g.off[m];
  const float *u = kc + static_cast<size_t>(h) * per_head + g.ucol[m] +
                   static_cast<size_t>(r) * g.len[m];
  float acc = 0.0f;
  for (int ch = 0; ch < g.len[m]; ++ch) acc = fmaf(q[ch], u[ch], acc);
  tables[(static_cast<size_t>(h) * c_q + c) * cs + col] = acc;
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

}  // namespace

hipError_t score_tables(int heads, int d, const int *off, const int *len,
                        int c_q, const int *c_m, const float *qc,
                        const float *kc, float *tables, hipStream_t s) {
  TableGeom g;
  int col = 0, ucol = 0;
  for (int m = 0; m < 3; ++m) {
    g.off[m] = off[m];
    g.len[m] = len[m];
    g.cm[m] = c_m[m];
    g.col[m] = col;
    g.ucol[m] = ucol;
    col += c_m[m];
    ucol += c_m[m] * len[m];
  }
  const int cs = col;
  hipLaunchKernelGGL(tables_kernel, dim3((cs + 127) / 128, c_q, heads),
                     dim3(128), 0, s, d, c_q, cs, ucol, g, qc, kc, tables);
  return hipGetLastError();
}

hipError_t score_logits(int heads, int n, int d, int c_q, const int *c_m,
                        const float *tables, const uint32_t *codes,
                        float *scores, hipStream_t s) {
  const int cs = c_m[0] + c_m[1] + c_m[2];
  const float sigma = static_cast<float>(1.0 / sqrt(static_cast<double>(d)));
  hipLaunchKernelGGL(logits_kernel, dim3((n + 255) / 256, c_q, heads),
                     dim3(256), 0, s, n, c_q, cs, c_m[0], c_m[0] + c_m[1],
                     sigma, tables, codes, scores);
  return hipGetLastError();
}

}  // namespace scope
