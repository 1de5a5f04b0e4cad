// K-means assignment on the matrix cores, exact with respect to the
// canonical assignment (argmin_r fl(||u_r||^2 - 2<x,u_r>) with fp32 fma-chain
// dot products in channel order, ties to the lowest r).
//
// bf16 points x are exact in bf16, so with centroids rounded to bf16 (u^) the
// products x_c u^_c are exact and a bf16 MFMA gives the approximate score
//   s~_r = fl(nu_r - 2 <x, u^_r>_mfma).
// Its distance to the canonical score c_r is bounded per point by
//   |s~_r - c_r| <= beta = 2|x| (E + 8 DXP 2^-24 Nmax) + 2^-23 (numax + 2.02 |x| Nmax)
// (E >= |u^_r - u_r|, Nmax >= |u_r| + E, numax >= |nu_r|; the first term is the
// bf16 rounding of the centroid, the second both fp32 accumulations, the
// third the two roundings of the final subtraction), inflated by 1%.  So the
// canonical argmin r* satisfies s~_{r*} <= min_r s~_r + 2 beta: every such
// r is a candidate, re-scored with the canonical arithmetic, and the smallest
// (score, r) wins.  Equal canonical scores are all candidates, so the
// lowest-index rule carries over exactly.
//
// Block = 8 waves x 32 points (one grouping chunk).  Pass 1 finds min s~ per
// point, pass 2 recomputes the products and collects candidates into an LDS
// list, then all lanes re-score the list; a point whose candidates overflow
// the list is re-scored against every centroid.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kMfmaPoints = 256;          // == kAssignBlock
constexpr int kUbfLds = 34816;            // bf16 codebook elements in LDS
                                          // (two blocks fit one CU)
constexpr int kCandCap = 1024;            // candidate (point, centroid) pairs
constexpr int kMaxCpad = 1024;

__device__ __forceinline__ uint16_t to_bf16(float f) {
  bf16x2 r;
  r[0] = static_cast<__bf16>(f);
  r[1] = static_cast<__bf16>(0.0f);
  return static_cast<uint16_t>(__builtin_bit_cast(uint32_t, r) & 0xFFFFu);
}

// ascending-order key of a float score
__device__ __forceinline__ uint32_t asc_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Per pass: bf16 codebook (zero padded), canonical squared norms (+inf for
// padding rows, which then never win) and the bound constants of each head.
template <int DXP>
__global__ __launch_bounds__(1024) void km_prep_kernel(
    const float *__restrict__ U, size_t u_hs, int C, int cpad, int dx,
    uint16_t *ubf, float *nu, float *bnd) {
  __shared__ float red[3][16];
  const int h = blockIdx.x, t = threadIdx.x;
  float e_max = 0.0f, n_max = 0.0f, nu_max = 0.0f;
  for (int r = t; r < cpad; r += blockDim.x) {
    uint16_t *dst = ubf + (static_cast<size_t>(h) * cpad + r) * DXP;
    if (r < C) {
      const float *u = U + h * u_hs + static_cast<size_t>(r) * dx;
      float nr = 0.0f;
      double e2 = 0.0, n2 = 0.0;
      for (int c = 0; c < dx; ++c) {
        nr = fmaf(u[c], u[c], nr);
        const uint16_t b = to_bf16(u[c]);
        const double df = static_cast<double>(bf16_to_f32(b)) - static_cast<double>(u[c]);
        e2 += df * df;
        n2 += static_cast<double>(u[c]) * static_cast<double>(u[c]);
        dst[c] = b;
      }
      for (int c = dx; c < DXP; ++c) dst[c] = 0;
      nu[static_cast<size_t>(h) * cpad + r] = nr;
      e_max = fmaxf(e_max, static_cast<float>(sqrt(e2)));
      n_max = fmaxf(n_max, static_cast<float>(sqrt(n2)));
      nu_max = fmaxf(nu_max, fabsf(nr));
    } else {
      for (int c = 0; c < DXP; ++c) dst[c] = 0;
      nu[static_cast<size_t>(h) * cpad + r] = INFINITY;
    }
  }
  e_max = wave_max(e_max);
  n_max = wave_max(n_max);
  nu_max = wave_max(nu_max);
  const int lane = t & 63, w = t >> 6;
  if (lane == 0) {
    red[0][w] = e_max;
    red[1][w] = n_max;
    red[2][w] = nu_max;
  }
  __syncthreads();
  if (t == 0) {
    float a = 0.0f, b = 0.0f, c = 0.0f;
    for (int i = 0; i < static_cast<int>(blockDim.x >> 6); ++i) {
      a = fmaxf(a, red[0][i]);
      b = fmaxf(b, red[1][i]);
      c = fmaxf(c, red[2][i]);
    }
    // small upward slack on top of the fp64 evaluation
    bnd[4 * h + 0] = a * 1.001f;
    bnd[4 * h + 1] = (b + a) * 1.001f;
    bnd[4 * h + 2] = c * 1.001f;
    bnd[4 * h + 3] = 0.0f;
  }
}

template <int DXP>
__global__ __launch_bounds__(512) void km_assign_mfma_kernel(
    const uint16_t *__restrict__ X, size_t x_hs, int ld, int col0, int dx,
    int n, const float *__restrict__ U, size_t u_hs,
    const uint16_t *__restrict__ ubf, const float *__restrict__ nu,
    const float *__restrict__ bnd, int C, int cpad, int32_t *assign,
    size_t a_hs, int32_t *chunk_hist, int nchunks) {
  constexpr int US = DXP + 8;   // LDS row stride of the bf16 codebook
  constexpr int KS = DXP / 16;  // MFMA k-steps
  __shared__ __attribute__((aligned(16))) uint16_t Us[kUbfLds];
  __shared__ float nus[kMaxCpad];
  __shared__ uint32_t cand[kCandCap];   // candidate pairs, then the histogram
  __shared__ unsigned long long best[kMfmaPoints];
  __shared__ int flag[kMfmaPoints];
  __shared__ int ncand;
  int *hist = reinterpret_cast<int *>(cand);
  const int h = blockIdx.y, t = threadIdx.x;
  const int lane = t & 63, w = t >> 6, l32 = lane & 31, hf = lane >> 5;
  const int p0 = blockIdx.x * kMfmaPoints;

  // stage the codebook (16-byte rows pieces) and norms
  const uint16_t *ub = ubf + static_cast<size_t>(h) * cpad * DXP;
  for (int e = t; e < cpad * (DXP / 8); e += 512) {
    const int r = e / (DXP / 8), q = e % (DXP / 8);
    *reinterpret_cast<uint4 *>(&Us[r * US + 8 * q]) =
        *reinterpret_cast<const uint4 *>(ub + static_cast<size_t>(r) * DXP + 8 * q);
  }
  for (int r = t; r < cpad; r += 512) nus[r] = nu[static_cast<size_t>(h) * cpad + r];
  if (t < kMfmaPoints) {
    best[t] = ~0ull;
    flag[t] = 0;
  }
  if (t == 0) ncand = 0;

  // this lane's point (column l32 of wave w) as MFMA B fragments
  const int pl = w * 32 + l32;
  const int i = p0 + pl;
  const bool valid = i < n;
  const uint16_t *xrow = X + h * x_hs + static_cast<size_t>(valid ? i : 0) * ld + col0;
  bf16x8 xf[KS];
  float ss = 0.0f;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    uint32_t wv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = 16 * s + 8 * hf + 2 * q;
      uint32_t v = 0;
      if (valid && c < dx) v = *reinterpret_cast<const uint32_t *>(xrow + c);
      wv[q] = v;
      const float a = __uint_as_float(v << 16), b = __uint_as_float(v & 0xFFFF0000u);
      ss = fmaf(a, a, ss);
      ss = fmaf(b, b, ss);
    }
    xf[s] = __builtin_bit_cast(bf16x8, make_uint4(wv[0], wv[1], wv[2], wv[3]));
  }
  ss += __shfl_xor(ss, 32);
  __syncthreads();

  // per-point bound; |x| rounded up generously
  const float E = bnd[4 * h + 0], Nmax = bnd[4 * h + 1], numax = bnd[4 * h + 2];
  const float nx = sqrtf(ss) * 1.0001f + 1e-30f;
  const float kappa = 8.0f * DXP * 0x1p-24f;
  const float beta = (2.0f * nx * (E + kappa * Nmax) +
                      0x1p-23f * (numax + 2.02f * nx * Nmax)) * 1.01f + 1e-30f;

  // pass 1: min approximate score per point
  float tau = INFINITY;
  for (int rb = 0; rb < cpad; rb += 32) {
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 a = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const uint4 *>(&Us[(rb + l32) * US + 16 * s + 8 * hf]));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xf[s], acc, 0, 0, 0);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int r = rb + 8 * (e >> 2) + 4 * hf + (e & 3);
      tau = fminf(tau, fmaf(-2.0f, acc[e], nus[r]));
    }
  }
  tau = fminf(tau, __shfl_xor(tau, 32));
  const float v = tau + 2.0f * beta;  // rounded up by more than its own rounding
  const float thr = v + fabsf(v) * 2e-6f + 1e-30f;

  // pass 2: candidates s~_r <= min + 2 beta
  for (int rb = 0; rb < cpad; rb += 32) {
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 a = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const uint4 *>(&Us[(rb + l32) * US + 16 * s + 8 * hf]));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xf[s], acc, 0, 0, 0);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int r = rb + 8 * (e >> 2) + 4 * hf + (e & 3);
      if (valid && r < C && fmaf(-2.0f, acc[e], nus[r]) <= thr) {
        const int slot = atomicAdd(&ncand, 1);
        if (slot < kCandCap)
          cand[slot] = (static_cast<uint32_t>(pl) << 16) | static_cast<uint32_t>(r);
        else
          flag[pl] = 1;
      }
    }
  }
  __syncthreads();

  // exact re-scoring of the candidates: point and centroid rows (both in L2)
  // are fetched 32 channels at a time with every load in flight, then the
  // canonical fma chain runs in channel order
  const int cnt = min(ncand, kCandCap);
  const float *Uh = U + h * u_hs;
  auto rescore = [&](int q, int r) {
    const float2 *u2 = reinterpret_cast<const float2 *>(Uh + static_cast<size_t>(r) * dx);
    const uint32_t *x2 = reinterpret_cast<const uint32_t *>(
        X + h * x_hs + static_cast<size_t>(p0 + q) * ld + col0);
    float dot = 0.0f;
#pragma unroll 1
    for (int c0 = 0; c0 < DXP; c0 += 32) {
      float2 uv[16];
      uint32_t xv[16];
#pragma unroll
      for (int k2 = 0; k2 < 16; ++k2) {
        const bool in = c0 + 2 * k2 < dx;
        uv[k2] = in ? u2[(c0 >> 1) + k2] : make_float2(0.0f, 0.0f);
        xv[k2] = in ? x2[(c0 >> 1) + k2] : 0u;
      }
#pragma unroll
      for (int k2 = 0; k2 < 16; ++k2) {
        if (c0 + 2 * k2 < dx) {
          dot = fmaf(__uint_as_float(xv[k2] << 16), uv[k2].x, dot);
          dot = fmaf(__uint_as_float(xv[k2] & 0xFFFF0000u), uv[k2].y, dot);
        }
      }
    }
    return fmaf(-2.0f, dot, nus[r]) + 0.0f;
  };
  for (int k = t; k < cnt; k += 512) {
    const uint32_t pr = cand[k];
    const int q = static_cast<int>(pr >> 16), r = static_cast<int>(pr & 0xFFFFu);
    const float sc = rescore(q, r);
    atomicMin(&best[q], (static_cast<unsigned long long>(asc_key(sc)) << 32) | static_cast<unsigned>(r));
  }
  __syncthreads();
  // points whose candidates did not fit: every centroid, canonically
  if (t < kMfmaPoints && flag[t] && p0 + t < n) {
    unsigned long long b = ~0ull;
    for (int r = 0; r < C; ++r) {
      const float sc = rescore(t, r);
      const unsigned long long key = (static_cast<unsigned long long>(asc_key(sc)) << 32) | static_cast<unsigned>(r);
      b = key < b ? key : b;
    }
    best[t] = b;
  }
  __syncthreads();
  int arg = 0;
  if (t < kMfmaPoints && p0 + t < n) {
    const unsigned long long b = best[t];
    arg = b == ~0ull ? 0 : static_cast<int>(b & 0xFFFFFFFFu);
    assign[h * a_hs + p0 + t] = arg;
  }
  if (chunk_hist) {
    for (int r = t; r < C; r += 512) hist[r] = 0;
    __syncthreads();
    if (t < kMfmaPoints && p0 + t < n) atomicAdd(&hist[arg], 1);
    __syncthreads();
    int32_t *out = chunk_hist + (static_cast<size_t>(h) * nchunks + blockIdx.x) * C;
    for (int r = t; r < C; r += 512) out[r] = hist[r];
  }
}

template <int DXP>
hipError_t launch_mfma(const KmProblem &p, bool with_hist, hipStream_t s) {
  hipLaunchKernelGGL(km_prep_kernel<DXP>, dim3(p.heads), dim3(1024), 0, s, p.u,
                     p.u_head_stride, p.C, p.cpad, p.dx, p.ubf, p.nu, p.bnd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nch = km_nchunks(p.n);
  hipLaunchKernelGGL(km_assign_mfma_kernel<DXP>, dim3(nch, p.heads), dim3(512), 0,
                     s, static_cast<const uint16_t *>(p.x), p.x_head_stride, p.ld,
                     p.col0, p.dx, p.n, p.u, p.u_head_stride, p.ubf, p.nu, p.bnd,
                     p.C, p.cpad, p.assign, p.a_head_stride,
                     with_hist ? p.chunk_hist : nullptr, nch);
  return hipGetLastError();
}

}  // namespace

int km_cpad(int C) { return (C + 31) / 32 * 32; }
int km_dxp(int dx) { return dx <= 16 ? 16 : dx <= 32 ? 32 : dx <= 48 ? 48 : dx <= 64 ? 64 : 128; }

bool km_mfma_ok(bool bf16, int ld, int col0, int dx, int C) {
  if (!bf16 || (ld & 1) || (col0 & 1) || (dx & 1) || dx > 128) return false;
  return km_cpad(C) * (km_dxp(dx) + 8) <= kUbfLds && km_cpad(C) <= kMaxCpad;
}

hipError_t km_assign_mfma(const KmProblem &p, bool with_hist, hipStream_t s) {
  switch (p.dxp) {
    case 16: return launch_mfma<16>(p, with_hist, s);
    case 32: return launch_mfma<32>(p, with_hist, s);
    case 48: return launch_mfma<48>(p, with_hist, s);
    case 64: return launch_mfma<64>(p, with_hist, s);
    default: return launch_mfma<128>(p, with_hist, s);
  }
}

}  // namespace scope
