// K-means assignment on the matrix cores, exact with respect to the
// canonical assignment (argmin_r fl(||u_r||^2 - 2<x,u_r>) with fp32 fma-chain
// dot products in channel order, ties to the lowest r).
//
// bf16 points x are exact in bf16.  Each centroid is split into two bf16
// terms, u ~ hi + lo (hi = bf16(u), lo = bf16(u - hi)), so every product
// x_c hi_c and x_c lo_c is exact.  The MFMA accumulator starts at -nu_r / 2
// and two bf16 MFMAs per k-step add the products, which gives the halved,
// negated score
//   a_r = fl(-nu_r / 2 + <x, hi_r + lo_r>_mfma),   argmin_r c_r = argmax_r -c_r / 2.
// Summed in any order with one fp32 rounding per addition, the 2 DXP
// products and the start value err by at most 2 DXP 2^-24 (numax / 2 +
// |x| Nmax); the canonical score adds its dot product's DXP 2^-24 |x| Nmax and
// one rounding of the final fma.  So, in the canonical scale,
//   |-2 a_r - c_r| <= beta = 2|x| (E + 8 DXP 2^-24 Nmax)
//                            + 2^-23 ((2 DXP + 1) numax + 2.02 |x| Nmax)
// (E >= |u_r - hi_r - lo_r|, Nmax >= |hi_r| + |lo_r| and |u_r|, numax >=
// |nu_r|; about twice the terms derived, for slack), inflated by 1%, and the
// canonical argmin r* satisfies a_{r*} >= max_r a_r - beta.
//
// One pass keeps, per point, the three largest a_r with the centroid index
// packed into the low mantissa bits (IB bits; this moves a value by less
// than delta = 2^(IB-23) |a|, added to the margin).  If the second-largest
// is more than beta + 2 delta below the largest, the largest's index is the
// only candidate and thus r*.  If only the third is, r* is one of the two
// largest, and the point's two half-wave lanes re-score one each with the
// canonical arithmetic.  For the very few points with three or more
// candidates, the wave recomputes the values, lists every candidate within
// the margin and re-scores them canonically.  In both cases the smallest
// canonical (score, r) wins, so equal scores keep the lowest index.
//
// Blocks are persistent per head: the two-term codebook is staged in LDS
// once, then each wave independently takes the block's next 32-point slice
// from a counter in LDS (so a wave slowed by a re-score does not hold up the
// others); chunk histograms for the grouping are accumulated with global
// atomics.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWavesPerBlock = 16;
constexpr int kUbfLds = 69632;            // two-term bf16 codebook elements in LDS
constexpr int kMaxCpad = 1024;
constexpr int kWaveCand = 64;             // candidate pairs per wave

__device__ __forceinline__ uint16_t to_bf16(float f) {
  bf16x2 r;
  r[0] = static_cast<__bf16>(f);
  r[1] = static_cast<__bf16>(0.0f);
  return static_cast<uint16_t>(__builtin_bit_cast(uint32_t, r) & 0xFFFFu);
}

// Channels c0 .. c0+7 of one bf16 row as four packed pairs, zero from dx on
// and for invalid rows.  A whole group is one 16-byte load when the rows are
// 16-byte aligned (vec), else four 4-byte loads (rows, ld, col0 and dx are
// even, so no pair straddles dx).
__device__ __forceinline__ uint4 load_group8(const uint16_t *xrow, int c0, int dx, bool valid, bool vec) {
  uint4 v = make_uint4(0, 0, 0, 0);
  if (vec && c0 + 8 <= dx) {
    if (valid) v = *reinterpret_cast<const uint4 *>(xrow + c0);
  } else {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = c0 + 2 * q;
      w[q] = valid && c < dx ? *reinterpret_cast<const uint32_t *>(xrow + c) : 0u;
    }
    v = make_uint4(w[0], w[1], w[2], w[3]);
  }
  return v;
}

// Canonical <x, u>: one fp32 fma per channel in ascending channel order, x
// in bf16 and u in fp32.  Both rows 16-byte aligned: eight channels per load
// step (the same chain), with the loads of four steps issued together; x
// 4-byte and u 8-byte aligned: two channels per step; then one at a time.
__device__ __forceinline__ float canon_dot(const uint16_t *xr, const float *u, int dx) {
  float dot = 0.0f;
  int c = 0;
  if (((reinterpret_cast<uintptr_t>(xr) | reinterpret_cast<uintptr_t>(u)) & 15) == 0) {
#pragma unroll 4
    for (; c + 8 <= dx; c += 8) {
      const uint4 xv = *reinterpret_cast<const uint4 *>(xr + c);
      const float4 u0 = *reinterpret_cast<const float4 *>(u + c);
      const float4 u1 = *reinterpret_cast<const float4 *>(u + c + 4);
      dot = fmaf(__uint_as_float(xv.x << 16), u0.x, dot);
      dot = fmaf(__uint_as_float(xv.x & 0xFFFF0000u), u0.y, dot);
      dot = fmaf(__uint_as_float(xv.y << 16), u0.z, dot);
      dot = fmaf(__uint_as_float(xv.y & 0xFFFF0000u), u0.w, dot);
      dot = fmaf(__uint_as_float(xv.z << 16), u1.x, dot);
      dot = fmaf(__uint_as_float(xv.z & 0xFFFF0000u), u1.y, dot);
      dot = fmaf(__uint_as_float(xv.w << 16), u1.z, dot);
      dot = fmaf(__uint_as_float(xv.w & 0xFFFF0000u), u1.w, dot);
    }
  }
  if (((reinterpret_cast<uintptr_t>(xr) & 3) | (reinterpret_cast<uintptr_t>(u) & 7)) == 0) {
#pragma unroll 4
    for (; c + 2 <= dx; c += 2) {
      const uint32_t xv = *reinterpret_cast<const uint32_t *>(xr + c);
      const float2 uv = *reinterpret_cast<const float2 *>(u + c);
      dot = fmaf(__uint_as_float(xv << 16), uv.x, dot);
      dot = fmaf(__uint_as_float(xv & 0xFFFF0000u), uv.y, dot);
    }
  }
  for (; c < dx; ++c) dot = fmaf(bf16_to_f32(xr[c]), u[c], dot);
  return dot;
}

// ascending-order key of a float score
__device__ __forceinline__ uint32_t asc_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Per pass: two-term bf16 codebook [cpad][2*DXP] (hi then lo, zero padded),
// canonical squared norms (FLT_MAX for padding rows, which never win), and
// per-row bound parts [cpad][2] = (|u - hi - lo|, max(|u|, |hi| + |lo|)),
// evaluated in fp64; the assignment kernel takes the per-head maxima.  One
// wave per row: lanes split the channels, lane 0 keeps the norm's fma chain
// in channel order.
template <int DXP>
__device__ __forceinline__ void km_prep_row(const float *__restrict__ U, size_t u_hs, int C,
                                            int cpad, int dx, uint16_t *ubf, float *nu,
                                            float *bnd) {
  const int h = blockIdx.y, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= cpad) return;
  uint16_t *dst = ubf + (static_cast<size_t>(h) * cpad + r) * (2 * DXP);
  const size_t row = static_cast<size_t>(h) * cpad + r;
  if (r >= C) {
    for (int c = lane; c < 2 * DXP; c += 64) dst[c] = 0;
    if (lane == 0) {
      nu[row] = 0x1.fffffep127f;
      bnd[2 * row + 0] = 0.0f;
      bnd[2 * row + 1] = 0.0f;
    }
    return;
  }
  const float *u = U + h * u_hs + static_cast<size_t>(r) * dx;
  double e2 = 0.0, n2 = 0.0, h2 = 0.0, l2 = 0.0;
  float xs[(DXP + 63) / 64];  // channel lane + 64 j of the row, 0 past dx
#pragma unroll
  for (int j = 0; j < (DXP + 63) / 64; ++j) {
    const int c = lane + 64 * j;
    xs[j] = c < dx ? u[c] : 0.0f;
  }
#pragma unroll
  for (int j = 0; j < (DXP + 63) / 64; ++j) {
    const int c = lane + 64 * j;
    if (c >= DXP) break;
    uint16_t bh = 0, bl = 0;
    if (c < dx) {
      const float x = xs[j];
      bh = to_bf16(x);
      const float rest = x - bf16_to_f32(bh);  // exact
      bl = to_bf16(rest);
      const double df = static_cast<double>(rest) - static_cast<double>(bf16_to_f32(bl));
      const double fh = bf16_to_f32(bh), fl = bf16_to_f32(bl);
      e2 += df * df;
      n2 += static_cast<double>(x) * static_cast<double>(x);
      h2 += fh * fh;
      l2 += fl * fl;
    }
    dst[c] = bh;
    dst[DXP + c] = bl;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    e2 += __shfl_xor(e2, o);
    n2 += __shfl_xor(n2, o);
    h2 += __shfl_xor(h2, o);
    l2 += __shfl_xor(l2, o);
  }
  // the canonical norm: one fma per channel in channel order, each channel
  // taken from the lane that loaded it
  float nr = 0.0f;
#pragma unroll
  for (int j = 0; j < (DXP + 63) / 64; ++j) {
    const int cend = dx - 64 * j < 64 ? dx - 64 * j : 64;
    for (int c = 0; c < cend; ++c) {
      const float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(xs[j]), c));
      nr = fmaf(v, v, nr);
    }
  }
  if (lane == 0) {
    nu[row] = nr;
    bnd[2 * row + 0] = static_cast<float>(sqrt(e2));
    bnd[2 * row + 1] = static_cast<float>(fmax(sqrt(n2), sqrt(h2) + sqrt(l2)));
  }
}

template <int DXP>
__global__ __launch_bounds__(256) void km_prep_kernel(
    const float *__restrict__ U, size_t u_hs, int C, int cpad, int dx,
    uint16_t *ubf, float *nu, float *bnd) {
  km_prep_row<DXP>(U, u_hs, C, cpad, dx, ubf, nu, bnd);
}

// The three subspaces' codebooks in one launch (blockIdx.z = subspace).
struct Prep3 {
  const float *U[3];
  size_t u_hs[3];
  int C[3], cpad[3], dx[3];
  uint16_t *ubf[3];
  float *nu[3], *bnd[3];
};

template <int D0, int D1, int D2>
__global__ __launch_bounds__(256) void km_prep3_kernel(Prep3 P) {
  const int m = blockIdx.z;
  if (m == 0)
    km_prep_row<D0>(P.U[0], P.u_hs[0], P.C[0], P.cpad[0], P.dx[0], P.ubf[0], P.nu[0], P.bnd[0]);
  else if (m == 1)
    km_prep_row<D1>(P.U[1], P.u_hs[1], P.C[1], P.cpad[1], P.dx[1], P.ubf[1], P.nu[1], P.bnd[1]);
  else
    km_prep_row<D2>(P.U[2], P.u_hs[2], P.C[2], P.cpad[2], P.dx[2], P.ubf[2], P.nu[2], P.bnd[2]);
}

// Keeps the compiler from moving this wave's LDS accesses across the call
// (the LDS completes one wave's operations in issue order).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The bound constants of one head's codebook (maxima of the per-row parts,
// with a small upward slack on top of their fp64 evaluation).
struct FilterBound {
  float E, Nmax, numax;
};

// The head's bound constants from the per-wave maxima in red.
template <int NW>
__device__ __forceinline__ FilterBound reduce_bound(const float (*red)[NW]) {
  float E = 0.0f, Nmax = 0.0f, numax = 0.0f;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    E = fmaxf(E, red[0][i]);
    Nmax = fmaxf(Nmax, red[1][i]);
    numax = fmaxf(numax, red[2][i]);
  }
  E = E * 1.001f + 1e-30f;
  Nmax *= 1.001f;
  numax *= 1.001f;
  return FilterBound{E, Nmax, numax};
}

// Stages head h's two-term codebook (16-byte pieces of each row; LDS row
// stride 2 DXP + 8), its norms and the accumulator start values -nu / 2
// into LDS and returns the head's bound constants.  Ends with a block
// barrier; the caller makes sure no wave still reads the previous contents.
template <int DXP, int NW = kWavesPerBlock>
__device__ __forceinline__ FilterBound stage_codebook(uint16_t *Us, float *nus, float *nhs,
                                                      float (*red)[NW],
                                                      const uint16_t *__restrict__ ubf,
                                                      const float *__restrict__ nu,
                                                      const float *__restrict__ bnd, int h,
                                                      int C, int cpad) {
  constexpr int US = 2 * DXP + 8;
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const uint16_t *ub = ubf + static_cast<size_t>(h) * cpad * (2 * DXP);
  for (int e = t; e < cpad * (DXP / 4); e += 64 * NW) {
    const int r = e / (DXP / 4), q = e % (DXP / 4);
    *reinterpret_cast<uint4 *>(&Us[r * US + 8 * q]) =
        *reinterpret_cast<const uint4 *>(ub + static_cast<size_t>(r) * (2 * DXP) + 8 * q);
  }
  // the head's bound constants: maxima of the per-row parts, with a small
  // upward slack on top of their fp64 evaluation
  float e_max = 0.0f, n_max = 0.0f, nu_max = 0.0f;
  for (int r = t; r < cpad; r += 64 * NW) {
    const size_t row = static_cast<size_t>(h) * cpad + r;
    const float v = nu[row];
    nus[r] = v;
    // exact for every norm at or above 2^-125 (smaller ones move by at most
    // 2^-150, far inside the margin); padding rows (nu = FLT_MAX) start at
    // -FLT_MAX / 2 and never win
    nhs[r] = -0.5f * v;
    if (r < C) {
      e_max = fmaxf(e_max, bnd[2 * row + 0]);
      n_max = fmaxf(n_max, bnd[2 * row + 1]);
      nu_max = fmaxf(nu_max, fabsf(v));
    }
  }
  e_max = wave_max(e_max);
  n_max = wave_max(n_max);
  nu_max = wave_max(nu_max);
  if (lane == 0) {
    red[0][w] = e_max;
    red[1][w] = n_max;
    red[2][w] = nu_max;
  }
  __syncthreads();
  return reduce_bound<NW>(red);
}

// One codebook's view of the rows: channels col0 .. col0+dx of X[h] (row
// stride ld), C centroids (padded to cpad) U[h] in fp32 for the canonical
// re-score, and where the assignment goes.
struct SliceArgs {
  const uint16_t *X;
  size_t x_hs;
  int ld, col0, dx, n, C, cpad;
  const float *U;
  size_t u_hs;
  int32_t *assign;
  size_t a_hs;
  int32_t *chunk_hist;
  int nchunks;
};

// The assignment of the 32 points of slice sl of head h by one wave, against
// the codebook staged in Us/nus/nhs with bound constants B (candidate
// scratch of this wave: cand, best, ncand).
template <int DXP>
__device__ __forceinline__ void assign_slice(const SliceArgs &A, const uint16_t *Us,
                                             const float *nus, const float *nhs, FilterBound B,
                                             int h, int sl,
                                             uint32_t *cand_w, unsigned long long *best_w,
                                             int *ncand_w) {
  constexpr int US = 2 * DXP + 8;  // LDS row stride of the two-term codebook
  constexpr int KS = DXP / 16;     // MFMA k-steps per term
  const int lane = threadIdx.x & 63, l32 = lane & 31, hf = lane >> 5;
  const uint16_t *X = A.X;
  const size_t x_hs = A.x_hs;
  const int ld = A.ld, col0 = A.col0, dx = A.dx, n = A.n, C = A.C, cpad = A.cpad;
  int32_t *assign = A.assign;
  const size_t a_hs = A.a_hs;
  int32_t *chunk_hist = A.chunk_hist;
  const int nchunks = A.nchunks;
  const float E = B.E, Nmax = B.Nmax, numax = B.numax;
  const float kappa = 8.0f * DXP * 0x1p-24f;
  // index bits packed into the low mantissa of the scores
  const int ib = 32 - __clz(cpad - 1);
  const uint32_t imask = (1u << ib) - 1u;
  const float dpack = __uint_as_float(static_cast<uint32_t>(127 + ib - 23) << 23);  // 2^(ib-23)
  // every row's first channel is 16-byte aligned
  const bool vec = ((reinterpret_cast<uintptr_t>(X + col0) & 15) | ((x_hs | static_cast<size_t>(ld)) & 7)) == 0;
  const float *Uh = A.U + h * A.u_hs;
  const int i = sl * 32 + l32;
  const bool valid = i < n;
  const uint16_t *xrow = X + h * x_hs + static_cast<size_t>(valid ? i : 0) * ld + col0;
  bf16x8 xf[KS];
  float ss = 0.0f;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const uint4 v4 = load_group8(xrow, 16 * s + 8 * hf, dx, valid, vec);
    const uint32_t wv[4] = {v4.x, v4.y, v4.z, v4.w};
    // |x|^2 only sizes the margin: two squares per dot2 (each rounding
    // within 2^-23 relative, far inside the 1e-4 slack below)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bf16x2 p2 = __builtin_bit_cast(bf16x2, wv[q]);
      ss = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, ss, false);
    }
    xf[s] = __builtin_bit_cast(bf16x8, v4);
  }
  ss += __shfl_xor(ss, 32);
  const float nx = sqrtf(ss) * 1.0001f + 1e-30f;
  const float beta = (2.0f * nx * (E + kappa * Nmax) +
                      0x1p-23f * ((2.0f * DXP + 1.0f) * numax + 2.02f * nx * Nmax)) * 1.01f + 1e-25f;

  // a_r of the 32 centroids rb .. rb+31 for the 32 points: the accumulator
  // starts at -nu_r / 2 (lane holds rows rb + 8(e/4) + 4hf + e%4)
  auto chain = [&](int rb) {
    f32x16 acc;
    const float *nh = nhs + rb + 4 * hf;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 v = *reinterpret_cast<const float4 *>(nh + 8 * q);
      acc[4 * q + 0] = v.x;
      acc[4 * q + 1] = v.y;
      acc[4 * q + 2] = v.z;
      acc[4 * q + 3] = v.w;
    }
    const uint16_t *urow = &Us[(rb + l32) * US + 8 * hf];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 a_hi = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(urow + 16 * s));
      const bf16x8 a_lo = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(urow + DXP + 16 * s));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_hi, xf[s], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_lo, xf[s], acc, 0, 0, 0);
    }
    return acc;
  };
  // one pass: the three largest packed values per point (each med3 keeps
  // the larger two of its inputs' lower pair; the start value lies below
  // every value of valid inputs).  The index packed here leaves out the
  // lane's 4 hf, which is the same for all of the lane's values (so their
  // order is that of the full index) and is added once after the pass.
  // The mask stays in a vector register so that the index, uniform across
  // the wave, can come from a scalar register.
  uint32_t vmask;
  asm volatile("v_mov_b32 %0, %1" : "=v"(vmask) : "s"(~imask));
  float m1 = -0x1.1p127f, m2 = -0x1.1p127f, m3 = -0x1.1p127f;
  auto fold = [&](const f32x16 &acc, int rb) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint32_t ru = static_cast<uint32_t>(
          __builtin_amdgcn_readfirstlane(rb + 8 * (e >> 2) + (e & 3)));
      const float sp = __uint_as_float((__float_as_uint(acc[e]) & vmask) | ru);
      m3 = __builtin_amdgcn_fmed3f(m2, m3, sp);
      m2 = __builtin_amdgcn_fmed3f(m1, m2, sp);
      m1 = __builtin_amdgcn_fmed3f(m1, sp, 0x1.1p127f);  // max without NaN quieting
    }
  };
  // software pipeline: the values of one block are folded while the MFMAs
  // of the next run; two accumulators alternate, so no copies
  f32x16 acc0 = chain(0), acc1;
  int rb = 32;
  for (; rb + 32 < cpad; rb += 64) {
    acc1 = chain(rb);
    fold(acc0, rb - 32);
    acc0 = chain(rb + 32);
    fold(acc1, rb);
  }
  if (rb < cpad) {
    acc1 = chain(rb);
    fold(acc0, rb - 32);
    fold(acc1, rb);
  } else {
    fold(acc0, rb - 32);
  }
  {
    const uint32_t add = 4u * static_cast<uint32_t>(hf);
    m1 = __uint_as_float(__float_as_uint(m1) + add);
    m2 = __uint_as_float(__float_as_uint(m2) + add);
    m3 = __uint_as_float(__float_as_uint(m3) + add);
    // the other half-wave's three into this one's (same multiset, same
    // result in both halves)
    const float o[3] = {__shfl_xor(m1, 32), __shfl_xor(m2, 32), __shfl_xor(m3, 32)};
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      m3 = __builtin_amdgcn_fmed3f(m2, m3, o[q]);
      m2 = __builtin_amdgcn_fmed3f(m1, m2, o[q]);
      m1 = __builtin_amdgcn_fmed3f(m1, o[q], 0x1.1p127f);
    }
  }
  // candidates: a_r >= max a - beta (halved scale: 2 x beta / 2), less the
  // two packing perturbations
  const float slack = (beta + 2.0f * dpack * fabsf(m1)) * 1.001f;
  const float lim = m1 - slack;
  const float thr = lim - fabsf(lim) * 2e-6f - 1e-30f;
  const bool needy = valid && !(m2 < thr);
  // three or more candidates (very rare)
  const bool wide = needy && !(m3 < thr);
  int arg = static_cast<int>(__float_as_uint(m1) & imask);

  if (__ballot(needy && !wide)) {
    // exactly two candidates, the two largest packed values: the point's
    // two half-wave lanes re-score one each canonically and exchange
    unsigned long long key = ~0ull;
    if (needy && !wide) {
      const int r = min(static_cast<int>(__float_as_uint(hf ? m2 : m1) & imask), C - 1);
      const uint16_t *xr = X + h * x_hs + static_cast<size_t>(i) * ld + col0;
      const float dot = canon_dot(xr, Uh + static_cast<size_t>(r) * dx, dx);
      const float sc = fmaf(-2.0f, dot, nus[r]) + 0.0f;
      key = (static_cast<unsigned long long>(asc_key(sc)) << 32) | static_cast<unsigned>(r);
    }
    const uint32_t ok_lo = __shfl_xor(static_cast<uint32_t>(key), 32);
    const uint32_t ok_hi = __shfl_xor(static_cast<uint32_t>(key >> 32), 32);
    const unsigned long long other = (static_cast<unsigned long long>(ok_hi) << 32) | ok_lo;
    if (needy && !wide) arg = static_cast<int>((key < other ? key : other) & 0xFFFFFFFFu);
  }
  if (__ballot(wide)) {
    // every candidate of the wide points, re-scored canonically
    wave_sync();
    if (lane == 0) *ncand_w = 0;
    if (lane < 32) best_w[lane] = ~0ull;
    wave_sync();
    bool over = false;
    for (int rb = 0; rb < cpad; rb += 32) {
      const f32x16 acc = chain(rb);
      if (wide) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const uint32_t r = static_cast<uint32_t>(rb + 8 * (e >> 2) + 4 * hf + (e & 3));
          const float sp = __uint_as_float((__float_as_uint(acc[e]) & ~imask) | r);
          if (static_cast<int>(r) < C && sp >= thr) {
            const int slot = atomicAdd(ncand_w, 1);
            if (slot < kWaveCand)
              cand_w[slot] = (static_cast<uint32_t>(l32) << 16) | r;
            else
              over = true;
          }
        }
      }
    }
    // a point whose candidates did not fit scans every centroid
    const bool full = __shfl_xor(static_cast<int>(over), 32) || over;
    wave_sync();
    const int cnt = min(*ncand_w, kWaveCand);
    for (int k = lane; k < cnt; k += 64) {
      const uint32_t pr = cand_w[k];
      const int q = static_cast<int>(pr >> 16), r = static_cast<int>(pr & 0xFFFFu);
      const uint16_t *xr = X + h * x_hs + static_cast<size_t>(sl * 32 + q) * ld + col0;
      const float *u = Uh + static_cast<size_t>(r) * dx;
      const float dot = canon_dot(xr, u, dx);
      const float sc = fmaf(-2.0f, dot, nus[r]) + 0.0f;
      atomicMin(&best_w[q], (static_cast<unsigned long long>(asc_key(sc)) << 32) | static_cast<unsigned>(r));
    }
    wave_sync();
    if (wide && hf == 0) {
      unsigned long long b = best_w[l32];
      if (full) {
        const uint16_t *xr = X + h * x_hs + static_cast<size_t>(i) * ld + col0;
        b = ~0ull;
        for (int r = 0; r < C; ++r) {
          const float *u = Uh + static_cast<size_t>(r) * dx;
          const float dot = canon_dot(xr, u, dx);
          const float sc = fmaf(-2.0f, dot, nus[r]) + 0.0f;
          const unsigned long long key = (static_cast<unsigned long long>(asc_key(sc)) << 32) | static_cast<unsigned>(r);
          b = key < b ? key : b;
        }
      }
      arg = b == ~0ull ? 0 : static_cast<int>(b & 0xFFFFFFFFu);
    }
    arg = __shfl(arg, l32);  // the lower half-wave holds the result
  }
  if (valid && hf == 0) {
    arg = min(max(arg, 0), C - 1);
    assign[h * a_hs + i] = arg;
    if (chunk_hist)
      atomicAdd(&chunk_hist[(static_cast<size_t>(h) * nchunks + (i / kAssignBlock)) * C + arg], 1);
  }
}

template <int DXP>
__global__ __launch_bounds__(64 * kWavesPerBlock) void km_assign_mfma_kernel(
    const uint16_t *__restrict__ X, size_t x_hs, int ld, int col0, int dx,
    int n, int heads, const float *__restrict__ U, size_t u_hs,
    const uint16_t *__restrict__ ubf, const float *__restrict__ nu,
    const float *__restrict__ bnd, int C, int cpad, int32_t *assign,
    size_t a_hs, int32_t *chunk_hist, int nchunks) {
  __shared__ __attribute__((aligned(16))) uint16_t Us[kUbfLds];
  __shared__ __attribute__((aligned(16))) float nus[kMaxCpad];
  __shared__ __attribute__((aligned(16))) float nhs[kMaxCpad];
  __shared__ uint32_t cand[kWavesPerBlock][kWaveCand];
  __shared__ unsigned long long best[kWavesPerBlock][32];
  __shared__ int ncand[kWavesPerBlock];
  __shared__ float red[3][kWavesPerBlock];
  __shared__ int next_slice;
  const int w = threadIdx.x >> 6;
  const SliceArgs A{X, x_hs, ld, col0, dx, n, C, cpad, U, u_hs, assign, a_hs, chunk_hist, nchunks};
  const int nslices = (n + 31) / 32;

  // this block's contiguous range of (head, slice) pairs
  const long long total = static_cast<long long>(heads) * nslices;
  const long long per = (total + gridDim.x - 1) / gridDim.x;
  long long beg = static_cast<long long>(blockIdx.x) * per;
  const long long end = beg + per < total ? beg + per : total;
  while (beg < end) {
    const int h = static_cast<int>(beg / nslices);
    const long long seg_end = end < static_cast<long long>(h + 1) * nslices
                                  ? end : static_cast<long long>(h + 1) * nslices;
    __syncthreads();
    if (threadIdx.x == 0) next_slice = 0;  // visible after the staging barrier
    const FilterBound B = stage_codebook<DXP>(Us, nus, nhs, red, ubf, nu, bnd, h, C, cpad);
    // a wave that is done takes the block's next slice
    const long long count = seg_end - beg;
    for (;;) {
      int u = 0;
      if ((threadIdx.x & 63) == 0) u = atomicAdd(&next_slice, 1);
      u = __builtin_amdgcn_readfirstlane(__shfl(u, 0));
      if (u >= count) break;
      const long long g = beg + u;
      assign_slice<DXP>(A, Us, nus, nhs, B, h, static_cast<int>(g - static_cast<long long>(h) * nslices),
                        cand[w], best[w], &ncand[w]);
    }
    beg = seg_end;
  }
}

// The three key subspaces in one pass over the rows: their codebooks are
// staged in LDS side by side (subspace m at element offset uoff[m] and norm
// offset noff[m]), and the block's waves take work units (slice, subspace)
// from a counter in LDS, in slice order.  A wave that is done takes the next
// unit whatever its subspace, so the subspaces' different costs balance
// out, and the three units of a slice start at about the same time, so a
// row fetched from HBM for one is found in cache by the others.
struct Sub3 {
  SliceArgs a[3];
  const uint16_t *ubf[3];
  const float *nu[3];
  const float *bnd[3];
  int uoff[3], noff[3];
};

template <int D0, int D1, int D2>
__global__ __launch_bounds__(64 * kWavesPerBlock) void km_assign_mfma3_kernel(
    const Sub3 *__restrict__ Sp, int n, int heads) {
  __shared__ __attribute__((aligned(16))) uint16_t Us[kUbfLds];
  __shared__ __attribute__((aligned(16))) float nus[kMaxCpad];
  __shared__ __attribute__((aligned(16))) float nhs[kMaxCpad];
  __shared__ uint32_t cand[kWavesPerBlock][kWaveCand];
  __shared__ unsigned long long best[kWavesPerBlock][32];
  __shared__ int ncand[kWavesPerBlock];
  __shared__ float red[3][3][kWavesPerBlock];
  __shared__ int next_unit;
  const int w = threadIdx.x >> 6;
  const int nslices = (n + 31) / 32;
  const long long total = static_cast<long long>(heads) * nslices;
  const long long per = (total + gridDim.x - 1) / gridDim.x;
  long long beg = static_cast<long long>(blockIdx.x) * per;
  const long long end = beg + per < total ? beg + per : total;
  while (beg < end) {
    const int h = static_cast<int>(beg / nslices);
    const long long seg_end = end < static_cast<long long>(h + 1) * nslices
                                  ? end : static_cast<long long>(h + 1) * nslices;
    __syncthreads();
    if (threadIdx.x == 0) next_unit = 0;  // visible after the staging barriers
    stage_codebook<D0>(Us + Sp->uoff[0], nus + Sp->noff[0], nhs + Sp->noff[0], red[0], Sp->ubf[0], Sp->nu[0],
                       Sp->bnd[0], h, Sp->a[0].C, Sp->a[0].cpad);
    stage_codebook<D1>(Us + Sp->uoff[1], nus + Sp->noff[1], nhs + Sp->noff[1], red[1], Sp->ubf[1], Sp->nu[1],
                       Sp->bnd[1], h, Sp->a[1].C, Sp->a[1].cpad);
    stage_codebook<D2>(Us + Sp->uoff[2], nus + Sp->noff[2], nhs + Sp->noff[2], red[2], Sp->ubf[2], Sp->nu[2],
                       Sp->bnd[2], h, Sp->a[2].C, Sp->a[2].cpad);
    const long long first = static_cast<long long>(h) * nslices;
    const FilterBound B0 = reduce_bound<kWavesPerBlock>(red[0]);
    const FilterBound B1 = reduce_bound<kWavesPerBlock>(red[1]);
    const FilterBound B2 = reduce_bound<kWavesPerBlock>(red[2]);
    const long long units = 3 * (seg_end - beg);
    for (;;) {
      int u = 0;
      if ((threadIdx.x & 63) == 0) u = atomicAdd(&next_unit, 1);
      u = __builtin_amdgcn_readfirstlane(__shfl(u, 0));
      if (u >= units) break;
      const long long g = beg + u / 3;
      const int m = u - 3 * (u / 3);
      if (m == 0)
        assign_slice<D0>(Sp->a[0], Us + Sp->uoff[0], nus + Sp->noff[0], nhs + Sp->noff[0], B0, h,
                         static_cast<int>(g - first), cand[w], best[w], &ncand[w]);
      else if (m == 1)
        assign_slice<D1>(Sp->a[1], Us + Sp->uoff[1], nus + Sp->noff[1], nhs + Sp->noff[1], B1, h,
                         static_cast<int>(g - first), cand[w], best[w], &ncand[w]);
      else
        assign_slice<D2>(Sp->a[2], Us + Sp->uoff[2], nus + Sp->noff[2], nhs + Sp->noff[2], B2, h,
                         static_cast<int>(g - first), cand[w], best[w], &ncand[w]);
    }
    beg = seg_end;
  }
}

// Codebooks larger than the LDS holds (e.g. 300 centroids at d = 128) are
// cut into chunks of at most CR rows, and every chunk gets its own
// persistent blocks, which keep the chunk in LDS for their whole range of
// slices (waves run independently, as above).  Per point, each chunk yields
// its four smallest packed scores (indices over the whole codebook), and
// chunk 0 also the point's norm bound.  The decision kernel below merges the
// lists, one point per thread.
template <int DXP>
__global__ __launch_bounds__(64 * kWavesPerBlock) void km_assign_mfma_part_kernel(
    const uint16_t *__restrict__ X, size_t x_hs, int ld, int col0, int dx,
    int n, int heads, const uint16_t *__restrict__ ubf, const float *__restrict__ nu,
    int cpad, int crows, float *part, float *pnx) {
  constexpr int US = 2 * DXP + 8;  // LDS row stride of the two-term codebook
  constexpr int KS = DXP / 16;     // MFMA k-steps per term
  __shared__ __attribute__((aligned(16))) uint16_t Us[kUbfLds];
  __shared__ float nus[kMaxCpad];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6, l32 = lane & 31, hf = lane >> 5;
  const int chunk = blockIdx.y, r0 = chunk * crows;
  const int rows = cpad - r0 < crows ? cpad - r0 : crows;  // a multiple of 32
  const int ib = 32 - __clz(cpad - 1);
  const uint32_t imask = (1u << ib) - 1u;
  const int nslices = (n + 31) / 32;
  // every row's first channel is 16-byte aligned
  const bool vec = ((reinterpret_cast<uintptr_t>(X + col0) & 15) | ((x_hs | static_cast<size_t>(ld)) & 7)) == 0;

  const long long total = static_cast<long long>(heads) * nslices;
  const long long per = (total + gridDim.x - 1) / gridDim.x;
  long long beg = static_cast<long long>(blockIdx.x) * per;
  const long long end = beg + per < total ? beg + per : total;
  while (beg < end) {
    const int h = static_cast<int>(beg / nslices);
    const long long seg_end = end < static_cast<long long>(h + 1) * nslices
                                  ? end : static_cast<long long>(h + 1) * nslices;
    // stage this head's chunk (rows r0 .. r0+rows) and its norms
    __syncthreads();
    const uint16_t *ub = ubf + (static_cast<size_t>(h) * cpad + r0) * (2 * DXP);
    for (int e = t; e < rows * (DXP / 4); e += 64 * kWavesPerBlock) {
      const int r = e / (DXP / 4), q = e % (DXP / 4);
      *reinterpret_cast<uint4 *>(&Us[r * US + 8 * q]) =
          *reinterpret_cast<const uint4 *>(ub + static_cast<size_t>(r) * (2 * DXP) + 8 * q);
    }
    for (int r = t; r < rows; r += 64 * kWavesPerBlock)
      nus[r] = nu[static_cast<size_t>(h) * cpad + r0 + r];
    __syncthreads();
    for (long long g = beg + w; g < seg_end; g += kWavesPerBlock) {
      const int sl = static_cast<int>(g - static_cast<long long>(h) * nslices);
      const int i = sl * 32 + l32;
      const bool valid = i < n;
      const uint16_t *xrow = X + h * x_hs + static_cast<size_t>(valid ? i : 0) * ld + col0;
      bf16x8 xf[KS];
      float ss = 0.0f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const uint4 v4 = load_group8(xrow, 16 * s + 8 * hf, dx, valid, vec);
        const uint32_t wv[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float a = __uint_as_float(wv[q] << 16), b = __uint_as_float(wv[q] & 0xFFFF0000u);
          ss = fmaf(a, a, ss);
          ss = fmaf(b, b, ss);
        }
        xf[s] = __builtin_bit_cast(bf16x8, v4);
      }
      ss += __shfl_xor(ss, 32);

      auto chain = [&](int rb) {  // rb: row within the chunk
        f32x16 acc;
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
        const uint16_t *urow = &Us[(rb + l32) * US + 8 * hf];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const bf16x8 a_hi = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(urow + 16 * s));
          const bf16x8 a_lo = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(urow + DXP + 16 * s));
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_hi, xf[s], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_lo, xf[s], acc, 0, 0, 0);
        }
        return acc;
      };
      // the four smallest packed scores, m1 <= m2 <= m3 <= m4
      float m1 = 0x1.1p127f, m2 = 0x1.1p127f, m3 = 0x1.1p127f, m4 = 0x1.1p127f;
      auto insert = [&](float sp) {
        m4 = __builtin_amdgcn_fmed3f(m3, m4, sp);
        m3 = __builtin_amdgcn_fmed3f(m2, m3, sp);
        m2 = __builtin_amdgcn_fmed3f(m1, m2, sp);
        m1 = fminf(m1, sp);
      };
      auto fold = [&](const f32x16 &acc, int rb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int rl = rb + 8 * (e >> 2) + 4 * hf + (e & 3);
          const float sc = fmaf(-2.0f, acc[e], nus[rl]);
          insert(__uint_as_float((__float_as_uint(sc) & ~imask) | static_cast<uint32_t>(r0 + rl)));
        }
      };
      f32x16 prev = chain(0);
      for (int rb = 32; rb < rows; rb += 32) {
        const f32x16 cur = chain(rb);
        fold(prev, rb - 32);
        prev = cur;
      }
      fold(prev, rows - 32);
      {  // the two half-waves saw disjoint centroids of the same points
        const float o1 = __shfl_xor(m1, 32), o2 = __shfl_xor(m2, 32);
        const float o3 = __shfl_xor(m3, 32), o4 = __shfl_xor(m4, 32);
        insert(o1);
        insert(o2);
        insert(o3);
        insert(o4);
      }
      if (valid && hf == 0) {
        *reinterpret_cast<float4 *>(part + ((static_cast<size_t>(chunk) * heads + h) * n + i) * 4) =
            make_float4(m1, m2, m3, m4);
        if (chunk == 0) pnx[static_cast<size_t>(h) * n + i] = sqrtf(ss) * 1.0001f + 1e-30f;
      }
    }
    beg = seg_end;
  }
}

// The decision for chunked codebooks, one point per thread: the chunks'
// lists merged into the four smallest packed scores, then the margin of the
// kernel above; with a runner-up inside it, the fourth score bounds the
// candidates to at most three, re-scored canonically, and only four or more
// candidates scan every centroid canonically.
__global__ __launch_bounds__(256) void km_assign_decide_kernel(
    const uint16_t *__restrict__ X, size_t x_hs, int ld, int col0, int dx, int n,
    int heads, const float *__restrict__ U, size_t u_hs, const float *__restrict__ nu,
    const float *__restrict__ bnd, int C, int cpad, int nparts,
    const float *__restrict__ part, const float *__restrict__ pnx, float kappa,
    int32_t *assign, size_t a_hs, int32_t *chunk_hist, int nchunks) {
  __shared__ float red[3][4];
  const int h = blockIdx.y, t = threadIdx.x, lane = t & 63, w = t >> 6;
  // the head's bound constants, as in the assignment kernel
  float e_max = 0.0f, n_max = 0.0f, nu_max = 0.0f;
  for (int r = t; r < C; r += 256) {
    const size_t row = static_cast<size_t>(h) * cpad + r;
    e_max = fmaxf(e_max, bnd[2 * row + 0]);
    n_max = fmaxf(n_max, bnd[2 * row + 1]);
    nu_max = fmaxf(nu_max, fabsf(nu[row]));
  }
  e_max = wave_max(e_max);
  n_max = wave_max(n_max);
  nu_max = wave_max(nu_max);
  if (lane == 0) {
    red[0][w] = e_max;
    red[1][w] = n_max;
    red[2][w] = nu_max;
  }
  __syncthreads();
  const float E = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3])) * 1.001f + 1e-30f;
  const float Nmax = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3])) * 1.001f;
  const float numax = fmaxf(fmaxf(red[2][0], red[2][1]), fmaxf(red[2][2], red[2][3])) * 1.001f;
  const int i = blockIdx.x * 256 + t;
  if (i >= n) return;
  const int ib = 32 - __clz(cpad - 1);
  const uint32_t imask = (1u << ib) - 1u;
  const float dpack = __uint_as_float(static_cast<uint32_t>(127 + ib - 23) << 23);
  float m1 = 0x1.1p127f, m2 = 0x1.1p127f, m3 = 0x1.1p127f, m4 = 0x1.1p127f;
  auto insert = [&](float sp) {
    m4 = __builtin_amdgcn_fmed3f(m3, m4, sp);
    m3 = __builtin_amdgcn_fmed3f(m2, m3, sp);
    m2 = __builtin_amdgcn_fmed3f(m1, m2, sp);
    m1 = fminf(m1, sp);
  };
  for (int k = 0; k < nparts; ++k) {
    const float4 v = *reinterpret_cast<const float4 *>(
        part + ((static_cast<size_t>(k) * heads + h) * n + i) * 4);
    insert(v.x);
    insert(v.y);
    insert(v.z);
    insert(v.w);
  }
  const float nx = pnx[static_cast<size_t>(h) * n + i];
  const float beta = (2.0f * nx * (E + kappa * Nmax) +
                      0x1p-23f * (numax + 2.02f * nx * Nmax)) * 1.01f + 1e-25f;
  const float slack = (2.0f * beta + 2.0f * dpack * fabsf(m1)) * 1.001f;
  const float lim = m1 + slack;
  const float thr = lim + fabsf(lim) * 2e-6f + 1e-30f;
  int arg = static_cast<int>(__float_as_uint(m1) & imask);
  if (!(m2 > thr)) {
    const uint16_t *xr = X + h * x_hs + static_cast<size_t>(i) * ld + col0;
    const float *Uh = U + h * u_hs;
    unsigned long long b = ~0ull;
    auto rescore = [&](int r) {
      r = min(r, C - 1);
      const float *u = Uh + static_cast<size_t>(r) * dx;
      const float dot = canon_dot(xr, u, dx);
      const float sc = fmaf(-2.0f, dot, nu[static_cast<size_t>(h) * cpad + r]) + 0.0f;
      const unsigned long long key =
          (static_cast<unsigned long long>(asc_key(sc)) << 32) | static_cast<unsigned>(r);
      b = key < b ? key : b;
    };
    if (m4 > thr) {
      // every candidate is among the three smallest
      rescore(arg);
      rescore(static_cast<int>(__float_as_uint(m2) & imask));
      if (m3 <= thr) rescore(static_cast<int>(__float_as_uint(m3) & imask));
    } else {
      for (int r = 0; r < C; ++r) rescore(r);
    }
    arg = static_cast<int>(b & 0xFFFFFFFFu);
  }
  arg = min(max(arg, 0), C - 1);
  assign[h * a_hs + i] = arg;
  if (chunk_hist)
    atomicAdd(&chunk_hist[(static_cast<size_t>(h) * nchunks + (i / kAssignBlock)) * C + arg], 1);
}

__global__ void km_zero_kernel(int32_t *p, size_t count) {
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    p[i] = 0;
}

template <int DXP>
hipError_t launch_mfma(const KmProblem &p, bool with_hist, hipStream_t s) {
  hipLaunchKernelGGL(km_prep_kernel<DXP>, dim3((p.cpad + 3) / 4, p.heads), dim3(256), 0, s, p.u,
                     p.u_head_stride, p.C, p.cpad, p.dx, p.ubf, p.nu, p.bnd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nch = km_nchunks(p.n);
  if (with_hist) {
    const size_t cnt = static_cast<size_t>(p.heads) * nch * p.C;
    hipLaunchKernelGGL(km_zero_kernel, dim3(static_cast<unsigned>((cnt + 255) / 256 < 4096 ? (cnt + 255) / 256 : 4096)),
                       dim3(256), 0, s, p.chunk_hist, cnt);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // persistent blocks, one per CU (the codebook fills most of the LDS),
  // each over a contiguous range of (head, 32-point slice) pairs
  const long long slices = static_cast<long long>(p.heads) * ((p.n + 31) / 32);
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  const int blocks = static_cast<int>(slices < static_cast<long long>(cus) * kWavesPerBlock
                                          ? (slices + kWavesPerBlock - 1) / kWavesPerBlock : cus);
  const uint16_t *x = static_cast<const uint16_t *>(p.x);
  if (p.cpad * (2 * DXP + 8) <= kUbfLds) {
    hipLaunchKernelGGL(km_assign_mfma_kernel<DXP>, dim3(blocks), dim3(64 * kWavesPerBlock), 0, s,
                       x, p.x_head_stride, p.ld, p.col0, p.dx, p.n, p.heads, p.u,
                       p.u_head_stride, p.ubf, p.nu, p.bnd, p.C, p.cpad, p.assign,
                       p.a_head_stride, with_hist ? p.chunk_hist : nullptr, nch);
    return hipGetLastError();
  }
  // chunked codebook: balanced chunks, the CUs shared among them
  const int nparts = km_parts(p.C, p.dx);
  const int crows = (p.cpad / 32 + nparts - 1) / nparts * 32;
  const int per_part = cus / nparts > 1 ? cus / nparts : 1;
  const long long need = (slices + kWavesPerBlock - 1) / kWavesPerBlock;
  const int bpp = static_cast<int>(need < per_part ? need : per_part);
  hipLaunchKernelGGL(km_assign_mfma_part_kernel<DXP>, dim3(bpp, nparts),
                     dim3(64 * kWavesPerBlock), 0, s, x, p.x_head_stride, p.ld, p.col0, p.dx,
                     p.n, p.heads, p.ubf, p.nu, p.cpad, crows, p.part, p.pnx);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(km_assign_decide_kernel, dim3((p.n + 255) / 256, p.heads), dim3(256), 0,
                     s, x, p.x_head_stride, p.ld, p.col0, p.dx, p.n, p.heads, p.u,
                     p.u_head_stride, p.nu, p.bnd, p.C, p.cpad, nparts, p.part, p.pnx,
                     8.0f * DXP * 0x1p-24f, p.assign, p.a_head_stride,
                     with_hist ? p.chunk_hist : nullptr, nch);
  return hipGetLastError();
}

__global__ void store_sub3_kernel(Sub3 S, Sub3 *dst) { *dst = S; }

template <int D0, int D1, int D2>
hipError_t launch_mfma3(const KmProblem (&p)[3], Sub3 *dev_args, bool store_args,
                        hipStream_t s) {
  // the three codebooks' two-term splits, norms and bound parts
  Prep3 P{};
  int cmax = 0;
  for (int m = 0; m < 3; ++m) {
    P.U[m] = p[m].u;
    P.u_hs[m] = p[m].u_head_stride;
    P.C[m] = p[m].C;
    P.cpad[m] = p[m].cpad;
    P.dx[m] = p[m].dx;
    P.ubf[m] = p[m].ubf;
    P.nu[m] = p[m].nu;
    P.bnd[m] = p[m].bnd;
    cmax = p[m].cpad > cmax ? p[m].cpad : cmax;
  }
  hipLaunchKernelGGL((km_prep3_kernel<D0, D1, D2>), dim3((cmax + 3) / 4, p[0].heads, 3),
                     dim3(256), 0, s, P);
  hipError_t e0 = hipGetLastError();
  if (e0 != hipSuccess) return e0;
  Sub3 S{};
  int uoff = 0, noff = 0;
  const int dxp[3] = {D0, D1, D2};
  for (int m = 0; m < 3; ++m) {
    const KmProblem &q = p[m];
    S.a[m] = SliceArgs{static_cast<const uint16_t *>(q.x), q.x_head_stride, q.ld, q.col0, q.dx,
                       q.n, q.C, q.cpad, q.u, q.u_head_stride, q.assign, q.a_head_stride,
                       nullptr, 0};
    S.ubf[m] = q.ubf;
    S.nu[m] = q.nu;
    S.bnd[m] = q.bnd;
    S.uoff[m] = uoff;
    S.noff[m] = noff;
    uoff += q.cpad * (2 * dxp[m] + 8);
    noff += q.cpad;
  }
  const long long slices = static_cast<long long>(p[0].heads) * ((p[0].n + 31) / 32);
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  const int blocks = static_cast<int>(slices < static_cast<long long>(cus) * kWavesPerBlock
                                          ? (slices + kWavesPerBlock - 1) / kWavesPerBlock : cus);
  // the arguments go to device memory, so each wave group loads only its
  // own; they hold only pointers and sizes, so one store per call suffices
  if (store_args) {
    hipLaunchKernelGGL(store_sub3_kernel, dim3(1), dim3(1), 0, s, S, dev_args);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((km_assign_mfma3_kernel<D0, D1, D2>), dim3(blocks), dim3(64 * kWavesPerBlock),
                     0, s, dev_args, p[0].n, p[0].heads);
  return hipGetLastError();
}

}  // namespace

bool km_assign3_ok(const KmProblem (&p)[3]) {
  int lds = 0, rows = 0;
  for (int m = 0; m < 3; ++m) {
    const KmProblem &q = p[m];
    if (!q.mfma || q.x != p[0].x || q.ld != p[0].ld || q.n != p[0].n ||
        q.heads != p[0].heads || q.x_head_stride != p[0].x_head_stride)
      return false;
    lds += q.cpad * (2 * q.dxp + 8);
    rows += q.cpad;
  }
  if (lds > kUbfLds || rows > kMaxCpad) return false;
  const int a = p[0].dxp, b = p[1].dxp, c = p[2].dxp;
  return (a == 16 && b == 64 && c == 64) || (a == 48 && b == 48 && c == 48) ||
         (a == 16 && b == 32 && c == 32);
}

size_t km_assign3_scratch_bytes() { return sizeof(Sub3); }

hipError_t km_assign3(const KmProblem (&p)[3], void *scratch, bool store_args,
                      hipStream_t s) {
  Sub3 *args = static_cast<Sub3 *>(scratch);
  const int a = p[0].dxp, b = p[1].dxp;
  if (a == 16 && b == 64) return launch_mfma3<16, 64, 64>(p, args, store_args, s);
  if (a == 48) return launch_mfma3<48, 48, 48>(p, args, store_args, s);
  return launch_mfma3<16, 32, 32>(p, args, store_args, s);
}

int km_cpad(int C) { return (C + 31) / 32 * 32; }
int km_dxp(int dx) { return dx <= 16 ? 16 : dx <= 32 ? 32 : dx <= 48 ? 48 : dx <= 64 ? 64 : 128; }

// Chunks of a codebook beyond the LDS (1 when it fits).
int km_parts(int C, int dx) {
  const int rows_max = kUbfLds / (2 * km_dxp(dx) + 8) / 32 * 32;
  return (km_cpad(C) + rows_max - 1) / rows_max;
}

size_t km_split_floats(int C, int dx, int heads, int n) {
  const int parts = km_parts(C, dx);
  if (parts <= 1) return 0;
  return static_cast<size_t>(heads) * n * (4 * static_cast<size_t>(parts) + 1);
}

// Codebooks beyond the LDS are split in chunks across blocks.
bool km_mfma_ok(bool bf16, int ld, int col0, int dx, int C) {
  if (!bf16 || (ld & 1) || (col0 & 1) || (dx & 1) || dx > 128) return false;
  return km_cpad(C) <= kMaxCpad;
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
