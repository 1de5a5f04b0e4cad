// Device-side helpers shared by the SCOPE kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/scope.h"

// Every kernel translation unit is compiled with -ffp-contract=off: the
// canonical arithmetic of the clustering, scoring and selection stages is
// spelled out with explicit fmaf, and nothing else may be fused.

namespace scope {

constexpr int kWave = 64;

// Status bits OR-ed into the optional device word.
constexpr int kStatusNonFinite = 1;
constexpr int kStatusRange = 2;
constexpr int kStatusBadInit = 4;

// Element loads: bf16 storage widens exactly to fp32.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ float load_elem(const float *p, size_t i) { return p[i]; }
__device__ __forceinline__ float load_elem(const uint16_t *p, size_t i) {
  return bf16_to_f32(p[i]);
}

// Round-to-nearest-even fp32 -> bf16 bits (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Wave-level reductions (wave64).
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
// Inclusive prefix sum over the 64 lanes.
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    T t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// ---------------------------------------------------------------------------
// Proxy-logit arithmetic (Eq. 6): ((P_T + P_H) + P_W) * sigma, then + 0 to
// fold -0 into +0.  P points at one concatenated table row.
// Code fields are clamped to their codebooks so a bad code cannot read
// outside the row.
__device__ __forceinline__ float proxy_logit(const float *P, int cT, int cTH,
                                             int cs, uint32_t code, float sigma) {
  const int zT = min(static_cast<int>(code & 1023u), cT - 1);
  const int zH = min(static_cast<int>((code >> 10) & 1023u), cTH - cT - 1);
  const int zW = min(static_cast<int>((code >> 20) & 1023u), cs - cTH - 1);
  float s = P[zT] + P[cT + zH];
  s = s + P[cTH + zW];
  s = s * sigma;
  return s + 0.0f;
}

// The same sum over the M subspaces of a general partition, left to right
// in subspace order (M = 3 gives the expression above), from one uint16
// code plane per subspace: z^m of key j at planes[m * n + j].  col[m] is
// the first table column of subspace m, col[M] the row length.
constexpr int kCodeMaxSub = 8;
struct CodePlanes {
  int M;
  int col[kCodeMaxSub + 1];
};
__device__ __forceinline__ float proxy_logit_planes(const float *P,
                                                    const CodePlanes &cp,
                                                    const uint16_t *planes,
                                                    size_t n, int j, float sigma) {
  float s = P[min(static_cast<int>(planes[j]), cp.col[1] - 1)];
#pragma unroll
  for (int m = 1; m < kCodeMaxSub; ++m) {
    if (m < cp.M) {
      const int z = min(static_cast<int>(planes[m * n + j]), cp.col[m + 1] - cp.col[m] - 1);
      s = s + P[cp.col[m] + z];
    }
  }
  s = s * sigma;
  return s + 0.0f;
}

// Rank key: logits in DEScending order map to ascending unsigned keys.
__device__ __forceinline__ uint32_t desc_key(float s) {
  uint32_t u = __float_as_uint(s);
  uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}
__device__ __forceinline__ float desc_key_value(uint32_t key) {
  uint32_t asc = ~key;
  uint32_t u = (asc & 0x80000000u) ? (asc & 0x7FFFFFFFu) : ~asc;
  return __uint_as_float(u);
}

// Fixed-point exponential of the proxy softmax: for y <= 0 returns about
// e^y * 2^32 as an integer.  z = y*log2(e) in fp32; below -40 the mass is 0;
// z = n + f with n = rint(z); 2^f from its Taylor series (coefficients
// (ln 2)^k / k! rounded to fp32, Horner with fmaf); then 2^(n+32) * p
// rounded to the nearest integer (ties to even), done exactly in integers.
__device__ __forceinline__ uint64_t fixexp(float y) {
  const float kLog2e = 0x1.715476p+0f;
  float z = y * kLog2e;
  if (!(z >= -40.0f)) return 0;
  float nr = rintf(z);
  float f = z - nr;
  float p = 0x1.ffcbfcp-17f;
  p = fmaf(p, f, 0x1.430912p-13f);
  p = fmaf(p, f, 0x1.5d87fep-10f);
  p = fmaf(p, f, 0x1.3b2ab6p-7f);
  p = fmaf(p, f, 0x1.c6b08ep-5f);
  p = fmaf(p, f, 0x1.ebfbep-3f);
  p = fmaf(p, f, 0x1.62e43p-1f);
  p = fmaf(p, f, 1.0f);
  // p in [0.70, 1.42] is a normal float: p = mant * 2^(pe - 23)
  uint32_t bits = __float_as_uint(p);
  int pe = static_cast<int>((bits >> 23) & 0xFFu) - 127;
  uint32_t mant = (bits & 0x7FFFFFu) | 0x800000u;
  int k = pe + static_cast<int>(nr) + 9;  // value = mant * 2^k
  if (k >= 0) return static_cast<uint64_t>(mant) << k;
  int s = -k;
  if (s >= 25) return 0;  // mant * 2^-s < 1/2
  uint32_t q = mant >> s;
  uint32_t rem = mant & ((1u << s) - 1u);
  uint32_t half = 1u << (s - 1);
  if (rem > half || (rem == half && (q & 1u))) q += 1u;
  return q;
}

// Exact ceil(rho * tot) for 0 < rho < 1 (finite) and tot < 2^63.
__device__ __forceinline__ uint64_t mass_target(float rho, uint64_t tot) {
  uint32_t bits = __float_as_uint(rho);
  int ex = static_cast<int>((bits >> 23) & 0xFFu);
  uint64_t m;
  int sh;  // rho = m / 2^sh
  if (ex == 0) {  // subnormal
    m = bits & 0x7FFFFFu;
    sh = 149;
  } else {
    m = (bits & 0x7FFFFFu) | 0x800000u;
    sh = 150 - ex;  // rho = m * 2^(ex - 127 - 23)
  }
  // m < 2^24 and tot < 2^63: for sh >= 100 the product is below 1, ceil 1
  if (sh >= 100) return tot ? 1 : 0;
  unsigned __int128 prod = static_cast<unsigned __int128>(m) * tot;
  unsigned __int128 one = static_cast<unsigned __int128>(1) << sh;
  return static_cast<uint64_t>((prod + one - 1) >> sh);
}

}  // namespace scope
