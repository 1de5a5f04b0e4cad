// K-means centroid update (Sec. 3.2 Eq. 2, Sec. 3.3 Eq. 3), canonical
// arithmetic: exact int64 sums of rint(x * 2^24) over each cluster's
// members, one fp64 division by count * 2^24 rounded to fp32; an empty
// cluster keeps its centroid.  Integer sums do not depend on the order in
// which members are added, so any accumulation order gives the canonical
// result.
//
// The rows are streamed once, in storage order.  A block owns a contiguous
// row range of one head and one channel window; for every row it adds the
// window's channels to the sums of the row's cluster in LDS (int64 LDS
// atomics) and counts the row.  All three key subspaces fit one window, so
// one pass over K updates T, H and W together; the query codebook is split
// over two windows.  Each block writes its sums to a slab laid out like the
// centroids; a second kernel reduces the slabs and divides.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

constexpr int kAccThreads = 1024;
constexpr int kAccWaves = kAccThreads / 64;

// rint(x * 2^24) as a two's complement int64, exact for |x| < 2^27: the
// fp64 value x * 2^24 + 1.5 * 2^52 is rounded once, to the nearest integer
// with ties to even (the spacing of doubles in [2^52, 2^53) is 1), and the
// low 52 bits of its encoding then hold 2^51 + rint(x * 2^24).  The high
// word minus the fixed exponent and 2^19 is the upper half of the result.
// Other x (flagged in the status word) give some value, never a trap.
__device__ __forceinline__ unsigned long long fixed24(float x) {
  const double d = fma(static_cast<double>(x), 0x1p24, 0x1.8p52);
  const unsigned long long bits = static_cast<unsigned long long>(__double_as_longlong(d));
  const uint32_t lo = static_cast<uint32_t>(bits);
  const uint32_t hi = static_cast<uint32_t>(bits >> 32) - 0x43380000u;
  return (static_cast<unsigned long long>(hi) << 32) | lo;
}

__device__ __forceinline__ void check_value(float x, int &bad) {
  if (!(fabsf(x) < 0x1p22f))
    bad |= isfinite(x) ? kStatusRange : (kStatusRange | kStatusNonFinite);
}

// Two adjacent channels of a row: one aligned load when VEC (every pair
// complete and aligned), else two loads, the second repeating the first
// where the pair has one channel.
template <typename T, bool VEC> struct Pair;
template <bool VEC> struct Pair<uint16_t, VEC> {
  typedef uint32_t type;
  static __device__ __forceinline__ type load(const uint16_t *p, bool two) {
    if (VEC) return *reinterpret_cast<const uint32_t *>(p);
    return static_cast<uint32_t>(p[0]) | (static_cast<uint32_t>(p[two ? 1 : 0]) << 16);
  }
  static __device__ __forceinline__ float first(type v) { return __uint_as_float(v << 16); }
  static __device__ __forceinline__ float second(type v) { return __uint_as_float(v & 0xFFFF0000u); }
};
template <bool VEC> struct Pair<float, VEC> {
  typedef float2 type;
  static __device__ __forceinline__ type load(const float *p, bool two) {
    if (VEC) return *reinterpret_cast<const float2 *>(p);
    return make_float2(p[0], p[two ? 1 : 0]);
  }
  static __device__ __forceinline__ float first(type v) { return v.x; }
  static __device__ __forceinline__ float second(type v) { return v.y; }
};

template <typename T, bool VEC, bool CHECK>
__global__ __launch_bounds__(kAccThreads) void km_accum_kernel(
    const T *__restrict__ X, size_t x_hs, int ld, int n, const AccPlan plan,
    const int32_t *__restrict__ assign, size_t a_hs, size_t a_ss,
    long long *slab, int32_t *cslab, int32_t *status) {
  __shared__ unsigned long long sums[kAccLds];
  __shared__ int cnts[kAccCnt];
  const int b = blockIdx.x, wi = blockIdx.y, h = blockIdx.z, t = threadIdx.x;
  const AccWindow &W = plan.win[wi];
  for (int e = t; e < W.elems; e += kAccThreads) sums[e] = 0ull;
  for (int e = t; e < W.cnt_elems; e += kAccThreads) cnts[e] = 0;
  __syncthreads();

  // lane -> (row within the wave's row group, piece, channel pair)
  const int lane = t & 63, wv = t >> 6;
  const int rpw = 64 / W.lanes;
  const int rr = lane / W.lanes, pl = lane % W.lanes;
  const bool active = rr < rpw;
  int p = 0, first = 0;
  while (p + 1 < W.npieces && pl >= first + (W.piece[p].width + 1) / 2) {
    first += (W.piece[p].width + 1) / 2;
    ++p;
  }
  // the piece's fields, held in registers for the row loop
  const int pm = W.piece[p].m, p_width = W.piece[p].width, p_lds = W.piece[p].lds;
  const int p_cnt = W.piece[p].cnt, p_sub0 = W.piece[p].sub0;
  const int j = 2 * (pl - first);                // channel of the pair in the piece
  const bool two = j + 1 < p_width;
  const int Cm = plan.C[pm];
  const T *xb = X + h * x_hs + plan.col0[pm] + p_sub0 + j;
  const int32_t *ab = assign + h * a_hs + pm * a_ss;
  const bool counter = p_cnt >= 0 && j == 0;
  int bad = 0;

  const int lo = static_cast<int>((static_cast<long long>(n) * b) / gridDim.x);
  const int hi = static_cast<int>((static_cast<long long>(n) * (b + 1)) / gridDim.x);
  const int step = kAccWaves * rpw;  // rows per block step
  constexpr int U = 4;
  for (int g = lo + wv * rpw + rr; g - rr < hi; g += U * step) {
    typename Pair<T, VEC>::type xv[U];
    int av[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = g + u * step;
      const int rc = (active && row < hi) ? row : lo;
      av[u] = ab[rc];
      xv[u] = Pair<T, VEC>::load(xb + static_cast<size_t>(rc) * ld, two);
    }
    // branch-free: rows past the range (and idle lanes) add zeros
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = g + u * step;
      const bool ok = active && row < hi;
      const int a = min(static_cast<unsigned>(av[u]), static_cast<unsigned>(Cm - 1));
      const int idx = p_lds + a * p_width + j;
      const float x0 = ok ? Pair<T, VEC>::first(xv[u]) : 0.0f;
      const float x1 = ok ? Pair<T, VEC>::second(xv[u]) : 0.0f;
      if (CHECK) {
        check_value(x0, bad);
        check_value(x1, bad);
      }
      atomicAdd(&sums[idx], fixed24(x0));
      if (VEC || two) atomicAdd(&sums[idx + 1], fixed24(x1));
      if (counter) atomicAdd(&cnts[p_cnt + a], ok ? 1 : 0);
    }
  }
  if (CHECK && status && bad) atomicOr(status, bad);
  __syncthreads();

  // this block's sums into its slab, in the centroids' layout
  long long *sl = slab + (static_cast<size_t>(h) * gridDim.x + b) * plan.S;
  for (int q = 0; q < W.npieces; ++q) {
    const AccPiece &Q = W.piece[q];
    const int m = Q.m, cnt = plan.C[m] * Q.width;
    for (int e = t; e < cnt; e += kAccThreads) {
      const int r = e / Q.width, k = e - r * Q.width;
      sl[plan.ucol[m] + static_cast<size_t>(r) * plan.dx[m] + Q.sub0 + k] =
          static_cast<long long>(sums[Q.lds + e]);
    }
    if (Q.cnt >= 0) {
      int32_t *cs = cslab + (static_cast<size_t>(h) * gridDim.x + b) * plan.SC + plan.ccol[m];
      for (int r = t; r < plan.C[m]; r += kAccThreads) cs[r] = cnts[Q.cnt + r];
    }
  }
}

// U[h][pos] = sum over blocks / (count * 2^24), for every centroid element
// pos of the slab layout; an empty cluster keeps its centroid.
__global__ __launch_bounds__(256) void km_accum_finalize_kernel(
    const AccPlan plan, int blocks, const long long *__restrict__ slab,
    const int32_t *__restrict__ cslab, float *U, size_t u_hs) {
  const int pos = blockIdx.x * 256 + threadIdx.x, h = blockIdx.y;
  if (pos >= plan.S) return;
  int m = 0;
  while (m + 1 < plan.nsub && pos >= plan.ucol[m + 1]) ++m;
  const int r = (pos - plan.ucol[m]) / plan.dx[m];
  long long tot = 0;
  int cnt = 0;
  for (int b = 0; b < blocks; ++b) {
    const size_t hb = static_cast<size_t>(h) * blocks + b;
    tot += slab[hb * plan.S + pos];
    cnt += cslab[hb * plan.SC + plan.ccol[m] + r];
  }
  if (cnt <= 0) return;
  const double den = static_cast<double>(cnt) * 16777216.0;
  U[h * u_hs + pos] = static_cast<float>(static_cast<double>(tot) / den);
}

}  // namespace

bool km_accum_plan(int nsub, const int *col0, const int *dx, const int *C,
                   int heads, int n, AccPlan *plan) {
  AccPlan P{};
  if (plan) *plan = P;  // nwin == 0 marks a failed plan
  if (nsub < 1 || nsub > 3) return false;
  P.nsub = nsub;
  int S = 0, SC = 0;
  for (int m = 0; m < nsub; ++m) {
    if (C[m] < 1 || C[m] > kAccCnt || dx[m] < 1 || C[m] > kAccLds / 2) return false;
    P.C[m] = C[m];
    P.dx[m] = dx[m];
    P.col0[m] = col0[m];
    P.ucol[m] = S;
    P.ccol[m] = SC;
    S += C[m] * dx[m];
    SC += C[m];
  }
  P.S = S;
  P.SC = SC;
  // greedy windows: each subspace's channels in pieces of even width while
  // the LDS budget, the 64 lanes (128 channels) and the piece slots allow
  int nw = 0;
  AccWindow cur{};
  auto flush = [&]() -> bool {
    if (cur.npieces == 0) return true;
    if (nw == kAccMaxWindows) return false;
    P.win[nw++] = cur;
    cur = AccWindow{};
    return true;
  };
  for (int m = 0; m < nsub; ++m) {
    int done = 0;
    while (done < dx[m]) {
      const int room_lds = (kAccLds - cur.elems) / C[m];
      const int room_lanes = 2 * (64 - cur.lanes);
      const bool counts_here = done == 0;
      const bool cnt_fits = !counts_here || cur.cnt_elems + C[m] <= kAccCnt;
      int w = dx[m] - done;
      if (w > room_lds) w = room_lds;
      if (w > room_lanes) w = room_lanes;
      if (w < dx[m] - done) w &= ~1;
      if (w < 1 || cur.npieces == kAccMaxPieces || !cnt_fits) {
        if (cur.npieces == 0) return false;
        if (!flush()) return false;
        continue;
      }
      AccPiece &pc = cur.piece[cur.npieces++];
      pc.m = m;
      pc.sub0 = done;
      pc.width = w;
      pc.lds = cur.elems;
      pc.cnt = counts_here ? cur.cnt_elems : -1;
      cur.elems += C[m] * w;
      if (counts_here) cur.cnt_elems += C[m];
      cur.lanes += (w + 1) / 2;
      done += w;
    }
  }
  if (!flush()) return false;
  P.nwin = nw;
  int blocks = kAccTargetBlocks / (heads * nw);
  const int by_rows = (n + 255) / 256;
  if (blocks > by_rows) blocks = by_rows;
  if (blocks < 1) blocks = 1;
  P.blocks = blocks;
  if (plan) *plan = P;
  return true;
}

size_t km_accum_slab_bytes(const AccPlan &p, int heads) {
  return static_cast<size_t>(heads) * p.blocks * p.S * sizeof(long long);
}
size_t km_accum_cslab_bytes(const AccPlan &p, int heads) {
  return static_cast<size_t>(heads) * p.blocks * p.SC * sizeof(int32_t);
}

hipError_t km_accum(const AccPlan &plan, const void *x, bool bf16, size_t x_hs,
                    int ld, int n, int heads, const int32_t *assign,
                    size_t a_hs, size_t a_ss, long long *slab, int32_t *cslab,
                    float *U, size_t u_hs, int32_t *status, hipStream_t s) {
  const dim3 grid(plan.blocks, plan.nwin, heads);
  const bool check = status != nullptr;
  // paired loads need complete pairs starting on pair boundaries
  bool vec = (ld % 2 == 0) && (x_hs % 2 == 0) &&
             reinterpret_cast<uintptr_t>(x) % (bf16 ? 4 : 8) == 0;
  for (int m = 0; m < plan.nsub; ++m) vec = vec && plan.col0[m] % 2 == 0 && plan.dx[m] % 2 == 0;
#define SCOPE_ACCUM(T, V, K)                                                     \
  hipLaunchKernelGGL((km_accum_kernel<T, V, K>), grid, dim3(kAccThreads), 0, s,  \
                     static_cast<const T *>(x), x_hs, ld, n, plan, assign, a_hs,  \
                     a_ss, slab, cslab, status)
#define SCOPE_ACCUM_T(T)                       \
  if (vec) {                                   \
    if (check) SCOPE_ACCUM(T, true, true);     \
    else SCOPE_ACCUM(T, true, false);          \
  } else {                                     \
    if (check) SCOPE_ACCUM(T, false, true);    \
    else SCOPE_ACCUM(T, false, false);         \
  }
  if (bf16) {
    SCOPE_ACCUM_T(uint16_t)
  } else {
    SCOPE_ACCUM_T(float)
  }
#undef SCOPE_ACCUM_T
#undef SCOPE_ACCUM
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(km_accum_finalize_kernel, dim3((plan.S + 255) / 256, heads),
                     dim3(256), 0, s, plan, plan.blocks, slab, cslab, U, u_hs);
  return hipGetLastError();
}

}  // namespace scope
