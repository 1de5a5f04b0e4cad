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
// atomics, laid out so the lanes of a row hit consecutive slots) and counts
// the row.  Lanes take 4 channels (8-byte loads) where the channel ranges
// allow, else 2.  All three key subspaces fit one window, so
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

// The int64 sums stay exact while n terms of magnitude below 2^(e+24) cannot
// reach 2^63: |x| < lim = 2^e with e = min(22, 39 - ceil(log2 n)).  Larger or
// non-finite inputs are flagged.
__device__ __forceinline__ void check_value(float x, float lim, int &bad) {
  if (!(fabsf(x) < lim))
    bad |= isfinite(x) ? kStatusRange : (kStatusRange | kStatusNonFinite);
}

// CPL (2 or 4) adjacent channels of a row as floats.  VEC: one aligned load
// of the whole chunk (every chunk complete); else scalar loads, repeating the
// first element past the `nvalid` channels the chunk has.
template <typename T, int CPL, bool VEC>
__device__ __forceinline__ void load_chunk(const T *p, int nvalid, float (&x)[CPL]) {
  if constexpr (sizeof(T) == 2) {
    if constexpr (VEC && CPL == 4) {
      const uint2 v = *reinterpret_cast<const uint2 *>(p);
      x[0] = __uint_as_float(v.x << 16);
      x[1] = __uint_as_float(v.x & 0xFFFF0000u);
      x[2] = __uint_as_float(v.y << 16);
      x[3] = __uint_as_float(v.y & 0xFFFF0000u);
    } else if constexpr (VEC) {
      const uint32_t v = *reinterpret_cast<const uint32_t *>(p);
      x[0] = __uint_as_float(v << 16);
      x[1] = __uint_as_float(v & 0xFFFF0000u);
    } else {
#pragma unroll
      for (int e = 0; e < CPL; ++e) x[e] = bf16_to_f32(p[e < nvalid ? e : 0]);
    }
  } else {
    if constexpr (VEC && CPL == 4) {
      const float4 v = *reinterpret_cast<const float4 *>(p);
      x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    } else if constexpr (VEC) {
      const float2 v = *reinterpret_cast<const float2 *>(p);
      x[0] = v.x; x[1] = v.y;
    } else {
#pragma unroll
      for (int e = 0; e < CPL; ++e) x[e] = p[e < nvalid ? e : 0];
    }
  }
}

template <typename T, int CPL, bool VEC, bool CHECK>
__global__ __launch_bounds__(kAccThreads) void km_accum_kernel(
    const T *__restrict__ X, size_t x_hs, int ld, int n, const AccPlan plan,
    const int32_t *__restrict__ assign, size_t a_hs, size_t a_ss,
    long long *slab, int32_t *cslab, int32_t *status, float lim) {
  // the last CPL sums are a sink for lanes that hold no channels
  __shared__ unsigned long long sums[kAccLds + 4];
  __shared__ int cnts[kAccCnt];
  const int b = blockIdx.x, wi = blockIdx.y, h = blockIdx.z, t = threadIdx.x;
  const AccWindow &W = plan.win[wi];
  for (int e = t; e < W.elems; e += kAccThreads) sums[e] = 0ull;
  for (int e = t; e < W.cnt_elems; e += kAccThreads) cnts[e] = 0;
  __syncthreads();

  // lanes per row: one per CPL channels of each piece
  int lanes = 0;
  for (int q = 0; q < W.npieces; ++q) lanes += (W.piece[q].width + CPL - 1) / CPL;
  // lane -> (row within the wave's row group, piece, channel chunk)
  const int lane = t & 63, wv = t >> 6;
  const int rpw = 64 / lanes;
  const int rr = lane / lanes, pl = lane % lanes;
  const bool active = rr < rpw;
  int p = 0, first = 0;
  while (p + 1 < W.npieces && pl >= first + (W.piece[p].width + CPL - 1) / CPL) {
    first += (W.piece[p].width + CPL - 1) / CPL;
    ++p;
  }
  // the piece's fields, held in registers for the row loop
  const int pm = W.piece[p].m, p_width = W.piece[p].width;
  const int p_cnt = W.piece[p].cnt, p_sub0 = W.piece[p].sub0;
  const int j = CPL * (pl - first);              // first channel of the chunk in the piece
  const int nvalid = min(CPL, p_width - j);
  const int Cm = plan.C[pm];
  const T *xb = X + h * x_hs + plan.col0[pm] + p_sub0 + j;
  const int32_t *ab = assign + h * a_hs + pm * a_ss;
  const bool counter = active && p_cnt >= 0 && j == 0;
  // LDS sums of a cluster's piece: with vector loads, element e of chunk c
  // at e * (width / CPL) + c, so for each e the lanes of a row add to
  // consecutive slots (no bank conflicts); idle lanes add into the sink
  const int e_stride = VEC ? p_width / CPL : 1;
  const int lds_base = active ? W.piece[p].lds + (VEC ? j / CPL : j) : kAccLds;
  const int lds_stride = active ? p_width : 0;
  int bad = 0;

  const int lo = static_cast<int>((static_cast<long long>(n) * b) / gridDim.x);
  const int hi = static_cast<int>((static_cast<long long>(n) * (b + 1)) / gridDim.x);
  const int step = kAccWaves * rpw;  // rows per block step
  constexpr int U = 4;
  // one group of U rows per lane; FULL: every row of the group is in range
  auto group = [&](int g, bool full) {
    float xv[U][CPL];
    int av[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = g + u * step;
      const int rc = (active && (full || row < hi)) ? row : lo;
      av[u] = ab[rc];
      load_chunk<T, CPL, VEC>(xb + static_cast<size_t>(rc) * ld, nvalid, xv[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = g + u * step;
      const bool ok = full || row < hi;
      const int a = min(static_cast<unsigned>(av[u]), static_cast<unsigned>(Cm - 1));
      const int idx = lds_base + a * lds_stride;
#pragma unroll
      for (int e = 0; e < CPL; ++e) {
        const float x = ok ? xv[u][e] : 0.0f;
        if (CHECK && e < nvalid) check_value(x, lim, bad);
        if (VEC || e < nvalid) atomicAdd(&sums[idx + (active ? e * e_stride : e)], fixed24(x));
      }
      if (counter) atomicAdd(&cnts[p_cnt + a], ok ? 1 : 0);
    }
  };
  int g = lo + wv * rpw + rr;
  for (; (g - rr) + (U - 1) * step + rpw - 1 < hi; g += U * step) group(g, true);
  if (g - rr < hi) group(g, false);
  if (CHECK && status && bad) atomicOr(status, bad);
  __syncthreads();

  // this block's sums into its slab, in the centroids' layout
  long long *sl = slab + (static_cast<size_t>(h) * gridDim.x + b) * plan.S;
  for (int q = 0; q < W.npieces; ++q) {
    const AccPiece &Q = W.piece[q];
    const int m = Q.m, cnt = plan.C[m] * Q.width;
    const int cw = Q.width / CPL;
    for (int e = t; e < cnt; e += kAccThreads) {
      const int r = e / Q.width, k = e - r * Q.width;
      const int off = VEC ? (k % CPL) * cw + k / CPL : k;
      sl[plan.ucol[m] + static_cast<size_t>(r) * plan.dx[m] + Q.sub0 + k] =
          static_cast<long long>(sums[Q.lds + r * Q.width + off]);
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
  if (nsub < 1 || nsub > kMaxSub) return false;
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
      // cuts fall on multiples of 64 channels where the room allows (whole
      // 128-byte lines of bf16 rows), else of 32, else of 4 (8-byte loads);
      // a window with less room than that is closed
      if (w < dx[m] - done) w &= w >= 64 ? ~63 : w >= 32 ? ~31 : ~3;
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
      const bool cut = w < dx[m] - done;
      done += w;
      if (cut && !flush()) return false;  // a cut closes its window
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
  int ce = 0;  // ceil(log2 n)
  while (ce < 31 && (1LL << ce) < n) ++ce;
  const float lim = ldexpf(1.0f, 39 - ce < 22 ? 39 - ce : 22);
  // vector loads need complete chunks starting on chunk boundaries
  auto aligned = [&](int cpl) {
    const size_t bytes = static_cast<size_t>(cpl) * (bf16 ? 2 : 4);
    if (ld % cpl || x_hs % cpl || reinterpret_cast<uintptr_t>(x) % bytes) return false;
    for (int w = 0; w < plan.nwin; ++w)
      for (int q = 0; q < plan.win[w].npieces; ++q) {
        const AccPiece &pc = plan.win[w].piece[q];
        if ((plan.col0[pc.m] + pc.sub0) % cpl || pc.width % cpl) return false;
      }
    return true;
  };
  const bool v4 = aligned(4), v2 = aligned(2);
#define SCOPE_ACCUM(T, CPL, V, K)                                                    \
  hipLaunchKernelGGL((km_accum_kernel<T, CPL, V, K>), grid, dim3(kAccThreads), 0, s, \
                     static_cast<const T *>(x), x_hs, ld, n, plan, assign, a_hs,      \
                     a_ss, slab, cslab, status, lim)
#define SCOPE_ACCUM_K(T, CPL, V)            \
  if (check) SCOPE_ACCUM(T, CPL, V, true);  \
  else SCOPE_ACCUM(T, CPL, V, false);
#define SCOPE_ACCUM_T(T)                    \
  if (v4) {                                 \
    SCOPE_ACCUM_K(T, 4, true)               \
  } else if (v2) {                          \
    SCOPE_ACCUM_K(T, 2, true)               \
  } else {                                  \
    SCOPE_ACCUM_K(T, 2, false)              \
  }
  if (bf16) {
    SCOPE_ACCUM_T(uint16_t)
  } else {
    SCOPE_ACCUM_T(float)
  }
#undef SCOPE_ACCUM_T
#undef SCOPE_ACCUM_K
#undef SCOPE_ACCUM
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(km_accum_finalize_kernel, dim3((plan.S + 255) / 256, heads),
                     dim3(256), 0, s, plan, plan.blocks, slab, cslab, U, u_hs);
  return hipGetLastError();
}

}  // namespace scope
