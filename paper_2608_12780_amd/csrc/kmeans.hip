// K-means kernels (Sec. 3.2 Eq. 2 for queries; Sec. 3.3 Eq. 3 for the key
// subspaces), canonical arithmetic:
//   assign: argmin_r fl(||u_r||^2 - 2<x, u_r>), dot products as fp32 fma
//           chains in ascending channel order, ties to the lowest r;
//   update: exact int64 sums of rint(x * 2^24) over the members, one fp64
//           division by count * 2^24, rounded to fp32; empty clusters keep
//           their centroid.
// This file: initialisation, the VALU assignment, and the grouping of the
// final query assignment (per-chunk cluster histograms -> column scan ->
// stable scatter into the cluster-grouped permutation);
// also the packing of key codes and the channel gather of general key
// partitions.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

template <typename T>
__global__ void km_init_kernel(const T *X, size_t x_hs, int ld, int col0,
                               int dx, int n, int C, const int32_t *init,
                               int init_stride, float *U, size_t u_hs,
                               int32_t *status) {
  const int r = blockIdx.x, h = blockIdx.y;
  const int def = static_cast<int>(((2LL * r + 1) * n) / (2LL * C));
  int row = def;
  if (init) {
    row = init[static_cast<size_t>(h) * init_stride + r];
    if (row < 0 || row >= n) {
      if (threadIdx.x == 0 && status) atomicOr(status, kStatusBadInit);
      row = def;
    }
  }
  const T *src = X + h * x_hs + static_cast<size_t>(row) * ld + col0;
  float *dst = U + h * u_hs + static_cast<size_t>(r) * dx;
  for (int c = threadIdx.x; c < dx; c += blockDim.x) dst[c] = load_elem(src, c);
}

// One point per thread, its channels held in registers (zero padded to DXP:
// a trailing fma(0, 0, acc) leaves the score unchanged).  Centroids are
// staged through LDS transposed, CB at a time, and read as wave-wide
// broadcasts.  Scores are compared in ascending centroid order with a
// strict '<', so ties go to the lowest index.
template <typename T, int DXP>
__global__ __launch_bounds__(kAssignBlock) void km_assign_kernel(
    const T *__restrict__ X, size_t x_hs, int ld, int col0, int dx, int n,
    const float *__restrict__ U, size_t u_hs, int C, int32_t *assign,
    size_t a_hs, int32_t *chunk_hist, int nchunks) {
  constexpr int CB = 64;
  __shared__ float Ut[DXP][CB];
  __shared__ float nu_s[CB];
  __shared__ int hist[1024];
  const int h = blockIdx.y, t = threadIdx.x;
  const int i = blockIdx.x * kAssignBlock + t;
  const bool valid = i < n;
  const T *xrow = X + h * x_hs + static_cast<size_t>(valid ? i : 0) * ld + col0;
  float xr[DXP];
#pragma unroll
  for (int c = 0; c < DXP; ++c) xr[c] = (c < dx) ? load_elem(xrow, c) : 0.0f;
  const float *Uh = U + h * u_hs;
  float best = INFINITY;
  int arg = 0;
  for (int r0 = 0; r0 < C; r0 += CB) {
    __syncthreads();
    for (int e = t; e < DXP * CB; e += kAssignBlock) {
      const int rr = e % CB, c = e / CB, r = r0 + rr;
      Ut[c][rr] = (r < C && c < dx) ? Uh[static_cast<size_t>(r) * dx + c] : 0.0f;
    }
    if (t < CB) {
      const int r = r0 + t;
      float nu = INFINITY;  // padding centroids never win
      if (r < C) {
        const float *u = Uh + static_cast<size_t>(r) * dx;
        nu = 0.0f;
        for (int c = 0; c < dx; ++c) nu = fmaf(u[c], u[c], nu);
      }
      nu_s[t] = nu;
    }
    __syncthreads();
    const int rend = min(CB, C - r0);
    for (int rr = 0; rr < rend; rr += 8) {
      float acc[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] = 0.0f;
#pragma unroll
      for (int c = 0; c < DXP; ++c) {
        const float4 u0 = *reinterpret_cast<const float4 *>(&Ut[c][rr]);
        const float4 u1 = *reinterpret_cast<const float4 *>(&Ut[c][rr + 4]);
        acc[0] = fmaf(xr[c], u0.x, acc[0]);
        acc[1] = fmaf(xr[c], u0.y, acc[1]);
        acc[2] = fmaf(xr[c], u0.z, acc[2]);
        acc[3] = fmaf(xr[c], u0.w, acc[3]);
        acc[4] = fmaf(xr[c], u1.x, acc[4]);
        acc[5] = fmaf(xr[c], u1.y, acc[5]);
        acc[6] = fmaf(xr[c], u1.z, acc[6]);
        acc[7] = fmaf(xr[c], u1.w, acc[7]);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float s = fmaf(-2.0f, acc[k], nu_s[rr + k]);
        if (s < best) {
          best = s;
          arg = r0 + rr + k;
        }
      }
    }
  }
  if (valid) assign[h * a_hs + i] = arg;
  if (chunk_hist) {
    __syncthreads();
    for (int r = t; r < C; r += kAssignBlock) hist[r] = 0;
    __syncthreads();
    if (valid) atomicAdd(&hist[arg], 1);
    __syncthreads();
    int32_t *out = chunk_hist + (static_cast<size_t>(h) * nchunks + blockIdx.x) * C;
    for (int r = t; r < C; r += kAssignBlock) out[r] = hist[r];
  }
}

// Column scan of the chunk histograms: counts[r] and, per chunk, the number
// of members of r in earlier chunks.  Block = (64-column group, head); each
// column is split into segments summed in parallel.
__global__ __launch_bounds__(1024) void km_colscan_kernel(
    int nchunks, int C, const int32_t *__restrict__ hist, int32_t *rel,
    int32_t *counts) {
  __shared__ int seg[1024];
  const int h = blockIdx.y, t = threadIdx.x;
  const int c0 = blockIdx.x * 64;
  const int cols = min(64, C - c0);
  const int nseg = 1024 / cols;
  const int col = c0 + t % cols, g = t / cols;
  const int seglen = (nchunks + nseg - 1) / nseg;
  const int k0 = g * seglen, k1 = min(nchunks, k0 + seglen);
  const int32_t *H = hist + static_cast<size_t>(h) * nchunks * C;
  int sum = 0;
  if (g < nseg) {
#pragma unroll 8
    for (int k = k0; k < k1; ++k) sum += H[static_cast<size_t>(k) * C + col];
  }
  seg[t] = sum;
  __syncthreads();
  if (t < cols) {
    int run = 0;
    for (int gg = 0; gg < nseg; ++gg) {
      const int v = seg[gg * cols + t];
      seg[gg * cols + t] = run;
      run += v;
    }
    counts[static_cast<size_t>(h) * C + col] = run;
  }
  __syncthreads();
  if (g < nseg) {
    int run = seg[t];
    int32_t *R = rel + static_cast<size_t>(h) * nchunks * C;
#pragma unroll 8
    for (int k = k0; k < k1; ++k) {
      R[static_cast<size_t>(k) * C + col] = run;
      run += H[static_cast<size_t>(k) * C + col];
    }
  }
}

// Exclusive prefix sum of counts[0..C) into off_s (block of 256 threads).
__device__ void block_offsets(const int32_t *counts, int C, int *off_s) {
  __shared__ int wtot[4];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int per = (C + 255) / 256;
  const int b = t * per;
  int local = 0;
  for (int e = 0; e < per; ++e)
    if (b + e < C) local += counts[b + e];
  const int incl = wave_incl_scan(local);
  if (lane == 63) wtot[w] = incl;
  __syncthreads();
  int base = 0;
  for (int ww = 0; ww < w; ++ww) base += wtot[ww];
  int run = base + incl - local;
  for (int e = 0; e < per; ++e) {
    if (b + e < C) {
      off_s[b + e] = run;
      run += counts[b + e];
    }
  }
  if (t == 255) off_s[C] = base + incl;
  __syncthreads();
}

// Stable scatter: point i of chunk k goes to
// offsets[a] + (members of a in earlier chunks) + (earlier members in chunk).
// The in-chunk rank uses an 11-round ballot match per wave plus per-wave
// counts in LDS.
__global__ __launch_bounds__(kAssignBlock) void km_scatter_kernel(
    int n, int C, int nchunks, const int32_t *__restrict__ assign, size_t a_hs,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ rel,
    int32_t *offsets, int32_t *perm, size_t p_hs) {
  __shared__ int off_s[1025];
  __shared__ int wcnt[4][1024];
  const int h = blockIdx.y, k = blockIdx.x, t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  block_offsets(counts + static_cast<size_t>(h) * C, C, off_s);
  if (k == 0)
    for (int r = t; r <= C; r += kAssignBlock)
      offsets[static_cast<size_t>(h) * (C + 1) + r] = off_s[r];
  const int i = k * kAssignBlock + t;
  const bool valid = i < n;
  const int a = valid ? assign[h * a_hs + i] : C;  // C: sentinel, never valid
  uint64_t same = ~0ull;
#pragma unroll
  for (int b = 0; b < 11; ++b) {
    const bool bit = (a >> b) & 1;
    const uint64_t bal = __ballot(bit);
    same &= bit ? bal : ~bal;
  }
  const int rank = __popcll(same & ((1ull << lane) - 1ull));
  const int total = __popcll(same);
  for (int e = t; e < 4 * C; e += kAssignBlock) wcnt[e / C][e % C] = 0;
  __syncthreads();
  if (valid && rank == 0) wcnt[w][a] = total;
  __syncthreads();
  if (valid) {
    int pre = 0;
    for (int ww = 0; ww < w; ++ww) pre += wcnt[ww][a];
    const int pos = off_s[a] + rel[(static_cast<size_t>(h) * nchunks + k) * C + a] + pre + rank;
    if (pos >= 0 && pos < n) perm[h * p_hs + pos] = i;
  }
}

// Composite key codes zT | zH << 10 | zW << 20 (Sec. 3.3).
__global__ void km_pack_kernel(const int32_t *__restrict__ a3, size_t a_hs,
                               size_t a_ss, int n, uint32_t *codes) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x, h = blockIdx.y;
  if (j >= n) return;
  const int32_t *A = a3 + h * a_hs;
  codes[static_cast<size_t>(h) * n + j] =
      static_cast<uint32_t>(A[j]) | (static_cast<uint32_t>(A[a_ss + j]) << 10) |
      (static_cast<uint32_t>(A[2 * a_ss + j]) << 20);
}

__global__ void km_codes16_kernel(const int32_t *__restrict__ a, size_t count,
                                  uint16_t *codes) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < count) codes[i] = static_cast<uint16_t>(a[i]);
}

template <typename T>
__global__ void gather_channels_kernel(const T *__restrict__ src, T *dst,
                                       size_t rows, int d, ChannelMap map) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= rows * d) return;
  const size_t r = i / d;
  const int t = static_cast<int>(i - r * d);
  dst[i] = src[r * d + map.chan[t]];
}

template <typename T>
hipError_t assign_dispatch(const KmProblem &p, bool with_hist, hipStream_t s) {
  const dim3 grid(km_nchunks(p.n), p.heads);
  const T *x = static_cast<const T *>(p.x);
  int32_t *hist = with_hist ? p.chunk_hist : nullptr;
  const int nch = km_nchunks(p.n);
#define SCOPE_ASSIGN(DXP)                                                      \
  hipLaunchKernelGGL((km_assign_kernel<T, DXP>), grid, dim3(kAssignBlock), 0, s, \
                     x, p.x_head_stride, p.ld, p.col0, p.dx, p.n, p.u,          \
                     p.u_head_stride, p.C, p.assign, p.a_head_stride, hist, nch)
  if (p.dx <= 16) SCOPE_ASSIGN(16);
  else if (p.dx <= 32) SCOPE_ASSIGN(32);
  else if (p.dx <= 48) SCOPE_ASSIGN(48);
  else if (p.dx <= 64) SCOPE_ASSIGN(64);
  else SCOPE_ASSIGN(128);
#undef SCOPE_ASSIGN
  return hipGetLastError();
}

}  // namespace

hipError_t km_init(const KmProblem &p, const int32_t *init, int init_stride,
                   int32_t *status, hipStream_t s) {
  const dim3 grid(p.C, p.heads);
  if (p.bf16)
    hipLaunchKernelGGL(km_init_kernel<uint16_t>, grid, dim3(64), 0, s,
                       static_cast<const uint16_t *>(p.x), p.x_head_stride,
                       p.ld, p.col0, p.dx, p.n, p.C, init, init_stride, p.u,
                       p.u_head_stride, status);
  else
    hipLaunchKernelGGL(km_init_kernel<float>, grid, dim3(64), 0, s,
                       static_cast<const float *>(p.x), p.x_head_stride, p.ld,
                       p.col0, p.dx, p.n, p.C, init, init_stride, p.u,
                       p.u_head_stride, status);
  return hipGetLastError();
}

hipError_t km_assign_mfma(const KmProblem &p, bool with_hist, hipStream_t s);

hipError_t km_assign(const KmProblem &p, bool with_hist, hipStream_t s) {
  if (p.mfma) return km_assign_mfma(p, with_hist, s);
  return p.bf16 ? assign_dispatch<uint16_t>(p, with_hist, s)
                : assign_dispatch<float>(p, with_hist, s);
}

hipError_t km_group(const KmProblem &p, hipStream_t s) {
  const int nch = km_nchunks(p.n);
  hipLaunchKernelGGL(km_colscan_kernel, dim3((p.C + 63) / 64, p.heads),
                     dim3(1024), 0, s, nch, p.C, p.chunk_hist, p.chunk_rel,
                     p.counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(km_scatter_kernel, dim3(nch, p.heads), dim3(kAssignBlock),
                     0, s, p.n, p.C, nch, p.assign, p.a_head_stride, p.counts,
                     p.chunk_rel, p.offsets, p.perm, p.a_head_stride);
  return hipGetLastError();
}

hipError_t km_pack_codes(const int32_t *a3, size_t a_head_stride,
                         size_t a_sub_stride, int n, int heads,
                         uint32_t *codes, hipStream_t s) {
  hipLaunchKernelGGL(km_pack_kernel, dim3((n + 255) / 256, heads), dim3(256),
                     0, s, a3, a_head_stride, a_sub_stride, n, codes);
  return hipGetLastError();
}

hipError_t km_codes16(const int32_t *assign, size_t count, uint16_t *codes,
                      hipStream_t s) {
  if (count == 0) return hipSuccess;
  hipLaunchKernelGGL(km_codes16_kernel, dim3(static_cast<unsigned>((count + 255) / 256)),
                     dim3(256), 0, s, assign, count, codes);
  return hipGetLastError();
}

hipError_t gather_channels(const void *src, void *dst, size_t rows, int d,
                           int elem_bytes, const ChannelMap &map, hipStream_t s) {
  const size_t count = rows * d;
  if (count == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((count + 255) / 256));
  if (elem_bytes == 2)
    hipLaunchKernelGGL(gather_channels_kernel<uint16_t>, grid, dim3(256), 0, s,
                       static_cast<const uint16_t *>(src), static_cast<uint16_t *>(dst),
                       rows, d, map);
  else
    hipLaunchKernelGGL(gather_channels_kernel<float>, grid, dim3(256), 0, s,
                       static_cast<const float *>(src), static_cast<float *>(dst), rows,
                       d, map);
  return hipGetLastError();
}

}  // namespace scope
