// Sparse attention over the selected keys (Eq. 11; Alg. 1 last step), and
// dense attention (Eq. 1) as the one-cluster special case.
//
// Work item = (head, query cluster c, chunk of up to 32*NW of its queries).
// The block gathers the cluster's selected keys 64 at a time: K rows into LDS
// row-major, V rows transposed (dim-major) so both products read operands
// straight from LDS.  Each wave owns 32 queries and runs
//   S^T (64 keys x 32 queries) = K_tile . Q^T       bf16 MFMA 32x32x16
//   online softmax in fp32 (exp2 domain), one query per lane column
//   O^T (d x 32 queries)      += V_tile^T . P^T      bf16 MFMA 32x32x16
// The S^T accumulator layout is reused directly as the B operand of the
// second product: the MFMA k-index order is matched by reading V^T with the
// same key permutation, so P never leaves registers.  K/V tiles are double
// buffered: the next tile's global loads are in flight during the MFMAs.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBN = 64;   // keys per tile
constexpr int kNW = 8;    // waves per block (32 queries each)
constexpr int kBM = 32 * kNW;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) {
  return __builtin_bit_cast(bf16x8, u);
}

// 8 consecutive input elements as packed bf16.
template <bool BF16IN>
__device__ __forceinline__ uint4 load8(const void *base, size_t elem) {
  if (BF16IN) {
    return *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(base) + elem);
  } else {
    const float4 a = *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem);
    const float4 b = *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem + 4);
    uint4 u;
    u.x = f32_to_bf16(a.x) | (static_cast<uint32_t>(f32_to_bf16(a.y)) << 16);
    u.y = f32_to_bf16(a.z) | (static_cast<uint32_t>(f32_to_bf16(a.w)) << 16);
    u.z = f32_to_bf16(b.x) | (static_cast<uint32_t>(f32_to_bf16(b.y)) << 16);
    u.w = f32_to_bf16(b.z) | (static_cast<uint32_t>(f32_to_bf16(b.w)) << 16);
    return u;
  }
}

template <int D, bool BF16IN>
__global__ __launch_bounds__(kNW * 64) void attn_kernel(
    int n, int c_q, int items_per_head, const void *__restrict__ qv,
    const void *__restrict__ kv, const void *__restrict__ vv, void *ov,
    const int32_t *__restrict__ offsets, const int32_t *__restrict__ perm,
    const int32_t *__restrict__ sel_idx, const int4 *__restrict__ items,
    float scale_log2) {
  constexpr int NT = kNW * 64;
  constexpr int KS = D + 8;     // K tile row stride (bf16 elements)
  constexpr int VS = kBN + 8;   // V^T tile row stride
  constexpr int C8 = D / 8;     // 16-byte chunks per row
  constexpr int CH = kBN * C8 / NT;
  static_assert(CH >= 1 && kBN * C8 % NT == 0, "tile/threads mismatch");
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kBN * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][D * VS];

  const int h = blockIdx.y;
  const int4 it = items[static_cast<size_t>(h) * items_per_head + blockIdx.x];
  const int c = it.x, row0 = it.y, rows = it.z, r = it.w;
  if (rows <= 0) return;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const size_t hoff = static_cast<size_t>(h) * n * D;

  // this lane's query row (column l32 of the wave's 32-query block)
  const int ql = w * 32 + l32;
  const bool qvalid = ql < rows;
  const bool wave_active = w * 32 < rows;
  int qi = 0;
  if (qvalid) {
    const int pb = offsets[static_cast<size_t>(h) * (c_q + 1) + c] + row0 + ql;
    qi = perm[static_cast<size_t>(h) * n + min(max(pb, 0), n - 1)];
    qi = min(max(qi, 0), n - 1);
  }
  bf16x8 qf[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    const uint4 u = qvalid ? load8<BF16IN>(qv, hoff + static_cast<size_t>(qi) * D + 16 * s + 8 * hf)
                           : make_uint4(0, 0, 0, 0);
    qf[s] = as_bf16x8(u);
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[db][e] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  const int32_t *sel = sel_idx + (static_cast<size_t>(h) * c_q + c) * n;
  const int ntiles = (r + kBN - 1) / kBN;

  uint4 kreg[CH], vreg[CH];
  auto gload = [&](int tile) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int id = t + i * NT;
      {  // K: row-major chunks
        const int key = id / C8, c8 = id % C8, kk = tile * kBN + key;
        if (kk < r) {
          const int row = min(max(sel[kk], 0), n - 1);
          kreg[i] = load8<BF16IN>(kv, hoff + static_cast<size_t>(row) * D + 8 * c8);
        } else {
          kreg[i] = make_uint4(0, 0, 0, 0);
        }
      }
      {  // V: key-fastest chunks (conflict-free transposed LDS writes)
        const int key = id % kBN, c8 = id / kBN, kk = tile * kBN + key;
        if (kk < r) {
          const int row = min(max(sel[kk], 0), n - 1);
          vreg[i] = load8<BF16IN>(vv, hoff + static_cast<size_t>(row) * D + 8 * c8);
        } else {
          vreg[i] = make_uint4(0, 0, 0, 0);
        }
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int id = t + i * NT;
      {
        const int key = id / C8, c8 = id % C8;
        *reinterpret_cast<uint4 *>(&Ks[buf][key * KS + 8 * c8]) = kreg[i];
      }
      {
        const int key = id % kBN, c8 = id / kBN;
        const uint32_t wv[4] = {vreg[i].x, vreg[i].y, vreg[i].z, vreg[i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          Vt[buf][(8 * c8 + 2 * e) * VS + key] = static_cast<uint16_t>(wv[e] & 0xFFFFu);
          Vt[buf][(8 * c8 + 2 * e + 1) * VS + key] = static_cast<uint16_t>(wv[e] >> 16);
        }
      }
    }
  };

  if (ntiles > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    if (tile + 1 < ntiles) gload(tile + 1);
    if (wave_active) {
      // S^T = K_tile . Q^T : two 32-key blocks
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.0f;
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
          const uint4 a = *reinterpret_cast<const uint4 *>(
              &Ks[buf][(kb * 32 + l32) * KS + 16 * s + 8 * hf]);
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), qf[s],
                                                             sacc[kb], 0, 0, 0);
        }
      }
      // online softmax; lane holds keys 32kb + 8i + 4hf + j of query l32
      const int kbase = tile * kBN;
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kbase + kb * 32 + 8 * (e >> 2) + 4 * hf + (e & 3);
          const float x = key < r ? sacc[kb][e] * scale_log2 : -INFINITY;
          sacc[kb][e] = x;
          mt = fmaxf(mt, x);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = fmaxf(m_run, mt);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float psum = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = __builtin_amdgcn_exp2f(sacc[kb][e] - m_new);
          sacc[kb][e] = p;
          psum += p;
        }
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
      // O^T += V_tile^T . P^T, 16 keys per step
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          uint4 pu;
          pu.x = f32_to_bf16(sacc[kb][8 * s2 + 0]) | (static_cast<uint32_t>(f32_to_bf16(sacc[kb][8 * s2 + 1])) << 16);
          pu.y = f32_to_bf16(sacc[kb][8 * s2 + 2]) | (static_cast<uint32_t>(f32_to_bf16(sacc[kb][8 * s2 + 3])) << 16);
          pu.z = f32_to_bf16(sacc[kb][8 * s2 + 4]) | (static_cast<uint32_t>(f32_to_bf16(sacc[kb][8 * s2 + 5])) << 16);
          pu.w = f32_to_bf16(sacc[kb][8 * s2 + 6]) | (static_cast<uint32_t>(f32_to_bf16(sacc[kb][8 * s2 + 7])) << 16);
          const bf16x8 pb = as_bf16x8(pu);
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const uint16_t *vrow = &Vt[buf][(db * 32 + l32) * VS + kb * 32 + 16 * s2];
            const uint2 lo = *reinterpret_cast<const uint2 *>(vrow + 4 * hf);
            const uint2 hi = *reinterpret_cast<const uint2 *>(vrow + 8 + 4 * hf);
            const uint4 a = make_uint4(lo.x, lo.y, hi.x, hi.y);
            oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), pb,
                                                               oacc[db], 0, 0, 0);
          }
        }
    }
    if (tile + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // lanes l and l^32 hold the two halves of one query's row sum
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!qvalid) return;
  const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
  // lane holds O^T[32db + 8i + 4hf + j][query l32]
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int dim = db * 32 + 8 * i + 4 * hf;
      const size_t at = hoff + static_cast<size_t>(qi) * D + dim;
      const float o0 = oacc[db][4 * i + 0] * inv, o1 = oacc[db][4 * i + 1] * inv;
      const float o2 = oacc[db][4 * i + 2] * inv, o3 = oacc[db][4 * i + 3] * inv;
      if (BF16IN) {
        uint2 u;
        u.x = f32_to_bf16(o0) | (static_cast<uint32_t>(f32_to_bf16(o1)) << 16);
        u.y = f32_to_bf16(o2) | (static_cast<uint32_t>(f32_to_bf16(o3)) << 16);
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(ov) + at) = u;
      } else {
        *reinterpret_cast<float4 *>(static_cast<float *>(ov) + at) = make_float4(o0, o1, o2, o3);
      }
    }
}

// Work list: per head, every cluster's queries cut into chunks of kBM rows,
// clusters in order; unused slots get rows = 0.
__global__ __launch_bounds__(1024) void attn_items_kernel(
    int n, int c_q, int items_per_head, const int32_t *__restrict__ offsets,
    const int32_t *__restrict__ sel_counts, int4 *items) {
  __shared__ int wtot[16];
  const int h = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int32_t *off = offsets + static_cast<size_t>(h) * (c_q + 1);
  int4 *out = items + static_cast<size_t>(h) * items_per_head;
  int run = 0;
  for (int c0 = 0; c0 < c_q; c0 += 1024) {
    const int c = c0 + t;
    int cnt = 0, rsel = 0;
    if (c < c_q) {
      cnt = min(max(off[c + 1] - off[c], 0), n);
      rsel = min(max(sel_counts[static_cast<size_t>(h) * c_q + c], 0), n);
    }
    const int k = (cnt + kBM - 1) / kBM;
    const int incl = wave_incl_scan(k);
    if (lane == 63) wtot[w] = incl;
    __syncthreads();
    int base = 0, tot = 0;
    for (int i = 0; i < 16; ++i) {
      if (i < w) base += wtot[i];
      tot += wtot[i];
    }
    __syncthreads();
    const int first = run + base + incl - k;
    for (int q = 0; q < k; ++q) {
      const int slot = first + q;
      if (slot < items_per_head)
        out[slot] = make_int4(c, q * kBM, min(kBM, cnt - q * kBM), rsel);
    }
    run += tot;
  }
  for (int slot = run + t; slot < items_per_head; slot += 1024)
    out[slot] = make_int4(0, 0, 0, 0);
}

template <int D>
hipError_t launch_attn(int heads, int n, bool bf16, const void *q,
                       const void *k, const void *v, void *o, int c_q,
                       const int32_t *offsets, const int32_t *perm,
                       const int32_t *sel_idx, const int4 *items, int iph,
                       float scale_log2, hipStream_t s) {
  const dim3 grid(iph, heads), block(kNW * 64);
  if (bf16)
    hipLaunchKernelGGL((attn_kernel<D, true>), grid, block, 0, s, n, c_q, iph, q,
                       k, v, o, offsets, perm, sel_idx, items, scale_log2);
  else
    hipLaunchKernelGGL((attn_kernel<D, false>), grid, block, 0, s, n, c_q, iph,
                       q, k, v, o, offsets, perm, sel_idx, items, scale_log2);
  return hipGetLastError();
}

}  // namespace

int attn_items_per_head(int n, int c_q) { return (n + kBM - 1) / kBM + c_q; }

hipError_t attention_run(int heads, int n, int d, bool bf16, const void *q,
                         const void *k, const void *v, void *o, int c_q,
                         const int32_t *offsets, const int32_t *perm,
                         const int32_t *sel_counts, const int32_t *sel_idx,
                         float scale, int4 *items, hipStream_t s) {
  const int iph = attn_items_per_head(n, c_q);
  hipLaunchKernelGGL(attn_items_kernel, dim3(heads), dim3(1024), 0, s, n, c_q,
                     iph, offsets, sel_counts, items);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const float sl2 = scale * 1.4426950408889634f;
  if (d == 128)
    return launch_attn<128>(heads, n, bf16, q, k, v, o, c_q, offsets, perm,
                            sel_idx, items, iph, sl2, s);
  return launch_attn<64>(heads, n, bf16, q, k, v, o, c_q, offsets, perm,
                         sel_idx, items, iph, sl2, s);
}

}  // namespace scope
