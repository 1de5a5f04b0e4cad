// Sparse attention over the selected keys (Eq. 11; Alg. 1 last step), and
// dense attention (Eq. 1) as the one-cluster special case.
//
// Work item = (head, query cluster c, chunk of up to 32*NW of its queries).
// The block gathers the cluster's selected keys 64 at a time, K and V rows
// both into LDS row-major.  Each wave owns 32 queries and runs
//   S^T (64 keys x 32 queries) = K_tile . Q^T       bf16 MFMA 32x32x16,
//                                 two 32-key chains interleaved
//   online softmax in fp32 (exp2 domain), one query per lane column, one
//                                 max / rescale decision per 64-key tile
//   O^T (d x 32 queries)      += V_tile^T . P^T      bf16 MFMA 32x32x16
// The S^T accumulator layout is reused directly as the B operand of the
// second product, so P never leaves registers; the matching V^T operand
// comes from the row-major V tile through transposing LDS reads
// (ds_read_b64_tr_b16).  K/V tiles are double buffered: the next tiles'
// gathers are in flight during the MFMAs.  bf16 gathers go through buffer
// resources, whose range checks turn every out-of-range index into a zero
// read instead of a fault.  At d = 128 with bf16 inputs (attn_kernel_dma)
// the buffer unit writes the gathered rows straight into LDS; fp32 inputs
// (rounded to bf16 on the way) and d = 64 stage rows through registers
// (attn_kernel).
#include <math.h>

#include <mutex>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kBN = 64;          // keys per tile
constexpr int kNW = 8;           // waves per block
constexpr int kQB = 1;           // 32-query column blocks per wave
constexpr int kBM = 32 * kQB * kNW;
constexpr float kRescale = 8.0f; // lazy rescale: running max may lag by 2^8

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) {
  return __builtin_bit_cast(bf16x8, u);
}

// Two floats -> packed bf16 (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  bf16x2 r;
  r[0] = static_cast<__bf16>(a);
  r[1] = static_cast<__bf16>(b);
  return __builtin_bit_cast(uint32_t, r);
}

// 8 consecutive input elements as packed bf16.
template <bool BF16IN>
__device__ __forceinline__ uint4 load8(const void *base, size_t elem) {
  if (BF16IN) {
    return *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(base) + elem);
  } else {
    const float4 a = *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem);
    const float4 b = *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem + 4);
    return make_uint4(pack_bf16(a.x, a.y), pack_bf16(a.z, a.w), pack_bf16(b.x, b.y),
                      pack_bf16(b.z, b.w));
  }
}

// Work items run in list order: heads one after the other and, within a
// head, by estimated cost, largest first, with a cluster's row chunks
// adjacent.  All XCDs work on the same head at a time, so one head's K/V
// (60 MB at 118800 x 128 bf16) is what the 256 MB memory-side cache has to
// hold.
//
// Block b runs on XCD b mod 8.  Runs of kRun consecutive work items (the
// chunks of one cluster, which gather the same K/V rows) go to one XCD so
// that they share its L2; windows of 8 * kRun items still follow the list
// order.  A partial last window keeps the identity map.
constexpr int kXcds = 8, kRun = 4;
__device__ __forceinline__ int xcd_item(int b, int total) {
  constexpr int W = kXcds * kRun;
  const int w0 = b / W * W;
  if (w0 + W > total) return b;
  const int r = b - w0;
  return w0 + (r % kXcds) * kRun + r / kXcds;
}

template <int D, bool BF16IN>
__global__ __launch_bounds__(kNW * 64) void attn_kernel(
    int n, int c_q, int items_per_head, int total_items,
    const void *__restrict__ qv, const void *__restrict__ kv,
    const void *__restrict__ vv, void *ov, const int32_t *__restrict__ offsets,
    const int32_t *__restrict__ perm, const int32_t *__restrict__ sel_idx,
    const int4 *__restrict__ items, float scale_log2) {
  constexpr int NT = kNW * 64;
  // LDS row strides (bf16 elements): K rows are read 16 bytes per lane, 16
  // consecutive rows at a time, so 16 bytes of padding keep them on distinct
  // banks; the transposing V reads take 64 bytes from each of four rows per
  // 32 lanes, so V rows are padded by 64 bytes (stride = 64 mod 256 bytes)
  constexpr int KS = D + 8;
  constexpr int KSV = D + 32;
  constexpr int C8 = D / 8;       // 16-byte chunks per row
  // staging: the first half of the block stages V (4 consecutive keys of one
  // 8-channel column per thread), the second half K (RK consecutive rows of
  // one 16-byte column per thread)
  constexpr int HALF = NT / 2;
  constexpr int RK = kBN * C8 / HALF;       // rows per staging thread
  static_assert(kBN * C8 % HALF == 0 && RK >= 1 && RK <= 4, "tile/threads mismatch");
  constexpr int NR = 4;                     // rows fetched per thread per tile
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kBN * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][kBN * KSV];

  const int item = xcd_item(static_cast<int>(blockIdx.x), total_items);
  if (item >= total_items) return;
  const int h = item / items_per_head;
  const int4 it = items[2 * item];  // work slots of this kernel hold one chunk
  const int c = it.x, row0 = it.y, rows = it.z, r = it.w;
  if (rows <= 0) return;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const size_t hoff = static_cast<size_t>(h) * n * D;

  // queries: wave w owns rows w*32*kQB + 32*qb + l32 of the chunk
  int qi[kQB];
  bool qvalid[kQB];
  bf16x8 qf[kQB][D / 16];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const int ql = w * 32 * kQB + 32 * qb + l32;
    qvalid[qb] = ql < rows;
    qi[qb] = 0;
    if (qvalid[qb]) {
      const int pb = offsets[static_cast<size_t>(h) * (c_q + 1) + c] + row0 + ql;
      qi[qb] = min(max(perm[static_cast<size_t>(h) * n + min(max(pb, 0), n - 1)], 0), n - 1);
    }
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
      qf[qb][s] = as_bf16x8(qvalid[qb] ? load8<BF16IN>(qv, hoff + static_cast<size_t>(qi[qb]) * D + 16 * s + 8 * hf)
                                       : make_uint4(0, 0, 0, 0));
  }
  const bool wave_active = w * 32 * kQB < rows;

  f32x16 oacc[kQB][D / 32];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) oacc[qb][db][e] = 0.0f;
  float m_run[kQB], l_run[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.0f;
  }

  const int32_t *sel = sel_idx + (static_cast<size_t>(h) * c_q + c) * n;
  const int ntiles = (r + kBN - 1) / kBN;

  // this thread's staging role (wave-uniform, kept in scalar registers):
  // the first half of the block stages V rows, the second K rows, both
  // row-major, RK consecutive rows of one 16-byte column per thread
  const bool is_v = __builtin_amdgcn_readfirstlane(t) < HALF;
  const int u = is_v ? t : t - HALF;
  const int c8 = u % C8;
  const int key0 = RK * (u / C8) % kBN;
  const bool stores = true;
  // transposing reads of V (ds_read_b64_tr_b16): source lane s supplies
  // row 4*(s/32) + (s%16)/4 and channels 16*((s/16)%2) + 4*(s%4) .. +3 of a
  // 16-key step; lane L then holds 4 consecutive keys of channel L%32
  const int tr_off = (4 * (lane >> 5) + ((lane & 15) >> 2)) * KSV + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const void *src = is_v ? vv : kv;
  // bf16 inputs are gathered through buffer resources: out-of-range offsets
  // (index slots past the key set, any bad row) read as zero in hardware,
  // so no index needs clamping; the host guarantees n * D * 2 < 2^32
  const __amdgpu_buffer_rsrc_t rsel = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t *>(sel), static_cast<short>(0), r * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t *>(static_cast<const uint16_t *>(src) + hoff), static_cast<short>(0),
      static_cast<int>(static_cast<uint32_t>(n) * (D * 2)), 0x00020000);

  // Software pipeline, two tiles deep: step T requests the row indices of
  // tile T+3 first and the rows of tile T+2 after its compute, so waiting for
  // indices never waits for rows in flight (vector loads complete in order)
  // and the rows have a whole step to arrive.  Every load is
  // unconditional with clamped indices, so the pipeline has no branches;
  // rows past the key set are fetched but masked (or never read).
  int selA[NR], selB[NR];
  uint4 dA[NR], dB[NR];
  auto load_sel = [&](int tile, int (&sx)[NR]) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      if constexpr (BF16IN)
        sx[i] = __builtin_amdgcn_raw_buffer_load_b32(rsel, (tile * kBN + key0 + i % RK) * 4, 0, 0);
      else
        sx[i] = sel[min(tile * kBN + key0 + i % RK, n - 1)];
    }
  };
  auto load_rows = [&](const int (&sx)[NR], uint4 (&dx)[NR]) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      if constexpr (BF16IN) {
        const auto v4 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, sx[i] * (D * 2) + 16 * c8, 0, 0);
        dx[i] = make_uint4(v4[0], v4[1], v4[2], v4[3]);
      } else {
        const int row = min(max(sx[i], 0), n - 1);
        dx[i] = load8<BF16IN>(src, hoff + static_cast<size_t>(row) * D + 8 * c8);
      }
    }
  };
  auto store_rows = [&](int buf, const uint4 (&dx)[NR]) {
    if (!stores) return;
    uint16_t *dst = is_v ? Vs[buf] : Ks[buf];
#pragma unroll
    for (int i = 0; i < RK; ++i)
      *reinterpret_cast<uint4 *>(&dst[(key0 + i) * (is_v ? KSV : KS) + 8 * c8]) = dx[i];
  };

  auto compute = [&](int tile, int buf) {
    if (!wave_active) return;
    // S^T for both 32-key blocks of the tile: two independent MFMA chains,
    // interleaved so the matrix pipe never waits on one accumulator
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.0f;
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4 *>(
            &Ks[buf][(kb * 32 + l32) * KS + 16 * s + 8 * hf]));
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[0][s], sacc[kb], 0, 0, 0);
      }
    // lane holds keys 32kb + 8(e/4) + 4hf + (e%4) of query column l32
    const int kbase = tile * kBN;
    if (kbase + kBN > r) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kbase + 32 * kb + 8 * (e >> 2) + 4 * hf + (e & 3) >= r) sacc[kb][e] = -INFINITY;
    }
    float mx0 = fmaxf(sacc[0][0], sacc[0][1]), mx1 = fmaxf(sacc[1][0], sacc[1][1]);
#pragma unroll
    for (int e = 2; e < 16; e += 2) {
      mx0 = fmaxf(fmaxf(mx0, sacc[0][e]), sacc[0][e + 1]);
      mx1 = fmaxf(fmaxf(mx1, sacc[1][e]), sacc[1][e + 1]);
    }
    float mx = fmaxf(mx0, mx1);
    {
      // the other half-wave holds the query's other keys
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    const float mt = mx * scale_log2;
    // rescale only when the running max falls too far behind; the branch is
    // wave-wide but each query decides for itself (alpha = 1 otherwise), so
    // a query's result never depends on its wave-mates
    const bool behind = mt > m_run[0] + kRescale;
    if (__ballot(behind)) {
      const float m_new = behind ? fmaxf(m_run[0], mt) : m_run[0];
      const float alpha = behind ? __builtin_amdgcn_exp2f(m_run[0] - m_new) : 1.0f;
      l_run[0] *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[0][db][e] *= alpha;
      m_run[0] = m_new;
    }
    const float neg_m = -m_run[0];
    uint4 pk[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float p[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) p[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], scale_log2, neg_m));
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        pk[kb][s2] = make_uint4(pack_bf16(p[8 * s2 + 0], p[8 * s2 + 1]),
                                pack_bf16(p[8 * s2 + 2], p[8 * s2 + 3]),
                                pack_bf16(p[8 * s2 + 4], p[8 * s2 + 5]),
                                pack_bf16(p[8 * s2 + 6], p[8 * s2 + 7]));
    }
    // the row sum of the bf16 weights the PV product uses, two per dot2
    {
      const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3F803F80u);
      float ps[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const uint4 w4 = pk[kb][s2];
          ps[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.x), one, ps[0], false);
          ps[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.y), one, ps[1], false);
          ps[2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.z), one, ps[2], false);
          ps[3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.w), one, ps[3], false);
        }
      l_run[0] += (ps[0] + ps[1]) + (ps[2] + ps[3]);
    }
    // O^T += V_tile^T . P^T in 16-key steps, four independent accumulators
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const uint16_t *vt = &Vs[buf][(kb * 32 + 16 * s2) * KSV + db * 32 + tr_off];
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(vt));
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(vt + 8 * KSV));
          const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
          const bf16x8 a = as_bf16x8(make_uint4(l2.x, l2.y, h2.x, h2.y));
          oacc[0][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              a, as_bf16x8(pk[kb][s2]), oacc[0][db], 0, 0, 0);
        }
  };

  // one pipeline step: compute tile T from LDS while tile T+1 (already in
  // registers `cur`) lands in the other LDS buffer; the rows of tile T+2
  // are requested after the compute (they have until the end of the next
  // step), so the MFMAs of this step never wait for them
  auto step = [&](int tile, int (&sel_next)[NR], uint4 (&cur)[NR],
                  int (&sel_far)[NR], uint4 (&far)[NR]) {
    load_sel(tile + 3, sel_next);
    compute(tile, tile & 1);
    load_rows(sel_far, far);
    store_rows((tile + 1) & 1, cur);
    __syncthreads();
  };

  if (ntiles > 0) {
    load_sel(0, selA);
    load_sel(1, selB);
    load_rows(selA, dA);   // tile 0
    load_sel(2, selA);
    load_rows(selB, dB);   // tile 1
    store_rows(0, dA);
  }
  __syncthreads();
  // registers: tile T+1 is in (T even ? dB : dA); the row indices of tile
  // T+2 in (T even ? selA : selB)
  for (int tile = 0; tile < ntiles; tile += 2) {
    step(tile, selB, dB, selA, dA);
    if (tile + 1 < ntiles) step(tile + 1, selA, dA, selB, dB);
  }

#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    // lanes l and l^32 hold the two halves of one query's row sum
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
    if (!qvalid[qb]) continue;
    const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
    // lane holds O^T[32db + 8i + 4hf + j][query]
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int dim = db * 32 + 8 * i + 4 * hf;
        const size_t at = hoff + static_cast<size_t>(qi[qb]) * D + dim;
        const float o0 = oacc[qb][db][4 * i + 0] * inv, o1 = oacc[qb][db][4 * i + 1] * inv;
        const float o2 = oacc[qb][db][4 * i + 2] * inv, o3 = oacc[qb][db][4 * i + 3] * inv;
        if (BF16IN) {
          *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(ov) + at) =
              make_uint2(pack_bf16(o0, o1), pack_bf16(o2, o3));
        } else {
          *reinterpret_cast<float4 *>(static_cast<float *>(ov) + at) = make_float4(o0, o1, o2, o3);
        }
      }
  }
}

// bf16 inputs at d = 128: the same computation with the K/V rows gathered
// straight into LDS by the buffer unit (one 1 KB load per 4 rows, no
// staging registers).  Rows land unpadded, so 16-byte slots are
// XOR-swizzled: slot = chunk ^ (row mod 16) in K tiles (16-row b128 reads)
// and chunk ^ 4 (row mod 4) in V tiles (4-row transposing reads).  A work
// slot may hold two chunks (A, B) of different clusters: A's waves come
// first, each chunk has its own tiles, and every wave gathers its share of
// both.  The four tile buffers (K and V, two steps) are distinct LDS
// objects, each holding the tiles of both chunks, so the compiler's waits
// for the loads into one never hold up the reads of another.
using DmaTile = uint16_t[2][kBN * 128];

template <bool PAIRED>
__device__ __forceinline__ void attn_dma_body(
    int n, int c_q, int h, int4 ia, int4 ib, const void *__restrict__ qv,
    const void *__restrict__ kv, const void *__restrict__ vv, void *ov,
    const int32_t *__restrict__ offsets, const int32_t *__restrict__ perm,
    const int32_t *__restrict__ sel_idx, float scale_log2, DmaTile &K0, DmaTile &K1,
    DmaTile &V0, DmaTile &V1) {
  constexpr int D = 128;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const size_t hoff = static_cast<size_t>(h) * n * D;
  // this wave's chunk: A's ceil(rows / 32) waves first, then B's
  const int wa = (ia.z + 31) >> 5;
  const int g = PAIRED && w >= wa ? 1 : 0;
  const int4 it = g ? ib : ia;
  const int c = it.x, row0 = it.y, rows = it.z, r = it.w;
  const int wl = w - (g ? wa : 0);

  // queries: wave wl of the chunk owns its rows 32 wl + l32
  const int ql = wl * 32 + l32;
  const bool qvalid = ql < rows;
  int qi = 0;
  if (qvalid) {
    const int pb = offsets[static_cast<size_t>(h) * (c_q + 1) + c] + row0 + ql;
    qi = min(max(perm[static_cast<size_t>(h) * n + min(max(pb, 0), n - 1)], 0), n - 1);
  }
  bf16x8 qf[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
    qf[s] = as_bf16x8(qvalid ? load8<true>(qv, hoff + static_cast<size_t>(qi) * D + 16 * s + 8 * hf)
                             : make_uint4(0, 0, 0, 0));
  const bool wave_active = wl * 32 < rows;

  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[db][e] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  // key tiles of each chunk; the block steps through the longer list
  const int ntA = (ia.w + kBN - 1) / kBN, ntB = PAIRED ? (ib.w + kBN - 1) / kBN : 0;
  const int ntiles = ntA > ntB ? ntA : ntB;
  const int nt_own = (r + kBN - 1) / kBN;
  auto sel_rsrc = [&](const int4 &e) {
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(sel_idx + (static_cast<size_t>(h) * c_q + e.x) * n),
        static_cast<short>(0), e.w * 4, 0x00020000);
  };
  const __amdgpu_buffer_rsrc_t rselA = sel_rsrc(ia);
  const __amdgpu_buffer_rsrc_t rselB = sel_rsrc(PAIRED ? ib : ia);
  const int nbytes = static_cast<int>(static_cast<uint32_t>(n) * (D * 2));
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t *>(static_cast<const uint16_t *>(kv) + hoff), static_cast<short>(0), nbytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t *>(static_cast<const uint16_t *>(vv) + hoff), static_cast<short>(0), nbytes, 0x00020000);

  // gathers: wave w brings rows 8w .. 8w+7 of each chunk's tile, four rows
  // (1 KB) per load; lane L covers row 8w + 4i + L/16, slot L%16, and
  // fetches the chunk that the swizzle puts there.  Past the end of a
  // chunk's key list its index loads read zeros, so its gathers fetch row 0
  // (the pairing matches key counts, so few such tiles).
  struct Idx {
    int a[2], b[2];
  };
  auto load_idx = [&](int tile, Idx &ix) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int at = (tile * kBN + 8 * w + 4 * i + (lane >> 4)) * 4;
      ix.a[i] = __builtin_amdgcn_raw_buffer_load_b32(rselA, at, 0, 0);
      ix.b[i] = PAIRED ? __builtin_amdgcn_raw_buffer_load_b32(rselB, at, 0, 0) : 0;
    }
  };
  auto gather_k = [&](uint16_t (*kbuf)[kBN * D], const Idx &ix) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = 8 * w + 4 * i + (lane >> 4), s = lane & 15;
      const int col = 16 * (s ^ (row & 15));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, kbuf[0] + (8 * w + 4 * i) * D, 16, ix.a[i] * (D * 2) + col, 0, 0, 0);
      if constexpr (PAIRED)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, kbuf[1] + (8 * w + 4 * i) * D, 16, ix.b[i] * (D * 2) + col, 0, 0, 0);
    }
  };
  auto gather_v = [&](uint16_t (*vbuf)[kBN * D], const Idx &ix) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = 8 * w + 4 * i + (lane >> 4), s = lane & 15;
      const int col = 16 * (s ^ (4 * (row & 3)));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, vbuf[0] + (8 * w + 4 * i) * D, 16, ix.a[i] * (D * 2) + col, 0, 0, 0);
      if constexpr (PAIRED)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, vbuf[1] + (8 * w + 4 * i) * D, 16, ix.b[i] * (D * 2) + col, 0, 0, 0);
    }
  };

  // transposing V reads: lane L supplies row rl = 4(L/32) + (L%16)/4 of a
  // 16-key step, chunk 4db + 2((L/16)%2) + (L%4)/2, half L%2
  const int rl = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int vch = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
  const int vsw = 4 * (rl & 3);
  const int vhalf = 4 * (lane & 1);   // elements

  // tile T of this wave's chunk from kt/vt0; the gathers of tile T+1 into
  // kn/vn are issued between the phases: K rows after the S MFMAs, V rows
  // before the PV MFMAs
  auto compute = [&](int tile, const uint16_t *kt, const uint16_t *vt0,
                     uint16_t (*kn)[kBN * D], uint16_t (*vn)[kBN * D], const Idx &ix) {
    if (!wave_active || tile >= nt_own) {
      gather_k(kn, ix);
      gather_v(vn, ix);
      return;
    }
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.0f;
    const int krow = l32;  // + 32 kb; the swizzle sees row mod 16 only
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int slot = (2 * s + hf) ^ (krow & 15);
        const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4 *>(
            &kt[(kb * 32 + krow) * D + 8 * slot]));
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], sacc[kb], 0, 0, 0);
      }
    // each K operand is read from LDS two MFMAs ahead of its use
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
    for (int i = 0; i < 14; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    gather_k(kn, ix);
    const int kbase = tile * kBN;
    if (kbase + kBN > r) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kbase + 32 * kb + 8 * (e >> 2) + 4 * hf + (e & 3) >= r) sacc[kb][e] = -INFINITY;
    }
    float mx0 = fmaxf(sacc[0][0], sacc[0][1]), mx1 = fmaxf(sacc[1][0], sacc[1][1]);
#pragma unroll
    for (int e = 2; e < 16; e += 2) {
      mx0 = fmaxf(fmaxf(mx0, sacc[0][e]), sacc[0][e + 1]);
      mx1 = fmaxf(fmaxf(mx1, sacc[1][e]), sacc[1][e + 1]);
    }
    float mx = fmaxf(mx0, mx1);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    const float mt = mx * scale_log2;
    const bool behind = mt > m_run + kRescale;
    if (__ballot(behind)) {
      const float m_new = behind ? fmaxf(m_run, mt) : m_run;
      const float alpha = behind ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
      m_run = m_new;
    }
    const float neg_m = -m_run;
    uint4 pk[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float p[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) p[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], scale_log2, neg_m));
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        pk[kb][s2] = make_uint4(pack_bf16(p[8 * s2 + 0], p[8 * s2 + 1]),
                                pack_bf16(p[8 * s2 + 2], p[8 * s2 + 3]),
                                pack_bf16(p[8 * s2 + 4], p[8 * s2 + 5]),
                                pack_bf16(p[8 * s2 + 6], p[8 * s2 + 7]));
    }
    {
      const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3F803F80u);
      float ps[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const uint4 w4 = pk[kb][s2];
          ps[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.x), one, ps[0], false);
          ps[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.y), one, ps[1], false);
          ps[2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.z), one, ps[2], false);
          ps[3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4.w), one, ps[3], false);
        }
      l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
    }
    gather_v(vn, ix);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const int vrow = kb * 32 + 16 * s2 + rl;  // hi: vrow + 8, same swizzle
          const int slot = (4 * db + vch) ^ vsw;
          const uint16_t *p0 = &vt0[vrow * D + 8 * slot + vhalf];
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p0));
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p0 + 8 * D));
          const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
          const bf16x8 a = as_bf16x8(make_uint4(l2.x, l2.y, h2.x, h2.y));
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(pk[kb][s2]), oacc[db], 0, 0, 0);
        }
  };

  // one step: indices of tile T+2 requested, tile T computed while tile T+1
  // is gathered into the free buffers; every wave's gathers land before the
  // barrier
  Idx cidx, nidx;
  auto step = [&](int tile, uint16_t (*kc)[kBN * D], uint16_t (*vc)[kBN * D],
                  uint16_t (*kn)[kBN * D], uint16_t (*vn)[kBN * D]) {
    load_idx(tile + 2, nidx);
    compute(tile, kc[g], vc[g], kn, vn, cidx);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's gathers are in LDS
    __syncthreads();
    cidx = nidx;
  };

  if (ntiles > 0) {
    Idx ix0;
    load_idx(0, ix0);
    load_idx(1, cidx);
    gather_k(K0, ix0);
    gather_v(V0, ix0);
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  for (int tile = 0; tile < ntiles; tile += 2) {
    step(tile, K0, V0, K1, V1);
    if (tile + 1 < ntiles) step(tile + 1, K1, V1, K0, V0);
  }

  // lanes l and l^32 hold the two halves of one query's row sum
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!qvalid) return;
  const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int dim = db * 32 + 8 * i + 4 * hf;
      const size_t at = hoff + static_cast<size_t>(qi) * D + dim;
      const float o0 = oacc[db][4 * i + 0] * inv, o1 = oacc[db][4 * i + 1] * inv;
      const float o2 = oacc[db][4 * i + 2] * inv, o3 = oacc[db][4 * i + 3] * inv;
      *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(ov) + at) =
          make_uint2(pack_bf16(o0, o1), pack_bf16(o2, o3));
    }
}

__global__ __launch_bounds__(kNW * 64) void attn_kernel_dma(
    int n, int c_q, int items_per_head, int total_items,
    const void *__restrict__ qv, const void *__restrict__ kv,
    const void *__restrict__ vv, void *ov, const int32_t *__restrict__ offsets,
    const int32_t *__restrict__ perm, const int32_t *__restrict__ sel_idx,
    const int4 *__restrict__ items, float scale_log2) {
  __shared__ __attribute__((aligned(16))) DmaTile K0;
  __shared__ __attribute__((aligned(16))) DmaTile K1;
  __shared__ __attribute__((aligned(16))) DmaTile V0;
  __shared__ __attribute__((aligned(16))) DmaTile V1;
  const int item = xcd_item(static_cast<int>(blockIdx.x), total_items);
  if (item >= total_items) return;
  const int h = item / items_per_head;
  const int4 ia = items[2 * item], ib = items[2 * item + 1];
  if (ia.z <= 0) return;
  // one block-uniform branch: a lone chunk gathers one set of tiles
  if (ib.z > 0)
    attn_dma_body<true>(n, c_q, h, ia, ib, qv, kv, vv, ov, offsets, perm, sel_idx, scale_log2,
                        K0, K1, V0, V1);
  else
    attn_dma_body<false>(n, c_q, h, ia, ib, qv, kv, vv, ov, offsets, perm, sel_idx, scale_log2,
                         K0, K1, V0, V1);
}

// Work list of one head.  Every cluster's queries are cut into chunks of kBM
// rows; a block runs one work slot of two entries (A, B), each (cluster,
// first row, rows, selected keys), B empty (rows = 0) or a second chunk that
// shares the block: A's chunk takes waves 0 .. ceil(rows_A / 32) - 1 and
// B's the next ones.  Slots: the clusters' full chunks in cluster order,
// then their remainder chunks (fewer than kBM rows), then empty slots.  With
// `pair`, remainders are paired so that the two chunks need at most kNW
// waves together: bucketed by their wave count w and ordered by key count
// within a bucket, bucket w (largest first) takes partners from bucket
// min(8 - w, w) down to 1 in key-count order, so paired chunks run similar
// numbers of key tiles.  Remainders left without a partner (among them every
// remainder of 8 waves) run alone.  Up to kSortMaxSlots slots per head, the
// head's slots are then reordered by estimated cost, largest first (ties
// keep their order, so a cluster's full chunks stay adjacent): the
// expensive blocks of each head start early and the cheap ones fill in
// behind them, which shortens the launch's tail.
constexpr int kPairMaxClusters = 2048;  // pairing up to this many clusters
constexpr int kSortMaxSlots = 2048;     // cost-ordered work lists up to this many slots
__global__ __launch_bounds__(1024) void attn_items_kernel(
    int n, int c_q, int items_per_head, int pair, const int32_t *__restrict__ offsets,
    const int32_t *__restrict__ sel_counts, int4 *items) {
  __shared__ int wtot[16];
  __shared__ int rem_w[kPairMaxClusters], rem_r[kPairMaxClusters], ord[kPairMaxClusters];
  __shared__ int bucket_n[kNW + 1], bucket_at[kNW + 1];
  __shared__ int4 seg[64];   // (A's first ordinal, B's first ordinal or -1, count, same bucket)
  __shared__ int seg_at[65], nseg, full_tot;
  __shared__ int4 staged[2 * kSortMaxSlots];
  __shared__ unsigned long long cost[kSortMaxSlots];
  const int h = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int32_t *off = offsets + static_cast<size_t>(h) * (c_q + 1);
  const int32_t *scnt = sel_counts + static_cast<size_t>(h) * c_q;
  int4 *out = items + static_cast<size_t>(h) * items_per_head * 2;
  const bool do_pair = pair && c_q <= kPairMaxClusters;
  const bool sorted = items_per_head <= kSortMaxSlots;
  auto count_of = [&](int c) { return min(max(off[c + 1] - off[c], 0), n); };
  auto keys_of = [&](int c) { return min(max(scnt[c], 0), n); };
  auto put = [&](int slot, int4 a, int4 b) {
    if (slot < items_per_head) {
      if (sorted) {
        staged[2 * slot] = a;
        staged[2 * slot + 1] = b;
      } else {
        out[2 * slot] = a;
        out[2 * slot + 1] = b;
      }
    }
  };
  // the staged slots, largest estimated cost first: a slot costs its key
  // tiles times the per-tile time of its wave count (about 1.45x for 5-8
  // waves against 1-4) and of a second chunk's gathers (about 1.15x).  The
  // first `used` slots hold chunks; the empty ones after them stay in place.
  auto emit_sorted = [&](int used) {
    if (!sorted) return;
    __syncthreads();
    for (int i = t; i < used; i += 1024) {
      const int4 a = staged[2 * i], b = staged[2 * i + 1];
      const int ta = (a.w + kBN - 1) / kBN, tb = b.z > 0 ? (b.w + kBN - 1) / kBN : 0;
      const int waves = (a.z + 31) / 32 + (b.z > 0 ? (b.z + 31) / 32 : 0);
      const uint32_t per = waves > 4 ? (b.z > 0 ? 196u : 171u) : (b.z > 0 ? 135u : 118u);
      const uint32_t k = static_cast<uint32_t>(ta > tb ? ta : tb) * per;
      // descending cost, then ascending slot: one unsigned comparison
      cost[i] = (static_cast<unsigned long long>(k) << 32) | static_cast<uint32_t>(~i);
    }
    __syncthreads();
    for (int i = t; i < items_per_head; i += 1024) {
      int rank = i;
      if (i < used) {
        const unsigned long long ci = cost[i];
        rank = 0;
#pragma unroll 8
        for (int j = 0; j < used; ++j) rank += cost[j] > ci ? 1 : 0;
      }
      out[2 * rank] = staged[2 * i];
      out[2 * rank + 1] = staged[2 * i + 1];
    }
  };
  const int4 none = make_int4(0, 0, 0, 0);
  if (t <= kNW) bucket_n[t] = 0;
  __syncthreads();
  // full chunks, in cluster order
  int run = 0;
  for (int c0 = 0; c0 < c_q; c0 += 1024) {
    const int c = c0 + t;
    int cnt = 0, rsel = 0;
    if (c < c_q) {
      cnt = count_of(c);
      rsel = keys_of(c);
    }
    const int k = cnt / kBM, rem = cnt - k * kBM;
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
    for (int q = 0; q < k; ++q) put(first + q, make_int4(c, q * kBM, kBM, rsel), none);
    run += tot;
    // remainders, bucketed by wave count for pairing
    if (do_pair && c < c_q) {
      rem_w[c] = rem > 0 ? (rem + 31) / 32 : 0;
      rem_r[c] = rsel;
      if (rem > 0) atomicAdd(&bucket_n[rem_w[c]], 1);
    }
  }
  if (t == 0) full_tot = run;
  __syncthreads();
  if (!do_pair) {
    // remainders alone, in cluster order, after the full chunks
    int at = 0;
    for (int c0 = 0; c0 < c_q; c0 += 1024) {
      const int c = c0 + t;
      int cnt = 0, rsel = 0;
      if (c < c_q) {
        cnt = count_of(c);
        rsel = keys_of(c);
      }
      const int rem = cnt % kBM, has = rem > 0 ? 1 : 0;
      const int incl = wave_incl_scan(has);
      if (lane == 63) wtot[w] = incl;
      __syncthreads();
      int base = 0, tot = 0;
      for (int i = 0; i < 16; ++i) {
        if (i < w) base += wtot[i];
        tot += wtot[i];
      }
      __syncthreads();
      if (has) put(full_tot + at + base + incl - 1, make_int4(c, cnt - rem, rem, rsel), none);
      at += tot;
    }
    for (int slot = full_tot + at + t; slot < items_per_head; slot += 1024) put(slot, none, none);
    emit_sorted(min(full_tot + at, items_per_head));
    return;
  }
  // ordinal of each remainder within (bucket ascending, keys ascending,
  // cluster ascending)
  if (t == 0) {
    int a = 0;
    for (int b = 0; b <= kNW; ++b) {
      bucket_at[b] = a;
      a += b == 0 ? 0 : bucket_n[b];
    }
  }
  __syncthreads();
  for (int c = t; c < c_q; c += 1024) {
    const int wc = rem_w[c];
    if (wc == 0) continue;
    const int rc = rem_r[c];
    int pos = bucket_at[wc];
    for (int o = 0; o < c_q; ++o)
      if (rem_w[o] == wc && (rem_r[o] < rc || (rem_r[o] == rc && o < c))) ++pos;
    ord[pos] = c;
  }
  // the pairing plan (at most kNW * kNW segments), one thread
  if (t == 0) {
    int nxt[kNW + 1], left[kNW + 1];
    for (int b = 0; b <= kNW; ++b) {
      nxt[b] = bucket_at[b];
      left[b] = b == 0 ? 0 : bucket_n[b];
    }
    int ns = 0;
    for (int wa = kNW; wa >= 1; --wa) {
      for (int wb = min(kNW - wa, wa); wb >= 1 && left[wa] > 0; --wb) {
        const int m = wb == wa ? left[wa] / 2 : min(left[wa], left[wb]);
        if (m <= 0) continue;
        seg[ns++] = make_int4(nxt[wa], nxt[wb], m, wb == wa ? 1 : 0);
        if (wb == wa) {
          nxt[wa] += 2 * m;
          left[wa] -= 2 * m;
        } else {
          nxt[wa] += m;
          left[wa] -= m;
          nxt[wb] += m;
          left[wb] -= m;
        }
      }
      if (left[wa] > 0) {  // no partner left: alone
        seg[ns++] = make_int4(nxt[wa], -1, left[wa], 0);
        nxt[wa] += left[wa];
        left[wa] = 0;
      }
    }
    int a = 0;
    for (int i = 0; i < ns; ++i) {
      seg_at[i] = a;
      a += seg[i].z;
    }
    seg_at[ns] = a;
    nseg = ns;
  }
  __syncthreads();
  const int total = seg_at[nseg];
  auto entry = [&](int c) {
    const int cnt = count_of(c), rem = cnt % kBM;
    return make_int4(c, cnt - rem, rem, rem_r[c]);
  };
  for (int i = t; i < total; i += 1024) {
    int s = 0;
    while (seg_at[s + 1] <= i) ++s;
    const int4 g = seg[s];
    const int j = i - seg_at[s];
    if (g.y < 0) {
      put(full_tot + i, entry(ord[g.x + j]), none);
    } else if (g.w) {
      put(full_tot + i, entry(ord[g.x + 2 * j]), entry(ord[g.x + 2 * j + 1]));
    } else {
      put(full_tot + i, entry(ord[g.x + j]), entry(ord[g.y + j]));
    }
  }
  for (int slot = full_tot + total + t; slot < items_per_head; slot += 1024) put(slot, none, none);
  emit_sorted(min(full_tot + total, items_per_head));
}

template <int D>
hipError_t launch_attn(int heads, int n, bool bf16, const void *q,
                       const void *k, const void *v, void *o, int c_q,
                       const int32_t *offsets, const int32_t *perm,
                       const int32_t *sel_idx, const int4 *items, int iph,
                       float scale_log2, hipStream_t s) {
  const int total = iph * heads;
  const dim3 grid(total), block(kNW * 64);
  if (bf16 && D == 128)
    hipLaunchKernelGGL(attn_kernel_dma, grid, block, 0, s, n, c_q, iph,
                       total, q, k, v, o, offsets, perm, sel_idx, items,
                       scale_log2);
  else if (bf16)
    hipLaunchKernelGGL((attn_kernel<D, true>), grid, block, 0, s, n, c_q, iph,
                       total, q, k, v, o, offsets, perm, sel_idx, items,
                       scale_log2);
  else
    hipLaunchKernelGGL((attn_kernel<D, false>), grid, block, 0, s, n, c_q, iph,
                       total, q, k, v, o, offsets, perm, sel_idx, items,
                       scale_log2);
  return hipGetLastError();
}

}  // namespace

// Work list of the no-allocation entry point: a fixed device array, one copy
// per GPU, held until the process ends.  Host code never passes `scratch`
// itself to a kernel (on the host it names a stand-in, not device memory);
// it looks up the array's device address once per device and uses that.
static __device__ __align__(256) int4 scratch[kAttnScratchItems];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
int4 *scratch_ptr[kMaxDevices];
}  // namespace

hipError_t attention_scratch(int4 **items) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    scratch_ptr[dev] = static_cast<int4 *>(p);
  }
  *items = scratch_ptr[dev];
  return hipSuccess;
}

// Work slots of one head: sum_c ceil(n_c / kBM) <= ceil(n / kBM) + c_q; each
// slot is two int4 entries.
int attn_items_per_head(int n, int c_q) { return (n + kBM - 1) / kBM + c_q; }

hipError_t attention_items(int heads, int n, int c_q, bool pair, const int32_t *offsets,
                           const int32_t *sel_counts, int4 *items, hipStream_t s) {
  hipLaunchKernelGGL(attn_items_kernel, dim3(heads), dim3(1024), 0, s, n, c_q,
                     attn_items_per_head(n, c_q), pair ? 1 : 0, offsets, sel_counts, items);
  return hipGetLastError();
}

hipError_t attention_run(int heads, int n, int d, bool bf16, const void *q,
                         const void *k, const void *v, void *o, int c_q,
                         const int32_t *offsets, const int32_t *perm,
                         const int32_t *sel_counts, const int32_t *sel_idx,
                         float scale, int4 *items, hipStream_t s) {
  const int iph = attn_items_per_head(n, c_q);
  // remainder chunks share blocks only in the LDS-DMA kernel
  const int pair = bf16 && d == 128 ? 1 : 0;
  hipLaunchKernelGGL(attn_items_kernel, dim3(heads), dim3(1024), 0, s, n, c_q,
                     iph, pair, offsets, sel_counts, items);
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
