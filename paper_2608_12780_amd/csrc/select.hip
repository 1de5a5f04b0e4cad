// Key selection (Sec. 3.4, Eq. 7-10; Alg. 3) without sorting.
//
// Ranking pi_c = keys by proxy logit descending, ties by ascending index.
// base kernel (one block per (cluster, head)):
//   M = max logit; every key's softmax mass E_j = fixexp(s_j - M) in units
//   of 2^-32; total and the exact target T = ceil(rho * total);
//   radix selection of the logit where the descending cumulative mass first
//   reaches T: one coarse pass over a monotone binning of M - s, one pass
//   that gathers the logits of the crossing bin into LDS, then three digit
//   rounds (11/11/10 bits) of the order-preserving key bits over that list
//   (over all keys again if the bin overflows the list); keys that tie at
//   the crossing logit all carry the same mass E*, so the Top-p count is
//   t = (#keys above) + ceil((T - mass above) / E*) (Eq. 7);
//   b = max(t, k_fix) (Eq. 8).  The coarse count histogram is kept for the
//   final kernel.
// Logits depend on a key only through its composite code (Eq. 6), so with
// packed codes the passes that only need per-logit counts and masses (max,
// coarse histogram, crossing-bin gathers and digit rounds) run over the
// head's distinct codes, each weighted by how many keys carry it (built once
// per call by hashing the codes into per-part LDS tables).  Only the final
// compaction, which emits key indices, visits every key.
// head kernel: k_head = ceil(sum n_c b_c / sum n_c) in integers (Eq. 9),
//   r_c = max(b_c, k_head) (Eq. 10), or for the Fig. 6 variants r_c = b_c
//   (fixed floor) or r_c = t_c (pure Top-p).
// final kernel: the rank-r_c logit by the same radix selection on counts
//   (reused from the base kernel when r_c == t_c; otherwise from the kept
//   coarse histogram, one gathering pass and the digit rounds), then an
//   ordered block compaction, eight keys per thread, emits every key above
//   it plus the lowest-index ties, in ascending key order.  With distinct
//   codes each key is classified by one LDS read: the row first writes two
//   bits per distinct code (above / tied with the rank-r_c logit; when the
//   row searches the crossing itself, in the same pass that lists the
//   crossing bin's codes), and the code build stores each key's index among
//   the distinct codes.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

constexpr int kSelBlock = 1024;
constexpr int kCoarseBins = kSelCoarseBins;
constexpr int kMaxTable = kSelMaxTable;
constexpr int kCand = 4096;  // logits of the crossing coarse bin held in LDS (two blocks per CU)

__device__ __forceinline__ int coarse_bin(float y) {
  // y = s - M <= 0; monotone non-increasing in s
  return static_cast<int>(fminf(-y * 64.0f, static_cast<float>(kCoarseBins - 1)));
}

// Inclusive prefix sum over the 64 lanes of 32-bit values with DPP moves:
// shifts by 1, 2, 4, 8 inside each row of 16 lanes, then the last lane of
// row 0 (2) added to row 1 (3), then the last lane of row 1 to rows 2 and 3.
// Lanes whose source falls outside the row read 0.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x111, 0xf, 0xf, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x112, 0xf, 0xf, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x114, 0xf, 0xf, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x118, 0xf, 0xf, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x142, 0xa, 0xf, false));
  v += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x143, 0xc, 0xf, false));
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_scan(T v) {
  if constexpr (sizeof(T) == 4) return static_cast<T>(wave_incl_scan_u32(static_cast<uint32_t>(v)));
  else return wave_incl_scan(v);
}

template <typename T>
__device__ T block_excl_scan(T v, T *total) {
  constexpr int kWaves = kSelBlock / 64;
  __shared__ __attribute__((aligned(16))) T ws[kWaves];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const T incl = wave_scan(v);
  if (lane == 63) ws[w] = incl;
  __syncthreads();
  T base = 0, tot = 0;
  if constexpr (sizeof(T) == 4 && kWaves == 16) {
    // lanes 0..15 scan the wave totals inside DPP row 0
    uint32_t x = lane < kWaves ? static_cast<uint32_t>(ws[lane]) : 0u;
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x111, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x112, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x114, 0xf, 0xf, false));
    x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x118, 0xf, 0xf, false));
    tot = static_cast<T>(__builtin_amdgcn_readlane(static_cast<int>(x), kWaves - 1));
    const int wu = __builtin_amdgcn_readfirstlane(w);  // the wave index, in a scalar register
    base = wu > 0 ? static_cast<T>(__builtin_amdgcn_readlane(static_cast<int>(x), wu - 1)) : T(0);
  } else {
#pragma unroll
    for (int i = 0; i < kWaves; ++i) {
      const T x = ws[i];
      if (i < w) base += x;
      tot += x;
    }
  }
  __syncthreads();
  *total = tot;
  return base + incl - v;
}

template <typename T>
__device__ T block_sum(T v) {
  T tot;
  block_excl_scan(v, &tot);
  return tot;
}

__device__ float block_max(float v) {
  __shared__ float ws[kSelBlock / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_max(v);
  if (lane == 0) ws[w] = v;
  __syncthreads();
  float m = ws[0];
#pragma unroll
  for (int i = 1; i < kSelBlock / 64; ++i) m = fmaxf(m, ws[i]);
  __syncthreads();
  return m;
}

struct Crossing {
  int bin;
  uint32_t cnt_before;
  uint64_t mass_before;
};

// Smallest bin b with base + sum_{b' <= b} w[b'] >= target, where w is the
// mass histogram (BY_MASS) or the count histogram.  Two bins per thread.
template <bool BY_MASS>
__device__ Crossing find_crossing(const uint32_t *hc, const uint64_t *hm,
                                  int nbins, uint64_t base, uint64_t target) {
  __shared__ Crossing res;
  const int t = threadIdx.x;
  const int b0 = 2 * t, b1 = 2 * t + 1;
  const uint32_t c0 = b0 < nbins ? hc[b0] : 0u, c1 = b1 < nbins ? hc[b1] : 0u;
  uint64_t w0, w1;
  if (BY_MASS) {
    w0 = b0 < nbins ? hm[b0] : 0ull;
    w1 = b1 < nbins ? hm[b1] : 0ull;
  } else {
    w0 = c0;
    w1 = c1;
  }
  uint64_t wt;
  uint32_t ct;
  const uint64_t wex = block_excl_scan<uint64_t>(w0 + w1, &wt);
  const uint32_t cex = block_excl_scan<uint32_t>(c0 + c1, &ct);
  const uint64_t a0 = base + wex, a1 = a0 + w0, a2 = a1 + w1;
  if (a0 < target && target <= a1) res = Crossing{b0, cex, wex};
  if (a1 < target && target <= a2) res = Crossing{b1, cex + c0, wex + w0};
  __syncthreads();
  const Crossing out = res;
  __syncthreads();
  return out;
}

// Where a cluster row's logits come from: the materialised scores, or the
// table row (staged in LDS) and the key codes, packed (three subspaces) or
// one uint16 plane per subspace.
constexpr int kFromScores = 0, kFromPacked = 1, kFromPlanes = 2, kFromUnique = 3;

struct CodeBooks {
  const uint32_t *packed;  // [heads][n], KIND == kFromPacked
  const uint16_t *planes;  // [heads][M][n], KIND == kFromPlanes
  const uint32_t *ucodes;  // [heads][n]: distinct packed codes, KIND == kFromUnique
  const uint32_t *umult;   // [heads][n]: keys carrying each of them
  const int *ucount;       // [heads]: number of distinct codes
  const uint32_t *uidx;    // [heads][upitch]: each key's distinct code, or null
  int upitch;              // n rounded up to a multiple of 4
  CodePlanes cp;           // M and the table columns of each subspace
};

// Entry j of a row: its logit and how many keys it stands for (1 except
// for distinct codes); count is the number of entries.
template <int KIND>
struct LogitSource {
  const float *P;          // LDS table row or global score row
  const uint32_t *packed;  // codes of this head (or its distinct codes)
  const uint32_t *mult;
  const uint16_t *planes;
  CodePlanes cp;
  size_t n;
  int count;
  float sigma;
  __device__ __forceinline__ float operator()(int j) const {
    if (KIND == kFromScores) return P[j];
    if (KIND == kFromPacked || KIND == kFromUnique)
      return proxy_logit(P, cp.col[1], cp.col[2], cp.col[3], packed[j], sigma);
    return proxy_logit_planes(P, cp, planes, n, j, sigma);
  }
  __device__ __forceinline__ uint32_t weight(int j) const {
    return KIND == kFromUnique ? mult[j] : 1u;
  }
};

template <int KIND>
__device__ LogitSource<KIND> make_source(float *lut, int h, int c, int n, int c_q,
                                         const CodeBooks &cb, float sigma,
                                         const float *scores, const float *tables) {
  LogitSource<KIND> src;
  src.cp = cb.cp;
  src.n = static_cast<size_t>(n);
  src.sigma = sigma;
  src.count = n;
  src.mult = nullptr;
  if (KIND == kFromUnique) {
    src.packed = cb.ucodes + static_cast<size_t>(h) * n;
    src.mult = cb.umult + static_cast<size_t>(h) * n;
    src.count = min(max(cb.ucount[h], 0), n);
  } else {
    src.packed = cb.packed ? cb.packed + static_cast<size_t>(h) * n : nullptr;
  }
  src.planes = cb.planes ? cb.planes + static_cast<size_t>(h) * cb.cp.M * n : nullptr;
  if (KIND != kFromScores) {
    const int cs = cb.cp.col[cb.cp.M];
    const float *row = tables + (static_cast<size_t>(h) * c_q + c) * cs;
    for (int e = threadIdx.x; e < cs; e += kSelBlock) lut[e] = row[e];
    __syncthreads();
    src.P = lut;
  } else {
    src.P = scores + (static_cast<size_t>(h) * c_q + c) * n;
  }
  return src;
}

// Radix refinement inside one coarse bin: three digit passes over the
// order-preserving key of every logit the source visits (all keys of the
// bin).  BY_MASS selects the mass target (Top-p) or the count target
// (rank).  Returns the exact crossing key and what lies above it.
template <bool BY_MASS, typename Visit>
__device__ void refine(Visit visit, float M, uint64_t target, uint32_t *hc,
                       uint64_t *hm, uint32_t *key_out, uint32_t *cnt_above,
                       uint64_t *mass_above) {
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  uint32_t prefix = 0, pmask = 0;
  for (int round = 0; round < 3; ++round) {
    const int sh = shifts[round], nb = 1 << widths[round];
    for (int b = threadIdx.x; b < nb; b += kSelBlock) {
      hc[b] = 0;
      if (BY_MASS) hm[b] = 0;
    }
    __syncthreads();
    visit([&](float s, uint32_t wt) {
      const uint32_t key = desc_key(s);
      if ((key & pmask) != prefix) return;
      const int dig = (key >> sh) & (nb - 1);
      atomicAdd(&hc[dig], wt);
      if (BY_MASS) {
        const uint64_t e = fixexp(s - M) * wt;
        if (e) atomicAdd(reinterpret_cast<unsigned long long *>(&hm[dig]),
                         static_cast<unsigned long long>(e));
      }
    });
    __syncthreads();
    const uint64_t base = BY_MASS ? *mass_above : static_cast<uint64_t>(*cnt_above);
    const Crossing x = find_crossing<BY_MASS>(hc, hm, nb, base, target);
    *cnt_above += x.cnt_before;
    if (BY_MASS) *mass_above += x.mass_before;
    prefix |= static_cast<uint32_t>(x.bin) << sh;
    pmask |= static_cast<uint32_t>(nb - 1) << sh;
  }
  *key_out = prefix;
}

// Gathers the logits of coarse bin `cbin` into cand (one LDS slot per key,
// reserved per wave); returns how many there are (more than kCand: the
// list is incomplete and the caller visits all keys instead).
template <int KIND, int CAP = kCand>
__device__ int gather_bin(const LogitSource<KIND> &src, float M, int cbin,
                          float *cand, uint32_t *candw, int *ncand) {
  if (threadIdx.x == 0) *ncand = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int n = src.count;
  // four entries per thread in flight (read at clamped positions; those
  // past the end are not in the bin)
  constexpr int kG = 4;
  for (int j0 = 0; j0 < n; j0 += kG * kSelBlock) {
    float sv[kG];
    uint32_t wv[kG];
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const int j = min(j0 + g * kSelBlock + static_cast<int>(threadIdx.x), n - 1);
      sv[g] = src(j);
      wv[g] = src.weight(j);
    }
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const int j = j0 + g * kSelBlock + static_cast<int>(threadIdx.x);
      const bool in = j < n && coarse_bin(sv[g] - M) == cbin;
      const uint64_t mask = __ballot(in);
      if (mask) {
        int first = 0;
        if (lane == static_cast<int>(__ffsll(static_cast<long long>(mask))) - 1)
          first = atomicAdd(ncand, __popcll(mask));
        first = __shfl(first, __ffsll(static_cast<long long>(mask)) - 1);
        const int slot = first + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
            static_cast<uint32_t>(mask >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u)));
        if (in && slot < CAP) {
          cand[slot] = sv[g];
          candw[slot] = wv[g];
        }
      }
    }
  }
  __syncthreads();
  const int cnt = *ncand;
  __syncthreads();
  return cnt;
}

// Exact crossing key inside coarse bin `cbin`: over the gathered list when
// it is complete, else over all keys.
template <int KIND, bool BY_MASS, int CAP = kCand>
__device__ void refine_bin(const LogitSource<KIND> &src, float M, int cbin,
                           uint64_t target, uint32_t *hc, uint64_t *hm, float *cand,
                           uint32_t *candw, int *ncand, uint32_t *key_out,
                           uint32_t *cnt_above, uint64_t *mass_above) {
  const int cnt = gather_bin<KIND, CAP>(src, M, cbin, cand, candw, ncand);
  if (cnt <= CAP) {
    refine<BY_MASS>([&](auto f) {
      for (int k = threadIdx.x; k < cnt; k += kSelBlock) f(cand[k], candw[k]);
    }, M, target, hc, hm, key_out, cnt_above, mass_above);
  } else {
    refine<BY_MASS>([&](auto f) {
      for (int j = threadIdx.x; j < src.count; j += kSelBlock) {
        const float s = src(j);
        if (coarse_bin(s - M) == cbin) f(s, src.weight(j));
      }
    }, M, target, hc, hm, key_out, cnt_above, mass_above);
  }
}

template <int KIND>
__global__ __launch_bounds__(kSelBlock) __attribute__((amdgpu_waves_per_eu(8))) void select_base_kernel(
    int n, int c_q, CodeBooks cb, float sigma, const float *__restrict__ scores,
    const float *__restrict__ tables, float rho, int k_fix, int32_t *base_counts, int32_t *topp_counts,
    float *row_max, uint32_t *row_state, uint32_t *coarse_hist) {
  __shared__ float lut[kMaxTable];
  __shared__ uint32_t hc[kCoarseBins];
  __shared__ uint64_t hm[kCoarseBins];
  __shared__ float cand[kCand];
  __shared__ uint32_t candw[kCand];
  __shared__ int ncand;
  const int c = blockIdx.x, h = blockIdx.y;
  const size_t row = static_cast<size_t>(h) * c_q + c;
  const LogitSource<KIND> src =
      make_source<KIND>(lut, h, c, n, c_q, cb, sigma, scores, tables);
  const int ne = src.count;
  // four logits per thread in flight; clamped positions repeat a real entry
  float mloc = -INFINITY;
  for (int j0 = threadIdx.x; j0 < ne; j0 += 4 * kSelBlock) {
    float v[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) v[g] = src(min(j0 + g * kSelBlock, ne - 1));
#pragma unroll
    for (int g = 0; g < 4; ++g) mloc = fmaxf(mloc, v[g]);
  }
  const float M = block_max(mloc);
  int t_p = n;
  uint32_t key_star = 0, above_star = 0;
  if (rho < 1.0f) {
    for (int b = threadIdx.x; b < kCoarseBins; b += kSelBlock) {
      hc[b] = 0;
      hm[b] = 0;
    }
    __syncthreads();
    // four consecutive entries per thread: a run of them in one bin costs
    // one pair of LDS atomics (integer sums, so the order does not matter)
    uint64_t tloc = 0;
    for (int j0 = 4 * threadIdx.x; j0 < ne; j0 += 4 * kSelBlock) {
      int cb = -1;
      uint32_t cc = 0;
      uint64_t cm = 0;
      float yv[4];
      uint32_t wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // loads at clamped positions, all four in flight
        const int j = min(j0 + i, ne - 1);
        yv[i] = src(j) - M;
        wv[i] = src.weight(j);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (j0 + i < ne) {
          const float y = yv[i];
          const uint32_t wt = wv[i];
          const int bin = coarse_bin(y);
          const uint64_t e = fixexp(y) * wt;
          tloc += e;
          if (bin != cb) {
            if (cc) atomicAdd(&hc[cb], cc);
            if (cm) atomicAdd(reinterpret_cast<unsigned long long *>(&hm[cb]),
                              static_cast<unsigned long long>(cm));
            cb = bin;
            cc = 0;
            cm = 0;
          }
          cc += wt;
          cm += e;
        }
      }
      if (cc) atomicAdd(&hc[cb], cc);
      if (cm) atomicAdd(reinterpret_cast<unsigned long long *>(&hm[cb]),
                        static_cast<unsigned long long>(cm));
    }
    const uint64_t tot = block_sum<uint64_t>(tloc);
    __syncthreads();
    // the coarse count histogram, for the rank selection of the final kernel
    for (int b = threadIdx.x; b < kCoarseBins; b += kSelBlock)
      coarse_hist[row * kCoarseBins + b] = hc[b];
    const uint64_t T = mass_target(rho, tot);
    const Crossing x = find_crossing<true>(hc, hm, kCoarseBins, 0, T);
    uint32_t cnt_above = x.cnt_before;
    uint64_t mass_above = x.mass_before;
    refine_bin<KIND, true, kCand>(src, M, x.bin, T, hc, hm, cand, candw, &ncand, &key_star,
                            &cnt_above, &mass_above);
    const float s_star = desc_key_value(key_star);
    const uint64_t e_star = fixexp(s_star - M);
    const uint64_t need = (T - mass_above + e_star - 1) / e_star;
    t_p = static_cast<int>(cnt_above + need);
    above_star = cnt_above;
  }
  if (threadIdx.x == 0) {
    const int b = t_p > k_fix ? t_p : k_fix;
    base_counts[row] = b;
    if (topp_counts) topp_counts[row] = t_p;
    row_max[row] = M;
    row_state[4 * row + 0] = static_cast<uint32_t>(t_p);
    row_state[4 * row + 1] = key_star;
    row_state[4 * row + 2] = above_star;
  }
}

__global__ __launch_bounds__(kSelBlock) void select_head_kernel(
    int c_q, const int32_t *__restrict__ counts, const int32_t *__restrict__ base,
    const uint32_t *__restrict__ row_state, int policy, int32_t *k_head,
    int32_t *sel_counts) {
  const int h = blockIdx.x;
  uint64_t num = 0, den = 0;
  for (int c = threadIdx.x; c < c_q; c += kSelBlock) {
    const uint64_t nc = static_cast<uint64_t>(max(counts[static_cast<size_t>(h) * c_q + c], 0));
    num += nc * static_cast<uint64_t>(base[static_cast<size_t>(h) * c_q + c]);
    den += nc;
  }
  num = block_sum<uint64_t>(num);
  den = block_sum<uint64_t>(den);
  const int kh = den ? static_cast<int>((num + den - 1) / den) : 0;
  if (threadIdx.x == 0) k_head[h] = kh;
  // r_c per policy: online (Eq. 10), fixed floor (Eq. 8), pure Top-p (Eq. 7)
  for (int c = threadIdx.x; c < c_q; c += kSelBlock) {
    const size_t row = static_cast<size_t>(h) * c_q + c;
    const int b = base[row];
    const int t = static_cast<int>(row_state[4 * row + 0]);
    sel_counts[row] = policy == 0 ? (b > kh ? b : kh) : policy == 1 ? b : t;
  }
}

// Class words of the compaction: the distinct codes u of a head in groups of
// 32, one uint2 per group: bit u%32 of .x is set when the code's logit ranks
// above the rank-r_c logit, of .y when it ties with it.  They replace the
// coarse histogram and candidate list in LDS once the crossing is known.
constexpr int kPoolWords = kCoarseBins + 2 * kCand;
constexpr int kClassCodes = kPoolWords / 2 * 32;  // distinct codes the words cover
// the merged crossing pass keeps class words, the coarse histogram and a
// list of the crossing bin's codes in the pool at once
constexpr int kMergedCand = 2048;
constexpr int kMergedClassWords = kPoolWords - kCoarseBins - kMergedCand;  // 32-bit words
constexpr int kMergedCodes = kMergedClassWords / 2 * 32;
static_assert(kMergedClassWords % 2 == 0 && kMergedCodes >= 65536, "merged pool layout");
// Keys per thread per compaction pass: with eight, the 16 waves' output
// slices take 32 KB of LDS; with the table row sized at launch (1.5 KB for
// three codebooks of 128) two blocks still fit on a CU.
constexpr int kSelKeys = 8;
static_assert(kSelKeys % 4 == 0 && kSelKeys * kSelBlock < 65536, "packed 16-bit counts");

template <int KIND, int RKIND>
__global__ __launch_bounds__(kSelBlock) __attribute__((amdgpu_waves_per_eu(8))) void select_final_kernel(
    int n, int c_q, CodeBooks cb, float sigma, const float *__restrict__ scores,
    const float *__restrict__ tables, const int32_t *__restrict__ sel_counts, const float *__restrict__ row_max,
    const uint32_t *__restrict__ row_state,
    const uint32_t *__restrict__ coarse_hist, int32_t *sel_idx) {
  extern __shared__ float lut[];  // the table row: cs floats, sized at launch
  __shared__ __attribute__((aligned(16))) uint32_t pool[kPoolWords];
  __shared__ int ncand;
  uint32_t *hc = pool;
  float *cand = reinterpret_cast<float *>(pool + kCoarseBins);
  uint32_t *candw = pool + kCoarseBins + kCand;
  const int c = blockIdx.x, h = blockIdx.y;
  const size_t row = static_cast<size_t>(h) * c_q + c;
  int32_t *out = sel_idx + row * n;
  const int r = min(sel_counts[row], n);
  if (r >= n) {
    for (int j = threadIdx.x; j < n; j += kSelBlock) out[j] = j;
    return;
  }
  if (r <= 0) return;
  const LogitSource<KIND> src =
      make_source<KIND>(lut, h, c, n, c_q, cb, sigma, scores, tables);
  const float M = row_max[row];
  uint32_t key_r = 0, above = 0;
  const bool have_key = static_cast<uint32_t>(r) == row_state[4 * row + 0];
  if (have_key) {
    key_r = row_state[4 * row + 1];
    above = row_state[4 * row + 2];
  }
  // with distinct codes the keys are classified through their code's class
  // bits (one LDS read per key); otherwise each key's logit is recomputed
  const int ucnt = RKIND == kFromUnique ? min(max(cb.ucount[h], 0), n) : 0;
  const bool by_class = RKIND == kFromUnique && cb.uidx != nullptr && ucnt > 0 && ucnt <= kClassCodes;
  // Without the key, and with few enough distinct codes, one pass over them
  // both classifies them by coarse bin (a code whose bin precedes the
  // crossing bin ranks above the rank-r_c logit, one after it below) and
  // lists the codes of the crossing bin; the digit rounds then find the key
  // among those and fix their bits.  Pool: class words, then the coarse
  // histogram, then the listed codes' indices.
  const bool merged = by_class && !have_key && ucnt <= kMergedCodes;
  const uint2 *cls = reinterpret_cast<const uint2 *>(pool);
  const uint32_t *kidx = by_class ? cb.uidx + static_cast<size_t>(h) * cb.upitch : nullptr;
  const uint32_t *uc = by_class ? cb.ucodes + static_cast<size_t>(h) * n : nullptr;
  const uint32_t *um = by_class ? cb.umult + static_cast<size_t>(h) * n : nullptr;
  const int lane = threadIdx.x & 63;
  auto ulogit = [&](uint32_t code) __attribute__((always_inline)) {
    return proxy_logit(src.P, cb.cp.col[1], cb.cp.col[2], cb.cp.col[3], code, sigma);
  };
  bool exact_build = by_class;   // class bits by exact comparison with key_r
  if (merged) {
    uint32_t *hm2 = pool + kMergedClassWords;
    uint32_t *candu = hm2 + kCoarseBins;
    for (int b = threadIdx.x; b < kCoarseBins; b += kSelBlock)
      hm2[b] = coarse_hist[row * kCoarseBins + b];
    if (threadIdx.x == 0) ncand = 0;
    __syncthreads();
    const Crossing x = find_crossing<false>(hm2, nullptr, kCoarseBins, 0,
                                            static_cast<uint64_t>(r));
    above = x.cnt_before;
    const int cbin = x.bin;
    uint2 *clsw = reinterpret_cast<uint2 *>(pool);
    constexpr int kG = 4;
    for (int u0 = 64 * kG * (threadIdx.x >> 6); u0 < ucnt; u0 += kG * kSelBlock) {
      uint32_t code[kG];
#pragma unroll
      for (int g = 0; g < kG; ++g) code[g] = uc[min(u0 + 64 * g + lane, ucnt - 1)];
#pragma unroll
      for (int g = 0; g < kG; ++g) {
        const int u = u0 + 64 * g + lane;
        const int bin = coarse_bin(ulogit(code[g]) - M);
        const bool in = u < ucnt && bin == cbin;
        const uint64_t ab = __ballot(u < ucnt && bin < cbin);
        const uint64_t cbm = __ballot(in);
        if (lane < 2 && u0 + 64 * g < ucnt)
          clsw[((u0 + 64 * g) >> 5) + lane] =
              make_uint2(static_cast<uint32_t>(lane == 0 ? ab : ab >> 32), 0u);
        if (cbm) {
          int first = 0;
          const int lead = static_cast<int>(__ffsll(static_cast<long long>(cbm))) - 1;
          if (lane == lead) first = atomicAdd(&ncand, __popcll(cbm));
          first = __shfl(first, lead);
          const int slot = first + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
              static_cast<uint32_t>(cbm >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(cbm), 0u)));
          if (in && slot < kMergedCand) candu[slot] = static_cast<uint32_t>(u);
        }
      }
    }
    __syncthreads();
    const int cnt = ncand;
    uint64_t unused = 0;
    if (cnt <= kMergedCand) {
      refine<false>([&](auto f) {
        for (int k2 = threadIdx.x; k2 < cnt; k2 += kSelBlock) {
          const uint32_t u = candu[k2];
          f(ulogit(uc[u]), um[u]);
        }
      }, M, static_cast<uint64_t>(r), hm2, nullptr, &key_r, &above, &unused);
      // the listed codes' bits, now that the key is known
      uint32_t *clsw32 = pool;
      for (int k2 = threadIdx.x; k2 < cnt; k2 += kSelBlock) {
        const uint32_t u = candu[k2];
        const uint32_t key = desc_key(ulogit(uc[u]));
        const uint32_t bit = 1u << (u & 31u);
        if (key < key_r) atomicOr(&clsw32[2 * (u >> 5)], bit);
        else if (key == key_r) atomicOr(&clsw32[2 * (u >> 5) + 1], bit);
      }
      exact_build = false;
    } else {
      // the crossing bin holds more codes than the list: digit rounds over
      // every distinct code of the bin, then the exact class build
      refine<false>([&](auto f) {
        for (int u = threadIdx.x; u < ucnt; u += kSelBlock) {
          const float sv = ulogit(uc[u]);
          if (coarse_bin(sv - M) == cbin) f(sv, um[u]);
        }
      }, M, static_cast<uint64_t>(r), hm2, nullptr, &key_r, &above, &unused);
    }
  } else if (!have_key) {
    // the coarse count histogram of the base kernel (same logits, same M)
    for (int b = threadIdx.x; b < kCoarseBins; b += kSelBlock)
      hc[b] = coarse_hist[row * kCoarseBins + b];
    __syncthreads();
    const Crossing x = find_crossing<false>(hc, nullptr, kCoarseBins, 0,
                                            static_cast<uint64_t>(r));
    above = x.cnt_before;
    uint64_t unused = 0;
    LogitSource<RKIND> rsrc;
    rsrc.P = src.P;
    rsrc.packed = src.packed;
    rsrc.mult = src.mult;
    rsrc.planes = src.planes;
    rsrc.cp = src.cp;
    rsrc.n = src.n;
    rsrc.count = src.count;
    rsrc.sigma = src.sigma;
    if (RKIND != KIND) {
      // the same table row (already in LDS), over the distinct codes
      rsrc.packed = cb.ucodes + static_cast<size_t>(h) * n;
      rsrc.mult = cb.umult + static_cast<size_t>(h) * n;
      rsrc.count = min(max(cb.ucount[h], 0), n);
    }
    refine_bin<RKIND, false, kCand>(rsrc, M, x.bin, static_cast<uint64_t>(r), hc, nullptr,
                             cand, candw, &ncand, &key_r, &above, &unused);
  }
  if (exact_build) {
    __syncthreads();  // the crossing search is done with the pool
    uint2 *clsw = reinterpret_cast<uint2 *>(pool);
    // four groups of 64 codes per wave in flight (codes read from clamped
    // positions; those past the list are masked out of the ballots)
    constexpr int kG = 4;
    for (int u0 = 64 * kG * (threadIdx.x >> 6); u0 < ucnt; u0 += kG * kSelBlock) {
      uint32_t code[kG];
#pragma unroll
      for (int g = 0; g < kG; ++g) code[g] = uc[min(u0 + 64 * g + lane, ucnt - 1)];
#pragma unroll
      for (int g = 0; g < kG; ++g) {
        const int u = u0 + 64 * g + lane;
        const uint32_t key = desc_key(ulogit(code[g]));
        const uint64_t ab = __ballot(u < ucnt && key < key_r);
        const uint64_t tb = __ballot(u < ucnt && key == key_r);
        if (lane < 2 && u0 + 64 * g < ucnt)
          clsw[((u0 + 64 * g) >> 5) + lane] =
              lane == 0 ? make_uint2(static_cast<uint32_t>(ab), static_cast<uint32_t>(tb))
                        : make_uint2(static_cast<uint32_t>(ab >> 32), static_cast<uint32_t>(tb >> 32));
      }
    }
  }
  __syncthreads();
  const int cls_last = max((ucnt + 31) / 32 - 1, 0);
  // Ordered compaction: every key above key_r and the first `need` ties in
  // index order, in ascending key order.  Each pass takes kSelKeys
  // consecutive keys per thread (their indices or codes read from clamped
  // positions, unconditionally, so a pass's loads are in flight together;
  // with class words the next pass's indices load during this one); one
  // block scan of the packed per-thread counts places them: a selected key
  // goes to (#above before it) + min(#ties before it, need).  A wave's keys
  // are consecutive and so are its outputs, which it stages in its LDS slice
  // and stores with consecutive lanes through a buffer resource spanning the
  // row's r outputs (offsets past it are dropped by the hardware).
  const uint32_t need = static_cast<uint32_t>(r) - above;
  const __amdgpu_buffer_rsrc_t rout =
      __builtin_amdgcn_make_buffer_rsrc(out, static_cast<short>(0), r * 4, 0x00020000);
  constexpr uint32_t kDropped = 0x80000000u;   // past any row (r * 4 < 2^31)
  uint32_t out_run = 0, ties_run = 0;
  constexpr int KPT = kSelKeys;
  __shared__ uint32_t stage_all[kSelBlock * KPT];
  uint32_t *stage = stage_all + (threadIdx.x >> 6) * 64 * KPT;
  // the pitch is a multiple of 4, so a group that starts before n lies in
  // the row; groups at or past n reread the row's last group
  auto load_idx = [&](int j, uint4 (&v)[KPT / 4]) {
#pragma unroll
    for (int g = 0; g < KPT / 4; ++g)
      v[g] = *reinterpret_cast<const uint4 *>(kidx + min(j + 4 * g, (n - 1) & ~3));
  };
  // one pass over keys j0 .. j0 + KPT * kSelBlock - 1 with this pass's
  // indices in cur; the next pass's are loaded into nxt meanwhile (two
  // buffers that trade places, so no register copy waits for the load)
  auto pass = [&](int j0, const uint4 (&cur)[KPT / 4], uint4 (&nxt)[KPT / 4]) __attribute__((always_inline)) {
    const int jb = j0 + KPT * threadIdx.x;
    uint32_t fa = 0, ft = 0;  // per-key flags, bit i = key jb + i
    if (by_class) {
      uint32_t uu[KPT];
#pragma unroll
      for (int g = 0; g < KPT / 4; ++g) {
        uu[4 * g + 0] = cur[g].x;
        uu[4 * g + 1] = cur[g].y;
        uu[4 * g + 2] = cur[g].z;
        uu[4 * g + 3] = cur[g].w;
      }
      // the next pass's indices are in flight during this pass's scan
      load_idx(jb + KPT * kSelBlock, nxt);
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const uint2 wd = cls[min(static_cast<int>(uu[i] >> 5), cls_last)];
        const uint32_t bit = uu[i] & 31u;
        fa |= ((wd.x >> bit) & 1u) << i;
        ft |= ((wd.y >> bit) & 1u) << i;
      }
    } else {
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const uint32_t key = desc_key(src(min(jb + i, n - 1)));
        fa |= static_cast<uint32_t>(key < key_r) << i;
        ft |= static_cast<uint32_t>(key == key_r) << i;
      }
    }
    // keys at or past n count for nothing
    const int valid = min(max(n - jb, 0), KPT);
    const uint32_t vmask = valid >= 32 ? 0xFFFFFFFFu : (1u << valid) - 1u;
    fa &= vmask;
    ft &= vmask;
    uint32_t tot;
    const uint32_t ex = block_excl_scan<uint32_t>((static_cast<uint32_t>(__popc(ft)) << 16) |
                                                      static_cast<uint32_t>(__popc(fa)), &tot);
    const uint32_t a_pre = ex & 0xFFFFu, t_pre = ex >> 16;
    const uint32_t remaining = need > ties_run ? need - ties_run : 0u;
    // this thread keeps its keys above and its first remaining - t_pre ties
    uint32_t sel = fa;
    if (ft) {
      uint32_t take = remaining > t_pre ? remaining - t_pre : 0u;
      uint32_t m = ft;
      while (take && m) {
        sel |= m & (0u - m);
        m &= m - 1u;
        --take;
      }
    }
    // a wave's keys are consecutive, so are its outputs: stage them in the
    // wave's LDS slice, then store the slice with consecutive lanes
    const uint32_t pos0 = out_run + a_pre + min(t_pre, remaining);
    const uint32_t wbase = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(pos0)));
    const uint32_t wend = static_cast<uint32_t>(
        __builtin_amdgcn_readlane(static_cast<int>(pos0 + static_cast<uint32_t>(__popc(sel))), 63));
    uint32_t at = pos0 - wbase;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      if ((sel >> i) & 1u) stage[at] = static_cast<uint32_t>(jb + i);
      at += (sel >> i) & 1u;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // a fixed count of stores (lanes past the wave's outputs store to an
    // offset past the row, which is dropped), so the wait for the next
    // pass's indices need not wait for these stores
    const uint32_t wcnt = wend - wbase;
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
      const uint32_t k = static_cast<uint32_t>(64 * q + lane);
      __builtin_amdgcn_raw_buffer_store_b32(stage[k], rout, k < wcnt ? (wbase + k) * 4u : kDropped, 0, 0);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    out_run += (tot & 0xFFFFu) + min(tot >> 16, remaining);
    ties_run += tot >> 16;
  };
  uint4 ia[KPT / 4], ib[KPT / 4];
  constexpr int kStep = KPT * kSelBlock;
  if (by_class) {
    load_idx(KPT * threadIdx.x, ia);
    for (int j0 = 0; j0 < n; j0 += 2 * kStep) {
      pass(j0, ia, ib);
      if (j0 + kStep < n) pass(j0 + kStep, ib, ia);
    }
  } else {
    for (int j0 = 0; j0 < n; j0 += kStep) pass(j0, ia, ib);
  }
}

// Distinct packed codes of every head.  Only the low 30 bits of a code (its
// three 10-bit fields) reach a logit, so they are the key; 0xFFFFFFFF marks
// a free slot.  The code space is hashed into P parts of a head; block
// (part, head) reads all of the head's codes and counts the ones of its
// part in an LDS table with open addressing, then stores the part's
// (code, count) pairs, each occupied slot's rank among them, and for every
// key of the part its (part, slot).  P is chosen so that the tables are at
// most 80% full even if every key has its own code; should a skewed part
// still fill its table, the head falls back to one entry per key (count 1),
// which the selection treats exactly like the keys themselves.
constexpr uint32_t kFreeSlot = 0xFFFFFFFFu;
constexpr int kPartSlots = 16384;   // LDS table of one part: 128 KB
constexpr int kSlotBits = 14;       // log2(kPartSlots)
constexpr int kGatherBlocks = 16;   // blocks per head that assemble the lists
// Every part reads all of a head's codes, so the build costs parts x n
// reads; beyond kMaxDistinctKeys keys the passes visit every key.
constexpr int kMaxParts = 32;
constexpr int kMaxDistinctKeys = 262144;

__device__ __forceinline__ uint32_t code_hash(uint32_t code) { return code * 0x9E3779B1u; }

__global__ void code_parts_clear_kernel(int *overflow, int heads) {
  for (int h = blockIdx.x * blockDim.x + threadIdx.x; h < heads; h += gridDim.x * blockDim.x)
    overflow[h] = 0;
}

__global__ __launch_bounds__(kSelBlock) void code_parts_kernel(
    const uint32_t *__restrict__ codes, int n, int parts, int upitch, uint32_t *stage_codes,
    uint32_t *stage_mult, uint32_t *stage_rank, int *part_count, uint32_t *key_slot,
    int *overflow) {
  __shared__ uint32_t lk[kPartSlots];
  __shared__ uint32_t lc[kPartSlots];
  __shared__ int full;
  const int p = blockIdx.x, h = blockIdx.y;
  for (int i = threadIdx.x; i < kPartSlots; i += kSelBlock) {
    lk[i] = kFreeSlot;
    lc[i] = 0;
  }
  if (threadIdx.x == 0) full = 0;
  __syncthreads();
  const uint32_t *hc = codes + static_cast<size_t>(h) * n;
  uint32_t *ks = key_slot + static_cast<size_t>(h) * upitch;
  // four codes per thread in flight (clamped positions; the extra ones are
  // skipped below)
  constexpr int kG = 4;
  for (int j0 = threadIdx.x; j0 < n; j0 += kG * kSelBlock) {
    uint32_t cv[kG];
#pragma unroll
    for (int g = 0; g < kG; ++g) cv[g] = hc[min(j0 + g * kSelBlock, n - 1)];
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const int j = j0 + g * kSelBlock;
      const uint32_t code = cv[g] & 0x3FFFFFFFu;
      const uint32_t hv = code_hash(code);
      if (j >= n || static_cast<int>((static_cast<uint64_t>(hv) * parts) >> 32) != p) continue;
      uint32_t slot = hv & (kPartSlots - 1);
      bool done = false;
      for (int probe = 0; probe < kPartSlots; ++probe) {
        const uint32_t prev = atomicCAS(&lk[slot], kFreeSlot, code);
        if (prev == kFreeSlot || prev == code) {
          atomicAdd(&lc[slot], 1u);
          ks[j] = (static_cast<uint32_t>(p) << kSlotBits) | slot;
          done = true;
          break;
        }
        slot = (slot + 1u) & (kPartSlots - 1);
      }
      if (!done) full = 1;
    }
  }
  __syncthreads();
  if (full) {
    if (threadIdx.x == 0) atomicOr(&overflow[h], 1);
    return;
  }
  // the part's pairs, in slot order
  constexpr int per = kPartSlots / kSelBlock;
  uint32_t mine = 0;
#pragma unroll
  for (int k = 0; k < per; ++k) mine += lk[threadIdx.x * per + k] != kFreeSlot;
  uint32_t total;
  uint32_t at = block_excl_scan<uint32_t>(mine, &total);
  const size_t base = (static_cast<size_t>(h) * parts + p) * kPartSlots;
#pragma unroll
  for (int k = 0; k < per; ++k) {
    const int i = threadIdx.x * per + k;
    if (lk[i] != kFreeSlot) {
      stage_codes[base + at] = lk[i];
      stage_mult[base + at] = lc[i];
      stage_rank[base + i] = at;
      ++at;
    }
  }
  if (threadIdx.x == 0) part_count[static_cast<size_t>(h) * parts + p] = static_cast<int>(total);
}

// Blocks (g, head): the parts' pairs concatenated into the head's list, and
// each key's (part, slot) turned into its index in that list; or one entry
// per key (its own index) after an overflow.
__global__ __launch_bounds__(kSelBlock) void code_parts_gather_kernel(
    const uint32_t *__restrict__ codes, int n, int parts, int upitch,
    const uint32_t *__restrict__ stage_codes, const uint32_t *__restrict__ stage_mult,
    const uint32_t *__restrict__ stage_rank, const int *__restrict__ part_count,
    const int *__restrict__ overflow, uint32_t *ucodes, uint32_t *umult, int *ucount,
    uint32_t *uidx) {
  __shared__ int pbase[kMaxParts + 1];
  const int g = blockIdx.x, h = blockIdx.y;
  const int first = g * kSelBlock + threadIdx.x, stride = gridDim.x * kSelBlock;
  uint32_t *uc = ucodes + static_cast<size_t>(h) * n;
  uint32_t *um = umult + static_cast<size_t>(h) * n;
  uint32_t *ui = uidx + static_cast<size_t>(h) * upitch;
  if (overflow[h]) {
    for (int j = first; j < n; j += stride) {
      uc[j] = codes[static_cast<size_t>(h) * n + j] & 0x3FFFFFFFu;
      um[j] = 1u;
      ui[j] = static_cast<uint32_t>(j);
    }
    if (g == 0 && threadIdx.x == 0) ucount[h] = n;
    return;
  }
  if (threadIdx.x == 0) {
    int off = 0;
    for (int q = 0; q < parts; ++q) {
      pbase[q] = off;
      off += part_count[static_cast<size_t>(h) * parts + q];
    }
    pbase[parts] = off;
  }
  __syncthreads();
  for (int q = 0; q < parts; ++q) {
    const int cnt = pbase[q + 1] - pbase[q];
    const size_t base = (static_cast<size_t>(h) * parts + q) * kPartSlots;
    for (int i = first; i < cnt; i += stride) {
      if (pbase[q] + i < n) {
        uc[pbase[q] + i] = stage_codes[base + i];
        um[pbase[q] + i] = stage_mult[base + i];
      }
    }
  }
  for (int j = first; j < n; j += stride) {
    const uint32_t e = ui[j];
    const int q = min(static_cast<int>(e >> kSlotBits), parts - 1);
    const uint32_t slot = e & (kPartSlots - 1);
    ui[j] = static_cast<uint32_t>(pbase[q]) +
            stage_rank[(static_cast<size_t>(h) * parts + q) * kPartSlots + slot];
  }
  if (g == 0 && threadIdx.x == 0) ucount[h] = pbase[parts] < n ? pbase[parts] : n;
}

__global__ void fixexp_kernel(const float *y, uint64_t *out, int64_t count) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < count) out[i] = fixexp(y[i]);
}

}  // namespace

int code_parts(int n) {
  // tables at most 80% full even if every key has its own code: at 720p
  // (n = 118800) 10 parts, so 24 heads' blocks run in one round on 256 CUs
  const long long p = (5LL * n + 4LL * kPartSlots - 1) / (4LL * kPartSlots);
  return p < 1 ? 1 : static_cast<int>(p);
}

bool use_distinct_codes(int n) { return n <= kMaxDistinctKeys && code_parts(n) <= kMaxParts; }

// Row pitch of the per-key index arrays: n rounded up to 4 entries, so the
// final kernel reads four keys' indices per 16-byte load.
static size_t key_pitch(int n) { return (static_cast<size_t>(n) + 3) & ~static_cast<size_t>(3); }

size_t select_dedup_words(int heads, int n) {
  if (!use_distinct_codes(n)) return 0;
  const size_t parts = static_cast<size_t>(code_parts(n));
  return static_cast<size_t>(heads) *
         (key_pitch(n) + 3 * parts * kPartSlots + parts + 2 * static_cast<size_t>(n) + 2);
}

hipError_t select_run(int heads, int n, int c_q, const Subspaces &sub, int d,
                      const float *scores, const float *tables,
                      const uint32_t *codes32, const uint16_t *codes16,
                      const int32_t *counts, float rho, int k_fix, int32_t *base,
                      int32_t *topp, int32_t *k_head, int32_t *sel_counts,
                      int32_t *sel_idx, float *row_max, uint32_t *row_state,
                      uint32_t *coarse_hist, uint32_t *dedup, int policy, hipStream_t s) {
  CodeBooks cb{};
  cb.packed = codes32;
  cb.planes = codes16;
  cb.cp.M = sub.M;
  for (int m = 0; m < sub.M; ++m) cb.cp.col[m + 1] = cb.cp.col[m] + sub.c[m];
  const int kind = scores ? kFromScores : codes16 ? kFromPlanes : kFromPacked;
  const float sigma = static_cast<float>(1.0 / sqrt(static_cast<double>(d)));
  const dim3 grid(c_q, heads), block(kSelBlock);
  hipError_t e = hipSuccess;
  const bool distinct = kind == kFromPacked && use_distinct_codes(n);
  if (distinct) {
    // the head's distinct codes, their multiplicities and each key's index
    // among them (the index array first: 16-byte aligned like the scratch)
    const int parts = code_parts(n);
    const int upitch = static_cast<int>(key_pitch(n));
    const size_t stage = static_cast<size_t>(heads) * parts * kPartSlots;
    uint32_t *uidx = dedup;
    uint32_t *stage_codes = uidx + static_cast<size_t>(heads) * upitch;
    uint32_t *stage_mult = stage_codes + stage;
    uint32_t *stage_rank = stage_mult + stage;
    uint32_t *ucodes = stage_rank + stage;
    uint32_t *umult = ucodes + static_cast<size_t>(heads) * n;
    int *part_count = reinterpret_cast<int *>(umult + static_cast<size_t>(heads) * n);
    int *ucount = part_count + static_cast<size_t>(heads) * parts;
    int *overflow = ucount + heads;
    hipLaunchKernelGGL(code_parts_clear_kernel, dim3((heads + 255) / 256), dim3(256), 0, s,
                       overflow, heads);
    hipLaunchKernelGGL(code_parts_kernel, dim3(parts, heads), dim3(kSelBlock), 0, s, codes32, n,
                       parts, upitch, stage_codes, stage_mult, stage_rank, part_count, uidx,
                       overflow);
    hipLaunchKernelGGL(code_parts_gather_kernel, dim3(kGatherBlocks, heads), dim3(kSelBlock), 0, s,
                       codes32, n, parts, upitch, stage_codes, stage_mult, stage_rank, part_count,
                       overflow, ucodes, umult, ucount, uidx);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    cb.ucodes = ucodes;
    cb.umult = umult;
    cb.ucount = ucount;
    cb.uidx = uidx;
    cb.upitch = upitch;
  }
#define SCOPE_SEL_BASE(K)                                                          \
  hipLaunchKernelGGL(select_base_kernel<K>, grid, block, 0, s, n, c_q, cb, sigma,  \
                     scores, tables, rho, k_fix, base, topp, row_max, row_state, \
                     coarse_hist)
  const size_t lut_bytes = kind == kFromScores ? 16 : static_cast<size_t>(cb.cp.col[cb.cp.M]) * 4;
#define SCOPE_SEL_FINAL(K, R)                                                      \
  hipLaunchKernelGGL((select_final_kernel<K, R>), grid, block, lut_bytes, s, n, c_q, cb, \
                     sigma, scores, tables, sel_counts, row_max, row_state,       \
                     coarse_hist, sel_idx)
  if (kind == kFromScores) SCOPE_SEL_BASE(kFromScores);
  else if (distinct) SCOPE_SEL_BASE(kFromUnique);
  else if (kind == kFromPacked) SCOPE_SEL_BASE(kFromPacked);
  else SCOPE_SEL_BASE(kFromPlanes);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_head_kernel, dim3(heads), block, 0, s, c_q, counts,
                     base, row_state, policy, k_head, sel_counts);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (kind == kFromScores) SCOPE_SEL_FINAL(kFromScores, kFromScores);
  else if (distinct) SCOPE_SEL_FINAL(kFromPacked, kFromUnique);
  else if (kind == kFromPacked) SCOPE_SEL_FINAL(kFromPacked, kFromPacked);
  else SCOPE_SEL_FINAL(kFromPlanes, kFromPlanes);
#undef SCOPE_SEL_BASE
#undef SCOPE_SEL_FINAL
  return hipGetLastError();
}

hipError_t debug_fixexp(const float *y, uint64_t *out, int64_t count,
                        hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = (count + 255) / 256;
  hipLaunchKernelGGL(fixexp_kernel, dim3(static_cast<unsigned>(blocks)),
                     dim3(256), 0, s, y, out, count);
  return hipGetLastError();
}

}  // namespace scope
