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
//   ordered block compaction, four keys per thread, emits every key above
//   it plus the lowest-index ties, in ascending key order.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

constexpr int kSelBlock = 1024;
constexpr int kCoarseBins = kSelCoarseBins;
constexpr int kMaxTable = kSelMaxTable;
constexpr int kCand = 8192;      // logits of the crossing coarse bin held in LDS
constexpr int kCandFinal = 4096; // the same in the final kernel (two blocks per CU)

__device__ __forceinline__ int coarse_bin(float y) {
  // y = s - M <= 0; monotone non-increasing in s
  return static_cast<int>(fminf(-y * 64.0f, static_cast<float>(kCoarseBins - 1)));
}

template <typename T>
__device__ T block_excl_scan(T v, T *total) {
  __shared__ T ws[kSelBlock / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const T incl = wave_incl_scan(v);
  if (lane == 63) ws[w] = incl;
  __syncthreads();
  T base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelBlock / 64; ++i) {
    const T x = ws[i];
    if (i < w) base += x;
    tot += x;
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
  for (int j0 = 0; j0 < n; j0 += kSelBlock) {
    const int j = j0 + threadIdx.x;
    float s = 0.0f;
    bool in = false;
    if (j < n) {
      s = src(j);
      in = coarse_bin(s - M) == cbin;
    }
    const uint64_t mask = __ballot(in);
    if (mask) {
      int first = 0;
      if (lane == static_cast<int>(__ffsll(static_cast<long long>(mask))) - 1)
        first = atomicAdd(ncand, __popcll(mask));
      first = __shfl(first, __ffsll(static_cast<long long>(mask)) - 1);
      const int slot = first + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
          static_cast<uint32_t>(mask >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u)));
      if (in && slot < CAP) {
        cand[slot] = s;
        candw[slot] = src.weight(j);
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
  __shared__ float cand[kCandFinal];
  __shared__ uint32_t candw[kCandFinal];
  __shared__ int ncand;
  const int c = blockIdx.x, h = blockIdx.y;
  const size_t row = static_cast<size_t>(h) * c_q + c;
  const LogitSource<KIND> src =
      make_source<KIND>(lut, h, c, n, c_q, cb, sigma, scores, tables);
  const int ne = src.count;
  float mloc = -INFINITY;
  for (int j = threadIdx.x; j < ne; j += kSelBlock) mloc = fmaxf(mloc, src(j));
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
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (j0 + i < ne) {
          const float y = src(j0 + i) - M;
          const uint32_t wt = src.weight(j0 + i);
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
    refine_bin<KIND, true, kCandFinal>(src, M, x.bin, T, hc, hm, cand, candw, &ncand, &key_star,
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

template <int KIND, int RKIND>
__global__ __launch_bounds__(kSelBlock) __attribute__((amdgpu_waves_per_eu(8))) void select_final_kernel(
    int n, int c_q, CodeBooks cb, float sigma, const float *__restrict__ scores,
    const float *__restrict__ tables, const int32_t *__restrict__ sel_counts, const float *__restrict__ row_max,
    const uint32_t *__restrict__ row_state,
    const uint32_t *__restrict__ coarse_hist, int32_t *sel_idx) {
  __shared__ float lut[kMaxTable];
  __shared__ uint32_t hc[kCoarseBins];
  __shared__ float cand[kCandFinal];
  __shared__ uint32_t candw[kCandFinal];
  __shared__ int ncand;
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
  uint32_t key_r, above;
  if (static_cast<uint32_t>(r) == row_state[4 * row + 0]) {
    key_r = row_state[4 * row + 1];
    above = row_state[4 * row + 2];
  } else {
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
    refine_bin<RKIND, false, kCandFinal>(rsrc, M, x.bin, static_cast<uint64_t>(r), hc, nullptr,
                             cand, candw, &ncand, &key_r, &above, &unused);
  }
  // ordered compaction, four consecutive keys per thread: keys above key_r
  // and the first `need` ties in index order
  const uint32_t need = static_cast<uint32_t>(r) - above;
  uint32_t out_run = 0, ties_run = 0;
  constexpr int KPT = 4;
  for (int j0 = 0; j0 < n; j0 += KPT * kSelBlock) {
    const int jb = j0 + KPT * threadIdx.x;
    uint32_t fa = 0, ft = 0;  // per-key flags, bit i = key jb + i
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      if (jb + i < n) {
        const uint32_t key = desc_key(src(jb + i));
        fa |= static_cast<uint32_t>(key < key_r) << i;
        ft |= static_cast<uint32_t>(key == key_r) << i;
      }
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan<uint32_t>((static_cast<uint32_t>(__popc(ft)) << 16) |
                                                      static_cast<uint32_t>(__popc(fa)), &tot);
    uint32_t a_pre = ex & 0xFFFFu, t_pre = ex >> 16;
    const uint32_t remaining = need > ties_run ? need - ties_run : 0u;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const bool a = (fa >> i) & 1u, tie = (ft >> i) & 1u;
      if (a || (tie && t_pre < remaining))
        out[out_run + a_pre + min(t_pre, remaining)] = jb + i;
      a_pre += a;
      t_pre += tie;
    }
    out_run += (tot & 0xFFFFu) + min(tot >> 16, remaining);
    ties_run += tot >> 16;
  }
}

// Distinct packed codes of every head.  Only the low 30 bits of a code (its
// three 10-bit fields) reach a logit, so they are the key; 0xFFFFFFFF marks
// a free slot.  The code space is hashed into P parts of a head; block
// (part, head) reads all of the head's codes and counts the ones of its
// part in an LDS table with open addressing, then stores the part's
// (code, count) pairs.  P is chosen so that the tables are at most half
// full even if every key has its own code; should a skewed part still fill
// its table, the head falls back to one entry per key (count 1), which the
// selection treats exactly like the keys themselves.
constexpr uint32_t kFreeSlot = 0xFFFFFFFFu;
constexpr int kPartSlots = 16384;   // LDS table of one part: 128 KB

__device__ __forceinline__ uint32_t code_hash(uint32_t code) { return code * 0x9E3779B1u; }

__global__ void code_parts_clear_kernel(int *overflow, int heads) {
  for (int h = blockIdx.x * blockDim.x + threadIdx.x; h < heads; h += gridDim.x * blockDim.x)
    overflow[h] = 0;
}

__global__ __launch_bounds__(kSelBlock) void code_parts_kernel(
    const uint32_t *__restrict__ codes, int n, int parts, uint32_t *stage_codes,
    uint32_t *stage_mult, int *part_count, int *overflow) {
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
  for (int j = threadIdx.x; j < n; j += kSelBlock) {
    const uint32_t code = hc[j] & 0x3FFFFFFFu;
    const uint32_t hv = code_hash(code);
    if (static_cast<int>((static_cast<uint64_t>(hv) * parts) >> 32) != p) continue;
    uint32_t slot = hv & (kPartSlots - 1);
    bool done = false;
    for (int probe = 0; probe < kPartSlots; ++probe) {
      const uint32_t prev = atomicCAS(&lk[slot], kFreeSlot, code);
      if (prev == kFreeSlot || prev == code) {
        atomicAdd(&lc[slot], 1u);
        done = true;
        break;
      }
      slot = (slot + 1u) & (kPartSlots - 1);
    }
    if (!done) full = 1;
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
      ++at;
    }
  }
  if (threadIdx.x == 0) part_count[static_cast<size_t>(h) * parts + p] = static_cast<int>(total);
}

// One block per head: the parts' pairs concatenated into the head's list,
// or one entry per key after an overflow.
__global__ __launch_bounds__(kSelBlock) void code_parts_gather_kernel(
    const uint32_t *__restrict__ codes, int n, int parts, const uint32_t *__restrict__ stage_codes,
    const uint32_t *__restrict__ stage_mult, const int *__restrict__ part_count,
    const int *__restrict__ overflow, uint32_t *ucodes, uint32_t *umult, int *ucount) {
  const int h = blockIdx.x;
  uint32_t *uc = ucodes + static_cast<size_t>(h) * n;
  uint32_t *um = umult + static_cast<size_t>(h) * n;
  if (overflow[h]) {
    for (int j = threadIdx.x; j < n; j += kSelBlock) {
      uc[j] = codes[static_cast<size_t>(h) * n + j] & 0x3FFFFFFFu;
      um[j] = 1u;
    }
    if (threadIdx.x == 0) ucount[h] = n;
    return;
  }
  int off = 0;
  for (int p = 0; p < parts; ++p) {
    const int cnt = part_count[static_cast<size_t>(h) * parts + p];
    const size_t base = (static_cast<size_t>(h) * parts + p) * kPartSlots;
    for (int i = threadIdx.x; i < cnt; i += kSelBlock) {
      if (off + i < n) {
        uc[off + i] = stage_codes[base + i];
        um[off + i] = stage_mult[base + i];
      }
    }
    off += cnt;
  }
  if (threadIdx.x == 0) ucount[h] = off < n ? off : n;
}

__global__ void fixexp_kernel(const float *y, uint64_t *out, int64_t count) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < count) out[i] = fixexp(y[i]);
}

}  // namespace

int code_parts(int n) {
  const long long p = (2LL * n + kPartSlots - 1) / kPartSlots;
  return p < 1 ? 1 : static_cast<int>(p);
}

// Every part reads all of a head's codes, so the build costs parts x n
// reads; beyond kMaxParts parts (n > 262144) the passes visit every key.
constexpr int kMaxParts = 32;
bool use_distinct_codes(int n) { return code_parts(n) <= kMaxParts; }

size_t select_dedup_words(int heads, int n) {
  if (!use_distinct_codes(n)) return 0;
  const size_t parts = static_cast<size_t>(code_parts(n));
  return static_cast<size_t>(heads) *
         (2 * parts * kPartSlots + parts + 2 * static_cast<size_t>(n) + 2);
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
    // the head's distinct codes and their multiplicities
    const int parts = code_parts(n);
    const size_t stage = static_cast<size_t>(heads) * parts * kPartSlots;
    uint32_t *stage_codes = dedup;
    uint32_t *stage_mult = stage_codes + stage;
    uint32_t *ucodes = stage_mult + stage;
    uint32_t *umult = ucodes + static_cast<size_t>(heads) * n;
    int *part_count = reinterpret_cast<int *>(umult + static_cast<size_t>(heads) * n);
    int *ucount = part_count + static_cast<size_t>(heads) * parts;
    int *overflow = ucount + heads;
    hipLaunchKernelGGL(code_parts_clear_kernel, dim3((heads + 255) / 256), dim3(256), 0, s,
                       overflow, heads);
    hipLaunchKernelGGL(code_parts_kernel, dim3(parts, heads), dim3(kSelBlock), 0, s, codes32, n,
                       parts, stage_codes, stage_mult, part_count, overflow);
    hipLaunchKernelGGL(code_parts_gather_kernel, dim3(heads), dim3(kSelBlock), 0, s, codes32, n,
                       parts, stage_codes, stage_mult, part_count, overflow, ucodes, umult,
                       ucount);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    cb.ucodes = ucodes;
    cb.umult = umult;
    cb.ucount = ucount;
  }
#define SCOPE_SEL_BASE(K)                                                          \
  hipLaunchKernelGGL(select_base_kernel<K>, grid, block, 0, s, n, c_q, cb, sigma,  \
                     scores, tables, rho, k_fix, base, topp, row_max, row_state, \
                     coarse_hist)
#define SCOPE_SEL_FINAL(K, R)                                                      \
  hipLaunchKernelGGL((select_final_kernel<K, R>), grid, block, 0, s, n, c_q, cb,   \
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
