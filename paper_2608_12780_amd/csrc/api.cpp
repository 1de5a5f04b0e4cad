// C ABI of the SCOPE layer: argument validation, workspace layout and the
// order of kernel launches for each stage.  Validation runs before any HIP
// call, so every error path works on a host without a GPU.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "../../include/scope.h"
#include "kernels.h"

namespace {

using scope::KmProblem;

constexpr size_t kAlign = 256;
constexpr int kMaxC = 1024;
constexpr int kMaxN = 1 << 24;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Carves consecutive aligned regions out of a workspace (or just sizes them
// when base is null).
struct Carver {
  char *base;
  size_t used = 0;
  explicit Carver(void *b) : base(static_cast<char *>(b)) {}
  template <typename T>
  T *take(size_t count) {
    T *p = base ? reinterpret_cast<T *>(base + used) : nullptr;
    used = align_up(used + count * sizeof(T));
    return p;
  }
};

// Sizes and dtype only (the partition calls ignore the range fields).
int32_t check_dims(const scope_shape *s) {
  if (!s) return SCOPE_ERR_INVALID_ARGUMENT;
  if (s->heads < 1 || s->n < 1 || s->d < 2) return SCOPE_ERR_INVALID_ARGUMENT;
  if (s->dtype != SCOPE_F32 && s->dtype != SCOPE_BF16) return SCOPE_ERR_UNSUPPORTED;
  if (s->n > kMaxN || s->d > 128 || s->heads > 65535) return SCOPE_ERR_UNSUPPORTED;
  if (static_cast<long long>(s->heads) * s->n > (1LL << 31) - 1) return SCOPE_ERR_UNSUPPORTED;
  return SCOPE_OK;
}

int32_t check_shape(const scope_shape *s) {
  const int32_t st = check_dims(s);
  if (st) return st;
  int total = 0;
  for (int m = 0; m < 3; ++m) {
    const int o = s->range_off[m], l = s->range_len[m];
    if (l < 1 || o < 0 || o + l > s->d) return SCOPE_ERR_INVALID_ARGUMENT;
    for (int q = 0; q < m; ++q) {
      const int o2 = s->range_off[q], l2 = s->range_len[q];
      if (o < o2 + l2 && o2 < o + l) return SCOPE_ERR_INVALID_ARGUMENT;  // overlap
    }
    total += l;
  }
  if (total != s->d) return SCOPE_ERR_INVALID_ARGUMENT;  // must cover all d
  return SCOPE_OK;
}

int32_t check_cm(const scope_shape *s, const int32_t *c_m) {
  if (!c_m) return SCOPE_ERR_INVALID_ARGUMENT;
  for (int m = 0; m < 3; ++m) {
    if (c_m[m] < 1 || c_m[m] > s->n) return SCOPE_ERR_INVALID_ARGUMENT;
    if (c_m[m] > kMaxC) return SCOPE_ERR_UNSUPPORTED;
  }
  return SCOPE_OK;
}

int32_t check_cq(const scope_shape *s, int32_t c_q) {
  if (c_q < 1 || c_q > s->n) return SCOPE_ERR_INVALID_ARGUMENT;
  if (c_q > kMaxC) return SCOPE_ERR_UNSUPPORTED;
  return SCOPE_OK;
}

int32_t check_ws(void *ws, size_t bytes, size_t need) {
  if (need == 0) return SCOPE_OK;
  if (!ws || bytes < need) return SCOPE_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return SCOPE_ERR_WORKSPACE;
  return SCOPE_OK;
}

bool aligned_data(const void *p, const scope_shape *s) {
  return reinterpret_cast<uintptr_t>(p) % (s->dtype == SCOPE_BF16 ? 2 : 4) == 0;
}

// --- workspace layouts (each call's regions start at offset 0) -----------
// Update plans; shapes were validated, so planning cannot fail for them.
scope::AccPlan query_plan(const scope_shape *s, int c_q) {
  scope::AccPlan p;
  const int col0 = 0, dx = s->d;
  scope::km_accum_plan(1, &col0, &dx, &c_q, s->heads, s->n, &p);
  return p;
}
scope::AccPlan key_plan(const scope_shape *s, const int32_t *c_m) {
  scope::AccPlan p;
  const int C[3] = {c_m[0], c_m[1], c_m[2]};
  scope::km_accum_plan(3, s->range_off, s->range_len, C, s->heads, s->n, &p);
  return p;
}

scope::Subspaces three_subspaces(const int32_t *c_m) {
  scope::Subspaces sub{};
  sub.M = 3;
  for (int m = 0; m < 3; ++m) sub.c[m] = c_m[m];
  return sub;
}

struct QueryWs {
  int32_t *hist, *rel;
  long long *slab;
  int32_t *cslab;
  uint16_t *ubf;
  float *nu, *bnd, *split;
};

// part/pnx of a chunked codebook inside one split buffer
void set_split(KmProblem &p, float *split) {
  p.part = split;
  p.pnx = split ? split + static_cast<size_t>(p.heads) * p.n * 4 * scope::km_parts(p.C, p.dx)
                : nullptr;
}
size_t query_ws(const scope_shape *s, int c_q, void *base, QueryWs *w) {
  Carver cv(base);
  const int nch = scope::km_nchunks(s->n);
  const scope::AccPlan plan = query_plan(s, c_q);
  QueryWs q;
  q.hist = cv.take<int32_t>(static_cast<size_t>(s->heads) * nch * c_q);
  q.rel = cv.take<int32_t>(static_cast<size_t>(s->heads) * nch * c_q);
  q.slab = cv.take<long long>(scope::km_accum_slab_bytes(plan, s->heads) / sizeof(long long));
  q.cslab = cv.take<int32_t>(scope::km_accum_cslab_bytes(plan, s->heads) / sizeof(int32_t));
  const int cpad = scope::km_cpad(c_q);
  q.ubf = cv.take<uint16_t>(static_cast<size_t>(s->heads) * cpad * 2 * scope::km_dxp(s->d));
  q.nu = cv.take<float>(static_cast<size_t>(s->heads) * cpad);
  q.bnd = cv.take<float>(static_cast<size_t>(s->heads) * cpad * 2);
  q.split = cv.take<float>(scope::km_split_floats(c_q, s->d, s->heads, s->n));
  if (w) *w = q;
  return cv.used;
}

struct KeyWs {
  int32_t *assign3;
  long long *slab;
  int32_t *cslab;
  uint16_t *ubf[3];
  float *nu[3], *bnd[3];
  float *split;  // shared by the subspaces, whose assignments run in turn
  char *args3;   // arguments of the one-pass assignment of the three subspaces
};
size_t key_ws(const scope_shape *s, const int32_t *c_m, void *base, KeyWs *w) {
  Carver cv(base);
  const size_t H = static_cast<size_t>(s->heads);
  const scope::AccPlan plan = key_plan(s, c_m);
  KeyWs k;
  k.assign3 = cv.take<int32_t>(H * 3 * s->n);
  k.slab = cv.take<long long>(scope::km_accum_slab_bytes(plan, s->heads) / sizeof(long long));
  k.cslab = cv.take<int32_t>(scope::km_accum_cslab_bytes(plan, s->heads) / sizeof(int32_t));
  for (int m = 0; m < 3; ++m) {
    const int C = c_m[m], dx = s->range_len[m];
    const int cpad = scope::km_cpad(C);
    k.ubf[m] = cv.take<uint16_t>(H * cpad * 2 * scope::km_dxp(dx));
    k.nu[m] = cv.take<float>(H * cpad);
    k.bnd[m] = cv.take<float>(H * cpad * 2);
  }
  size_t split = 0;
  for (int m = 0; m < 3; ++m) {
    const size_t f = scope::km_split_floats(c_m[m], s->range_len[m], s->heads, s->n);
    split = f > split ? f : split;
  }
  k.split = cv.take<float>(split);
  k.args3 = cv.take<char>(scope::km_assign3_scratch_bytes());
  if (w) *w = k;
  return cv.used;
}

struct SelectWs {
  float *row_max;
  uint32_t *row_state;
  uint32_t *coarse_hist;
  uint32_t *dedup;
};
size_t select_ws(const scope_shape *s, int c_q, void *base, SelectWs *w) {
  Carver cv(base);
  SelectWs sw;
  sw.row_max = cv.take<float>(static_cast<size_t>(s->heads) * c_q);
  sw.row_state = cv.take<uint32_t>(static_cast<size_t>(s->heads) * c_q * 4);
  sw.coarse_hist = cv.take<uint32_t>(static_cast<size_t>(s->heads) * c_q * scope::kSelCoarseBins);
  sw.dedup = cv.take<uint32_t>(scope::select_dedup_words(s->heads, s->n));
  if (w) *w = sw;
  return cv.used;
}

size_t attn_ws(const scope_shape *s, int c_q, void *base, int4 **items) {
  Carver cv(base);
  int4 *it = cv.take<int4>(2 * static_cast<size_t>(s->heads) * scope::attn_items_per_head(s->n, c_q));
  if (items) *items = it;
  return cv.used;
}

// --- general key partitions ----------------------------------------------
int32_t check_partition(const scope_shape *s, const scope_partition *p) {
  if (!p || p->m < 1) return SCOPE_ERR_INVALID_ARGUMENT;
  if (p->m > scope::kMaxSub) return SCOPE_ERR_UNSUPPORTED;
  int total = 0, cs = 0;
  for (int m = 0; m < p->m; ++m) {
    if (p->len[m] < 1 || p->c[m] < 1 || p->c[m] > s->n) return SCOPE_ERR_INVALID_ARGUMENT;
    if (p->c[m] > kMaxC) return SCOPE_ERR_UNSUPPORTED;
    total += p->len[m];
    cs += p->c[m];
  }
  if (total != s->d) return SCOPE_ERR_INVALID_ARGUMENT;
  bool seen[SCOPE_MAX_D] = {};
  int t = 0;
  for (int m = 0; m < p->m; ++m)
    for (int k = 0; k < p->len[m]; ++k, ++t) {
      const int ch = p->channels[t];
      if (ch < 0 || ch >= s->d || seen[ch]) return SCOPE_ERR_INVALID_ARGUMENT;
      if (k > 0 && ch <= p->channels[t - 1]) return SCOPE_ERR_INVALID_ARGUMENT;
      seen[ch] = true;
    }
  if (cs > scope::kSelMaxTable) return SCOPE_ERR_UNSUPPORTED;
  return SCOPE_OK;
}

// The sets are the ranges [0, len0), [len0, len0 + len1), ...: no reordering.
bool partition_in_order(const scope_shape *s, const scope_partition *p) {
  for (int t = 0; t < s->d; ++t)
    if (p->channels[t] != t) return false;
  return true;
}

struct PartGeom {
  int M;
  int off[scope::kMaxSub], len[scope::kMaxSub], C[scope::kMaxSub];
  size_t per_head;  // centroid floats of one head
};
PartGeom part_geom(const scope_partition *p) {
  PartGeom g{};
  g.M = p->m;
  int off = 0;
  for (int m = 0; m < p->m; ++m) {
    g.off[m] = off;  // position of subspace m in the reordered channels
    g.len[m] = p->len[m];
    g.C[m] = p->c[m];
    off += p->len[m];
    g.per_head += static_cast<size_t>(p->c[m]) * p->len[m];
  }
  return g;
}
scope::Subspaces part_subspaces(const PartGeom &g) {
  scope::Subspaces sub{};
  sub.M = g.M;
  for (int m = 0; m < g.M; ++m) sub.c[m] = g.C[m];
  return sub;
}
scope::ChannelMap part_map(const scope_shape *s, const scope_partition *p) {
  scope::ChannelMap map{};
  for (int t = 0; t < s->d; ++t) map.chan[t] = p->channels[t];
  return map;
}
scope::AccPlan part_plan(const scope_shape *s, const PartGeom &g) {
  scope::AccPlan plan;
  scope::km_accum_plan(g.M, g.off, g.len, g.C, s->heads, s->n, &plan);
  return plan;
}

struct PartKeyWs {
  void *kp;  // channel-reordered K, or null
  int32_t *assign;
  long long *slab;
  int32_t *cslab;
  uint16_t *ubf[scope::kMaxSub];
  float *nu[scope::kMaxSub], *bnd[scope::kMaxSub];
  float *split;
};
size_t part_key_ws(const scope_shape *s, const scope_partition *p, void *base,
                   PartKeyWs *w) {
  Carver cv(base);
  const size_t H = static_cast<size_t>(s->heads);
  const PartGeom g = part_geom(p);
  const scope::AccPlan plan = part_plan(s, g);
  PartKeyWs k{};
  if (!partition_in_order(s, p)) {
    const size_t elems = H * s->n * s->d;
    k.kp = s->dtype == SCOPE_BF16 ? static_cast<void *>(cv.take<uint16_t>(elems))
                                  : static_cast<void *>(cv.take<float>(elems));
  }
  k.assign = cv.take<int32_t>(H * g.M * s->n);
  k.slab = cv.take<long long>(scope::km_accum_slab_bytes(plan, s->heads) / sizeof(long long));
  k.cslab = cv.take<int32_t>(scope::km_accum_cslab_bytes(plan, s->heads) / sizeof(int32_t));
  for (int m = 0; m < g.M; ++m) {
    const int cpad = scope::km_cpad(g.C[m]);
    k.ubf[m] = cv.take<uint16_t>(H * cpad * 2 * scope::km_dxp(g.len[m]));
    k.nu[m] = cv.take<float>(H * cpad);
    k.bnd[m] = cv.take<float>(H * cpad * 2);
  }
  size_t split = 0;
  for (int m = 0; m < g.M; ++m) {
    const size_t f = scope::km_split_floats(g.C[m], g.len[m], s->heads, s->n);
    split = f > split ? f : split;
  }
  k.split = cv.take<float>(split);
  if (w) *w = k;
  return cv.used;
}

// channel-reordered query centroids for the tables
size_t part_table_ws(const scope_shape *s, int c_q, void *base, float **qp) {
  Carver cv(base);
  float *q = cv.take<float>(static_cast<size_t>(s->heads) * c_q * s->d);
  if (qp) *qp = q;
  return cv.used;
}

#define SCOPE_TRY(expr)                                  \
  do {                                                   \
    if ((expr) != hipSuccess) return SCOPE_ERR_HIP;      \
  } while (0)

}  // namespace

extern "C" {

int32_t scope_abi_version(void) { return SCOPE_ABI_VERSION; }

const char *scope_status_string(int32_t status) {
  switch (status) {
    case SCOPE_OK: return "ok";
    case SCOPE_ERR_INVALID_ARGUMENT: return "invalid argument";
    case SCOPE_ERR_UNSUPPORTED: return "unsupported argument";
    case SCOPE_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case SCOPE_ERR_HIP: return "HIP launch failure";
    case SCOPE_ERR_SCRATCH_LIMIT:
      return "problem exceeds the fixed work list of the no-allocation entry point";
    default: return "unknown status";
  }
}

int32_t scope_workspace_size(const scope_shape *shape, int32_t c_q,
                             const int32_t c_m[3], size_t *bytes) {
  int32_t st = check_shape(shape);
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if ((st = check_cm(shape, c_m))) return st;
  if (!bytes) return SCOPE_ERR_INVALID_ARGUMENT;
  if (query_plan(shape, c_q).nwin == 0 || key_plan(shape, c_m).nwin == 0)
    return SCOPE_ERR_UNSUPPORTED;
  size_t need = query_ws(shape, c_q, nullptr, nullptr);
  size_t k = key_ws(shape, c_m, nullptr, nullptr);
  size_t s = select_ws(shape, c_q, nullptr, nullptr);
  size_t a = attn_ws(shape, c_q, nullptr, nullptr);
  if (k > need) need = k;
  if (s > need) need = s;
  if (a > need) need = a;
  *bytes = need;
  return SCOPE_OK;
}

}  // extern "C"

namespace {

// Query clustering; `warm` starts from the centroids already in q_centroids
// instead of the rows init_idx.
int32_t cluster_queries(const scope_shape *shape, const void *q, int32_t c_q, int32_t iters,
                        const int32_t *init_idx, bool warm, float *q_centroids,
                        int32_t *assign, int32_t *counts, int32_t *offsets, int32_t *perm,
                        void *workspace, size_t ws_bytes, int32_t *dev_status, void *stream) {
  int32_t st = check_shape(shape);
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if (iters < 1) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!q || !q_centroids || !assign || !counts || !offsets || !perm)
    return SCOPE_ERR_INVALID_ARGUMENT;
  if (!aligned_data(q, shape)) return SCOPE_ERR_INVALID_ARGUMENT;
  if (query_plan(shape, c_q).nwin == 0) return SCOPE_ERR_UNSUPPORTED;
  QueryWs w;
  const size_t need = query_ws(shape, c_q, nullptr, nullptr);
  if ((st = check_ws(workspace, ws_bytes, need))) return st;
  query_ws(shape, c_q, workspace, &w);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = shape->n, d = shape->d;
  KmProblem p{};
  p.x = q;
  p.bf16 = shape->dtype == SCOPE_BF16;
  p.x_head_stride = static_cast<size_t>(n) * d;
  p.ld = d;
  p.col0 = 0;
  p.dx = d;
  p.n = n;
  p.C = c_q;
  p.u = q_centroids;
  p.u_head_stride = static_cast<size_t>(c_q) * d;
  p.assign = assign;
  p.a_head_stride = static_cast<size_t>(n);
  p.counts = counts;
  p.offsets = offsets;
  p.perm = perm;
  p.chunk_hist = w.hist;
  p.chunk_rel = w.rel;
  p.heads = shape->heads;
  p.mfma = scope::km_mfma_ok(p.bf16, p.ld, p.col0, p.dx, p.C);
  p.cpad = scope::km_cpad(p.C);
  p.dxp = scope::km_dxp(p.dx);
  p.ubf = w.ubf;
  p.nu = w.nu;
  p.bnd = w.bnd;
  set_split(p, w.split);
  const scope::AccPlan plan = query_plan(shape, c_q);
  if (!warm) SCOPE_TRY(scope::km_init(p, init_idx, c_q, dev_status, s));
  // the returned grouping is that of the last assignment, taken before the
  // last update
  for (int it = 0; it < iters; ++it) {
    const bool last = it + 1 == iters;
    SCOPE_TRY(scope::km_assign(p, last, s));
    if (last) SCOPE_TRY(scope::km_group(p, s));
    SCOPE_TRY(scope::km_accum(plan, q, p.bf16, p.x_head_stride, d, n, shape->heads,
                              assign, p.a_head_stride, 0, w.slab, w.cslab,
                              q_centroids, p.u_head_stride, it == 0 ? dev_status : nullptr,
                              s));
  }
  return SCOPE_OK;
}

// Key subspace clustering; `warm` starts from the codebooks already in
// k_centroids instead of the rows init_idx.
int32_t cluster_key_subspaces(const scope_shape *shape, const void *k, const int32_t c_m[3],
                              int32_t iters, const int32_t *init_idx, int32_t init_stride,
                              bool warm, float *k_centroids, uint32_t *codes, void *workspace,
                              size_t ws_bytes, int32_t *dev_status, void *stream) {
  int32_t st = check_shape(shape);
  if (st) return st;
  if ((st = check_cm(shape, c_m))) return st;
  if (iters < 1) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!k || !k_centroids || !codes) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!aligned_data(k, shape)) return SCOPE_ERR_INVALID_ARGUMENT;
  if (init_idx) {
    const int mx = c_m[0] > c_m[1] ? (c_m[0] > c_m[2] ? c_m[0] : c_m[2])
                                   : (c_m[1] > c_m[2] ? c_m[1] : c_m[2]);
    if (init_stride < mx) return SCOPE_ERR_INVALID_ARGUMENT;
  }
  if (key_plan(shape, c_m).nwin == 0) return SCOPE_ERR_UNSUPPORTED;
  const size_t need = key_ws(shape, c_m, nullptr, nullptr);
  if ((st = check_ws(workspace, ws_bytes, need))) return st;
  KeyWs w;
  key_ws(shape, c_m, workspace, &w);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = shape->n, d = shape->d;
  KmProblem p[3];
  size_t ucol = 0;
  size_t per_head = 0;
  for (int m = 0; m < 3; ++m) per_head += static_cast<size_t>(c_m[m]) * shape->range_len[m];
  for (int m = 0; m < 3; ++m) {
    KmProblem &pm = p[m];
    pm = KmProblem{};
    pm.x = k;
    pm.bf16 = shape->dtype == SCOPE_BF16;
    pm.x_head_stride = static_cast<size_t>(n) * d;
    pm.ld = d;
    pm.col0 = shape->range_off[m];
    pm.dx = shape->range_len[m];
    pm.n = n;
    pm.C = c_m[m];
    pm.u = k_centroids + ucol;
    pm.u_head_stride = per_head;
    pm.assign = w.assign3 + static_cast<size_t>(m) * n;
    pm.a_head_stride = static_cast<size_t>(3) * n;
    pm.heads = shape->heads;
    pm.mfma = scope::km_mfma_ok(pm.bf16, pm.ld, pm.col0, pm.dx, pm.C);
    pm.cpad = scope::km_cpad(pm.C);
    pm.dxp = scope::km_dxp(pm.dx);
    pm.ubf = w.ubf[m];
    pm.nu = w.nu[m];
    pm.bnd = w.bnd[m];
    set_split(pm, w.split);
    ucol += static_cast<size_t>(c_m[m]) * pm.dx;
    const int32_t *init = init_idx ? init_idx + static_cast<size_t>(m) * init_stride : nullptr;
    // init rows of head h, subspace m live at init_idx[(h*3 + m)*init_stride]
    if (!warm) SCOPE_TRY(scope::km_init(pm, init, 3 * init_stride, dev_status, s));
  }
  const scope::AccPlan plan = key_plan(shape, c_m);
  // the three assignments in one pass over K when the codebooks fit the LDS
  // together, else one pass per subspace
  const bool fused = scope::km_assign3_ok(p);
  bool args_stored = false;
  auto assign_all = [&]() -> hipError_t {
    if (fused) {
      const hipError_t e = scope::km_assign3(p, w.args3, !args_stored, s);
      args_stored = true;
      return e;
    }
    for (int m = 0; m < 3; ++m) {
      const hipError_t e = scope::km_assign(p[m], false, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  };
  for (int it = 0; it < iters; ++it) {
    SCOPE_TRY(assign_all());
    SCOPE_TRY(scope::km_accum(plan, k, p[0].bf16, p[0].x_head_stride, d, n, shape->heads,
                              w.assign3, static_cast<size_t>(3) * n, n, w.slab, w.cslab,
                              k_centroids, per_head, it == 0 ? dev_status : nullptr, s));
  }
  SCOPE_TRY(assign_all());
  SCOPE_TRY(scope::km_pack_codes(w.assign3, static_cast<size_t>(3) * n, n, n,
                                 shape->heads, codes, s));
  return SCOPE_OK;
}

}  // namespace

extern "C" {

int32_t scope_cluster_queries(const scope_shape *shape, const void *q, int32_t c_q,
                              int32_t iters, const int32_t *init_idx, float *q_centroids,
                              int32_t *assign, int32_t *counts, int32_t *offsets,
                              int32_t *perm, void *workspace, size_t ws_bytes,
                              int32_t *dev_status, void *stream) {
  return cluster_queries(shape, q, c_q, iters, init_idx, false, q_centroids, assign, counts,
                         offsets, perm, workspace, ws_bytes, dev_status, stream);
}

int32_t scope_cluster_queries_warm(const scope_shape *shape, const void *q, int32_t c_q,
                                   int32_t iters, float *q_centroids, int32_t *assign,
                                   int32_t *counts, int32_t *offsets, int32_t *perm,
                                   void *workspace, size_t ws_bytes, int32_t *dev_status,
                                   void *stream) {
  return cluster_queries(shape, q, c_q, iters, nullptr, true, q_centroids, assign, counts,
                         offsets, perm, workspace, ws_bytes, dev_status, stream);
}

int32_t scope_cluster_key_subspaces(const scope_shape *shape, const void *k,
                                    const int32_t c_m[3], int32_t iters,
                                    const int32_t *init_idx, int32_t init_stride,
                                    float *k_centroids, uint32_t *codes, void *workspace,
                                    size_t ws_bytes, int32_t *dev_status, void *stream) {
  return cluster_key_subspaces(shape, k, c_m, iters, init_idx, init_stride, false, k_centroids,
                               codes, workspace, ws_bytes, dev_status, stream);
}

int32_t scope_cluster_key_subspaces_warm(const scope_shape *shape, const void *k,
                                         const int32_t c_m[3], int32_t iters,
                                         float *k_centroids, uint32_t *codes,
                                         void *workspace, size_t ws_bytes,
                                         int32_t *dev_status, void *stream) {
  return cluster_key_subspaces(shape, k, c_m, iters, nullptr, 0, true, k_centroids, codes,
                               workspace, ws_bytes, dev_status, stream);
}

int32_t scope_proxy_scores(const scope_shape *shape, const float *q_centroids,
                           int32_t c_q, const float *k_centroids,
                           const int32_t c_m[3], const uint32_t *codes,
                           float *tables, float *scores, void *stream) {
  int32_t st = check_shape(shape);
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if ((st = check_cm(shape, c_m))) return st;
  if (!q_centroids || !k_centroids || !tables) return SCOPE_ERR_INVALID_ARGUMENT;
  if (scores && !codes) return SCOPE_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const scope::Subspaces sub = three_subspaces(c_m);
  SCOPE_TRY(scope::score_tables(shape->heads, shape->d, shape->range_off,
                                shape->range_len, c_q, sub, q_centroids,
                                k_centroids, tables, s));
  if (scores)
    SCOPE_TRY(scope::score_logits(shape->heads, shape->n, shape->d, c_q, sub,
                                  tables, codes, nullptr, scores, s));
  return SCOPE_OK;
}

int32_t scope_select_policy(const scope_shape *shape, int32_t c_q,
                            const int32_t c_m[3], const float *scores,
                            const float *tables, const uint32_t *codes,
                            const int32_t *counts, float rho, int32_t k_fix,
                            int32_t *base_counts, int32_t *topp_counts,
                            int32_t *k_head, int32_t *sel_counts,
                            int32_t *sel_idx, void *workspace, size_t ws_bytes,
                            int32_t policy, void *stream) {
  int32_t st = check_shape(shape);
  if (policy != SCOPE_POLICY_ONLINE && policy != SCOPE_POLICY_FIXED &&
      policy != SCOPE_POLICY_TOPP)
    return SCOPE_ERR_INVALID_ARGUMENT;
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if ((st = check_cm(shape, c_m))) return st;
  if (!scores && (!tables || !codes)) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!counts || !base_counts || !k_head || !sel_counts || !sel_idx)
    return SCOPE_ERR_INVALID_ARGUMENT;
  if (!(rho > 0.0f && rho <= 1.0f)) return SCOPE_ERR_INVALID_ARGUMENT;  // rejects NaN
  if (k_fix < 1 || k_fix > shape->n) return SCOPE_ERR_INVALID_ARGUMENT;
  const size_t need = select_ws(shape, c_q, nullptr, nullptr);
  if ((st = check_ws(workspace, ws_bytes, need))) return st;
  SelectWs w;
  select_ws(shape, c_q, workspace, &w);
  SCOPE_TRY(scope::select_run(shape->heads, shape->n, c_q, three_subspaces(c_m),
                              shape->d, scores, tables, codes, nullptr, counts,
                              rho, k_fix,
                              base_counts, topp_counts, k_head, sel_counts,
                              sel_idx, w.row_max, w.row_state, w.coarse_hist, w.dedup, policy,
                              static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

int32_t scope_select(const scope_shape *shape, int32_t c_q,
                     const int32_t c_m[3], const float *scores,
                     const float *tables, const uint32_t *codes,
                     const int32_t *counts, float rho, int32_t k_fix,
                     int32_t *base_counts, int32_t *topp_counts,
                     int32_t *k_head, int32_t *sel_counts, int32_t *sel_idx,
                     void *workspace, size_t ws_bytes, void *stream) {
  return scope_select_policy(shape, c_q, c_m, scores, tables, codes, counts, rho,
                             k_fix, base_counts, topp_counts, k_head, sel_counts,
                             sel_idx, workspace, ws_bytes, SCOPE_POLICY_ONLINE,
                             stream);
}

int32_t scope_partition_workspace_size(const scope_shape *shape, int32_t c_q,
                                       const scope_partition *part,
                                       size_t *bytes) {
  int32_t st = check_dims(shape);
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if ((st = check_partition(shape, part))) return st;
  if (!bytes) return SCOPE_ERR_INVALID_ARGUMENT;
  if (query_plan(shape, c_q).nwin == 0 || part_plan(shape, part_geom(part)).nwin == 0)
    return SCOPE_ERR_UNSUPPORTED;
  size_t need = query_ws(shape, c_q, nullptr, nullptr);
  for (size_t x : {part_key_ws(shape, part, nullptr, nullptr),
                   part_table_ws(shape, c_q, nullptr, nullptr),
                   select_ws(shape, c_q, nullptr, nullptr),
                   attn_ws(shape, c_q, nullptr, nullptr)})
    if (x > need) need = x;
  *bytes = need;
  return SCOPE_OK;
}

int32_t scope_cluster_key_partition(const scope_shape *shape, const void *k,
                                    const scope_partition *part, int32_t iters,
                                    const int32_t *init_idx,
                                    int32_t init_stride, float *k_centroids,
                                    uint16_t *codes, void *workspace,
                                    size_t ws_bytes, int32_t *dev_status,
                                    void *stream) {
  int32_t st = check_dims(shape);
  if (st) return st;
  if ((st = check_partition(shape, part))) return st;
  if (iters < 1) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!k || !k_centroids || !codes) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!aligned_data(k, shape)) return SCOPE_ERR_INVALID_ARGUMENT;
  const PartGeom g = part_geom(part);
  if (init_idx) {
    int mx = 0;
    for (int m = 0; m < g.M; ++m) mx = g.C[m] > mx ? g.C[m] : mx;
    if (init_stride < mx) return SCOPE_ERR_INVALID_ARGUMENT;
  }
  const scope::AccPlan plan = part_plan(shape, g);
  if (plan.nwin == 0) return SCOPE_ERR_UNSUPPORTED;
  const size_t need = part_key_ws(shape, part, nullptr, nullptr);
  if ((st = check_ws(workspace, ws_bytes, need))) return st;
  PartKeyWs w;
  part_key_ws(shape, part, workspace, &w);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = shape->n, d = shape->d, M = g.M;
  const bool bf16 = shape->dtype == SCOPE_BF16;
  const void *x = k;
  if (w.kp) {
    SCOPE_TRY(scope::gather_channels(k, w.kp, static_cast<size_t>(shape->heads) * n, d,
                                     bf16 ? 2 : 4, part_map(shape, part), s));
    x = w.kp;
  }
  KmProblem p[scope::kMaxSub];
  size_t ucol = 0;
  for (int m = 0; m < M; ++m) {
    KmProblem &pm = p[m];
    pm = KmProblem{};
    pm.x = x;
    pm.bf16 = bf16;
    pm.x_head_stride = static_cast<size_t>(n) * d;
    pm.ld = d;
    pm.col0 = g.off[m];
    pm.dx = g.len[m];
    pm.n = n;
    pm.C = g.C[m];
    pm.u = k_centroids + ucol;
    pm.u_head_stride = g.per_head;
    pm.assign = w.assign + static_cast<size_t>(m) * n;
    pm.a_head_stride = static_cast<size_t>(M) * n;
    pm.heads = shape->heads;
    pm.mfma = scope::km_mfma_ok(pm.bf16, pm.ld, pm.col0, pm.dx, pm.C);
    pm.cpad = scope::km_cpad(pm.C);
    pm.dxp = scope::km_dxp(pm.dx);
    pm.ubf = w.ubf[m];
    pm.nu = w.nu[m];
    pm.bnd = w.bnd[m];
    set_split(pm, w.split);
    ucol += static_cast<size_t>(g.C[m]) * pm.dx;
    // rows of head h, subspace m at init_idx[(h*M + m)*init_stride]
    const int32_t *init = init_idx ? init_idx + static_cast<size_t>(m) * init_stride : nullptr;
    SCOPE_TRY(scope::km_init(pm, init, M * init_stride, dev_status, s));
  }
  for (int it = 0; it < iters; ++it) {
    for (int m = 0; m < M; ++m) SCOPE_TRY(scope::km_assign(p[m], false, s));
    SCOPE_TRY(scope::km_accum(plan, x, bf16, p[0].x_head_stride, d, n, shape->heads,
                              w.assign, static_cast<size_t>(M) * n, n, w.slab, w.cslab,
                              k_centroids, g.per_head, it == 0 ? dev_status : nullptr, s));
  }
  for (int m = 0; m < M; ++m) SCOPE_TRY(scope::km_assign(p[m], false, s));
  SCOPE_TRY(scope::km_codes16(w.assign, static_cast<size_t>(shape->heads) * M * n, codes, s));
  return SCOPE_OK;
}

int32_t scope_proxy_scores_partition(const scope_shape *shape,
                                     const float *q_centroids, int32_t c_q,
                                     const float *k_centroids,
                                     const scope_partition *part,
                                     const uint16_t *codes, float *tables,
                                     float *scores, void *workspace,
                                     size_t ws_bytes, void *stream) {
  int32_t st = check_dims(shape);
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if ((st = check_partition(shape, part))) return st;
  if (!q_centroids || !k_centroids || !tables) return SCOPE_ERR_INVALID_ARGUMENT;
  if (scores && !codes) return SCOPE_ERR_INVALID_ARGUMENT;
  const bool in_order = partition_in_order(shape, part);
  if (!in_order &&
      (st = check_ws(workspace, ws_bytes, part_table_ws(shape, c_q, nullptr, nullptr))))
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const PartGeom g = part_geom(part);
  const scope::Subspaces sub = part_subspaces(g);
  const float *qc = q_centroids;
  if (!in_order) {
    float *qp = nullptr;
    part_table_ws(shape, c_q, workspace, &qp);
    SCOPE_TRY(scope::gather_channels(q_centroids, qp, static_cast<size_t>(shape->heads) * c_q,
                                     shape->d, 4, part_map(shape, part), s));
    qc = qp;
  }
  SCOPE_TRY(scope::score_tables(shape->heads, shape->d, g.off, g.len, c_q, sub, qc,
                                k_centroids, tables, s));
  if (scores)
    SCOPE_TRY(scope::score_logits(shape->heads, shape->n, shape->d, c_q, sub, tables,
                                  nullptr, codes, scores, s));
  return SCOPE_OK;
}

int32_t scope_select_partition(const scope_shape *shape, int32_t c_q,
                               const scope_partition *part,
                               const float *scores, const float *tables,
                               const uint16_t *codes, const int32_t *counts,
                               float rho, int32_t k_fix, int32_t *base_counts,
                               int32_t *topp_counts, int32_t *k_head,
                               int32_t *sel_counts, int32_t *sel_idx,
                               void *workspace, size_t ws_bytes, int32_t policy,
                               void *stream) {
  int32_t st = check_dims(shape);
  if (policy != SCOPE_POLICY_ONLINE && policy != SCOPE_POLICY_FIXED &&
      policy != SCOPE_POLICY_TOPP)
    return SCOPE_ERR_INVALID_ARGUMENT;
  if (st) return st;
  if ((st = check_cq(shape, c_q))) return st;
  if ((st = check_partition(shape, part))) return st;
  if (!scores && (!tables || !codes)) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!counts || !base_counts || !k_head || !sel_counts || !sel_idx)
    return SCOPE_ERR_INVALID_ARGUMENT;
  if (!(rho > 0.0f && rho <= 1.0f)) return SCOPE_ERR_INVALID_ARGUMENT;
  if (k_fix < 1 || k_fix > shape->n) return SCOPE_ERR_INVALID_ARGUMENT;
  const size_t need = select_ws(shape, c_q, nullptr, nullptr);
  if ((st = check_ws(workspace, ws_bytes, need))) return st;
  SelectWs w;
  select_ws(shape, c_q, workspace, &w);
  SCOPE_TRY(scope::select_run(shape->heads, shape->n, c_q, part_subspaces(part_geom(part)),
                              shape->d, scores, tables, nullptr, codes, counts, rho,
                              k_fix, base_counts, topp_counts, k_head, sel_counts,
                              sel_idx, w.row_max, w.row_state, w.coarse_hist, w.dedup, policy,
                              static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

}  // extern "C"

namespace {

int32_t check_attention(const scope_shape *shape, const void *q, const void *k,
                        const void *v, int32_t c_q, const int32_t *offsets,
                        const int32_t *perm, const int32_t *sel_counts,
                        const int32_t *sel_idx, float scale, const void *o) {
  int32_t st = check_shape(shape);
  if (st) return st;
  if (shape->d != 64 && shape->d != 128) return SCOPE_ERR_UNSUPPORTED;
  // the bf16 gather addresses one head's K or V with 32-bit byte offsets
  if (shape->dtype == SCOPE_BF16 &&
      static_cast<uint64_t>(shape->n) * shape->d * 2 >= (1ull << 32))
    return SCOPE_ERR_UNSUPPORTED;
  if (c_q < 1 || c_q > shape->n) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!q || !k || !v || !o || !offsets || !perm || !sel_counts || !sel_idx)
    return SCOPE_ERR_INVALID_ARGUMENT;
  // rows are read and written as 16-byte vectors
  for (const void *p : {q, k, v, o})
    if (reinterpret_cast<uintptr_t>(p) % 16) return SCOPE_ERR_INVALID_ARGUMENT;
  if (!(scale == scale) || isinf(scale)) return SCOPE_ERR_INVALID_ARGUMENT;
  return SCOPE_OK;
}

float attention_scale(const scope_shape *shape, float scale) {
  return scale > 0.0f ? scale
                      : static_cast<float>(1.0 / sqrt(static_cast<double>(shape->d)));
}

}  // namespace

extern "C" {

int32_t scope_sparse_attention_noalloc(const scope_shape *shape, const void *q,
                                       const void *k, const void *v,
                                       int32_t c_q, const int32_t *offsets,
                                       const int32_t *perm,
                                       const int32_t *sel_counts,
                                       const int32_t *sel_idx, float scale,
                                       void *o, void *stream) {
  int32_t st = check_attention(shape, q, k, v, c_q, offsets, perm, sel_counts,
                               sel_idx, scale, o);
  if (st) return st;
  // two 16-byte entries per work slot
  const size_t entries = 2 * static_cast<size_t>(shape->heads) *
                         scope::attn_items_per_head(shape->n, c_q);
  if (entries > scope::kAttnScratchItems) return SCOPE_ERR_SCRATCH_LIMIT;
  int4 *list = nullptr;
  SCOPE_TRY(scope::attention_scratch(&list));
  SCOPE_TRY(scope::attention_run(shape->heads, shape->n, shape->d,
                                 shape->dtype == SCOPE_BF16, q, k, v, o, c_q,
                                 offsets, perm, sel_counts, sel_idx,
                                 attention_scale(shape, scale), list,
                                 static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

int32_t scope_sparse_attention(const scope_shape *shape, const void *q,
                               const void *k, const void *v, int32_t c_q,
                               const int32_t *offsets, const int32_t *perm,
                               const int32_t *sel_counts,
                               const int32_t *sel_idx, float scale, void *o,
                               void *workspace, size_t ws_bytes,
                               void *stream) {
  int32_t st = check_attention(shape, q, k, v, c_q, offsets, perm, sel_counts,
                               sel_idx, scale, o);
  if (st) return st;
  const size_t need = attn_ws(shape, c_q, nullptr, nullptr);
  if ((st = check_ws(workspace, ws_bytes, need))) return st;
  int4 *items = nullptr;
  attn_ws(shape, c_q, workspace, &items);
  SCOPE_TRY(scope::attention_run(shape->heads, shape->n, shape->d,
                                 shape->dtype == SCOPE_BF16, q, k, v, o, c_q,
                                 offsets, perm, sel_counts, sel_idx,
                                 attention_scale(shape, scale), items,
                                 static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

int32_t scope_debug_copy(const void *src, void *dst, size_t bytes, void *stream) {
  if (bytes % 16) return SCOPE_ERR_INVALID_ARGUMENT;
  if (bytes == 0) return SCOPE_OK;
  if (!src || !dst || reinterpret_cast<uintptr_t>(src) % 16 ||
      reinterpret_cast<uintptr_t>(dst) % 16)
    return SCOPE_ERR_INVALID_ARGUMENT;
  const uintptr_t a = reinterpret_cast<uintptr_t>(src), b = reinterpret_cast<uintptr_t>(dst);
  if (a < b + bytes && b < a + bytes) return SCOPE_ERR_INVALID_ARGUMENT;
  SCOPE_TRY(scope::peak_copy(src, dst, bytes, static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

int32_t scope_debug_mfma_loop(float *out, int32_t blocks, int32_t iters, void *stream) {
  if (!out || blocks < 1 || blocks > (1 << 20) || iters < 1) return SCOPE_ERR_INVALID_ARGUMENT;
  SCOPE_TRY(scope::peak_mfma(out, blocks, iters, static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

int32_t scope_debug_attention_items(int32_t heads, int32_t n, int32_t c_q, int32_t pair,
                                    const int32_t *offsets, const int32_t *sel_counts,
                                    int32_t *items, int64_t capacity,
                                    int32_t *items_per_head, void *stream) {
  if (heads < 1 || heads > 65535 || n < 1 || n > kMaxN || c_q < 1 || c_q > n)
    return SCOPE_ERR_INVALID_ARGUMENT;
  if (!offsets || !sel_counts || !items || !items_per_head ||
      reinterpret_cast<uintptr_t>(items) % 16)
    return SCOPE_ERR_INVALID_ARGUMENT;
  const int iph = scope::attn_items_per_head(n, c_q);
  if (capacity < 0 || static_cast<uint64_t>(capacity) < 8ull * heads * iph)
    return SCOPE_ERR_INVALID_ARGUMENT;
  *items_per_head = iph;
  SCOPE_TRY(scope::attention_items(heads, n, c_q, pair != 0, offsets, sel_counts,
                                   reinterpret_cast<int4 *>(items),
                                   static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

int32_t scope_debug_fixexp(const float *y, uint64_t *out, int64_t count,
                           void *stream) {
  if (count < 0 || (count > 0 && (!y || !out))) return SCOPE_ERR_INVALID_ARGUMENT;
  SCOPE_TRY(scope::debug_fixexp(y, out, count, static_cast<hipStream_t>(stream)));
  return SCOPE_OK;
}

}  // extern "C"
