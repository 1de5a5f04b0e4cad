"""The SCOPE layer as five library calls on buffers allocated once.

ScopeLayer owns every output and the workspace for one problem size and runs
Alg. 1 end to end through the C ABI: query clustering, key-subspace
clustering, score tables, selection and sparse attention.  Nothing here
computes; it allocates device memory and sequences the calls.
"""
from __future__ import annotations

import torch

from . import binding as B


class ScopeLayer:
    def __init__(self, heads, n, d, ranges, c_q, c_m, iters, rho, k_fix,
                 dtype="bf16", device="cuda", materialize_scores=False,
                 workspace=True):
        self.heads, self.n, self.d = int(heads), int(n), int(d)
        self.ranges = (tuple(map(int, ranges[0])), tuple(map(int, ranges[1])))
        self.c_q = int(c_q)
        self.c_m = tuple(int(c) for c in c_m)
        self.iters, self.rho, self.k_fix = int(iters), float(rho), int(k_fix)
        self.dtype = B.BF16 if dtype == "bf16" else B.F32
        self.tdtype = torch.bfloat16 if self.dtype == B.BF16 else torch.float32
        self.shape = B.make_shape(heads, n, d, self.dtype, self.ranges)
        H, N, D, C = self.heads, self.n, self.d, self.c_q
        cs = sum(self.c_m)
        per_head = sum(self.c_m[m] * self.ranges[1][m] for m in range(3))
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.q_centroids = torch.empty(H, C, D, **f32)
        self.assign = torch.empty(H, N, **i32)
        self.counts = torch.empty(H, C, **i32)
        self.offsets = torch.empty(H, C + 1, **i32)
        self.perm = torch.empty(H, N, **i32)
        self.k_centroids = torch.empty(H, per_head, **f32)
        self.codes = torch.empty(H, N, **i32)
        self.tables = torch.empty(H, C, cs, **f32)
        self.scores = torch.empty(H, C, N, **f32) if materialize_scores else None
        self.base_counts = torch.empty(H, C, **i32)
        self.topp_counts = torch.empty(H, C, **i32)
        self.k_head = torch.empty(H, **i32)
        self.sel_counts = torch.empty(H, C, **i32)
        self.sel_idx = torch.empty(H, C, N, **i32)
        self.out = torch.empty(H, N, D, dtype=self.tdtype, device=device)
        self.workspace = (B.alloc_workspace(self.shape, C, self.c_m, device)
                          if workspace else None)
        self.status = torch.zeros(1, **i32)

    # the five stages -------------------------------------------------------
    def cluster_queries(self, q, init_q=None, stream=None, warm=False, iters=None):
        """warm: start from the centroids this layer holds (calls 1w)."""
        it = self.iters if iters is None else int(iters)
        if warm:
            B.scope_cluster_queries_warm(self.shape, q, self.c_q, it, self.q_centroids,
                                         self.assign, self.counts, self.offsets, self.perm,
                                         self.workspace, self.status, stream)
            return
        B.scope_cluster_queries(self.shape, q, self.c_q, it, init_q,
                                self.q_centroids, self.assign, self.counts,
                                self.offsets, self.perm, self.workspace,
                                self.status, stream)

    def cluster_keys(self, k, init_k=None, stream=None, warm=False, iters=None):
        """warm: start from the codebooks this layer holds (call 2w)."""
        it = self.iters if iters is None else int(iters)
        if warm:
            B.scope_cluster_key_subspaces_warm(self.shape, k, self.c_m, it, self.k_centroids,
                                               self.codes, self.workspace, self.status, stream)
            return
        stride = init_k.shape[-1] if init_k is not None else 0
        B.scope_cluster_key_subspaces(self.shape, k, self.c_m, it,
                                      init_k, stride, self.k_centroids,
                                      self.codes, self.workspace, self.status,
                                      stream)

    def proxy_scores(self, stream=None):
        B.scope_proxy_scores(self.shape, self.q_centroids, self.c_q,
                             self.k_centroids, self.c_m, self.codes,
                             self.tables, self.scores, stream)

    def select(self, stream=None, use_scores=False, policy="online", rho=None):
        """policy "online" is call 4 (Eq. 10); "fixed" and "topp" are the
        Fig. 6 variants through call 4b.  rho overrides the layer's."""
        rho = self.rho if rho is None else rho
        args = (self.shape, self.c_q, self.c_m,
                self.scores if use_scores else None, self.tables,
                self.codes, self.counts, rho, self.k_fix,
                self.base_counts, self.topp_counts, self.k_head,
                self.sel_counts, self.sel_idx, self.workspace)
        if policy == "online":
            B.scope_select(*args, stream)
        else:
            B.scope_select_policy(*args, policy, stream)

    def attend(self, q, k, v, scale=0.0, stream=None):
        B.scope_sparse_attention(self.shape, q, k, v, self.c_q, self.offsets,
                                 self.perm, self.sel_counts, self.sel_idx,
                                 scale, self.out, self.workspace, stream)

    def forward(self, q, k, v, init_q=None, init_k=None, stream=None,
                marks=None, warm=False, warm_iters=None):
        """Runs the layer; `marks(i)` (if given) is called before stage i and
        after the last one, e.g. to record timing events.  warm: the
        clusterings start from the centroids the layer holds (the previous
        denoising step's), with warm_iters iterations (default: iters)."""
        steps = (lambda: self.cluster_queries(q, init_q, stream, warm, warm_iters),
                 lambda: self.cluster_keys(k, init_k, stream, warm, warm_iters),
                 lambda: self.proxy_scores(stream),
                 lambda: self.select(stream),
                 lambda: self.attend(q, k, v, 0.0, stream))
        for i, f in enumerate(steps):
            if marks:
                marks(i)
            f()
        if marks:
            marks(len(steps))
        return self.out


class SparsitySchedule:
    """Where the layer runs across a DiT's layers and denoising steps (Sec. 4
    setup): the first attention layer stays dense at every step, and the
    other layers stay dense during the first `dense_fraction` of the steps
    (20% for the Wan models, 10% for HunyuanVideo), SCOPE afterwards.  The
    first SCOPE step of a layer clusters from seeded rows; later steps may
    warm-start from the previous step's centroids."""

    def __init__(self, steps, dense_fraction, dense_layers=(0,)):
        self.steps = int(steps)
        self.dense_fraction = float(dense_fraction)
        self.dense_layers = frozenset(int(x) for x in dense_layers)
        # the dense prefix in whole steps, ceil(fraction * steps) exactly
        from fractions import Fraction
        f = Fraction(str(dense_fraction)) * self.steps
        self.dense_steps = -((-f.numerator) // f.denominator)

    def dense(self, layer, step):
        return layer in self.dense_layers or step < self.dense_steps

    def warm(self, layer, step):
        """True when the previous step of this layer also ran SCOPE."""
        return not self.dense(layer, step) and step > self.dense_steps


def _dummy_ranges(d):
    """Three valid ranges for the calls that check but do not use them."""
    a = d // 3 // 2 * 2
    ln = (a, a, d - 2 * a)
    return (0, ln[0], ln[0] + ln[1]), ln


class ScopePartitionLayer(ScopeLayer):
    """The layer with the keys split into any M disjoint channel sets (App. B;
    the partition ablation of Table 3), through the partition calls: codes
    are one uint16 plane per subspace (held in an int16 tensor)."""

    def __init__(self, heads, n, d, sets, c_q, c_m, iters, rho, k_fix,
                 dtype="bf16", device="cuda", materialize_scores=False):
        self.sets = [tuple(map(int, x)) for x in sets]
        self.part = B.make_partition(self.sets, c_m)
        M = len(self.sets)
        # the query and attention calls see three placeholder ranges
        super().__init__(heads, n, d, _dummy_ranges(d), c_q, (1, 1, 1), iters,
                         rho, k_fix, dtype, device, materialize_scores,
                         workspace=False)
        self.c_m = tuple(int(c) for c in c_m)
        H, N, C = self.heads, self.n, self.c_q
        per_head = sum(self.c_m[m] * len(self.sets[m]) for m in range(M))
        self.k_centroids = torch.empty(H, per_head, dtype=torch.float32, device=device)
        self.codes = torch.empty(H, M, N, dtype=torch.int16, device=device)
        self.tables = torch.empty(H, C, sum(self.c_m), dtype=torch.float32, device=device)
        self.workspace = B.alloc_partition_workspace(self.shape, C, self.part, device)

    def cluster_keys(self, k, init_k=None, stream=None, warm=False, iters=None):
        if warm:
            raise NotImplementedError("warm starts are offered for the three RoPE ranges only")
        stride = init_k.shape[-1] if init_k is not None else 0
        B.scope_cluster_key_partition(self.shape, k, self.part,
                                      self.iters if iters is None else int(iters), init_k,
                                      stride, self.k_centroids, self.codes,
                                      self.workspace, self.status, stream)

    def proxy_scores(self, stream=None):
        B.scope_proxy_scores_partition(self.shape, self.q_centroids, self.c_q,
                                       self.k_centroids, self.part, self.codes,
                                       self.tables, self.scores, self.workspace,
                                       stream)

    def select(self, stream=None, use_scores=False, policy="online", rho=None):
        rho = self.rho if rho is None else rho
        B.scope_select_partition(self.shape, self.c_q, self.part,
                                 self.scores if use_scores else None, self.tables,
                                 self.codes, self.counts, rho, self.k_fix,
                                 self.base_counts, self.topp_counts, self.k_head,
                                 self.sel_counts, self.sel_idx, self.workspace,
                                 policy, stream)


class DenseAttention:
    """Dense attention (Eq. 1) through the same attention call: one cluster
    holding every query, whose key set is every key."""

    def __init__(self, heads, n, d, dtype="bf16", device="cuda"):
        self.heads, self.n, self.d = int(heads), int(n), int(d)
        self.dtype = B.BF16 if dtype == "bf16" else B.F32
        tdt = torch.bfloat16 if self.dtype == B.BF16 else torch.float32
        self.shape = B.make_shape(heads, n, d, self.dtype, _dummy_ranges(d))
        i32 = dict(dtype=torch.int32, device=device)
        H, N = self.heads, self.n
        self.offsets = torch.tensor([0, N], **i32).repeat(H, 1).contiguous()
        self.perm = torch.arange(N, **i32).repeat(H, 1).contiguous()
        self.sel_counts = torch.full((H, 1), N, **i32)
        self.sel_idx = torch.arange(N, **i32).repeat(H, 1).reshape(H, 1, N).contiguous()
        self.out = torch.empty(H, N, d, dtype=tdt, device=device)
        self.workspace = B.alloc_workspace(self.shape, 1, (1, 1, 1), device)

    def forward(self, q, k, v, scale=0.0, stream=None):
        B.scope_sparse_attention(self.shape, q, k, v, 1, self.offsets,
                                 self.perm, self.sel_counts, self.sel_idx,
                                 scale, self.out, self.workspace, stream)
        return self.out
