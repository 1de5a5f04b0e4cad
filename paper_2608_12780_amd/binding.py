"""Thin Python binding of libscope.so (argument marshalling only).

Each ``scope_*`` function mirrors the C entry point of the same name in
include/scope.h: it takes torch tensors that already live on the GPU, checks
their dtype, size and contiguity, passes their device pointers and the
current HIP stream to the library, and raises ScopeError on a non-zero
status.  Every stage of the layer runs in the library's HIP kernels; this
module computes nothing.  It fails loudly if the library is not built.
"""
from __future__ import annotations

import ctypes
import os

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
# SCOPE_LIBRARY selects another build of the library (e.g. libscope_san.so)
LIB_PATH = os.environ.get("SCOPE_LIBRARY") or os.path.join(PKG, "libscope.so")

F32, BF16 = 0, 1
ENTRY_POINTS = (
    "scope_abi_version", "scope_status_string", "scope_workspace_size",
    "scope_cluster_queries", "scope_cluster_key_subspaces",
    "scope_proxy_scores", "scope_select", "scope_select_policy",
    "scope_sparse_attention", "scope_debug_fixexp",
    "scope_partition_workspace_size", "scope_cluster_key_partition",
    "scope_proxy_scores_partition", "scope_select_partition",
    "scope_sparse_attention_noalloc", "scope_debug_copy", "scope_debug_mfma_loop",
    "scope_cluster_queries_warm", "scope_cluster_key_subspaces_warm",
    "scope_debug_attention_items",
)
MAX_SUBSPACES, MAX_D = 8, 128
POLICIES = {"online": 0, "fixed": 1, "topp": 2}


class ScopeError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn}: {status_string(status)} (status {status})")


class Shape(ctypes.Structure):
    _fields_ = [("heads", ctypes.c_int32), ("n", ctypes.c_int32),
                ("d", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("range_off", ctypes.c_int32 * 3),
                ("range_len", ctypes.c_int32 * 3)]


def make_shape(heads, n, d, dtype, ranges) -> Shape:
    off, ln = ranges
    return Shape(int(heads), int(n), int(d), int(dtype),
                 (ctypes.c_int32 * 3)(*map(int, off)),
                 (ctypes.c_int32 * 3)(*map(int, ln)))


class Partition(ctypes.Structure):
    """A general key partition: M channel sets and their codebook sizes."""
    _fields_ = [("m", ctypes.c_int32), ("c", ctypes.c_int32 * MAX_SUBSPACES),
                ("len", ctypes.c_int32 * MAX_SUBSPACES),
                ("channels", ctypes.c_int32 * MAX_D)]


def make_partition(sets, c_m) -> Partition:
    """sets: M sequences of channel indices (each ascending); c_m: M sizes."""
    sets = [list(map(int, x)) for x in sets]
    if len(sets) != len(c_m) or not 1 <= len(sets) <= MAX_SUBSPACES:
        raise ValueError("need 1..8 channel sets, one codebook size each")
    chan = [ch for x in sets for ch in x]
    if len(chan) > MAX_D:
        raise ValueError("more than 128 channels")
    p = Partition()
    p.m = len(sets)
    for m, x in enumerate(sets):
        p.c[m] = int(c_m[m])
        p.len[m] = len(x)
    for t, ch in enumerate(chan):
        p.channels[t] = ch
    return p


_lib = None


def lib() -> ctypes.CDLL:
    """Load libscope.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2608_12780_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        P, I, Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        SP = ctypes.POINTER(Shape)
        L.scope_abi_version.restype = I
        L.scope_status_string.argtypes = [I]
        L.scope_status_string.restype = ctypes.c_char_p
        L.scope_workspace_size.argtypes = [SP, I, P, ctypes.POINTER(Z)]
        L.scope_cluster_queries.argtypes = [SP, P, I, I, P, P, P, P, P, P, P, Z, P, P]
        L.scope_cluster_key_subspaces.argtypes = [SP, P, P, I, P, I, P, P, P, Z, P, P]
        L.scope_cluster_queries_warm.argtypes = [SP, P, I, I, P, P, P, P, P, P, Z, P, P]
        L.scope_cluster_key_subspaces_warm.argtypes = [SP, P, P, I, P, P, P, Z, P, P]
        L.scope_proxy_scores.argtypes = [SP, P, I, P, P, P, P, P, P]
        L.scope_select.argtypes = [SP, I, P, P, P, P, P, ctypes.c_float, I, P, P,
                                   P, P, P, P, Z, P]
        L.scope_select_policy.argtypes = [SP, I, P, P, P, P, P, ctypes.c_float, I, P,
                                          P, P, P, P, P, Z, I, P]
        L.scope_sparse_attention.argtypes = [SP, P, P, P, I, P, P, P, P,
                                             ctypes.c_float, P, P, Z, P]
        L.scope_sparse_attention_noalloc.argtypes = [SP, P, P, P, I, P, P, P, P,
                                                     ctypes.c_float, P, P]
        L.scope_debug_fixexp.argtypes = [P, P, ctypes.c_int64, P]
        L.scope_debug_copy.argtypes = [P, P, Z, P]
        L.scope_debug_mfma_loop.argtypes = [P, I, I, P]
        L.scope_debug_attention_items.argtypes = [I, I, I, I, P, P, P, ctypes.c_int64,
                                                  ctypes.POINTER(I), P]
        PP = ctypes.POINTER(Partition)
        L.scope_partition_workspace_size.argtypes = [SP, I, PP, ctypes.POINTER(Z)]
        L.scope_cluster_key_partition.argtypes = [SP, P, PP, I, P, I, P, P, P, Z, P, P]
        L.scope_proxy_scores_partition.argtypes = [SP, P, I, P, PP, P, P, P, P, Z, P]
        L.scope_select_partition.argtypes = [SP, I, PP, P, P, P, P, ctypes.c_float, I,
                                             P, P, P, P, P, P, Z, I, P]
        for name in ENTRY_POINTS[2:]:
            getattr(L, name).restype = I
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().scope_status_string(int(status)).decode()


def _check(fn, status):
    if status != 0:
        raise ScopeError(fn, status)


def _cm(c_m):
    return (ctypes.c_int32 * 3)(*map(int, c_m))


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t, dtype=None, numel=None, name="tensor", optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} needs {numel} elements, has {t.numel()}")
    return ctypes.c_void_p(t.data_ptr())


def _data_dtype(shape: Shape):
    return torch.bfloat16 if shape.dtype == BF16 else torch.float32


def scope_workspace_size(shape: Shape, c_q: int, c_m) -> int:
    out = ctypes.c_size_t(0)
    _check("scope_workspace_size",
           lib().scope_workspace_size(ctypes.byref(shape), int(c_q), _cm(c_m),
                                      ctypes.byref(out)))
    return int(out.value)


def alloc_workspace(shape: Shape, c_q: int, c_m, device="cuda"):
    """A uint8 workspace tensor (torch's allocator aligns to >= 256 bytes)."""
    return torch.empty(max(scope_workspace_size(shape, c_q, c_m), 1),
                       dtype=torch.uint8, device=device)


def scope_cluster_queries(shape, q, c_q, iters, init_idx, q_centroids, assign,
                          counts, offsets, perm, workspace, dev_status=None,
                          stream=None):
    H, N, D = shape.heads, shape.n, shape.d
    _check("scope_cluster_queries", lib().scope_cluster_queries(
        ctypes.byref(shape), _ptr(q, _data_dtype(shape), H * N * D, "q"),
        int(c_q), int(iters),
        _ptr(init_idx, torch.int32, H * c_q, "init_idx", optional=True),
        _ptr(q_centroids, torch.float32, H * c_q * D, "q_centroids"),
        _ptr(assign, torch.int32, H * N, "assign"),
        _ptr(counts, torch.int32, H * c_q, "counts"),
        _ptr(offsets, torch.int32, H * (c_q + 1), "offsets"),
        _ptr(perm, torch.int32, H * N, "perm"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _ptr(dev_status, torch.int32, 1, "dev_status", optional=True),
        _stream(stream)))


def scope_cluster_queries_warm(shape, q, c_q, iters, q_centroids, assign, counts, offsets,
                               perm, workspace, dev_status=None, stream=None):
    """Call 1w: q_centroids holds the starting centroids and receives the result."""
    H, N, D = shape.heads, shape.n, shape.d
    _check("scope_cluster_queries_warm", lib().scope_cluster_queries_warm(
        ctypes.byref(shape), _ptr(q, _data_dtype(shape), H * N * D, "q"),
        int(c_q), int(iters),
        _ptr(q_centroids, torch.float32, H * c_q * D, "q_centroids"),
        _ptr(assign, torch.int32, H * N, "assign"),
        _ptr(counts, torch.int32, H * c_q, "counts"),
        _ptr(offsets, torch.int32, H * (c_q + 1), "offsets"),
        _ptr(perm, torch.int32, H * N, "perm"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _ptr(dev_status, torch.int32, 1, "dev_status", optional=True),
        _stream(stream)))


def scope_cluster_key_subspaces_warm(shape, k, c_m, iters, k_centroids, codes, workspace,
                                     dev_status=None, stream=None):
    """Call 2w: k_centroids holds the starting codebooks and receives the result."""
    H, N, D = shape.heads, shape.n, shape.d
    per_head = sum(int(c_m[m]) * shape.range_len[m] for m in range(3))
    _check("scope_cluster_key_subspaces_warm", lib().scope_cluster_key_subspaces_warm(
        ctypes.byref(shape), _ptr(k, _data_dtype(shape), H * N * D, "k"),
        _cm(c_m), int(iters),
        _ptr(k_centroids, torch.float32, H * per_head, "k_centroids"),
        _ptr(codes, torch.int32, H * N, "codes"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _ptr(dev_status, torch.int32, 1, "dev_status", optional=True),
        _stream(stream)))


def scope_cluster_key_subspaces(shape, k, c_m, iters, init_idx, init_stride,
                                k_centroids, codes, workspace, dev_status=None,
                                stream=None):
    H, N, D = shape.heads, shape.n, shape.d
    per_head = sum(int(c_m[m]) * shape.range_len[m] for m in range(3))
    _check("scope_cluster_key_subspaces", lib().scope_cluster_key_subspaces(
        ctypes.byref(shape), _ptr(k, _data_dtype(shape), H * N * D, "k"),
        _cm(c_m), int(iters),
        _ptr(init_idx, torch.int32, H * 3 * int(init_stride), "init_idx",
             optional=True), int(init_stride),
        _ptr(k_centroids, torch.float32, H * per_head, "k_centroids"),
        _ptr(codes, torch.int32, H * N, "codes"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _ptr(dev_status, torch.int32, 1, "dev_status", optional=True),
        _stream(stream)))


def scope_proxy_scores(shape, q_centroids, c_q, k_centroids, c_m, codes,
                       tables, scores=None, stream=None):
    H, N, D = shape.heads, shape.n, shape.d
    cs = int(sum(c_m))
    per_head = sum(int(c_m[m]) * shape.range_len[m] for m in range(3))
    _check("scope_proxy_scores", lib().scope_proxy_scores(
        ctypes.byref(shape),
        _ptr(q_centroids, torch.float32, H * c_q * D, "q_centroids"), int(c_q),
        _ptr(k_centroids, torch.float32, H * per_head, "k_centroids"), _cm(c_m),
        _ptr(codes, torch.int32, H * N, "codes", optional=scores is None),
        _ptr(tables, torch.float32, H * c_q * cs, "tables"),
        _ptr(scores, torch.float32, H * c_q * N, "scores", optional=True),
        _stream(stream)))


def scope_select(shape, c_q, c_m, scores, tables, codes, counts, rho, k_fix,
                 base_counts, topp_counts, k_head, sel_counts, sel_idx,
                 workspace, stream=None):
    scope_select_policy(shape, c_q, c_m, scores, tables, codes, counts, rho, k_fix,
                        base_counts, topp_counts, k_head, sel_counts, sel_idx,
                        workspace, "online", stream, name="scope_select")


def scope_select_policy(shape, c_q, c_m, scores, tables, codes, counts, rho, k_fix,
                        base_counts, topp_counts, k_head, sel_counts, sel_idx,
                        workspace, policy="online", stream=None, name="scope_select_policy"):
    H, N = shape.heads, shape.n
    cs = int(sum(c_m))
    fn = lib().scope_select if name == "scope_select" else lib().scope_select_policy
    extra = () if name == "scope_select" else (POLICIES[policy],)
    _check(name, fn(
        ctypes.byref(shape), int(c_q), _cm(c_m),
        _ptr(scores, torch.float32, H * c_q * N, "scores", optional=True),
        _ptr(tables, torch.float32, H * c_q * cs, "tables", optional=True),
        _ptr(codes, torch.int32, H * N, "codes", optional=True),
        _ptr(counts, torch.int32, H * c_q, "counts"), float(rho), int(k_fix),
        _ptr(base_counts, torch.int32, H * c_q, "base_counts"),
        _ptr(topp_counts, torch.int32, H * c_q, "topp_counts", optional=True),
        _ptr(k_head, torch.int32, H, "k_head"),
        _ptr(sel_counts, torch.int32, H * c_q, "sel_counts"),
        _ptr(sel_idx, torch.int32, H * c_q * N, "sel_idx"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        *extra, _stream(stream)))


def scope_sparse_attention(shape, q, k, v, c_q, offsets, perm, sel_counts,
                           sel_idx, scale, o, workspace, stream=None):
    H, N, D = shape.heads, shape.n, shape.d
    dt = _data_dtype(shape)
    _check("scope_sparse_attention", lib().scope_sparse_attention(
        ctypes.byref(shape), _ptr(q, dt, H * N * D, "q"),
        _ptr(k, dt, H * N * D, "k"), _ptr(v, dt, H * N * D, "v"), int(c_q),
        _ptr(offsets, torch.int32, H * (c_q + 1), "offsets"),
        _ptr(perm, torch.int32, H * N, "perm"),
        _ptr(sel_counts, torch.int32, H * c_q, "sel_counts"),
        _ptr(sel_idx, torch.int32, H * c_q * N, "sel_idx"), float(scale),
        _ptr(o, dt, H * N * D, "o"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _stream(stream)))


def scope_sparse_attention_noalloc(shape, q, k, v, c_q, offsets, perm, sel_counts,
                                   sel_idx, scale, o, stream=None):
    H, N, D = shape.heads, shape.n, shape.d
    dt = _data_dtype(shape)
    _check("scope_sparse_attention_noalloc", lib().scope_sparse_attention_noalloc(
        ctypes.byref(shape), _ptr(q, dt, H * N * D, "q"),
        _ptr(k, dt, H * N * D, "k"), _ptr(v, dt, H * N * D, "v"), int(c_q),
        _ptr(offsets, torch.int32, H * (c_q + 1), "offsets"),
        _ptr(perm, torch.int32, H * N, "perm"),
        _ptr(sel_counts, torch.int32, H * c_q, "sel_counts"),
        _ptr(sel_idx, torch.int32, H * c_q * N, "sel_idx"), float(scale),
        _ptr(o, dt, H * N * D, "o"), _stream(stream)))


def scope_debug_copy(src, dst, stream=None):
    """Copies src into dst (same byte size) with the library's copy kernel."""
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise ValueError("src and dst must have the same byte size")
    _check("scope_debug_copy", lib().scope_debug_copy(
        _ptr(src, None, None, "src"), _ptr(dst, None, None, "dst"), n, _stream(stream)))


def scope_debug_mfma_loop(out, blocks, iters, stream=None):
    _check("scope_debug_mfma_loop", lib().scope_debug_mfma_loop(
        _ptr(out, torch.float32, int(blocks) * 256, "out"), int(blocks), int(iters),
        _stream(stream)))


def scope_debug_attention_items(heads, n, c_q, offsets, sel_counts, pair=True, stream=None):
    """The sparse attention's work list: an int32 device tensor
    [heads][slots][2][4] of (cluster, first row, rows, selected keys)."""
    s = ctypes.c_int32(0)
    slots = -(-int(n) // 256) + int(c_q)
    items = torch.empty(int(heads) * slots * 8, dtype=torch.int32, device=offsets.device)
    _check("scope_debug_attention_items", lib().scope_debug_attention_items(
        int(heads), int(n), int(c_q), 1 if pair else 0,
        _ptr(offsets, torch.int32, int(heads) * (int(c_q) + 1), "offsets"),
        _ptr(sel_counts, torch.int32, int(heads) * int(c_q), "sel_counts"),
        _ptr(items, torch.int32, None, "items"), items.numel(), ctypes.byref(s),
        _stream(stream)))
    return items.view(int(heads), s.value, 2, 4)


def scope_debug_fixexp(y, out, stream=None):
    _check("scope_debug_fixexp", lib().scope_debug_fixexp(
        _ptr(y, torch.float32, None, "y"), _ptr(out, torch.int64, y.numel(), "out"),
        y.numel(), _stream(stream)))


def scope_partition_workspace_size(shape: Shape, c_q: int, part: Partition) -> int:
    out = ctypes.c_size_t(0)
    _check("scope_partition_workspace_size",
           lib().scope_partition_workspace_size(ctypes.byref(shape), int(c_q),
                                                ctypes.byref(part), ctypes.byref(out)))
    return int(out.value)


def alloc_partition_workspace(shape: Shape, c_q: int, part: Partition, device="cuda"):
    return torch.empty(max(scope_partition_workspace_size(shape, c_q, part), 1),
                       dtype=torch.uint8, device=device)


def _part_sizes(part: Partition):
    per_head = sum(int(part.c[m]) * int(part.len[m]) for m in range(part.m))
    cs = sum(int(part.c[m]) for m in range(part.m))
    return per_head, cs


def scope_cluster_key_partition(shape, k, part, iters, init_idx, init_stride,
                                k_centroids, codes, workspace, dev_status=None,
                                stream=None):
    """codes: int16 tensor holding the uint16 codes [heads][M][n]."""
    H, N, D = shape.heads, shape.n, shape.d
    per_head, _ = _part_sizes(part)
    _check("scope_cluster_key_partition", lib().scope_cluster_key_partition(
        ctypes.byref(shape), _ptr(k, _data_dtype(shape), H * N * D, "k"),
        ctypes.byref(part), int(iters),
        _ptr(init_idx, torch.int32, H * part.m * int(init_stride), "init_idx",
             optional=True), int(init_stride),
        _ptr(k_centroids, torch.float32, H * per_head, "k_centroids"),
        _ptr(codes, torch.int16, H * part.m * N, "codes"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _ptr(dev_status, torch.int32, 1, "dev_status", optional=True),
        _stream(stream)))


def scope_proxy_scores_partition(shape, q_centroids, c_q, k_centroids, part, codes,
                                 tables, scores, workspace, stream=None):
    H, N, D = shape.heads, shape.n, shape.d
    per_head, cs = _part_sizes(part)
    _check("scope_proxy_scores_partition", lib().scope_proxy_scores_partition(
        ctypes.byref(shape),
        _ptr(q_centroids, torch.float32, H * c_q * D, "q_centroids"), int(c_q),
        _ptr(k_centroids, torch.float32, H * per_head, "k_centroids"),
        ctypes.byref(part),
        _ptr(codes, torch.int16, H * part.m * N, "codes", optional=scores is None),
        _ptr(tables, torch.float32, H * c_q * cs, "tables"),
        _ptr(scores, torch.float32, H * c_q * N, "scores", optional=True),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _stream(stream)))


def scope_select_partition(shape, c_q, part, scores, tables, codes, counts, rho,
                           k_fix, base_counts, topp_counts, k_head, sel_counts,
                           sel_idx, workspace, policy="online", stream=None):
    H, N = shape.heads, shape.n
    _, cs = _part_sizes(part)
    _check("scope_select_partition", lib().scope_select_partition(
        ctypes.byref(shape), int(c_q), ctypes.byref(part),
        _ptr(scores, torch.float32, H * c_q * N, "scores", optional=True),
        _ptr(tables, torch.float32, H * c_q * cs, "tables", optional=True),
        _ptr(codes, torch.int16, H * part.m * N, "codes", optional=True),
        _ptr(counts, torch.int32, H * c_q, "counts"), float(rho), int(k_fix),
        _ptr(base_counts, torch.int32, H * c_q, "base_counts"),
        _ptr(topp_counts, torch.int32, H * c_q, "topp_counts", optional=True),
        _ptr(k_head, torch.int32, H, "k_head"),
        _ptr(sel_counts, torch.int32, H * c_q, "sel_counts"),
        _ptr(sel_idx, torch.int32, H * c_q * N, "sel_idx"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        POLICIES[policy], _stream(stream)))
