"""The C ABI on a host without a GPU: the library loads, exports every entry
point include/scope.h declares, and rejects bad arguments before touching
the GPU (fake device pointers are never dereferenced on these paths)."""
import ctypes
import os
import re

import pytest

from paper_2608_12780_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = ctypes.c_void_p(1 << 20)     # never dereferenced by validation


def declared_entry_points():
    hdr = open(os.path.join(ROOT, "include", "scope.h")).read()
    return re.findall(r"^\w[\w\s\*]*?\b(scope_\w+)\s*\(", hdr, re.M)


def hy_shape(**kw):
    a = dict(heads=24, n=118800, d=128, dtype=B.BF16,
             ranges=((0, 16, 72), (16, 56, 56)))
    a.update(kw)
    return B.make_shape(a["heads"], a["n"], a["d"], a["dtype"], a["ranges"])


def test_library_exports_every_declared_symbol():
    names = declared_entry_points()
    assert set(names) == set(B.ENTRY_POINTS)
    L = B.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.scope_abi_version() == 2


def test_status_strings():
    for s in (OK, INVALID, UNSUPPORTED, WORKSPACE, 4, 5, 99):
        assert isinstance(B.status_string(s), str) and B.status_string(s)


def ws_size(shape, c_q=256, c_m=(128, 128, 128)):
    out = ctypes.c_size_t(0)
    st = B.lib().scope_workspace_size(ctypes.byref(shape), c_q,
                                      (ctypes.c_int32 * 3)(*c_m), ctypes.byref(out))
    return st, out.value


def test_workspace_size_and_shape_validation():
    st, size = ws_size(hy_shape())
    assert st == OK and 10 ** 7 < size < 10 ** 9 and size % 256 == 0
    bad = [
        (hy_shape(heads=0), INVALID),
        (hy_shape(n=0), INVALID),
        (hy_shape(d=256, ranges=((0, 16, 72), (16, 56, 184))), UNSUPPORTED),
        (hy_shape(dtype=7), UNSUPPORTED),
        (hy_shape(ranges=((0, 16, 72), (16, 56, 50))), INVALID),     # not covering d
        (hy_shape(ranges=((0, 10, 72), (16, 56, 56))), INVALID),     # overlap
        (hy_shape(ranges=((0, 16, 72), (16, 0, 56))), INVALID),      # empty range
        (hy_shape(ranges=((0, 16, 100), (16, 56, 56))), INVALID),    # out of d
    ]
    for shape, want in bad:
        assert ws_size(shape)[0] == want
    assert ws_size(hy_shape(), c_q=0)[0] == INVALID
    assert ws_size(hy_shape(), c_q=2048)[0] == UNSUPPORTED
    assert ws_size(hy_shape(), c_m=(128, 0, 128))[0] == INVALID
    assert ws_size(hy_shape(), c_m=(128, 2000, 128))[0] == UNSUPPORTED
    assert ws_size(hy_shape(n=100), c_q=101)[0] == INVALID          # C > n


def call_queries(shape, c_q=256, iters=10, ws=FAKE, ws_bytes=1 << 40, q=FAKE):
    return B.lib().scope_cluster_queries(
        ctypes.byref(shape), q, c_q, iters, None, FAKE, FAKE, FAKE, FAKE, FAKE,
        ws, ws_bytes, None, None)


def test_cluster_queries_validation():
    sh = hy_shape()
    assert call_queries(sh, iters=0) == INVALID
    assert call_queries(sh, c_q=0) == INVALID
    assert call_queries(sh, q=None) == INVALID
    assert call_queries(sh, ws=None) == WORKSPACE
    assert call_queries(sh, ws_bytes=16) == WORKSPACE
    assert call_queries(sh, ws=ctypes.c_void_p((1 << 20) + 8)) == WORKSPACE
    assert call_queries(sh, q=ctypes.c_void_p((1 << 20) + 1)) == INVALID


def test_cluster_keys_validation():
    L = B.lib()
    sh = hy_shape()
    cm = (ctypes.c_int32 * 3)(128, 128, 128)

    def call(c_m=cm, iters=10, init=None, stride=0, ws_bytes=1 << 40):
        return L.scope_cluster_key_subspaces(ctypes.byref(sh), FAKE, c_m, iters,
                                             init, stride, FAKE, FAKE, FAKE,
                                             ws_bytes, None, None)
    assert call(iters=0) == INVALID
    assert call(c_m=(ctypes.c_int32 * 3)(128, 0, 128)) == INVALID
    assert call(init=FAKE, stride=64) == INVALID          # stride < max c_m
    assert call(ws_bytes=100) == WORKSPACE


def test_select_validation():
    L = B.lib()
    sh = hy_shape()
    cm = (ctypes.c_int32 * 3)(128, 128, 128)

    def call(rho=0.9, k_fix=11880, scores=None, tables=FAKE, codes=FAKE):
        return L.scope_select(ctypes.byref(sh), 256, cm, scores, tables, codes,
                              FAKE, ctypes.c_float(rho), k_fix, FAKE, None, FAKE,
                              FAKE, FAKE, FAKE, 1 << 40, None)
    for rho in (0.0, -0.5, 1.5, float("nan"), float("inf")):
        assert call(rho=rho) == INVALID
    assert call(k_fix=0) == INVALID
    assert call(k_fix=118801) == INVALID
    assert call(tables=None) == INVALID            # neither scores nor tables
    assert call(codes=None) == INVALID
    # the policy variant rejects unknown policies before anything else
    sh = hy_shape()
    cm = (ctypes.c_int32 * 3)(128, 128, 128)
    for bad in (-1, 3, 99):
        assert L.scope_select_policy(ctypes.byref(sh), 256, cm, FAKE, FAKE, FAKE, FAKE,
                                     ctypes.c_float(0.9), 100, FAKE, None, FAKE, FAKE,
                                     FAKE, FAKE, 1 << 40, bad, None) == INVALID


def test_attention_validation():
    L = B.lib()

    def call(shape, scale=0.0, q=FAKE, c_q=256):
        return L.scope_sparse_attention(ctypes.byref(shape), q, FAKE, FAKE, c_q,
                                        FAKE, FAKE, FAKE, FAKE,
                                        ctypes.c_float(scale), FAKE, FAKE, 1 << 40,
                                        None)
    assert call(hy_shape(d=96, ranges=((0, 32, 64), (32, 32, 32)))) == UNSUPPORTED
    assert call(hy_shape(), scale=float("nan")) == INVALID
    assert call(hy_shape(), q=None) == INVALID
    assert call(hy_shape(), q=ctypes.c_void_p((1 << 20) + 8)) == INVALID   # 16B rows
    assert call(hy_shape(), c_q=0) == INVALID
    # bf16 gathers use 32-bit byte offsets within one head: n * d * 2 < 2^32
    assert call(hy_shape(n=1 << 24)) == UNSUPPORTED


def test_noalloc_attention_validation():
    """The no-allocation call validates like the workspace call and rejects
    problems whose work list exceeds its fixed array, before any GPU work."""
    L = B.lib()

    def call(shape, scale=0.0, q=FAKE, c_q=256):
        return L.scope_sparse_attention_noalloc(ctypes.byref(shape), q, FAKE, FAKE, c_q,
                                                FAKE, FAKE, FAKE, FAKE,
                                                ctypes.c_float(scale), FAKE, None)
    assert call(hy_shape(d=96, ranges=((0, 32, 64), (32, 32, 32)))) == UNSUPPORTED
    assert call(hy_shape(), scale=float("nan")) == INVALID
    assert call(hy_shape(), q=None) == INVALID
    assert call(hy_shape(), c_q=0) == INVALID
    # heads * (ceil(n / 256) + c_q) work slots of two entries against the
    # fixed list
    items = lambda sh, c_q: 2 * sh.heads * (-(-sh.n // 256) + c_q)
    big = hy_shape(heads=96)
    assert items(big, 256) > 65536
    assert call(big) == 5
    assert "no-allocation" in B.status_string(5)
    assert items(hy_shape(), 256) <= 65536


def test_proxy_scores_and_fixexp_validation():
    L = B.lib()
    sh = hy_shape()
    cm = (ctypes.c_int32 * 3)(128, 128, 128)
    assert L.scope_proxy_scores(ctypes.byref(sh), None, 256, FAKE, cm, FAKE, FAKE,
                                None, None) == INVALID
    assert L.scope_proxy_scores(ctypes.byref(sh), FAKE, 256, FAKE, cm, None, FAKE,
                                FAKE, None) == INVALID   # scores need codes
    assert L.scope_debug_fixexp(None, FAKE, 5, None) == INVALID
    assert L.scope_debug_fixexp(FAKE, FAKE, -1, None) == INVALID
    assert L.scope_debug_fixexp(None, None, 0, None) == OK   # empty: no launch


def test_work_list_diagnostic_validation():
    L = B.lib()
    S = ctypes.c_int32(-1)
    slots = -(-118800 // 256) + 256
    need = 24 * slots * 8
    call = lambda heads=24, n=118800, c_q=256, off=FAKE, sel=FAKE, items=FAKE, cap=need, s=S: \
        L.scope_debug_attention_items(heads, n, c_q, 1, off, sel, items, cap,
                                      None if s is None else ctypes.byref(s), None)
    assert call(heads=0) == INVALID
    assert call(n=0) == INVALID
    assert call(c_q=0) == INVALID
    assert call(c_q=118801) == INVALID          # more clusters than rows
    assert call(off=None) == INVALID
    assert call(sel=None) == INVALID
    assert call(items=None) == INVALID
    assert call(items=ctypes.c_void_p((1 << 20) + 4)) == INVALID   # not 16-byte aligned
    assert call(cap=need - 1) == INVALID
    assert call(s=None) == INVALID
    assert S.value == -1                        # nothing written before a rejection


def test_binding_rejects_host_tensors():
    torch = pytest.importorskip("torch")
    sh = hy_shape(heads=1, n=64, d=64, ranges=((0, 16, 40), (16, 24, 24)))
    q = torch.zeros(64, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        B.scope_cluster_queries(sh, q, 8, 2, None, q, q, q, q, q, q)


def part(sets=None, c=None):
    sets = sets if sets is not None else [range(0, 16), range(16, 72), range(72, 128)]
    c = c if c is not None else [333] * len(sets)
    return B.make_partition(sets, c)


def part_ws(shape, p, c_q=300):
    out = ctypes.c_size_t(0)
    st = B.lib().scope_partition_workspace_size(ctypes.byref(shape), c_q, ctypes.byref(p),
                                                ctypes.byref(out))
    return st, out.value


def test_partition_workspace_and_validation():
    sh = hy_shape()
    st, in_order = part_ws(sh, part())
    assert st == OK and in_order % 256 == 0
    # reordered channels: a copy of K (heads * n * d bf16) on top
    rnd = [sorted(range(0, 128, 3)), sorted(set(range(128)) - set(range(0, 128, 3)))]
    st, reordered = part_ws(sh, part(rnd, [333, 333]))
    assert st == OK and reordered >= 24 * 118800 * 128 * 2
    # the shape's ranges are not used by the partition calls
    assert part_ws(hy_shape(ranges=((0, 0, 0), (0, 0, 0))), part())[0] == OK
    bad = [
        (part([range(0, 64), range(63, 127)]), INVALID),              # overlap
        (part([range(0, 64), range(64, 127)]), INVALID),              # channel 127 missing
        (part([[1, 0] + list(range(2, 64)), range(64, 128)]), INVALID),  # not ascending
        (part([range(0, 64), range(64, 128)], [333, 0]), INVALID),
        (part([range(0, 64), range(64, 128)], [333, 1025]), UNSUPPORTED),
        (part([range(16 * m, 16 * m + 16) for m in range(8)], [400] * 8), UNSUPPORTED),  # LUT
    ]
    for p, want in bad:
        assert part_ws(sh, p)[0] == want
    p = part([range(16 * m, 16 * m + 16) for m in range(8)], [384] * 8)
    assert part_ws(sh, p)[0] == OK
    p.m = 9
    assert part_ws(sh, p)[0] == UNSUPPORTED
    p.m = 0
    assert part_ws(sh, p)[0] == INVALID
    assert B.lib().scope_partition_workspace_size(ctypes.byref(sh), 300, None,
                                                  ctypes.byref(ctypes.c_size_t())) == INVALID


def test_partition_calls_validation():
    L, sh, p = B.lib(), hy_shape(), part()
    def keys(iters=10, init=None, stride=0, ws=FAKE, ws_bytes=1 << 40, pp=p):
        return L.scope_cluster_key_partition(ctypes.byref(sh), FAKE, ctypes.byref(pp) if pp else None,
                                             iters, init, stride, FAKE, FAKE, ws, ws_bytes,
                                             None, None)
    assert keys(iters=0) == INVALID
    assert keys(pp=None) == INVALID
    assert keys(init=FAKE, stride=100) == INVALID              # stride < max c
    assert keys(ws=None) == WORKSPACE
    assert keys(ws_bytes=1000) == WORKSPACE
    def scores(ws=None, ws_bytes=0, pp=p, codes=FAKE, sc=FAKE):
        return L.scope_proxy_scores_partition(ctypes.byref(sh), FAKE, 300, FAKE,
                                              ctypes.byref(pp), codes, FAKE, sc, ws,
                                              ws_bytes, None)
    assert scores(codes=None) == INVALID                        # scores need codes
    rnd = part([sorted(range(0, 128, 2)), sorted(range(1, 128, 2))], [64, 64])
    assert scores(pp=rnd) == WORKSPACE                          # reordering needs it
    def select(policy=0, rho=0.9, tables=FAKE, codes=FAKE, ws=FAKE):
        return L.scope_select_partition(ctypes.byref(sh), 300, ctypes.byref(p), None, tables,
                                        codes, FAKE, rho, 11880, FAKE, None, FAKE, FAKE,
                                        FAKE, ws, 1 << 40, policy, None)
    assert select(policy=3) == INVALID
    assert select(rho=0.0) == INVALID
    assert select(codes=None) == INVALID
    assert select(ws=None) == WORKSPACE
