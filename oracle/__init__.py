"""CPU oracle for the SCOPE attention layer -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU library never does, and this package never
imports the GPU library: the two share no code.

The arithmetic lives in ``scope_oracle.c`` (plain C, compiled by ``build``);
this module only marshals numpy arrays into it.  See that file's header for
the canonical evaluation each stage follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "scope_oracle.c")
# SCOPE_ORACLE_LIBRARY selects another build (e.g. the sanitizer build)
LIB = os.environ.get("SCOPE_ORACLE_LIBRARY") or os.path.join(HERE, "libscope_oracle.so")
SAN_LIB = os.path.join(HERE, "libscope_oracle_san.so")

CFLAGS = ["-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
          "-fopenmp", "-mfma", "-fPIC", "-shared"]
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-fno-omit-frame-pointer", "-g"]


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile the oracle with gcc into oracle/libscope_oracle.so, or with
    sanitize into libscope_oracle_san.so under ASan and UBSan."""
    out = SAN_LIB if sanitize else LIB
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        flags = CFLAGS + (SAN_FLAGS if sanitize else [])
        subprocess.check_call(["gcc", *flags, "-o", tmp, SRC, "-lm"])
        os.replace(tmp, out)
    return out


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        L.oracle_num_threads.restype = I
        L.oracle_kmeans.argtypes = [P, ctypes.c_long, I, I, I, I, P, I, P, P, P]
        L.oracle_group.argtypes = [P, I, I, P, P, P]
        L.oracle_assign_rows.argtypes = [P, ctypes.c_long, I, I, P, I, P]
        L.oracle_mean_rows.argtypes = [P, ctypes.c_long, I, I, P, I, P, P]
        L.oracle_cluster_queries.argtypes = [I, I, I, P, I, I, P, P, P, P, P, P]
        L.oracle_cluster_key_subspaces.argtypes = [I, I, I, P, P, P, P, I, P, I,
                                                   P, P, P]
        L.oracle_tables.argtypes = [I, I, P, P, I, P, P, P, P]
        L.oracle_cluster_key_partition.argtypes = [I, I, I, I, P, P, P, P, I, P, I,
                                                   P, P, P]
        L.oracle_tables_partition.argtypes = [I, I, I, P, P, I, P, P, P, P]
        L.oracle_proxy_scores_partition.argtypes = [I, I, I, I, I, P, P, P, P]
        L.oracle_proxy_scores.argtypes = [I, I, I, I, P, P, P, P]
        L.oracle_sigma.argtypes = [I]
        L.oracle_sigma.restype = ctypes.c_float
        L.oracle_fixexp.argtypes = [ctypes.c_float]
        L.oracle_fixexp.restype = ctypes.c_uint64
        L.oracle_fixexp_batch.argtypes = [P, P, ctypes.c_long]
        L.oracle_mass_target.argtypes = [ctypes.c_float, ctypes.c_uint64]
        L.oracle_mass_target.restype = ctypes.c_uint64
        L.oracle_select.argtypes = [I, I, I, P, P, ctypes.c_float, I, I, P, P, P,
                                    P, P]
        L.oracle_attention.argtypes = [I, I, I, P, P, P, I, P, P, P, P,
                                       ctypes.c_double, P, P]
        L.oracle_cluster_queries_from.argtypes = [I, I, I, P, I, I, P, P, P, P, P]
        L.oracle_cluster_key_subspaces_from.argtypes = [I, I, I, P, P, P, P, I, P, P, P]
        L.oracle_kmeans_from.argtypes = [P, ctypes.c_long, I, I, I, I, I, P, P, P]
        for name in ("oracle_cluster_queries_from", "oracle_cluster_key_subspaces_from",
                     "oracle_kmeans_from"):
            getattr(L, name).restype = I
        D = ctypes.c_double
        L.oracle_block_proxy.argtypes = [I, I, I, P, P, I, D, P]
        L.oracle_matched_retention.argtypes = [I, I, P, P, I, I, P, P]
        L.oracle_recall_at_density.argtypes = [I, I, P, P, I, P]
        for name in ("oracle_block_proxy", "oracle_matched_retention",
                     "oracle_recall_at_density"):
            getattr(L, name).restype = I
        for name in ("oracle_kmeans", "oracle_group", "oracle_assign_rows",
                     "oracle_mean_rows", "oracle_cluster_queries",
                     "oracle_cluster_key_subspaces", "oracle_tables",
                     "oracle_proxy_scores", "oracle_select", "oracle_attention",
                     "oracle_cluster_key_partition", "oracle_tables_partition",
                     "oracle_proxy_scores_partition"):
            getattr(L, name).restype = I
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def _check(status, what):
    if status == 1:
        raise ValueError(f"oracle {what}: invalid argument")
    if status == 3:
        raise MemoryError(f"oracle {what}: out of memory")
    return status  # 2 = fixed-point range exceeded (reported, not raised)


def num_threads() -> int:
    return lib().oracle_num_threads()


def kmeans(X, C, iters, init, final_assign):
    """Canonical Lloyd k-means of the rows of X (n x dx)."""
    X = _c(X, np.float32)
    n, dx = X.shape
    init = _c(init, np.int32)
    U = np.empty((C, dx), np.float32)
    a = np.empty(n, np.int32)
    cnt = np.empty(C, np.int32)
    st = lib().oracle_kmeans(_p(X), dx, n, dx, C, iters, _p(init),
                             int(final_assign), _p(U), _p(a), _p(cnt))
    _check(st, "kmeans")
    return U, a, cnt, st


def assign_rows(X, U):
    """One canonical assignment step: nearest centroid of every row of X."""
    X = _c(X, np.float32)
    U = _c(U, np.float32)
    a = np.empty(X.shape[0], np.int32)
    _check(lib().oracle_assign_rows(_p(X), X.shape[1], X.shape[0], X.shape[1],
                                    _p(U), U.shape[0], _p(a)), "assign_rows")
    return a


def mean_rows(X, assign, U_prev):
    """One canonical update step: fixed-point means of the members."""
    X = _c(X, np.float32)
    U = np.array(U_prev, dtype=np.float32, copy=True)
    a = _c(assign, np.int32)
    cnt = np.empty(U.shape[0], np.int32)
    st = lib().oracle_mean_rows(_p(X), X.shape[1], X.shape[0], X.shape[1], _p(a),
                                U.shape[0], _p(U), _p(cnt))
    _check(st, "mean_rows")
    return U, cnt


def group(assign, C):
    assign = _c(assign, np.int32)
    n = assign.shape[0]
    counts = np.empty(C, np.int32)
    offsets = np.empty(C + 1, np.int32)
    perm = np.empty(n, np.int32)
    _check(lib().oracle_group(_p(assign), n, C, _p(counts), _p(offsets),
                              _p(perm)), "group")
    return counts, offsets, perm


def cluster_queries(q, c_q, iters, init):
    """Alg. 1: per-head query k-means plus grouping.  q: [heads][n][d]."""
    q = _c(q, np.float32)
    heads, n, d = q.shape
    init = _c(init, np.int32).reshape(heads, c_q)
    cen = np.empty((heads, c_q, d), np.float32)
    g = np.empty((heads, n), np.int32)
    cnt = np.empty((heads, c_q), np.int32)
    off = np.empty((heads, c_q + 1), np.int32)
    perm = np.empty((heads, n), np.int32)
    st = lib().oracle_cluster_queries(heads, n, d, _p(q), c_q, iters, _p(init),
                                      _p(cen), _p(g), _p(cnt), _p(off),
                                      _p(perm))
    _check(st, "cluster_queries")
    return dict(centroids=cen, assign=g, counts=cnt, offsets=off, perm=perm,
                status=st)


def cluster_queries_from(q, c_q, iters, centroids):
    """Query clustering warm-started from the given centroids [heads][c_q][d]."""
    q = _c(q, np.float32)
    heads, n, d = q.shape
    cen = np.array(centroids, dtype=np.float32, copy=True).reshape(heads, c_q, d)
    g = np.empty((heads, n), np.int32)
    cnt = np.empty((heads, c_q), np.int32)
    off = np.empty((heads, c_q + 1), np.int32)
    perm = np.empty((heads, n), np.int32)
    st = lib().oracle_cluster_queries_from(heads, n, d, _p(q), c_q, iters, _p(cen), _p(g),
                                           _p(cnt), _p(off), _p(perm))
    _check(st, "cluster_queries_from")
    return dict(centroids=cen, assign=g, counts=cnt, offsets=off, perm=perm, status=st)


def cluster_key_subspaces_from(k, ranges, c_m, iters, centroids):
    """Key subspace clustering warm-started from the given codebooks
    [heads][sum_m c_m len_m] (U^T, U^H, U^W back to back)."""
    k = _c(k, np.float32)
    heads, n, d = k.shape
    off = _c(ranges[0], np.int32)
    ln = _c(ranges[1], np.int32)
    cm = _c(c_m, np.int32)
    cen = np.array(centroids, dtype=np.float32, copy=True).reshape(heads, -1)
    codes = np.empty((heads, n), np.uint32)
    a3 = np.empty((heads, 3, n), np.int32)
    st = lib().oracle_cluster_key_subspaces_from(heads, n, d, _p(off), _p(ln), _p(k), _p(cm),
                                                 iters, _p(cen), _p(codes), _p(a3))
    _check(st, "cluster_key_subspaces_from")
    return dict(centroids=cen, codes=codes, assign3=a3, status=st)


def cluster_key_subspaces(k, ranges, c_m, iters, init):
    """Alg. 2: k-means of the T/H/W key subspaces, packed composite codes."""
    k = _c(k, np.float32)
    heads, n, d = k.shape
    off = _c(ranges[0], np.int32)
    ln = _c(ranges[1], np.int32)
    cm = _c(c_m, np.int32)
    init = _c(init, np.int32)
    stride = init.shape[-1]
    if init.shape != (heads, 3, stride) or stride < int(cm.max()):
        raise ValueError("init must be [heads][3][stride >= max c_m]")
    per_head = int(sum(int(cm[m]) * int(ln[m]) for m in range(3)))
    cen = np.empty((heads, per_head), np.float32)
    codes = np.empty((heads, n), np.uint32)
    a3 = np.empty((heads, 3, n), np.int32)
    st = lib().oracle_cluster_key_subspaces(heads, n, d, _p(off), _p(ln), _p(k),
                                            _p(cm), iters, _p(init), stride,
                                            _p(cen), _p(codes), _p(a3))
    _check(st, "cluster_key_subspaces")
    return dict(centroids=cen, codes=codes, assign3=a3, status=st)


def tables(q_centroids, k_centroids, ranges, c_m):
    """Eq. 5 score tables, [heads][c_q][C_T + C_H + C_W]."""
    qc = _c(q_centroids, np.float32)
    kc = _c(k_centroids, np.float32)
    heads, c_q, d = qc.shape
    cm = _c(c_m, np.int32)
    P = np.empty((heads, c_q, int(cm.sum())), np.float32)
    lib().oracle_tables(heads, d, _p(_c(ranges[0], np.int32)),
                        _p(_c(ranges[1], np.int32)), c_q, _p(cm), _p(qc),
                        _p(kc), _p(P))
    return P


def proxy_scores(tables_, codes, d, c_m):
    """Eq. 6 proxy logits, [heads][c_q][n]."""
    P = _c(tables_, np.float32)
    codes = _c(codes, np.uint32)
    heads, c_q, _ = P.shape
    n = codes.shape[1]
    S = np.empty((heads, c_q, n), np.float32)
    lib().oracle_proxy_scores(heads, n, d, c_q, _p(_c(c_m, np.int32)), _p(P),
                              _p(codes), _p(S))
    return S


def _partition(sets):
    """Channel sets I_1..I_M -> (M, concatenated channels, lengths)."""
    sets = [np.asarray(x, np.int32).ravel() for x in sets]
    return (len(sets), _c(np.concatenate(sets), np.int32),
            _c([x.size for x in sets], np.int32))


def cluster_key_partition(k, sets, c_m, iters, init):
    """App. B / Table 3: k-means of K[:, I_m] for any disjoint channel sets
    I_1..I_M (each ascending, together all d channels).  Codes per subspace,
    [heads][M][n] uint16; centroids per head U^1..U^M back to back.
    init: [heads][M][stride]."""
    k = _c(k, np.float32)
    heads, n, d = k.shape
    M, chan, ln = _partition(sets)
    cm = _c(c_m, np.int32)
    init = _c(init, np.int32)
    stride = init.shape[-1]
    if init.shape != (heads, M, stride) or stride < int(cm.max()):
        raise ValueError("init must be [heads][M][stride >= max c_m]")
    per_head = int(sum(int(cm[m]) * int(ln[m]) for m in range(M)))
    cen = np.empty((heads, per_head), np.float32)
    codes = np.empty((heads, M, n), np.uint16)
    a = np.empty((heads, M, n), np.int32)
    st = lib().oracle_cluster_key_partition(heads, n, d, M, _p(chan), _p(ln), _p(k),
                                            _p(cm), iters, _p(init), stride,
                                            _p(cen), _p(codes), _p(a))
    _check(st, "cluster_key_partition")
    return dict(centroids=cen, codes=codes, assign=a, status=st)


def tables_partition(q_centroids, k_centroids, sets, c_m):
    """Eq. 5 over M subspaces: [heads][c_q][C_1 + ... + C_M]."""
    qc = _c(q_centroids, np.float32)
    kc = _c(k_centroids, np.float32)
    heads, c_q, d = qc.shape
    M, chan, ln = _partition(sets)
    cm = _c(c_m, np.int32)
    P = np.empty((heads, c_q, int(cm.sum())), np.float32)
    _check(lib().oracle_tables_partition(heads, d, M, _p(chan), _p(ln), c_q, _p(cm),
                                         _p(qc), _p(kc), _p(P)), "tables_partition")
    return P


def proxy_scores_partition(tables_, codes, d, c_m):
    """Eq. 6 over M subspaces, codes [heads][M][n]: [heads][c_q][n]."""
    P = _c(tables_, np.float32)
    codes = _c(codes, np.uint16)
    heads, M, n = codes.shape
    c_q = P.shape[1]
    S = np.empty((heads, c_q, n), np.float32)
    _check(lib().oracle_proxy_scores_partition(heads, n, d, M, c_q,
                                               _p(_c(c_m, np.int32)), _p(P),
                                               _p(codes), _p(S)), "proxy_scores_partition")
    return S


def sigma(d: int) -> float:
    return float(lib().oracle_sigma(d))


def fixexp(y):
    y = _c(np.atleast_1d(y), np.float32)
    out = np.empty(y.shape, np.uint64)
    lib().oracle_fixexp_batch(_p(y), _p(out), y.size)
    return out


def mass_target(rho: float, tot: int) -> int:
    return int(lib().oracle_mass_target(float(np.float32(rho)), int(tot)))


POLICIES = {"online": 0, "fixed": 1, "topp": 2}


def select(scores, counts, rho, k_fix, policy="online"):
    """Alg. 3: base counts, k_head, r_c and key sets (ascending indices).
    policy: "online" (Eq. 10), or the Fig. 6 ablations "fixed" (r_c = b_c,
    no top-up) and "topp" (r_c = t_c)."""
    S = _c(scores, np.float32)
    heads, c_q, n = S.shape
    counts = _c(counts, np.int32).reshape(heads, c_q)
    base = np.empty((heads, c_q), np.int32)
    kh = np.empty(heads, np.int32)
    sc = np.empty((heads, c_q), np.int32)
    idx = np.full((heads, c_q, n), -1, np.int32)
    topp = np.empty((heads, c_q), np.int32)
    _check(lib().oracle_select(heads, n, c_q, _p(S), _p(counts),
                               float(np.float32(rho)), int(k_fix), POLICIES[policy],
                               _p(base), _p(kh), _p(sc), _p(idx), _p(topp)), "select")
    return dict(base_counts=base, k_head=kh, sel_counts=sc, sel_idx=idx,
                topp=topp)


def attention(q, k, v, offsets, perm, sel_counts, sel_idx, scale=None,
              row_mask=None):
    """Eq. 11 in fp64 (Eq. 1 when every key set is all keys)."""
    q = _c(q, np.float32)
    k = _c(k, np.float32)
    v = _c(v, np.float32)
    heads, n, d = q.shape
    offsets = _c(offsets, np.int32)
    c_q = offsets.shape[-1] - 1
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((heads, n, d), np.float32)
    mask = None if row_mask is None else _c(row_mask, np.uint8)
    lib().oracle_attention(heads, n, d, _p(q), _p(k), _p(v), c_q, _p(offsets),
                           _p(_c(perm, np.int32)), _p(_c(sel_counts, np.int32)),
                           _p(_c(sel_idx, np.int32)), float(scale), _p(mask),
                           _p(out))
    return out


def dense_attention(q, k, v, scale=None, row_mask=None):
    """Eq. 1 through the same routine: one cluster holding every query and
    every key."""
    heads, n, d = np.shape(q)
    offsets = np.tile(np.array([0, n], np.int32), (heads, 1))
    perm = np.tile(np.arange(n, dtype=np.int32), (heads, 1))
    sc = np.full((heads, 1), n, np.int32)
    idx = np.tile(np.arange(n, dtype=np.int32), (heads, 1, 1))
    return attention(q, k, v, offsets, perm, sc, idx, scale, row_mask)


def layer_partition(q, k, v, sets, c_q, c_m, iters, init_q, init_k, rho, k_fix,
                    policy="online"):
    """The layer with the keys split into the channel sets I_1..I_M."""
    d = np.shape(q)[2]
    qr = cluster_queries(q, c_q, iters, init_q)
    kr = cluster_key_partition(k, sets, c_m, iters, init_k)
    P = tables_partition(qr["centroids"], kr["centroids"], sets, c_m)
    S = proxy_scores_partition(P, kr["codes"], d, c_m)
    sel = select(S, qr["counts"], rho, k_fix, policy)
    O = attention(q, k, v, qr["offsets"], qr["perm"], sel["sel_counts"],
                  sel["sel_idx"])
    return dict(q=qr, k=kr, tables=P, scores=S, sel=sel, out=O)


def layer(q, k, v, ranges, c_q, c_m, iters, init_q, init_k, rho, k_fix,
          policy="online"):
    """The whole layer of Alg. 1 for every head; returns every intermediate."""
    d = np.shape(q)[2]
    qr = cluster_queries(q, c_q, iters, init_q)
    kr = cluster_key_subspaces(k, ranges, c_m, iters, init_k)
    P = tables(qr["centroids"], kr["centroids"], ranges, c_m)
    S = proxy_scores(P, kr["codes"], d, c_m)
    sel = select(S, qr["counts"], rho, k_fix, policy)
    O = attention(q, k, v, qr["offsets"], qr["perm"], sel["sel_counts"],
                  sel["sel_idx"])
    return dict(q=qr, k=kr, tables=P, scores=S, sel=sel, out=O)


# --- proxy comparison measurements (App. C, Fig. 9; Fig. 2) ---------------

def block_proxy(qrep, k, block, scale):
    """Block-wise proxy scores [rows][n]: each key scored by the mean of its
    block of `block` consecutive tokens against the row's query
    representative (qrep [rows][d]), times scale; fp64 arithmetic."""
    qrep = _c(qrep, np.float32)
    k = _c(k, np.float32)
    rows, d = qrep.shape
    n = k.shape[0]
    out = np.empty((rows, n), np.float32)
    _check(lib().oracle_block_proxy(rows, n, d, _p(qrep), _p(k), int(block), float(scale),
                                    _p(out)), "block_proxy")
    return out


def _ceil_frac(x, m):
    """ceil(x * m) for a decimal fraction x, in exact rationals."""
    from fractions import Fraction
    v = Fraction(str(x)) * m
    return -(-v.numerator // v.denominator)


def matched_retention(exact, proxy, top_frac=0.1, target=0.958):
    """Per row: retained fraction and oracle recall when keys are taken in
    proxy order until `target` of the exact top `top_frac` is held (whole
    tie groups of the proxy kept); kt = ceil(top_frac n), need =
    ceil(target kt)."""
    exact = _c(exact, np.float32)
    proxy = _c(proxy, np.float32)
    rows, n = exact.shape
    kt = max(1, _ceil_frac(top_frac, n))
    need = max(1, _ceil_frac(target, kt))
    ret = np.empty(rows, np.float64)
    rec = np.empty(rows, np.float64)
    _check(lib().oracle_matched_retention(rows, n, _p(exact), _p(proxy), kt, need, _p(ret),
                                          _p(rec)), "matched_retention")
    return ret, rec


def recall_at_density(p_exact, proxy, density):
    """Per row: exact attention mass held by the first max(1, round(density
    n)) keys in proxy order."""
    p = _c(p_exact, np.float64)
    proxy = _c(proxy, np.float32)
    rows, n = proxy.shape
    count = max(1, int(round(density * n)))
    out = np.empty(rows, np.float64)
    _check(lib().oracle_recall_at_density(rows, n, _p(p), _p(proxy), count, _p(out)),
           "recall_at_density")
    return out

