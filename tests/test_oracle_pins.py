"""Pins of the CPU oracle against facts the method and mathematics fix.

Nothing here re-types the oracle's formulas: every expectation comes from a
hand-worked fixture (tests/golden), a closed form, a textbook routine evaluated
another way (float64 numpy, exact rationals), an invariant, or brute force.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2608_12780_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
LN2 = math.log(2.0)


def _expr(e):
    e = e.strip()
    if e.endswith("ln2"):
        k = e[:-3]
        k = {"": 1.0, "-": -1.0}.get(k, None) if k in ("", "-") else float(k)
        return k * LN2
    return float(e)


# --------------------------------------------------------------------------
# k-means (Sec. 3.2 Eq. 2, Sec. 3.3 Eq. 3)

def _dyadic(rng, shape, scale_bits=10, lim=16):
    return (rng.integers(-lim << scale_bits, lim << scale_bits, size=shape)
            / float(1 << scale_bits)).astype(np.float32)


def test_kmeans_one_cluster_is_the_exact_mean(oracle_lib):
    rng = np.random.default_rng(11)
    X = _dyadic(rng, (37, 5))
    U, a, cnt, st = oracle.kmeans(X, 1, 3, [5], final_assign=False)
    assert st == 0 and (a == 0).all() and cnt[0] == 37
    for ch in range(5):
        exact = sum(Fraction(float(x)) for x in X[:, ch]) / 37
        # the mean of Eq. 2, rounded once to double and once to fp32
        assert U[0, ch] == np.float32(float(exact))
        assert abs(Fraction(float(U[0, ch])) - exact) <= abs(exact) * Fraction(1, 1 << 23)


def test_kmeans_separated_blobs_have_known_labels(oracle_lib):
    rng = np.random.default_rng(12)
    centers = np.array([[0, 0, 0], [40, 0, 0], [0, 40, 0], [0, 0, 40]], np.float32)
    lab = rng.integers(0, 4, size=200)
    X = (centers[lab] + rng.standard_normal((200, 3))).astype(np.float32)
    init = [int(np.flatnonzero(lab == b)[0]) for b in (2, 0, 3, 1)]
    U, a, cnt, _ = oracle.kmeans(X, 4, 4, init, final_assign=True)
    blob_of = np.array([2, 0, 3, 1])
    assert (blob_of[a] == lab).all()
    for r in range(4):
        np.testing.assert_allclose(U[r], X[lab == blob_of[r]].mean(0), atol=1e-5)


def test_kmeans_identity_start_with_c_equal_n(oracle_lib):
    rng = np.random.default_rng(13)
    X = inputs.bf16_widen(inputs.bf16_bits(rng.standard_normal((40, 6)).astype(np.float32)))
    U, a, cnt, _ = oracle.kmeans(X, 40, 2, np.arange(40), final_assign=True)
    assert (a == np.arange(40)).all() and (cnt == 1).all()
    assert np.array_equal(U, X)   # bf16 values are exact in 2^-24 fixed point


def _f64_sqdist(X, U):
    X = X.astype(np.float64)
    U = U.astype(np.float64)
    return (X * X).sum(1)[:, None] - 2 * X @ U.T + (U * U).sum(1)[None, :]


def test_kmeans_labels_are_argmins_of_returned_centroids(oracle_lib):
    # Eq. 3 holds for the returned codebook (keys end on an assignment)
    rng = np.random.default_rng(14)
    X = rng.standard_normal((500, 12)).astype(np.float32)
    init = rng.choice(500, 16, replace=False)
    U, a, cnt, _ = oracle.kmeans(X, 16, 5, init, final_assign=True)
    D = _f64_sqdist(X, U)
    best = D.argmin(1)
    srt = np.sort(D, 1)
    gap = srt[:, 1] - srt[:, 0]
    scale = np.linalg.norm(X, axis=1) * np.linalg.norm(U, axis=1).max()
    clear = gap > 1e-4 * scale
    assert clear.mean() > 0.95
    assert (best[clear] == a[clear]).all()
    assert (np.bincount(a, minlength=16) == cnt).all()


def test_kmeans_centroids_are_member_means(oracle_lib):
    # Eq. 2 holds for the returned clusters (queries end on an update)
    rng = np.random.default_rng(15)
    X = _dyadic(rng, (300, 7), scale_bits=12, lim=4)
    init = rng.choice(300, 9, replace=False)
    U, a, cnt, _ = oracle.kmeans(X, 9, 4, init, final_assign=False)
    for r in range(9):
        mem = X[a == r]
        assert len(mem) == cnt[r]
        if len(mem) == 0:
            continue
        for ch in range(7):
            exact = sum(Fraction(float(x)) for x in mem[:, ch]) / len(mem)
            assert U[r, ch] == np.float32(float(exact))


def test_kmeans_objective_does_not_increase(oracle_lib):
    rng = np.random.default_rng(16)
    X = rng.standard_normal((800, 16)).astype(np.float32)
    init = rng.choice(800, 10, replace=False)
    prev = np.inf
    for it in range(1, 7):
        U, a, _, _ = oracle.kmeans(X, 10, it, init, final_assign=False)
        obj = ((X.astype(np.float64) - U[a].astype(np.float64)) ** 2).sum()
        assert obj <= prev * (1 + 1e-6)
        prev = obj


def test_kmeans_matches_float64_lloyd_on_clear_data(oracle_lib):
    # textbook Lloyd in float64, same start; on clustered data no label is a
    # near-tie, so both evaluations must give the same labels.
    rng = np.random.default_rng(17)
    centers = rng.standard_normal((8, 10)) * 6
    lab = rng.integers(0, 8, size=400)
    X = (centers[lab] + rng.standard_normal((400, 10))).astype(np.float32)
    init = rng.choice(400, 8, replace=False)
    U64 = X[init].astype(np.float64)
    for _ in range(6):
        a64 = _f64_sqdist(X, U64).argmin(1)
        for r in range(8):
            if (a64 == r).any():
                U64[r] = X[a64 == r].astype(np.float64).mean(0)
    U, a, _, _ = oracle.kmeans(X, 8, 6, init, final_assign=False)
    assert (a == a64).all()
    np.testing.assert_allclose(U, U64, rtol=1e-6, atol=1e-6)


def test_kmeans_empty_cluster_keeps_centroid(oracle_lib):
    X = np.array([[0.0], [0.0], [10.0], [10.0], [100.0]], np.float32)
    # two starting rows are equal: the higher-index duplicate never wins a tie
    U, a, cnt, _ = oracle.kmeans(X, 3, 1, [0, 1, 4], final_assign=False)
    assert a.tolist() == [0, 0, 0, 0, 2] and cnt.tolist() == [4, 0, 1]
    assert U[:, 0].tolist() == [5.0, 0.0, 100.0]
    # the kept centroid then wins the two zeros back
    U, a, cnt, _ = oracle.kmeans(X, 3, 2, [0, 1, 4], final_assign=False)
    assert a.tolist() == [1, 1, 0, 0, 2] and U[:, 0].tolist() == [10.0, 0.0, 100.0]


def test_kmeans_fixed_point_range_depends_on_n(oracle_lib):
    """The int64 sums of rint(x 2^24) are exact while n terms cannot reach
    2^63.  The mean of n equal rows is that row exactly when the sums hold
    it; where n such terms would overflow, the range status (2) is
    reported.  At n = 2^17 the largest float below 2^22 is inside the range
    (2^17 (2^46 - 2^22) < 2^63); at n = 2^18 it is not, and the largest
    float below 2^21 is."""
    below22 = np.nextafter(np.float32(2.0 ** 22), np.float32(0))
    below21 = np.nextafter(np.float32(2.0 ** 21), np.float32(0))
    for n, x, want in ((1 << 17, below22, 0), (1 << 18, below22, 2), (1 << 18, below21, 0)):
        X = np.full((n, 1), x, np.float32)
        U, a, cnt, st = oracle.kmeans(X, 1, 1, np.array([0], np.int32), False)
        assert st == want, (n, x)
        if want == 0:
            assert U[0, 0] == x and cnt[0] == n
    # a non-finite value is outside every range
    X = np.ones((8, 2), np.float32)
    X[3, 1] = np.inf
    assert oracle.kmeans(X, 1, 1, np.array([0], np.int32), False)[3] == 2


def test_group_is_a_stable_sort(oracle_lib):
    rng = np.random.default_rng(18)
    g = rng.integers(0, 13, size=1000).astype(np.int32)
    counts, offsets, perm = oracle.group(g, 13)
    assert (perm == np.argsort(g, kind="stable")).all()
    assert (counts == np.bincount(g, minlength=13)).all()
    assert offsets[0] == 0 and (np.diff(offsets) == counts).all() and offsets[-1] == 1000


def test_cluster_queries_sizes_sum_to_n(oracle_lib):
    cfg = inputs.CONFIGS["tiny"]
    x = inputs.generate(cfg)
    r = oracle.cluster_queries(x.q, cfg.c_q, cfg.iters, x.init_q)
    assert (r["counts"].sum(1) == cfg.n).all()
    for h in range(cfg.heads):
        assert sorted(r["perm"][h]) == list(range(cfg.n))
        g = r["assign"][h]
        assert (g[r["perm"][h]] == np.repeat(np.arange(cfg.c_q), r["counts"][h])).all()


# --------------------------------------------------------------------------
# score tables and lookup-and-sum (Eq. 5-6; App. B exactness)

def test_lookup_golden_example(oracle_lib):
    gx = json.load(open(os.path.join(GOLDEN, "lookup_exactness_example.json")))
    ranges = (gx["offsets"], gx["lengths"])
    qc = np.array(gx["q_centroid"], np.float32)[None, None, :]
    kc = np.concatenate([np.ravel(gx["U_T"]), np.ravel(gx["U_H"]),
                         np.ravel(gx["U_W"])]).astype(np.float32)[None]
    P = oracle.tables(qc, kc, ranges, [2, 2, 2])
    assert P[0, 0].tolist() == gx["tables"]
    codes = np.array([[c[0] | (c[1] << 10) | (c[2] << 20) for c in gx["codes"]]],
                     np.uint32)
    S = oracle.proxy_scores(P, codes, gx["d"], [2, 2, 2])
    assert S[0, 0].tolist() == gx["logits"]


def test_lookup_sum_equals_full_centroid_dot(oracle_lib):
    # App. B: sum_m P_m[c, z_j^m] = <qbar_c, khat_j>; exact on dyadic data
    rng = np.random.default_rng(21)
    d, cq, n = 16, 5, 64
    ranges = ((0, 4, 10), (4, 6, 6))
    cm = [3, 4, 5]
    qc = (rng.integers(-8, 8, size=(1, cq, d)) / 4).astype(np.float32)
    U = [(rng.integers(-8, 8, size=(cm[m], ranges[1][m])) / 4).astype(np.float32)
         for m in range(3)]
    kc = np.concatenate([u.ravel() for u in U])[None]
    z = np.stack([rng.integers(0, cm[m], size=n) for m in range(3)], 1)
    codes = (z[:, 0] | (z[:, 1] << 10) | (z[:, 2] << 20)).astype(np.uint32)[None]
    P = oracle.tables(qc, kc, ranges, cm)
    S = oracle.proxy_scores(P, codes, d, cm)
    khat = np.concatenate([U[m][z[:, m]] for m in range(3)], 1).astype(np.float64)
    full = qc[0].astype(np.float64) @ khat.T            # exact for these values
    sums = (P[0][:, z[:, 0]].astype(np.float64) + P[0][:, cm[0] + z[:, 1]]
            + P[0][:, cm[0] + cm[1] + z[:, 2]])
    assert np.array_equal(sums, full)
    assert np.array_equal(S[0], (full * 0.25).astype(np.float32))  # 1/sqrt(16)


def test_identity_codebooks_give_exact_centroid_key_scores(oracle_lib):
    # C_m = N with identity starts: khat_j = k_j, so the proxy equals the direct
    # score Qbar K^T / sqrt(d) of App. B (exact on dyadic data)
    rng = np.random.default_rng(22)
    d, n, cq = 9, 30, 4
    ranges = ((0, 3, 6), (3, 3, 3))
    k = (rng.integers(-6, 7, size=(1, n, d)) / 2).astype(np.float32)
    qc = (rng.integers(-6, 7, size=(1, cq, d)) / 2).astype(np.float32)
    for m in range(3):  # keep every subspace slice distinct
        sl = slice(ranges[0][m], ranges[0][m] + 3)
        k[0, :, sl] += (np.arange(n)[:, None] * np.array([8, 0, 0]))
    init = np.tile(np.arange(n, dtype=np.int32), (1, 3, 1))
    kr = oracle.cluster_key_subspaces(k, ranges, [n, n, n], 2, init)
    z = kr["codes"][0]
    assert ((z & 1023) == np.arange(n)).all()
    P = oracle.tables(qc, kr["centroids"], ranges, [n, n, n])
    S = oracle.proxy_scores(P, kr["codes"], d, [n, n, n])
    direct = qc[0].astype(np.float64) @ k[0].astype(np.float64).T
    sig = np.float32(1.0 / math.sqrt(d))
    assert np.array_equal(S[0], (direct.astype(np.float32) * sig).astype(np.float32))


def test_table_mac_count_ratio_is_n_over_c():
    # App. B: direct scoring C_q*N*d MACs vs tables C_q*sum(C_m d_m); with
    # equal C_m = C the ratio is N / C.
    for cfg in inputs.CONFIGS.values():
        if cfg.name == "tiny":
            continue
        direct = cfg.c_q * cfg.n * cfg.d
        table = cfg.c_q * sum(cfg.c_m * dm for dm in cfg.split)
        assert Fraction(direct, table) == Fraction(cfg.n, cfg.c_m)


# --------------------------------------------------------------------------
# fixed-point exponential and Top-p target (Eq. 7 arithmetic)

def test_fixexp_error_bound(oracle_lib):
    # every 37th fp32 bit pattern from -0 down to -28
    bits = np.arange(0x80000000, int(np.float32(-28.0).view(np.uint32)) + 1, 37,
                     dtype=np.int64)
    y = np.concatenate([bits.astype(np.uint32).view(np.float32),
                        np.float32([0.0, -0.0, -1e-30, -0.5, -27.7, -28.0])])
    E = oracle.fixexp(y).astype(np.float64)
    ref = np.exp(y.astype(np.float64))
    bound = (np.abs(y) * 2.0 ** -23 + 8 * 2.0 ** -24) * ref + 2.0 ** -33
    err = np.abs(E / 2.0 ** 32 - ref)
    assert (err <= bound).all(), float((err / bound).max())
    assert oracle.fixexp(np.float32([0.0]))[0] == 1 << 32
    assert (oracle.fixexp(np.float32([-27.75, -30.0, -1e9])) == 0).all()


def test_mass_target_is_exact_ceiling(oracle_lib):
    rng = np.random.default_rng(31)
    rhos = list(np.float32(rng.uniform(0, 1, 200))) + [np.float32(x) for x in
                                                        (1e-30, 0.5, 0.9, 0.95, 0.999999)]
    tots = [int(x) for x in rng.integers(1, 1 << 50, 200)] + [1, 3, 1 << 32, (1 << 49) + 7]
    for r in rhos:
        for t in tots[::7]:
            want = math.ceil(Fraction(float(r)) * t)
            assert oracle.mass_target(r, t) == want


# --------------------------------------------------------------------------
# selection (Eq. 7-10, Alg. 3)

def _referee_select(S, counts, rho, k_fix, policy="online"):
    """Alg. 3 by the definition, in exact rationals over the oracle's
    integer softmax masses (policy: Eq. 10, or the Fig. 6 ablations)."""
    cq, n = S.shape
    t, b = [], []
    ranks = []
    for c in range(cq):
        s = S[c]
        pi = sorted(range(n), key=lambda j: (-float(s[j]), j))
        ranks.append(pi)
        E = [int(e) for e in oracle.fixexp(s - s.max())]
        tot = sum(E)
        if rho >= 1:
            tc = n
        else:
            acc = 0
            tc = None
            for l, j in enumerate(pi):
                acc += E[j]
                if Fraction(acc, tot) >= Fraction(float(np.float32(rho))):
                    tc = l + 1
                    break
        t.append(tc)
        b.append(max(tc, k_fix))
    kh = math.ceil(Fraction(sum(int(counts[c]) * b[c] for c in range(cq)),
                            int(sum(counts))))
    r = {"online": [max(bc, kh) for bc in b], "fixed": list(b), "topp": list(t)}[policy]
    sets = [sorted(ranks[c][:r[c]]) for c in range(cq)]
    return t, b, kh, r, sets


def test_select_golden_worked_example(oracle_lib):
    gx = json.load(open(os.path.join(GOLDEN, "select_worked_example.json")))
    S = np.array([[_expr(e) for e in row] for row in gx["logit_expressions"]],
                 np.float32)[None]
    counts = np.array(gx["cluster_sizes"], np.int32)[None]
    for case in gx["cases"]:
        r = oracle.select(S, counts, case["rho"], case["k_fix"])
        assert r["topp"][0].tolist() == case["t"]
        assert r["base_counts"][0].tolist() == case["b"]
        assert int(r["k_head"][0]) == case["k_head"]
        assert r["sel_counts"][0].tolist() == case["r"]
        for c, want in enumerate(case["S"]):
            assert r["sel_idx"][0, c, :len(want)].tolist() == want


@pytest.mark.parametrize("seed", range(40))
def test_select_brute_force_small(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 11))
    cq = int(rng.integers(1, 5))
    pool = rng.normal(0, 3, size=4).astype(np.float32)      # forces ties
    S = pool[rng.integers(0, 4, size=(cq, n))]
    if seed % 3 == 0:
        S = rng.normal(0, 2, size=(cq, n)).astype(np.float32)
    g = rng.integers(0, cq, size=n)
    counts = np.bincount(g, minlength=cq).astype(np.int32)
    rho = float(np.float32(rng.choice([0.3, 0.5, 0.9, 0.95, 1.0, rng.uniform()])))
    k_fix = int(rng.integers(1, n + 1))
    policy = ("online", "fixed", "topp")[seed % 3]
    r = oracle.select(S[None], counts[None], rho, k_fix, policy)
    t, b, kh, rr, sets = _referee_select(S, counts, rho, k_fix, policy)
    assert r["topp"][0].tolist() == t
    assert r["base_counts"][0].tolist() == b
    assert int(r["k_head"][0]) == kh
    assert r["sel_counts"][0].tolist() == rr
    for c in range(cq):
        assert r["sel_idx"][0, c, :rr[c]].tolist() == sets[c]
    # Eq. 9 closed form as a per-query average of b_{g_i}
    assert kh == math.ceil(Fraction(sum(b[gi] for gi in g), n))


def test_select_policies_nest(oracle_lib):
    """Top-p sets are contained in the fixed-floor sets, which are contained
    in the online sets; each is a prefix of the same ranking."""
    rng = np.random.default_rng(7)
    n, cq = 300, 5
    S = rng.normal(0, 2, size=(1, cq, n)).astype(np.float32)
    counts = rng.integers(1, 50, size=(1, cq)).astype(np.int32)
    out = {p: oracle.select(S, counts, 0.8, 40, p) for p in ("topp", "fixed", "online")}
    t, b = out["online"]["topp"][0], out["online"]["base_counts"][0]
    kh = int(out["online"]["k_head"][0])
    assert out["topp"]["sel_counts"][0].tolist() == t.tolist()
    assert out["fixed"]["sel_counts"][0].tolist() == b.tolist()
    assert out["online"]["sel_counts"][0].tolist() == np.maximum(b, kh).tolist()
    for c in range(cq):
        sets = [set(out[p]["sel_idx"][0, c, :out[p]["sel_counts"][0, c]].tolist())
                for p in ("topp", "fixed", "online")]
        assert sets[0] <= sets[1] <= sets[2]


def test_select_invariants_and_float64_softmax(oracle_lib):
    rng = np.random.default_rng(41)
    n, cq = 700, 6
    S = np.round(rng.normal(0, 2.5, size=(cq, n)), 2).astype(np.float32)
    counts = rng.multinomial(n, np.ones(cq) / cq).astype(np.int32)
    rho, k_fix = 0.9, 35
    r = oracle.select(S[None], counts[None], rho, k_fix)
    kh = int(r["k_head"][0])
    for c in range(cq):
        s = S[c].astype(np.float64)
        t = int(r["topp"][0, c])
        b = int(r["base_counts"][0, c])
        rc = int(r["sel_counts"][0, c])
        sel = r["sel_idx"][0, c, :rc]
        assert rc == len(set(sel.tolist())) and (np.diff(sel) > 0).all()
        assert rc >= b >= k_fix and rc >= kh
        assert b == max(t, k_fix) and (rc == b if b >= kh else rc == kh)
        pi = sorted(range(n), key=lambda j: (-s[j], j))
        assert sorted(pi[:rc]) == sel.tolist()     # a prefix of pi_c
        assert set(pi[:t]) <= set(sel.tolist())      # Top-p set inside S_c
        # real softmax in float64 agrees unless the crossing is a near-tie
        w = np.exp(s - s.max())
        cum = np.cumsum(w[pi]) / w.sum()
        t64 = int(np.searchsorted(cum, rho) + 1)
        if abs(cum[t64 - 1] - rho) > 1e-6 and (t64 < 2 or abs(cum[t64 - 2] - rho) > 1e-6):
            assert t == t64


def test_select_closed_forms(oracle_lib):
    n = 257
    flat = np.zeros((1, 2, n), np.float32)
    counts = np.array([[200, 57]], np.int32)
    # rho = 1 keeps every key; k_fix = n keeps every key
    for rho, k_fix in ((1.0, 1), (0.5, n)):
        r = oracle.select(flat, counts, rho, k_fix)
        assert (r["sel_counts"] == n).all()
        assert (r["sel_idx"][0, :, :] == np.arange(n)).all()
    # all-equal logits: the Top-p count is ceil(rho * n)
    for rho in (0.1, 0.5, 0.9, 0.95):
        r = oracle.select(flat, counts, rho, 1)
        want = math.ceil(Fraction(float(np.float32(rho))) * n)
        assert (r["topp"] == want).all()
    # one dominant key (others carry zero mass): t = 1
    dom = np.full((1, 1, n), -100.0, np.float32)
    dom[0, 0, 123] = 0.0
    r = oracle.select(dom, np.array([[n]], np.int32), 0.9, 1)
    assert r["topp"][0, 0] == 1 and r["sel_idx"][0, 0, 0] == 123


# --------------------------------------------------------------------------
# attention (Eq. 1, Eq. 11)

def _np_attention(q, k, v, scale):
    s = q.astype(np.float64) @ k.astype(np.float64).T * scale
    s -= s.max(1, keepdims=True)
    p = np.exp(s)
    return (p @ v.astype(np.float64)) / p.sum(1, keepdims=True)


def test_dense_attention_matches_textbook(oracle_lib):
    rng = np.random.default_rng(51)
    q, k, v = (rng.standard_normal((2, 90, 24)).astype(np.float32) for _ in range(3))
    out = oracle.dense_attention(q, k, v)
    for h in range(2):
        ref = _np_attention(q[h], k[h], v[h], 1 / math.sqrt(24))
        np.testing.assert_allclose(out[h], ref, rtol=2e-7, atol=2e-7)


def test_dense_attention_matches_torch_sdpa(oracle_lib):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(52)
    q, k, v = (rng.standard_normal((3, 70, 16)).astype(np.float32) for _ in range(3))
    out = oracle.dense_attention(q, k, v)
    ref = torch.nn.functional.scaled_dot_product_attention(
        *(torch.from_numpy(x).double()[None] for x in (q, k, v)))[0].numpy()
    np.testing.assert_allclose(out, ref, rtol=2e-7, atol=2e-7)


def test_sparse_attention_matches_masked_textbook(oracle_lib):
    rng = np.random.default_rng(53)
    n, d, cq = 60, 8, 5
    q, k, v = (rng.standard_normal((1, n, d)).astype(np.float32) for _ in range(3))
    g = rng.integers(0, cq, size=n)
    counts, offsets, perm = oracle.group(g.astype(np.int32), cq)
    sel_counts = rng.integers(1, n + 1, size=cq).astype(np.int32)
    sel_idx = np.full((cq, n), -1, np.int32)
    for c in range(cq):
        sel_idx[c, :sel_counts[c]] = np.sort(rng.choice(n, sel_counts[c], replace=False))
    out = oracle.attention(q, k, v, offsets[None], perm[None], sel_counts[None],
                           sel_idx[None])
    for i in range(n):
        S = sel_idx[g[i], :sel_counts[g[i]]]
        ref = _np_attention(q[0, i:i + 1], k[0, S], v[0, S], 1 / math.sqrt(d))
        np.testing.assert_allclose(out[0, i], ref[0], rtol=2e-7, atol=2e-7)


def test_single_key_returns_its_value(oracle_lib):
    rng = np.random.default_rng(54)
    q, k, v = (rng.standard_normal((1, 10, 4)).astype(np.float32) for _ in range(3))
    offsets = np.array([[0, 10]], np.int32)
    perm = np.arange(10, dtype=np.int32)[None]
    idx = np.full((1, 1, 10), -1, np.int32)
    idx[0, 0, 0] = 7
    out = oracle.attention(q, k, v, offsets, perm, np.array([[1]], np.int32), idx)
    assert np.array_equal(out[0], np.repeat(v[0, 7:8], 10, 0))


# --------------------------------------------------------------------------
# whole layer

def test_layer_with_rho_one_equals_dense(oracle_lib):
    cfg = inputs.CONFIGS["tiny"]
    x = inputs.generate(cfg)
    r = oracle.layer(x.q, x.k, x.v, cfg.ranges, cfg.c_q, [cfg.c_m] * 3, cfg.iters,
                     x.init_q, x.init_k, 1.0, cfg.k_fix)
    assert (r["sel"]["sel_counts"] == cfg.n).all()
    dense = oracle.dense_attention(x.q, x.k, x.v)
    np.testing.assert_allclose(r["out"], dense, rtol=1e-6, atol=1e-6)


def test_layer_tiny_is_deterministic_and_consistent(oracle_lib):
    cfg = inputs.CONFIGS["tiny"]
    x = inputs.generate(cfg)
    args = (x.q, x.k, x.v, cfg.ranges, cfg.c_q, [cfg.c_m] * 3, cfg.iters,
            x.init_q, x.init_k, cfg.rho, cfg.k_fix)
    a = oracle.layer(*args)
    b = oracle.layer(*args)
    assert np.array_equal(a["out"], b["out"])
    assert np.array_equal(a["sel"]["sel_idx"], b["sel"]["sel_idx"])
    codes = a["k"]["codes"]
    assert (codes >> 30 == 0).all() and ((codes & 1023) < cfg.c_m).all()


# --------------------------------------------------------------------------
# general key partitions (App. B; Table 3)

def _planes(codes, M=3):
    return np.stack([(codes >> (10 * m)) & 1023 for m in range(M)], 1).astype(np.uint16)


def test_partition_with_rope_sets_reduces_to_the_three_ranges(oracle_lib):
    cfg = inputs.CONFIGS["tiny"]
    x = inputs.generate(cfg)
    sets = inputs.partition_sets(cfg, "3-rope")
    cm = [cfg.c_m] * 3
    a = oracle.cluster_key_subspaces(x.k, cfg.ranges, cm, cfg.iters, x.init_k)
    b = oracle.cluster_key_partition(x.k, sets, cm, cfg.iters, x.init_k)
    assert np.array_equal(a["centroids"].view(np.uint32), b["centroids"].view(np.uint32))
    assert np.array_equal(_planes(a["codes"]), b["codes"])
    qc = oracle.cluster_queries(x.q, cfg.c_q, cfg.iters, x.init_q)["centroids"]
    Pa = oracle.tables(qc, a["centroids"], cfg.ranges, cm)
    Pb = oracle.tables_partition(qc, b["centroids"], sets, cm)
    assert np.array_equal(Pa.view(np.uint32), Pb.view(np.uint32))
    Sa = oracle.proxy_scores(Pa, a["codes"], cfg.d, cm)
    Sb = oracle.proxy_scores_partition(Pb, b["codes"], cfg.d, cm)
    assert np.array_equal(Sa.view(np.uint32), Sb.view(np.uint32))


@pytest.mark.parametrize("seed", range(3))
def test_partition_equals_ranges_of_channel_permuted_inputs(oracle_lib, seed):
    # relabelling the channels so that the random sets become consecutive
    # ranges leaves every dot product (same channels, same order) unchanged
    cfg = inputs.CONFIGS["tiny"]
    x = inputs.generate(cfg)
    sets = inputs.partition_sets(cfg, "3-random", seed)
    perm = np.concatenate(sets)
    ln = [len(s) for s in sets]
    ranges = ((0, ln[0], ln[0] + ln[1]), tuple(ln))
    cm = [7, 5, 8]
    init = x.init_k
    a = oracle.cluster_key_partition(x.k, sets, cm, 4, init)
    b = oracle.cluster_key_subspaces(x.k[:, :, perm], ranges, cm, 4, init)
    assert np.array_equal(a["centroids"].view(np.uint32), b["centroids"].view(np.uint32))
    assert np.array_equal(a["codes"], _planes(b["codes"]))
    qc = oracle.cluster_queries(x.q, cfg.c_q, 3, x.init_q)["centroids"]
    Pa = oracle.tables_partition(qc, a["centroids"], sets, cm)
    Pb = oracle.tables(qc[:, :, perm], b["centroids"], ranges, cm)
    assert np.array_equal(Pa.view(np.uint32), Pb.view(np.uint32))
    Sa = oracle.proxy_scores_partition(Pa, a["codes"], cfg.d, cm)
    Sb = oracle.proxy_scores(Pb, b["codes"], cfg.d, cm)
    assert np.array_equal(Sa.view(np.uint32), Sb.view(np.uint32))


@pytest.mark.parametrize("M", [1, 2, 5, 8])
def test_partition_lookup_sum_equals_full_centroid_dot(oracle_lib, M):
    # App. B for M subspaces: sum_m P_m[c, z^m] = <qbar_c, khat_j>, where khat_j
    # puts each subspace centroid back on its channels; exact on dyadic data
    rng = np.random.default_rng(40 + M)
    d, cq, n = 16, 4, 50
    perm = rng.permutation(d)
    cuts = np.sort(rng.choice(np.arange(1, d), M - 1, replace=False))
    sets = [np.sort(s) for s in np.split(perm, cuts)]
    cm = [int(rng.integers(2, 6)) for _ in range(M)]
    qc = (rng.integers(-8, 8, size=(1, cq, d)) / 4).astype(np.float32)
    U = [(rng.integers(-8, 8, size=(cm[m], len(sets[m]))) / 4).astype(np.float32)
         for m in range(M)]
    kc = np.concatenate([u.ravel() for u in U])[None]
    z = np.stack([rng.integers(0, cm[m], size=n) for m in range(M)], 0)
    P = oracle.tables_partition(qc, kc, sets, cm)
    S = oracle.proxy_scores_partition(P, z.astype(np.uint16)[None], d, cm)
    khat = np.zeros((n, d))
    for m in range(M):
        khat[:, sets[m]] = U[m][z[m]]
    full = qc[0].astype(np.float64) @ khat.T
    col = np.concatenate([[0], np.cumsum(cm)])
    sums = sum(P[0][:, col[m] + z[m]].astype(np.float64) for m in range(M))
    assert np.array_equal(sums, full)
    assert np.array_equal(S[0], (full * 0.25).astype(np.float32))


def test_partition_codes_are_argmins_of_returned_centroids(oracle_lib):
    # each subspace is k-means of K[:, I_m]: labels are exact argmins of the
    # returned centroids (fp64 distances where the margin is clear)
    rng = np.random.default_rng(7)
    n, d = 300, 12
    sets = [np.array([0, 5, 7]), np.array([1, 2, 3, 4, 6, 8]), np.array([9, 10, 11])]
    cm = [4, 6, 3]
    k = rng.standard_normal((1, n, d)).astype(np.float32)
    init = np.stack([inputs.init_rows(rng, n, 6) for _ in range(3)])[None]
    r = oracle.cluster_key_partition(k, sets, cm, 6, init)
    U = np.split(r["centroids"][0], np.cumsum([cm[m] * len(sets[m]) for m in range(3)])[:-1])
    for m in range(3):
        Um = U[m].reshape(cm[m], len(sets[m])).astype(np.float64)
        X = k[0][:, sets[m]].astype(np.float64)
        D = ((X[:, None, :] - Um[None]) ** 2).sum(-1)
        srt = np.sort(D, 1)
        clear = srt[:, 1] - srt[:, 0] > 1e-4
        assert np.array_equal(r["codes"][0, m][clear], D.argmin(1)[clear])
        # a final assignment over the returned centroids changes no label
        assert np.array_equal(r["codes"][0, m], oracle.assign_rows(X.astype(np.float32),
                                                                   U[m].reshape(cm[m], -1)))


def test_partition_rejects_bad_sets(oracle_lib):
    k = np.zeros((1, 20, 6), np.float32)
    init = np.zeros((1, 2, 4), np.int32)
    init[:] = np.arange(4)
    for sets in ([[0, 1, 2], [2, 3, 4, 5]],      # overlap
                 [[0, 1], [2, 3, 4]],            # channel 5 missing
                 [[1, 0, 2], [3, 4, 5]],         # not ascending
                 [[0, 1, 2], [3, 4, 6]]):        # out of range
        with pytest.raises(ValueError):
            oracle.cluster_key_partition(k, sets, [2, 2], 1, init)


# --------------------------------------------------------------------------
# Proxy comparison measurements (App. C, Fig. 9; Fig. 2)

def test_proxy_recall_golden_example(oracle_lib):
    g = json.load(open(os.path.join(GOLDEN, "proxy_recall_example.json")))
    exact = np.array([g["exact"]] * 2, np.float32)
    proxy = np.array(g["proxy_rows"], np.float32)
    ret, rec = oracle.matched_retention(exact, proxy, g["top_frac"], g["target"])
    assert [Fraction(x) for x in g["retention"]] == [Fraction(v).limit_denominator(1000) for v in ret]
    assert [Fraction(x) for x in g["recall"]] == [Fraction(v).limit_denominator(1000) for v in rec]
    p = exact.astype(np.float64) / g["p_exact_denominator"]
    mass = oracle.recall_at_density(p, proxy, g["density"])
    assert np.allclose(mass, [float(Fraction(x)) for x in g["mass"]], rtol=0, atol=1e-15)
    b = g["block"]
    out = oracle.block_proxy(np.array([b["q"]], np.float32), np.array(b["k"], np.float32),
                             b["block"], b["scale"])
    assert out[0].tolist() == b["proxy"]


def _retention_referee(exact, proxy, kt, need):
    """The protocol by brute force over explicit rankings, exact counts."""
    n = len(exact)
    o_rank = sorted(range(n), key=lambda j: (-float(exact[j]), j))
    oset = set(o_rank[:kt])
    p_rank = sorted(range(n), key=lambda j: (-float(proxy[j]), j))
    hits = 0
    for pos, j in enumerate(p_rank):
        hits += j in oset
        if hits >= need:
            break
    s_star = float(proxy[p_rank[pos]])
    kept = [j for j in range(n) if float(proxy[j]) >= s_star]
    return Fraction(len(kept), n), Fraction(len(oset & set(kept)), kt)


@pytest.mark.parametrize("seed", range(6))
def test_matched_retention_brute_force(oracle_lib, seed):
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(3, 13))
    rows = 8
    # small integer scores: many ties in both rankings
    exact = rng.integers(-3, 4, (rows, n)).astype(np.float32)
    proxy = rng.integers(-2, 3, (rows, n)).astype(np.float32)
    top_frac, target = [0.1, 0.3, 0.5][seed % 3], [0.5, 0.958, 1.0][seed % 3]
    ret, rec = oracle.matched_retention(exact, proxy, top_frac, target)
    ceil = lambda f: -((-f.numerator) // f.denominator)
    kt = max(1, ceil(Fraction(str(top_frac)) * n))
    need = max(1, ceil(Fraction(str(target)) * kt))
    for r in range(rows):
        want_ret, want_rec = _retention_referee(exact[r], proxy[r], kt, need)
        assert Fraction(ret[r]).limit_denominator(10000) == want_ret
        assert Fraction(rec[r]).limit_denominator(10000) == want_rec
    # density: mass of the first k keys of the proxy ranking
    p = rng.random((rows, n))
    for dens in (0.1, 0.5, 1.0):
        k = max(1, int(round(dens * n)))
        got = oracle.recall_at_density(p, proxy, dens)
        for r in range(rows):
            order = sorted(range(n), key=lambda j: (-float(proxy[r, j]), j))[:k]
            assert abs(got[r] - sum(p[r, j] for j in order)) < 1e-12


def test_proxy_recall_closed_forms(oracle_lib):
    rng = np.random.default_rng(41)
    rows, n = 5, 200
    exact = rng.standard_normal((rows, n)).astype(np.float32)
    # the exact scores as their own proxy (no ties): the first `need` keys
    # are all oracle keys, so exactly `need` keys are kept
    ret, rec = oracle.matched_retention(exact, exact, 0.1, 0.958)
    kt, need = 20, 20  # ceil(0.1 * 200), ceil(0.958 * 20)
    assert np.allclose(ret, need / n) and np.allclose(rec, need / kt)
    # a constant proxy keeps every key (one tie group)
    ret, rec = oracle.matched_retention(exact, np.zeros_like(exact), 0.1, 0.5)
    assert np.all(ret == 1.0) and np.all(rec == 1.0)
    # blocks of one token: the proxy is the direct representative score
    k = rng.standard_normal((n, 16)).astype(np.float32)
    q = rng.standard_normal((rows, 16)).astype(np.float32)
    direct = (q.astype(np.float64) @ k.T.astype(np.float64) * 0.25).astype(np.float32)
    assert np.array_equal(oracle.block_proxy(q, k, 1, 0.25), direct)
    # one block over all tokens: every key gets the score of the mean key
    one = oracle.block_proxy(q, k, n, 0.25)
    mean = (q.astype(np.float64) @ k.astype(np.float64).mean(0) * 0.25).astype(np.float32)
    assert np.allclose(one, mean[:, None], rtol=1e-6, atol=1e-6)


# --------------------------------------------------------------------------
# Warm starts across denoising steps (Sec. 4 setup)

def test_kmeans_warm_start_continues_the_iteration(oracle_lib):
    """Lloyd's state is its centroids: I1 iterations, then I2 more from the
    returned centroids, equal I1 + I2 iterations from the start, for the
    queries (ending on an update) and the key subspaces (ending on an
    assignment)."""
    cfg = inputs.CONFIGS["tiny"]
    x = inputs.generate(cfg)
    cm = (cfg.c_m,) * 3
    a = oracle.cluster_queries(x.q, cfg.c_q, 2, x.init_q)
    b = oracle.cluster_queries_from(x.q, cfg.c_q, 3, a["centroids"])
    c = oracle.cluster_queries(x.q, cfg.c_q, 5, x.init_q)
    for key in ("centroids", "assign", "counts", "offsets", "perm"):
        assert np.array_equal(b[key], c[key]), key
    ka = oracle.cluster_key_subspaces(x.k, cfg.ranges, cm, 2, x.init_k)
    kb = oracle.cluster_key_subspaces_from(x.k, cfg.ranges, cm, 3, ka["centroids"])
    kc = oracle.cluster_key_subspaces(x.k, cfg.ranges, cm, 5, x.init_k)
    assert np.array_equal(kb["centroids"], kc["centroids"])
    assert np.array_equal(kb["codes"], kc["codes"])


def test_kmeans_warm_start_hand_example(oracle_lib):
    """Points 0, 1, 10, 11 (one channel) from centroids 2 and 9: one step
    assigns {0, 1} and {10, 11} and moves the centroids to their means 0.5
    and 10.5, a fixed point of every later step."""
    q = np.array([[[0.0], [1.0], [10.0], [11.0]]], np.float32)
    r = oracle.cluster_queries_from(q, 2, 1, np.array([[[2.0], [9.0]]], np.float32))
    assert r["centroids"].ravel().tolist() == [0.5, 10.5]
    assert r["assign"].ravel().tolist() == [0, 0, 1, 1]
    r2 = oracle.cluster_queries_from(q, 2, 4, r["centroids"])
    assert np.array_equal(r2["centroids"], r["centroids"])


def test_sparsity_schedule():
    """First layer dense at every step; the other layers dense for the first
    ceil(fraction * steps) steps (Sec. 4: 20% Wan, 10% HunyuanVideo)."""
    from paper_2608_12780_amd.layer import SparsitySchedule
    wan = SparsitySchedule(50, 0.2)
    assert wan.dense_steps == 10
    assert all(wan.dense(0, s) for s in range(50))
    assert [wan.dense(7, s) for s in (9, 10, 49)] == [True, False, False]
    assert [wan.warm(7, s) for s in (9, 10, 11)] == [False, False, True]
    hy = SparsitySchedule(50, 0.1)
    assert hy.dense_steps == 5 and not hy.dense(3, 5) and hy.dense(3, 4)
    assert SparsitySchedule(7, 0.1).dense_steps == 1

