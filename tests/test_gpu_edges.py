"""GPU edge cases of the C ABI against the oracle.

* The data-dependent status word of the clustering calls (non-finite input,
  values outside the exact fixed-point range of the k-means means, a bad
  initial row), planted in otherwise ordinary inputs.
* The selection's crossing-bin fallback when the coarse bin that holds the
  Top-p mass crossing (Eq. 7) or the rank-r_c crossing (Eq. 10) contains more
  distinct key codes than the on-chip candidate list: the passes then visit
  every distinct code of the head.  Checked bit for bit against the oracle's
  selection on the oracle's proxy logits.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle  # noqa: E402
from paper_2608_12780_amd import binding as B  # noqa: E402
from paper_2608_12780_amd import inputs  # noqa: E402

import gpu_harness as G  # noqa: E402

# status bits of the device word (include/scope.h)
NONFINITE, RANGE, BADINIT = 1, 2, 4

# the selection's on-chip candidate list (logits of one coarse bin)
CAND_CAP = 4096
COARSE_BINS = 2048


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    oracle.lib()


SMALL = inputs.LayerConfig("status", 1, (3, 8, 10), 64, (16, 24, 24), 8, 6, 3, 0.9,
                           24, "bf16", 4, 71)


def range_limit(n):
    """The bound of the exact fixed-point sums, 2^min(22, 39 - ceil(log2 n))."""
    L = int(np.ceil(np.log2(n))) if n > 1 else 0
    return float(2.0 ** min(22, 39 - L))


def _cluster(cfg, x, init_q=None, init_k=None):
    layer = G.make_layer(cfg, materialize=False)
    q, k, _ = G.to_device(x)
    layer.cluster_queries(q, torch.from_numpy(x.init_q if init_q is None else init_q).cuda())
    torch.cuda.synchronize()
    st_q = int(layer.status.item())
    layer.status.zero_()
    layer.cluster_keys(k, torch.from_numpy(x.init_k if init_k is None else init_k).cuda())
    torch.cuda.synchronize()
    st_k = int(layer.status.item())
    return layer, st_q, st_k


def _set(x, which, h, row, ch, value):
    a = getattr(x, which)
    a[h, row, ch] = value
    if x.q_bits is not None:
        getattr(x, which + "_bits")[h] = inputs.bf16_bits(a[h])
        a[h] = inputs.bf16_widen(getattr(x, which + "_bits")[h])


def test_status_clean_inputs_report_nothing():
    x = inputs.generate(SMALL)
    _, st_q, st_k = _cluster(SMALL, x)
    assert st_q == 0 and st_k == 0


def test_status_non_finite_query():
    # fp32 storage: a NaN and an infinity in the queries set bits 0 and 1
    cfg = SMALL.with_(name="status_nan", dtype="f32")
    x = inputs.generate(cfg)
    x.q[0, 17, 5] = np.nan
    x.q[0, 40, 0] = np.inf
    _, st_q, st_k = _cluster(cfg, x)
    ref = oracle.cluster_queries(x.q, cfg.c_q, cfg.iters, x.init_q)
    assert ref["status"] == 2  # the oracle's range status
    assert st_q == NONFINITE | RANGE, st_q
    assert st_k == 0


@pytest.mark.parametrize("which", ["q", "k"])
def test_status_out_of_fixed_point_range(which):
    # |x| = 2^22 in bf16 storage: bit 1 only, as the oracle reports it
    x = inputs.generate(SMALL)
    _set(x, which, 0, 33, 20, 2.0 ** 22)
    assert abs(getattr(x, which)[0, 33, 20]) >= range_limit(SMALL.n)
    _, st_q, st_k = _cluster(SMALL, x)
    if which == "q":
        ref = oracle.cluster_queries(x.q, SMALL.c_q, SMALL.iters, x.init_q)
        assert ref["status"] == 2
        assert (st_q, st_k) == (RANGE, 0)
    else:
        ref = oracle.cluster_key_subspaces(x.k, SMALL.ranges, (SMALL.c_m,) * 3, SMALL.iters,
                                           x.init_k)
        assert ref["status"] == 2
        assert (st_q, st_k) == (0, RANGE)


def test_status_range_bound_tightens_with_n():
    """Above 2^17 rows the exact range shrinks: at n = 140800 (ceil(log2 n)
    = 18) it is 2^21, so 1.5 * 2^21 is flagged (it would not be at n <=
    2^17), and the oracle reports the same."""
    cfg = inputs.LayerConfig("status_big", 1, (11, 40, 320), 64, (16, 24, 24), 4, 4, 1,
                             0.9, 14080, "bf16", 2, 73)
    assert cfg.n > 2 ** 17 and range_limit(cfg.n) == 2.0 ** 21
    x = inputs.generate(cfg)
    _set(x, "q", 0, 1000, 3, 1.5 * 2.0 ** 21)
    layer = G.make_layer(cfg, materialize=False)
    q, _, _ = G.to_device(x)
    layer.cluster_queries(q, torch.from_numpy(x.init_q).cuda())
    torch.cuda.synchronize()
    ref = oracle.cluster_queries(x.q, cfg.c_q, cfg.iters, x.init_q)
    assert ref["status"] == 2
    assert int(layer.status.item()) == RANGE
    # and the same value at n <= 2^17 is inside the range: nothing flagged
    x2 = inputs.generate(SMALL)
    _set(x2, "q", 0, 5, 3, 1.5 * 2.0 ** 21)
    _, st_q, _ = _cluster(SMALL, x2)
    assert st_q == 0


def test_status_bad_initial_rows_fall_back_to_the_default_row():
    """An out-of-range starting row sets bit 2 and is replaced by the
    documented default row floor((2r + 1) n / (2C)); the result equals the
    oracle started from that row."""
    x = inputs.generate(SMALL)
    n, C, Cm = SMALL.n, SMALL.c_q, SMALL.c_m
    init_q = x.init_q.copy()
    init_k = x.init_k.copy()
    init_q[0, 3] = n          # past the end
    init_k[0, 1, 2] = -7      # negative, H subspace
    layer, st_q, st_k = _cluster(SMALL, x, init_q, init_k)
    assert st_q == BADINIT and st_k == BADINIT
    fixed_q = init_q.copy()
    fixed_q[0, 3] = inputs.default_init_rows(n, C)[3]
    fixed_k = init_k.copy()
    fixed_k[0, 1, 2] = inputs.default_init_rows(n, Cm)[2]
    ref_q = oracle.cluster_queries(x.q, C, SMALL.iters, fixed_q)
    ref_k = oracle.cluster_key_subspaces(x.k, SMALL.ranges, (Cm,) * 3, SMALL.iters, fixed_k)
    assert np.array_equal(layer.assign.cpu().numpy(), ref_q["assign"])
    assert np.array_equal(layer.q_centroids.cpu().numpy().view(np.uint32),
                          ref_q["centroids"].view(np.uint32))
    assert np.array_equal(layer.codes.cpu().numpy().view(np.uint32), ref_k["codes"])


# --- crossing bins beyond the candidate list ------------------------------

def _coarse_bin(y):
    # the selection's monotone binning of y = s - M <= 0 (bins of 1/64)
    return np.minimum(np.floor(-y.astype(np.float32) * np.float32(64)), COARSE_BINS - 1)


def _ranked(scores_row):
    """keys in the order pi_c (logit descending, index ascending)"""
    return np.lexsort((np.arange(scores_row.size), -scores_row.astype(np.float64)))


def _distinct_in_bin(scores_row, codes_row, key_rank):
    """distinct codes whose logit falls in the coarse bin of the key at rank
    key_rank (1-based) of pi_c"""
    M = scores_row.max()
    order = _ranked(scores_row)
    b = _coarse_bin(np.float32(scores_row[order[key_rank - 1]] - M))
    inb = _coarse_bin((scores_row - M).astype(np.float32)) == b
    return int(b), np.unique(codes_row[inb] & 0x3FFFFFFF).size


def test_topp_crossing_bin_beyond_the_candidate_list():
    """Every logit within 1/64 of the maximum: the Top-p crossing (Eq. 7,
    about 0.7 n) and the rank crossing of r_c = k_fix = 25000 (Eq. 8 and 10)
    both lie in coarse bin 0, which holds about 24000 distinct codes."""
    rng = np.random.default_rng(81)
    H, C, n, d, c_m = 1, 4, 30000, 64, (32, 32, 64)
    tables = (rng.random((H, C, sum(c_m))) * 0.01).astype(np.float32)
    codes = (rng.integers(0, c_m[0], (H, n)) | (rng.integers(0, c_m[1], (H, n)) << 10)
             | (rng.integers(0, c_m[2], (H, n)) << 20)).astype(np.uint32)
    counts = np.array([[9000, 1000, 12000, 8000]], np.int32)
    S = oracle.proxy_scores(tables, codes, d, c_m)
    k_fix = 25000
    ref = oracle.select(S, counts, 0.7, k_fix)
    for c in range(C):
        for rank in (int(ref["topp"][0, c]), int(ref["sel_counts"][0, c])):
            b, nd = _distinct_in_bin(S[0, c], codes[0], rank)
            assert b == 0 and nd > CAND_CAP, (c, rank, b, nd)
    # every cluster keeps more than its Top-p count (the rank target)
    assert (ref["sel_counts"] == k_fix).all() and (ref["topp"] < k_fix).all()
    G.say(f"[edges] bin-0 crossing: k_head {int(ref['k_head'][0])}, "
          f"t {ref['topp'][0].tolist()}, r {ref['sel_counts'][0].tolist()}")
    G.select_from_codes(tables, codes, counts, d, c_m, 0.7, k_fix)


def test_rank_crossing_in_the_clamped_last_bin_beyond_the_candidate_list():
    """Keys whose T code is 0 score about 12.5; every other key scores below
    -40, more than 32 under the maximum, so all of them share the clamped
    last coarse bin (over 20000 distinct codes).  k_fix = 20000 puts every
    cluster's rank crossing (Eq. 8 and 10) in that bin."""
    rng = np.random.default_rng(83)
    H, C, n, d, c_m = 1, 3, 30000, 64, (32, 32, 64)
    tables = np.empty((H, C, sum(c_m)), np.float32)
    tables[..., :c_m[0]] = rng.uniform(-400.0, -330.0, (H, C, c_m[0]))
    tables[..., 0] = 100.0
    tables[..., c_m[0]:] = rng.uniform(-1.0, 1.0, (H, C, c_m[1] + c_m[2]))
    codes = (rng.integers(0, c_m[0], (H, n)) | (rng.integers(0, c_m[1], (H, n)) << 10)
             | (rng.integers(0, c_m[2], (H, n)) << 20)).astype(np.uint32)
    counts = np.array([[10000, 15000, 5000]], np.int32)
    k_fix = 20000
    S = oracle.proxy_scores(tables, codes, d, c_m)
    ref = oracle.select(S, counts, 0.9, k_fix)
    for c in range(C):
        assert ref["sel_counts"][0, c] == k_fix > ref["topp"][0, c]
        b, nd = _distinct_in_bin(S[0, c], codes[0], k_fix)
        assert b == COARSE_BINS - 1 and nd > CAND_CAP, (c, b, nd)
    G.select_from_codes(tables, codes, counts, d, c_m, 0.9, k_fix)
