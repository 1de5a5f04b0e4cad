"""GPU parity: the HIP library through the C ABI against the CPU oracle.

Integer results (assignments, counts, permutation, codes, selected sets) and
the canonical fp32 results (centroids, tables, proxy logits) must match bit
for bit; attention output must be within max-abs 2e-2 and mean-rel 1e-2 of
the oracle's fp64 attention on the same bf16-rounded Q/K/V and key sets.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle  # noqa: E402
from paper_2608_12780_amd import binding as B  # noqa: E402
from paper_2608_12780_amd import inputs  # noqa: E402
from paper_2608_12780_amd.layer import DenseAttention  # noqa: E402

import gpu_harness as G  # noqa: E402

MID_HY = inputs.LayerConfig("mid_hy", 2, (5, 19, 23), 128, (16, 56, 56), 32, 16,
                            4, 0.9, inputs.ceil_tenth(5 * 19 * 23), "bf16", 8, 7)
MID_WAN = inputs.LayerConfig("mid_wan", 1, (4, 10, 13), 128, (44, 42, 42), 16, 8,
                             3, 0.9, inputs.ceil_tenth(520), "bf16", 8, 8)
# d = 64 in bf16: 16- and 32-channel codebooks on the matrix cores and the
# d = 64 attention kernel inside the sparse layer
MID_D64 = inputs.LayerConfig("mid_d64", 2, (4, 12, 17), 64, (16, 24, 24), 24, 12,
                             3, 0.9, inputs.ceil_tenth(4 * 12 * 17), "bf16", 6, 10)
# the paper's operating point: C_q = 300 and C_m = 333 (not powers of two).
# Both take the matrix-core assignment: the 300 x 128 query codebook does
# not fit one block's LDS and is split into two chunks (km_assign_mfma_part
# plus km_assign_decide); the 333-centroid subspace codebooks (16 and 56
# channels) are padded to 352 rows and fit it whole.
PAPER_POINT = inputs.LayerConfig("paper_point", 1, (6, 20, 24), 128, (16, 56, 56), 300, 333,
                                 3, 0.9, inputs.ceil_tenth(6 * 20 * 24), "bf16", 8, 9)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    oracle.lib()


def check_layer(cfg, use_scores=False, policy="online"):
    G.say(f"[parity] {cfg.name}: heads={cfg.heads} n={cfg.n} d={cfg.d} "
          f"split={cfg.split} c_q={cfg.c_q} c_m={cfg.c_m} iters={cfg.iters}")
    x = inputs.generate(cfg)
    layer = G.make_layer(cfg)
    gpu = G.run_gpu(layer, x, use_scores=use_scores, policy=policy)
    ref = G.oracle_all(x, cfg.c_q, (cfg.c_m,) * 3, cfg.iters, cfg.rho, cfg.k_fix, policy)
    assert gpu["status"] == 0
    # query clustering (Eq. 2)
    assert np.array_equal(gpu["assign"], ref["q"]["assign"])
    assert np.array_equal(gpu["counts"], ref["q"]["counts"])
    assert np.array_equal(gpu["offsets"], ref["q"]["offsets"])
    assert np.array_equal(gpu["perm"], ref["q"]["perm"])
    assert np.array_equal(gpu["centroids"].view(np.uint32),
                          ref["q"]["centroids"].view(np.uint32))
    # key subspaces (Eq. 3-4)
    assert np.array_equal(gpu["codes"], ref["k"]["codes"])
    assert np.array_equal(gpu["k_centroids"].view(np.uint32),
                          ref["k"]["centroids"].view(np.uint32))
    # tables and proxy logits (Eq. 5-6)
    assert np.array_equal(gpu["tables"].view(np.uint32), ref["tables"].view(np.uint32))
    assert np.array_equal(gpu["scores"].view(np.uint32), ref["scores"].view(np.uint32))
    # selection (Eq. 7-10)
    G.assert_same_selection(gpu, ref["sel"])
    # attention (Eq. 11) against fp64 on the same bf16 operands
    qr, kr, vr = (G.bf16_round(a) for a in (x.q, x.k, x.v))
    att = oracle.attention(qr, kr, vr, ref["q"]["offsets"], ref["q"]["perm"],
                           ref["sel"]["sel_counts"], ref["sel"]["sel_idx"])
    mx, mr = G.assert_attention_close(gpu["out"], att)
    G.say(f"[parity] {cfg.name}: attention max-abs {mx:.3e} mean-rel {mr:.3e}; "
          f"k_head {gpu['k_head'].tolist()}")
    return gpu, ref


def test_fixexp_matches_oracle_exhaustively():
    """Every fp32 y in [-28, 0] (and a band below): GPU == oracle, bit for bit."""
    lo = 0x80000000
    hi = int(np.float32(-30.0).view(np.uint32))
    step = 1 << 26
    for start in range(lo, hi + 1, step):
        bits = np.arange(start, min(start + step, hi + 1), dtype=np.uint32)
        y = bits.view(np.float32)
        yd = torch.from_numpy(y).cuda()
        out = torch.empty(y.size, dtype=torch.int64, device="cuda")
        B.scope_debug_fixexp(yd, out)
        got = out.cpu().numpy().view(np.uint64)
        want = oracle.fixexp(y)
        bad = np.flatnonzero(got != want)
        assert bad.size == 0, (y[bad[:5]], got[bad[:5]], want[bad[:5]])
    G.say("[parity] fixexp: all fp32 in [-30, 0] identical")


def test_tiny_layer():
    check_layer(inputs.CONFIGS["tiny"])


def test_mid_layer_hunyuan_split_ragged():
    check_layer(MID_HY)


def test_mid_layer_wan_split():
    check_layer(MID_WAN)


def test_paper_operating_point_cluster_counts():
    check_layer(PAPER_POINT)


def test_mid_layer_d64_bf16():
    check_layer(MID_D64)


@pytest.mark.parametrize("policy", ["fixed", "topp"])
def test_selection_policies_of_the_ablation(policy):
    # the Fig. 6 variants: fixed floor without top-up, pure Top-p
    gpu, ref = check_layer(MID_HY.with_(name=f"mid_{policy}"), policy=policy)
    want = ref["sel"]["base_counts"] if policy == "fixed" else ref["sel"]["topp"]
    assert np.array_equal(gpu["sel_counts"], want)


@pytest.mark.parametrize("rho", [0.5, 0.95])
def test_mid_layer_stress_temperatures(rho):
    # per-head temperatures on Q spread the proxy softmax from flat to peaked
    check_layer(MID_HY.with_(name=f"mid_stress_{rho}", stress=True, rho=rho, seed=11))


def test_selection_from_materialised_scores_is_identical():
    cfg = MID_HY
    x = inputs.generate(cfg)
    a = G.run_gpu(G.make_layer(cfg), x, use_scores=False)
    b = G.run_gpu(G.make_layer(cfg), x, use_scores=True)
    for key in ("base", "topp", "k_head", "sel_counts", "out"):
        assert np.array_equal(a[key], b[key]), key
    r = a["sel_counts"]
    for h, c in np.ndindex(r.shape):
        assert np.array_equal(a["sel_idx"][h, c, :r[h, c]], b["sel_idx"][h, c, :r[h, c]])


def test_layer_is_deterministic():
    cfg = MID_HY
    x = inputs.generate(cfg)
    layer = G.make_layer(cfg)
    a = G.run_gpu(layer, x)
    b = G.run_gpu(layer, x)
    for key, va in a.items():
        if isinstance(va, np.ndarray):
            assert np.array_equal(va.view(np.uint8), b[key].view(np.uint8)), key


def test_rho_one_keeps_every_key_and_equals_dense_mode():
    cfg = MID_HY.with_(rho=1.0, heads=1)
    x = inputs.generate(cfg)
    gpu = G.run_gpu(G.make_layer(cfg), x)
    assert (gpu["sel_counts"] == cfg.n).all()
    assert (gpu["sel_idx"] == np.arange(cfg.n)).all()
    q, k, v = G.to_device(x)
    dense = DenseAttention(1, cfg.n, cfg.d, "bf16").forward(q, k, v)
    torch.cuda.synchronize()
    # identical key tiles in identical order: bit-identical to dense mode
    assert np.array_equal(gpu["out"], dense.float().cpu().numpy())
    ref = oracle.dense_attention(x.q, x.k, x.v)
    G.assert_attention_close(gpu["out"], ref)


def test_single_selected_key_returns_its_value():
    cfg = MID_HY.with_(rho=1e-7, k_fix=1, heads=1)
    x = inputs.generate(cfg)
    gpu = G.run_gpu(G.make_layer(cfg), x)
    assert (gpu["sel_counts"] == 1).all() and (gpu["k_head"] == 1).all()
    perm, off = gpu["perm"][0], gpu["offsets"][0]
    for c in range(cfg.c_q):
        j = gpu["sel_idx"][0, c, 0]
        rows = perm[off[c]:off[c + 1]]
        assert np.array_equal(gpu["out"][0, rows], np.repeat(x.v[0, j][None], len(rows), 0))


def test_empty_clusters():
    # many duplicate query rows: equal starting centroids tie and the higher
    # index never wins, so some clusters stay empty (n_c = 0)
    cfg = MID_WAN.with_(name="dups", c_q=24)
    x = inputs.generate(cfg)
    rng = np.random.default_rng(3)
    proto = x.q[0, rng.choice(cfg.n, 6, replace=False)]
    x.q[0] = proto[rng.integers(0, 6, cfg.n)]
    x.q_bits[0] = inputs.bf16_bits(x.q[0])
    gpu, ref = check_layer_inputs(cfg, x)
    assert (gpu["counts"] == 0).any()


def check_layer_inputs(cfg, x):
    layer = G.make_layer(cfg)
    gpu = G.run_gpu(layer, x)
    ref = G.oracle_all(x, cfg.c_q, (cfg.c_m,) * 3, cfg.iters, cfg.rho, cfg.k_fix)
    assert np.array_equal(gpu["assign"], ref["q"]["assign"])
    assert np.array_equal(gpu["perm"], ref["q"]["perm"])
    assert np.array_equal(gpu["centroids"].view(np.uint32),
                          ref["q"]["centroids"].view(np.uint32))
    assert np.array_equal(gpu["codes"], ref["k"]["codes"])
    G.assert_same_selection(gpu, ref["sel"])
    qr, kr, vr = (G.bf16_round(a) for a in (x.q, x.k, x.v))
    att = oracle.attention(qr, kr, vr, ref["q"]["offsets"], ref["q"]["perm"],
                           ref["sel"]["sel_counts"], ref["sel"]["sel_idx"])
    G.assert_attention_close(gpu["out"], att)
    return gpu, ref


@pytest.mark.parametrize("d,n", [(64, 700), (128, 1000)])
def test_dense_mode_matches_oracle(d, n):
    rng = np.random.default_rng(d + n)
    qkv = [G.bf16_round(rng.standard_normal((2, n, d)).astype(np.float32) * s)
           for s in (1.5, 1.5, 1.0)]
    dev = [torch.from_numpy(a).cuda().to(torch.bfloat16) for a in qkv]
    out = DenseAttention(2, n, d, "bf16").forward(*dev).float().cpu().numpy()
    ref = oracle.dense_attention(*qkv)
    mx, mr = G.assert_attention_close(out, ref)
    G.say(f"[parity] dense d={d} n={n}: max-abs {mx:.3e} mean-rel {mr:.3e}")


def _partition_case(cfg, kind, c_m, seed=1):
    x = inputs.generate(cfg)
    sets = inputs.partition_sets(cfg, kind, seed)
    M = len(sets)
    init_k = (x.init_k if kind == "3-rope" and max(c_m) <= cfg.c_m
              else inputs.partition_init(cfg, M, max(c_m)))
    G.say(f"[parity] partition {kind}: M={M} c_m={list(c_m)} sizes={[len(s) for s in sets]}")
    gpu = G.run_gpu(G.make_partition_layer(cfg, sets, c_m), x, init_k=init_k)
    ref = oracle.layer_partition(x.q, x.k, x.v, sets, cfg.c_q, c_m, cfg.iters, x.init_q,
                                 init_k, cfg.rho, cfg.k_fix)
    assert gpu["status"] == 0
    assert np.array_equal(gpu["perm"], ref["q"]["perm"])
    assert np.array_equal(gpu["codes"], ref["k"]["codes"])
    assert np.array_equal(gpu["k_centroids"].view(np.uint32),
                          ref["k"]["centroids"].view(np.uint32))
    assert np.array_equal(gpu["tables"].view(np.uint32), ref["tables"].view(np.uint32))
    assert np.array_equal(gpu["scores"].view(np.uint32), ref["scores"].view(np.uint32))
    G.assert_same_selection(gpu, ref["sel"])
    qr, kr, vr = (G.bf16_round(a) for a in (x.q, x.k, x.v))
    att = oracle.attention(qr, kr, vr, ref["q"]["offsets"], ref["q"]["perm"],
                           ref["sel"]["sel_counts"], ref["sel"]["sel_idx"])
    mx, mr = G.assert_attention_close(gpu["out"], att)
    G.say(f"[parity] partition {kind}: attention max-abs {mx:.3e} mean-rel {mr:.3e}")
    return gpu, x


@pytest.mark.parametrize("kind,c_m", [
    ("1", (40,)), ("2", (16, 24)), ("3-random", (20, 40, 33)), ("3-rope", (16, 16, 16)),
    ("4", (16,) * 4), ("8", (5, 9, 16, 33, 7, 12, 16, 3)), ("1", (333,)),
])
def test_key_partitions_of_the_ablation(kind, c_m):
    # Table 3 variants: any disjoint channel sets, M <= 8, codebooks of any
    # size (C = 333 over all 128 channels takes the matrix-core assignment
    # with the codebook split into two LDS chunks)
    _partition_case(MID_HY, kind, c_m)


def test_rope_partition_equals_the_three_range_calls():
    cfg = MID_HY
    gpu_p, x = _partition_case(cfg, "3-rope", (cfg.c_m,) * 3)
    gpu_r = G.run_gpu(G.make_layer(cfg), x)
    packed = gpu_r["codes"]
    planes = np.stack([(packed >> (10 * m)) & 1023 for m in range(3)], 1).astype(np.uint16)
    assert np.array_equal(gpu_p["codes"], planes)
    for key in ("k_centroids", "tables", "scores", "sel_counts", "out"):
        assert np.array_equal(gpu_p[key], gpu_r[key]), key
    # entries past r_c are left untouched by selection
    r = gpu_r["sel_counts"]
    for h, c in np.ndindex(r.shape):
        assert np.array_equal(gpu_p["sel_idx"][h, c, :r[h, c]], gpu_r["sel_idx"][h, c, :r[h, c]])


def test_partition_selection_from_codes_equals_from_scores():
    cfg = MID_WAN
    x = inputs.generate(cfg)
    sets = inputs.partition_sets(cfg, "3-random", 2)
    init_k = inputs.partition_init(cfg, 3, cfg.c_m)
    a = G.run_gpu(G.make_partition_layer(cfg, sets, (cfg.c_m,) * 3), x, init_k=init_k)
    b = G.run_gpu(G.make_partition_layer(cfg, sets, (cfg.c_m,) * 3), x, use_scores=True,
                  init_k=init_k)
    for key in ("base", "topp", "k_head", "sel_counts", "out"):
        assert np.array_equal(a[key], b[key]), key
    r = a["sel_counts"]
    for h, c in np.ndindex(r.shape):
        assert np.array_equal(a["sel_idx"][h, c, :r[h, c]], b["sel_idx"][h, c, :r[h, c]])


def _queries_case(cfg, x):
    layer = G.make_layer(cfg)
    q, _, _ = G.to_device(x)
    layer.cluster_queries(q, torch.from_numpy(x.init_q).cuda())
    torch.cuda.synchronize()
    ref = oracle.cluster_queries(x.q, cfg.c_q, cfg.iters, x.init_q)
    assert int(layer.status.item()) == 0
    assert np.array_equal(layer.assign.cpu().numpy(), ref["assign"])
    assert np.array_equal(layer.perm.cpu().numpy(), ref["perm"])
    assert np.array_equal(layer.q_centroids.cpu().numpy().view(np.uint32),
                          ref["centroids"].view(np.uint32))
    return ref


@pytest.mark.parametrize("d,c_q", [(128, 300), (64, 600), (128, 1000)])
def test_codebooks_streamed_through_lds_in_chunks(d, c_q):
    # bf16 codebooks beyond the assignment kernel's LDS: 300 x 128 (two
    # chunks), 600 x 64 (a ragged last chunk), 1000 x 128 (four chunks)
    split = (16, 56, 56) if d == 128 else (16, 24, 24)
    cfg = MID_HY.with_(name=f"chunked_{d}_{c_q}", d=d, split=split, c_q=c_q, heads=2,
                       iters=4, seed=13)
    G.say(f"[parity] chunked codebook d={d} c_q={c_q} n={cfg.n}")
    _queries_case(cfg, inputs.generate(cfg))


def test_chunked_codebook_with_tied_centroids():
    # six distinct query rows repeated: hundreds of equal centroids, so
    # points have four or more tied candidates and scan every centroid
    cfg = MID_HY.with_(name="chunked_ties", c_q=300, heads=1, iters=3, seed=17)
    x = inputs.generate(cfg)
    rng = np.random.default_rng(5)
    proto = x.q[0, rng.choice(cfg.n, 6, replace=False)]
    x.q[0] = proto[rng.integers(0, 6, cfg.n)]
    x.q_bits[0] = inputs.bf16_bits(x.q[0])
    ref = _queries_case(cfg, x)
    assert (ref["counts"] == 0).sum() >= 290


_select_from_codes = G.select_from_codes


def test_selection_with_heavily_shared_codes():
    """The passes over distinct codes weight each by its key count: 20000 keys
    sharing 300 codes give the oracle's sets exactly."""
    rng = np.random.default_rng(21)
    H, C, n, d, c_m = 2, 6, 20000, 64, (32, 32, 64)
    tables = rng.standard_normal((H, C, sum(c_m))).astype(np.float32) * 4
    pool = (rng.integers(0, c_m[0], 300) | (rng.integers(0, c_m[1], 300) << 10)
            | (rng.integers(0, c_m[2], 300) << 20)).astype(np.uint32)
    codes = pool[rng.integers(0, 300, (H, n))]
    counts = rng.multinomial(n, np.ones(C) / C, size=H).astype(np.int32)
    _select_from_codes(tables, codes, counts, d, c_m, 0.9, (n + 9) // 10)


def test_selection_when_one_dedup_part_overflows():
    """Head 0's 40000 distinct codes all hash to the same part of the
    distinct-code build (more than its table holds): that head falls back to
    one entry per key; head 1 (ordinary codes) keeps the distinct list.  Both
    must give the oracle's sets."""
    rng = np.random.default_rng(22)
    H, C, n, d, c_m = 2, 4, 40000, 64, (1024, 1024, 1024)
    parts = (5 * n + 4 * 16384 - 1) // (4 * 16384)  # the build's part count
    cand = np.arange(0, 1 << 22, dtype=np.uint64)
    hv = (cand * np.uint64(0x9E3779B1)) & np.uint64(0xFFFFFFFF)
    same_part = cand[((hv * np.uint64(parts)) >> np.uint64(32)) == 0][:n].astype(np.uint32)
    assert same_part.size == n
    codes = np.empty((H, n), np.uint32)
    codes[0] = rng.permutation(same_part)
    codes[1] = rng.integers(0, 1 << 30, n, dtype=np.uint32) & np.uint32(0x000FFFFF)
    tables = rng.standard_normal((H, C, sum(c_m))).astype(np.float32) * 3
    counts = rng.multinomial(n, np.ones(C) / C, size=H).astype(np.int32)
    _select_from_codes(tables, codes, counts, d, c_m, 0.7, (n + 9) // 10)


def test_selection_beyond_the_distinct_code_limit():
    """Above 262144 keys the selection passes visit every key instead of the
    distinct codes: 270000 keys, codes from a small pool, against the oracle."""
    rng = np.random.default_rng(23)
    H, C, n, d, c_m = 1, 4, 270000, 64, (16, 16, 32)
    tables = rng.standard_normal((H, C, sum(c_m))).astype(np.float32) * 2
    codes = (rng.integers(0, c_m[0], (H, n)) | (rng.integers(0, c_m[1], (H, n)) << 10)
             | (rng.integers(0, c_m[2], (H, n)) << 20)).astype(np.uint32)
    counts = rng.multinomial(n, np.ones(C) / C, size=H).astype(np.int32)
    _select_from_codes(tables, codes, counts, d, c_m, 0.8, (n + 9) // 10)


def test_selection_between_the_merged_and_the_class_bit_limits():
    """130000 keys, every code distinct: the final kernel keeps the class
    bits (up to 163840 codes) but has too many codes for the single pass that
    also lists the rank crossing's candidates (up to 98304), so rows that
    search their crossing gather it, run the digit rounds and classify in a
    second pass.  Against the oracle."""
    rng = np.random.default_rng(25)
    H, C, n, d, c_m = 1, 6, 130000, 64, (64, 64, 64)
    flat = rng.permutation(64 ** 3)[:n].astype(np.uint32)
    codes = ((flat % 64) | (((flat // 64) % 64) << 10) | ((flat // 4096) << 20)).reshape(H, n)
    assert 98304 < np.unique(codes).size == n <= 163840
    tables = rng.standard_normal((H, C, sum(c_m))).astype(np.float32) * 2
    counts = rng.multinomial(n, np.ones(C) / C, size=H).astype(np.int32)
    gpu = _select_from_codes(tables, codes.astype(np.uint32), counts, d, c_m, 0.8, (n + 9) // 10)
    # some rows search their own crossing (r_c differs from the Top-p count)
    assert (gpu["sel_counts"] != gpu["topp"]).any()


def test_selection_with_more_distinct_codes_than_the_class_bits_hold():
    """200000 keys, every code distinct: the distinct-code passes run (16
    parts), but the final compaction's LDS class bits cover 163840 codes, so
    it classifies each key from its own logit instead.  Against the oracle."""
    rng = np.random.default_rng(24)
    H, C, n, d, c_m = 1, 4, 200000, 64, (64, 64, 64)
    flat = rng.permutation(64 ** 3)[:n].astype(np.uint32)
    codes = ((flat % 64) | (((flat // 64) % 64) << 10) | ((flat // 4096) << 20)).reshape(H, n)
    assert np.unique(codes).size == n > 163840
    tables = rng.standard_normal((H, C, sum(c_m))).astype(np.float32) * 2
    counts = rng.multinomial(n, np.ones(C) / C, size=H).astype(np.int32)
    _select_from_codes(tables, codes.astype(np.uint32), counts, d, c_m, 0.8, (n + 9) // 10)


def test_points_at_exactly_zero_score():
    """A point whose score against its best centroid is exactly zero (centroid
    u = (2, 0, ...), point x = (1, 5, 0, ...): |u|^2 - 2<x, u> = 0) packs its
    index into a zero, i.e. a denormal.  The matrix-core assignment must still
    return that index (regression: scaling the packed value by -2 shifted a
    denormal's mantissa and doubled the index)."""
    cfg = MID_WAN.with_(name="zero_score", c_q=16, c_m=8, iters=2, seed=31)
    x = inputs.generate(cfg)
    (t_off, h_off, w_off), (t_len, h_len, w_len) = cfg.ranges

    def plant(a, bits, lo, ln):
        # row 0 -> (2, 0, ...) and row 1 -> (1, 5, 0, ...) on channels [lo, lo + ln)
        a[0, 0, lo:lo + ln] = 0.0
        a[0, 1, lo:lo + ln] = 0.0
        a[0, 0, lo] = 2.0
        a[0, 1, lo] = 1.0
        a[0, 1, lo + 1] = 5.0
        bits[0] = inputs.bf16_bits(a[0])

    plant(x.q, x.q_bits, 0, cfg.d)
    for lo, ln in ((t_off, t_len), (h_off, h_len), (w_off, w_len)):
        plant(x.k, x.k_bits, lo, ln)
    # centroid 1 starts at row 0; no other start row is 0 or 1
    def starts(row, c):
        others = [r for r in row.tolist() if r not in (0, 1)]
        extra = [r for r in range(2, cfg.n) if r not in others]
        out = [others.pop(0) if others else extra.pop(0) for _ in range(c)]
        out[1] = 0
        return np.asarray(out, np.int32)
    x.init_q[0] = starts(x.init_q[0], cfg.c_q)
    for m in range(3):
        x.init_k[0, m] = starts(x.init_k[0, m], cfg.c_m)
    gpu, ref = check_layer_inputs(cfg, x)
    assert ref["q"]["assign"][0, 1] == 1 or ref["q"]["counts"][0, 1] > 0


def test_exact_two_and_three_way_ties():
    """Exact ties in the first assignment, in the query clustering and in every
    key subspace.  Centroid 5 starts at e0, centroid 2 at e1 and centroid 7
    at -e0 (unit vectors on the first two channels of the range).  The zero
    point then scores exactly 1 against all three (three candidates within
    the matrix-core margin: the full re-scoring path).  e0 + e1 scores
    exactly -1 against centroids 5 and 2 (two candidates: the two half-wave
    lanes re-score one each).  The canonical rule (lowest index: 2 both
    times) must win; a wrong pick moves the centroids and fails the
    bit-exact comparison."""
    cfg = MID_WAN.with_(name="exact_ties", c_q=16, c_m=8, iters=2, seed=37)
    x = inputs.generate(cfg)
    (t_off, h_off, w_off), (t_len, h_len, w_len) = cfg.ranges

    def plant(a, bits, lo, ln):
        rows = {0: (1.0, 0.0), 1: (0.0, 1.0), 2: (-1.0, 0.0), 3: (0.0, 0.0), 4: (1.0, 1.0)}
        for r, (v0, v1) in rows.items():
            a[0, r, lo:lo + ln] = 0.0
            a[0, r, lo] = v0
            a[0, r, lo + 1] = v1
        bits[0] = inputs.bf16_bits(a[0])

    plant(x.q, x.q_bits, 0, cfg.d)
    for lo, ln in ((t_off, t_len), (h_off, h_len), (w_off, w_len)):
        plant(x.k, x.k_bits, lo, ln)

    def starts(row, c):
        # slots 5, 2, 7 start at rows 0, 1, 2; no other slot starts at rows 0-4
        others = [r for r in row.tolist() if r > 4]
        extra = [r for r in range(5, cfg.n) if r not in others]
        out = [others.pop(0) if others else extra.pop(0) for _ in range(c)]
        out[5], out[2], out[7] = 0, 1, 2
        return np.asarray(out, np.int32)

    x.init_q[0] = starts(x.init_q[0], cfg.c_q)
    for m in range(3):
        x.init_k[0, m] = starts(x.init_k[0, m], cfg.c_m)
    check_layer_inputs(cfg, x)


@pytest.mark.parametrize("grid,d,split,c_q,c_m,k_fix,dtype", [
    ((1, 1, 7), 64, (16, 24, 24), 3, 2, 2, "bf16"),       # fewer keys than a wave slice
    ((1, 3, 5), 64, (16, 24, 24), 1, 1, 1, "bf16"),       # one query cluster, one centroid per subspace
    ((1, 2, 9), 128, (16, 56, 56), 18, 18, 18, "bf16"),   # as many clusters as tokens, k_fix = N
    ((2, 3, 11), 64, (16, 24, 24), 5, 4, 66, "f32"),      # k_fix = N keeps every key
    ((3, 7, 13), 128, (44, 42, 42), 7, 5, 1, "bf16"),     # k_fix = 1, ragged tiles everywhere
])
def test_extreme_small_shapes(grid, d, split, c_q, c_m, k_fix, dtype):
    n = grid[0] * grid[1] * grid[2]
    cfg = inputs.LayerConfig(f"edge_{n}_{c_q}_{c_m}", 2, grid, d, split, c_q, c_m, 2, 0.9,
                             k_fix, dtype, 2, 40 + n)
    gpu, ref = check_layer(cfg)
    if k_fix == n:
        assert (gpu["sel_counts"] == n).all()


def _attention_case(sizes, keys, heads=2, d=128, seed=0):
    """Sparse attention on a given clustering (cluster sizes, per cluster a
    key count) with random permutation and random ascending key sets."""
    rng = np.random.default_rng(seed)
    n = int(sum(sizes))
    c_q = len(sizes)
    qkv = [G.bf16_round(rng.standard_normal((heads, n, d)).astype(np.float32) * s)
           for s in (1.5, 1.5, 1.0)]
    offsets = np.zeros((heads, c_q + 1), np.int32)
    offsets[:, 1:] = np.cumsum(sizes)
    perm = np.stack([rng.permutation(n) for _ in range(heads)]).astype(np.int32)
    sel_counts = np.zeros((heads, c_q), np.int32)
    sel_idx = np.zeros((heads, c_q, n), np.int32)
    for h in range(heads):
        for c, r in enumerate(keys):
            r = int(min(r, n))
            sel_counts[h, c] = r
            sel_idx[h, c, :r] = np.sort(rng.choice(n, r, replace=False))
    shape = B.make_shape(heads, n, d, B.BF16, ((0, 16, 72), (16, 56, 56)))
    dev = [torch.from_numpy(a).cuda().to(torch.bfloat16) for a in qkv]
    o = torch.empty_like(dev[0])
    # the attention call needs only its work list: two 16-byte entries per
    # slot, heads * (ceil(n / 256) + c_q) slots (clustering with this many
    # clusters is beyond the workspace-size call)
    ws = torch.empty(2 * heads * (-(-n // 256) + c_q) * 16 + 256, dtype=torch.uint8,
                     device="cuda")
    t = lambda a: torch.from_numpy(a).cuda()
    B.scope_sparse_attention(shape, *dev, c_q, t(offsets), t(perm), t(sel_counts),
                             t(sel_idx), 0.0, o, ws)
    torch.cuda.synchronize()
    ref = oracle.attention(*qkv, offsets, perm, sel_counts, sel_idx)
    return G.assert_attention_close(o.float().cpu().numpy(), ref)


def test_attention_pairs_remainder_chunks_of_every_width():
    # clusters with 0-2 full 256-query chunks and remainders of every wave
    # count 1..8 (1 .. 255 rows), several per count, with equal, close and
    # very different key counts, so that the work list pairs remainders of
    # complementary widths, leaves some alone and runs pairs whose key
    # lists end at different tiles
    rems = [1, 17, 32, 33, 60, 64, 65, 96, 97, 100, 128, 129, 150, 160, 161, 192,
            193, 200, 224, 225, 240, 255, 5, 31, 70, 130, 190, 230, 40, 250, 3, 120]
    sizes = [256 * (i % 3) + rm for i, rm in enumerate(rems)]
    pool = [1, 63, 64, 65, 640, 640, 640, 641, 700, 1000, 2049, 5000]
    keys = [pool[(7 * i) % len(pool)] for i in range(len(sizes))]
    mx, mr = _attention_case(sizes, keys)
    G.say(f"[parity] paired work slots: max-abs {mx:.3e} mean-rel {mr:.3e}")


def test_attention_remainders_alone_above_the_pairing_limit():
    # more clusters than the work list pairs (2,048): every remainder chunk
    # runs alone, after the full chunks
    rng = np.random.default_rng(11)
    sizes = [int(x) for x in rng.integers(0, 9, 2100)]
    sizes[5], sizes[700] = 300, 600
    keys = [int(x) for x in rng.integers(1, 200, 2100)]
    mx, mr = _attention_case(sizes, keys, heads=1, seed=2)
    G.say(f"[parity] {len(sizes)} clusters, unpaired remainders: max-abs {mx:.3e} mean-rel {mr:.3e}")
