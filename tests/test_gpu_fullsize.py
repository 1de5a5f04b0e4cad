"""Full-size parity in the benchmark's launch configuration.

The whole layer runs on every head of a 480p/720p workload exactly as
bench.py runs it; the oracle then recomputes sampled heads end to end
(clustering, tables, logits, selection: bit-exact) and attention for sampled
query rows (tolerance).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle  # noqa: E402
from paper_2608_12780_amd import inputs  # noqa: E402
from paper_2608_12780_amd.layer import ScopeLayer  # noqa: E402

import gpu_harness as G  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()


@pytest.mark.parametrize("name,heads", [("hy720", (13, 2)), ("wan720", (7,)), ("wan480", (31,))])
def test_full_size_layer_sampled_heads(name, heads):
    cfg = inputs.CONFIGS[name]
    G.say(f"[fullsize] {name}: heads={cfg.heads} n={cfg.n} split={cfg.split}; "
          f"oracle heads {heads}")
    x = inputs.generate(cfg)
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype)
    q, k, v = G.to_device(x)
    layer.forward(q, k, v, torch.from_numpy(x.init_q).cuda(),
                  torch.from_numpy(x.init_k).cuda())
    torch.cuda.synchronize()
    assert int(layer.status.item()) == 0
    gpus = {}
    for head in heads:
        g = lambda t: t[head:head + 1].cpu().numpy()
        gpus[head] = dict(assign=g(layer.assign), counts=g(layer.counts), offsets=g(layer.offsets),
                          perm=g(layer.perm), centroids=g(layer.q_centroids),
                          k_centroids=g(layer.k_centroids), codes=g(layer.codes).view(np.uint32),
                          tables=g(layer.tables), base=g(layer.base_counts),
                          topp=g(layer.topp_counts), k_head=g(layer.k_head),
                          sel_counts=g(layer.sel_counts), sel_idx=g(layer.sel_idx),
                          out=layer.out[head:head + 1].float().cpu().numpy())
    del layer, q, k, v
    torch.cuda.empty_cache()
    G.say(f"[fullsize] {name}: GPU layer done")
    for head in heads:
        check_head(cfg, x, head, gpus.pop(head), name)


def check_head(cfg, x, head, gpu, name):
    G.say(f"[fullsize] {name}: oracle on head {head}")
    hq, hk, hv = x.q[head:head + 1], x.k[head:head + 1], x.v[head:head + 1]
    cm = (cfg.c_m,) * 3
    qr = oracle.cluster_queries(hq, cfg.c_q, cfg.iters, x.init_q[head:head + 1])
    assert np.array_equal(gpu["assign"], qr["assign"])
    assert np.array_equal(gpu["counts"], qr["counts"])
    assert np.array_equal(gpu["offsets"], qr["offsets"])
    assert np.array_equal(gpu["perm"], qr["perm"])
    assert np.array_equal(gpu["centroids"].view(np.uint32), qr["centroids"].view(np.uint32))
    kr = oracle.cluster_key_subspaces(hk, cfg.ranges, cm, cfg.iters, x.init_k[head:head + 1])
    assert np.array_equal(gpu["codes"], kr["codes"])
    assert np.array_equal(gpu["k_centroids"].view(np.uint32), kr["centroids"].view(np.uint32))
    P = oracle.tables(qr["centroids"], kr["centroids"], cfg.ranges, cm)
    assert np.array_equal(gpu["tables"].view(np.uint32), P.view(np.uint32))
    S = oracle.proxy_scores(P, kr["codes"], cfg.d, cm)
    sel = oracle.select(S, qr["counts"], cfg.rho, cfg.k_fix)
    del S
    G.assert_same_selection(gpu, sel)
    G.say(f"[fullsize] {name}: head {head} clustering, tables and selection bit-exact; "
          f"k_head {int(gpu['k_head'][0])}")

    # attention for 4 x 32 sampled rows of 4 sampled clusters
    rng = np.random.default_rng(head)
    counts = qr["counts"][0]
    clusters = rng.choice(np.flatnonzero(counts > 0), 4, replace=False)
    mask = np.zeros((1, cfg.n), np.uint8)
    off, perm = qr["offsets"][0], qr["perm"][0]
    for c in clusters:
        members = perm[off[c]:off[c + 1]]
        mask[0, rng.choice(members, min(32, len(members)), replace=False)] = 1
    ref = oracle.attention(hq, hk, hv, qr["offsets"], qr["perm"], sel["sel_counts"],
                           sel["sel_idx"], row_mask=mask)
    rows = np.flatnonzero(mask[0])
    mx, mr = G.assert_attention_close(gpu["out"][0, rows], ref[0, rows])
    G.say(f"[fullsize] {name}: head {head} attention on {len(rows)} rows max-abs {mx:.3e} "
          f"mean-rel {mr:.3e}")


def test_full_size_paper_operating_point():
    # C_q = 300 and C_m = 333 at the HunyuanVideo-720p-like shape: the query
    # codebook is streamed through LDS in chunks
    cfg = inputs.CONFIGS["hy720"].with_(c_q=300, c_m=333, heads=3)
    G.say(f"[fullsize] paper point: heads={cfg.heads} n={cfg.n} c_q=300 c_m=333")
    x = inputs.generate(cfg)
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype)
    q, k, v = G.to_device(x)
    layer.forward(q, k, v, torch.from_numpy(x.init_q).cuda(),
                  torch.from_numpy(x.init_k).cuda())
    torch.cuda.synchronize()
    assert int(layer.status.item()) == 0
    head = 1
    g = lambda t: t[head:head + 1].cpu().numpy()
    gpu = dict(assign=g(layer.assign), counts=g(layer.counts), offsets=g(layer.offsets),
               perm=g(layer.perm), centroids=g(layer.q_centroids),
               k_centroids=g(layer.k_centroids), codes=g(layer.codes).view(np.uint32),
               tables=g(layer.tables), base=g(layer.base_counts), topp=g(layer.topp_counts),
               k_head=g(layer.k_head), sel_counts=g(layer.sel_counts), sel_idx=g(layer.sel_idx),
               out=layer.out[head:head + 1].float().cpu().numpy())
    del layer, q, k, v
    torch.cuda.empty_cache()
    check_head(cfg, x, head, gpu, "paper point")


def test_full_size_random_partition():
    # a random three-way channel split (the gather path) with 333 centroids
    # per subspace, full HunyuanVideo-720p-like size, two heads
    from paper_2608_12780_amd.layer import ScopePartitionLayer
    cfg = inputs.CONFIGS["hy720"].with_(c_q=300, c_m=333, heads=2)
    sets = inputs.partition_sets(cfg, "3-random")
    init_k = inputs.partition_init(cfg, 3, 333)
    G.say(f"[fullsize] random partition: sizes {[len(s) for s in sets]}")
    x = inputs.generate(cfg)
    layer = ScopePartitionLayer(cfg.heads, cfg.n, cfg.d, sets, cfg.c_q, (333,) * 3,
                                cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype)
    q, k, v = G.to_device(x)
    layer.forward(q, k, v, torch.from_numpy(x.init_q).cuda(), torch.from_numpy(init_k).cuda())
    torch.cuda.synchronize()
    assert int(layer.status.item()) == 0
    head = 0
    g = lambda t: t[head:head + 1].cpu().numpy()
    codes, kcen, tables = g(layer.codes).view(np.uint16), g(layer.k_centroids), g(layer.tables)
    counts, qcen = g(layer.counts), g(layer.q_centroids)
    gsel = dict(base=g(layer.base_counts), topp=g(layer.topp_counts), k_head=g(layer.k_head),
                sel_counts=g(layer.sel_counts), sel_idx=g(layer.sel_idx))
    del layer, q, k, v
    torch.cuda.empty_cache()
    hk = x.k[head:head + 1]
    qr = oracle.cluster_queries(x.q[head:head + 1], cfg.c_q, cfg.iters, x.init_q[head:head + 1])
    assert np.array_equal(counts, qr["counts"])
    assert np.array_equal(qcen.view(np.uint32), qr["centroids"].view(np.uint32))
    kr = oracle.cluster_key_partition(hk, sets, (333,) * 3, cfg.iters, init_k[head:head + 1])
    assert np.array_equal(codes, kr["codes"])
    assert np.array_equal(kcen.view(np.uint32), kr["centroids"].view(np.uint32))
    P = oracle.tables_partition(qr["centroids"], kr["centroids"], sets, (333,) * 3)
    assert np.array_equal(tables.view(np.uint32), P.view(np.uint32))
    S = oracle.proxy_scores_partition(P, kr["codes"], cfg.d, (333,) * 3)
    sel = oracle.select(S, qr["counts"], cfg.rho, cfg.k_fix)
    del S
    G.assert_same_selection(gsel, sel)
    G.say(f"[fullsize] random partition: head {head} bit-exact, k_head {int(gsel['k_head'][0])}")


@pytest.mark.parametrize("name", ["hy720", "wan720"])
def test_full_size_every_head_matrix_core_assignment_is_canonical(name):
    """Every head at full size: the bf16 clustering (matrix-core assignment,
    exact by its filter and canonical re-score) against the same clustering
    of the bf16 values widened to fp32, which takes the plain canonical
    fp32 assignment kernel.  Query assignments, centroids, permutation and
    key codes and centroids must be identical on all heads."""
    cfg = inputs.CONFIGS[name]
    G.say(f"[fullsize] {name}: every head, matrix-core vs canonical assignment")
    x = inputs.generate(cfg)
    iq = torch.from_numpy(x.init_q).cuda()
    ik = torch.from_numpy(x.init_k).cuda()
    res = {}
    for dtype in ("bf16", "f32"):
        layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                           cfg.iters, cfg.rho, cfg.k_fix, dtype=dtype)
        if dtype == "bf16":
            q, k, _ = G.to_device(x)
        else:
            q, k = torch.from_numpy(x.q).cuda(), torch.from_numpy(x.k).cuda()
        layer.cluster_queries(q, iq)
        layer.cluster_keys(k, ik)
        torch.cuda.synchronize()
        assert int(layer.status.item()) == 0
        res[dtype] = {key: getattr(layer, key).cpu().numpy() for key in
                      ("assign", "counts", "perm", "q_centroids", "codes", "k_centroids")}
        del layer, q, k
        torch.cuda.empty_cache()
        G.say(f"[fullsize] {name}: {dtype} clustering done")
    for key in res["bf16"]:
        a, b = res["bf16"][key], res["f32"][key]
        bad = np.flatnonzero((a.view(np.uint32) != b.view(np.uint32)).reshape(cfg.heads, -1).any(1))
        assert bad.size == 0, (key, bad.tolist())


def test_full_size_every_head_selection_from_codes_equals_from_scores():
    """Every head of the HunyuanVideo-720p-like layer: the selection fused
    from the tables and codes (passes over each head's distinct codes)
    against the selection from the materialised logits (passes over every
    key).  Counts, k_head and every key set must be identical."""
    cfg = inputs.CONFIGS["hy720"]
    x = inputs.generate(cfg)
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype, materialize_scores=True)
    q, k, _ = G.to_device(x)
    layer.cluster_queries(q, torch.from_numpy(x.init_q).cuda())
    layer.cluster_keys(k, torch.from_numpy(x.init_k).cuda())
    layer.proxy_scores()
    res = []
    for use_scores in (False, True):
        layer.select(use_scores=use_scores)
        torch.cuda.synchronize()
        res.append({key: getattr(layer, key).clone() for key in
                    ("base_counts", "topp_counts", "k_head", "sel_counts")})
        res[-1]["sel_idx"] = layer.sel_idx.clone()
        G.say(f"[fullsize] hy720 selection from {'scores' if use_scores else 'codes'} done")
    a, b = res
    for key in ("base_counts", "topp_counts", "k_head", "sel_counts"):
        assert torch.equal(a[key], b[key]), key
    # compare the valid prefix of every key set on the GPU
    r = a["sel_counts"]
    pos = torch.arange(cfg.n, device=r.device).view(1, 1, -1)
    valid = pos < r.unsqueeze(-1)
    assert torch.equal(torch.where(valid, a["sel_idx"], -1), torch.where(valid, b["sel_idx"], -1))


def test_full_size_stress_every_rho_flattest_and_most_peaked_heads():
    """The selection stress workload at full size (24 heads, N = 118800) in
    the benchmark's launch configuration, for every rho of the sweep.  The
    oracle recomputes the head with the smallest temperature (the flattest
    proxy softmax: the largest Top-p counts and crossing bins) and the one
    with the largest: clustering, tables and selection bit for bit at each
    rho, attention on sampled rows within tolerance."""
    cfg = inputs.CONFIGS["stress"]
    x = inputs.generate(cfg)
    heads = (int(np.argmin(x.tau)), int(np.argmax(x.tau)))
    G.say(f"[fullsize] stress: heads {heads} tau {[round(float(x.tau[h]), 3) for h in heads]}")
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype)
    q, k, v = G.to_device(x)
    layer.cluster_queries(q, torch.from_numpy(x.init_q).cuda())
    layer.cluster_keys(k, torch.from_numpy(x.init_k).cuda())
    layer.proxy_scores()
    torch.cuda.synchronize()
    assert int(layer.status.item()) == 0
    sl = lambda t, h: t[h:h + 1].cpu().numpy()
    clus = {h: dict(assign=sl(layer.assign, h), counts=sl(layer.counts, h),
                    offsets=sl(layer.offsets, h), perm=sl(layer.perm, h),
                    centroids=sl(layer.q_centroids, h), k_centroids=sl(layer.k_centroids, h),
                    codes=sl(layer.codes, h).view(np.uint32), tables=sl(layer.tables, h))
            for h in heads}
    rhos = (0.5, 0.7, 0.9, 0.95)
    sels = {}
    for rho in rhos:
        layer.select(rho=rho)
        layer.attend(q, k, v)
        torch.cuda.synchronize()
        for h in heads:
            sels[h, rho] = dict(base=sl(layer.base_counts, h), topp=sl(layer.topp_counts, h),
                                k_head=sl(layer.k_head, h), sel_counts=sl(layer.sel_counts, h),
                                sel_idx=sl(layer.sel_idx, h),
                                out=layer.out[h:h + 1].float().cpu().numpy())
        G.say(f"[fullsize] stress: GPU rho {rho} done, k_head "
              f"{[int(sels[h, rho]['k_head'][0]) for h in heads]}")
    del layer, q, k, v
    torch.cuda.empty_cache()
    cm = (cfg.c_m,) * 3
    for h in heads:
        gpu = clus.pop(h)
        hq, hk, hv = x.q[h:h + 1], x.k[h:h + 1], x.v[h:h + 1]
        qr = oracle.cluster_queries(hq, cfg.c_q, cfg.iters, x.init_q[h:h + 1])
        for key in ("assign", "counts", "offsets", "perm"):
            assert np.array_equal(gpu[key], qr[key]), key
        assert np.array_equal(gpu["centroids"].view(np.uint32), qr["centroids"].view(np.uint32))
        kr = oracle.cluster_key_subspaces(hk, cfg.ranges, cm, cfg.iters, x.init_k[h:h + 1])
        assert np.array_equal(gpu["codes"], kr["codes"])
        assert np.array_equal(gpu["k_centroids"].view(np.uint32), kr["centroids"].view(np.uint32))
        P = oracle.tables(qr["centroids"], kr["centroids"], cfg.ranges, cm)
        assert np.array_equal(gpu["tables"].view(np.uint32), P.view(np.uint32))
        S = oracle.proxy_scores(P, kr["codes"], cfg.d, cm)
        G.say(f"[fullsize] stress: head {h} clustering and tables bit-exact")
        rng = np.random.default_rng(100 + h)
        counts, off, perm = qr["counts"][0], qr["offsets"][0], qr["perm"][0]
        clusters = rng.choice(np.flatnonzero(counts > 0), 3, replace=False)
        mask = np.zeros((1, cfg.n), np.uint8)
        for c in clusters:
            members = perm[off[c]:off[c + 1]]
            mask[0, rng.choice(members, min(16, len(members)), replace=False)] = 1
        rows = np.flatnonzero(mask[0])
        for rho in rhos:
            g = sels.pop((h, rho))
            sel = oracle.select(S, qr["counts"], rho, cfg.k_fix)
            G.assert_same_selection(g, sel)
            ref = oracle.attention(hq, hk, hv, qr["offsets"], qr["perm"], sel["sel_counts"],
                                   sel["sel_idx"], row_mask=mask)
            mx, mr = G.assert_attention_close(g["out"][0, rows], ref[0, rows])
            kept = float((sel["sel_counts"][0].astype(np.float64) * counts).sum()) / cfg.n ** 2
            G.say(f"[fullsize] stress: head {h} rho {rho}: selection bit-exact, k_head "
                  f"{int(sel['k_head'][0])}, kept {kept:.3f}; attention on {len(rows)} rows "
                  f"max-abs {mx:.3e} mean-rel {mr:.3e}")
        del S
