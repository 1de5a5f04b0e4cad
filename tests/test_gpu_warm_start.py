"""Warm-started clustering (calls 1w and 2w) through the C ABI against the
oracle: from given centroids the GPU and the oracle agree bit for bit, and
I1 iterations followed by I2 warm ones equal I1 + I2 cold ones.  A
perturbed copy of the inputs stands in for the next denoising step."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle  # noqa: E402
from paper_2608_12780_amd import inputs  # noqa: E402

import gpu_harness as G  # noqa: E402

MID = inputs.LayerConfig("warm_mid", 2, (5, 19, 23), 128, (16, 56, 56), 32, 16,
                         2, 0.9, inputs.ceil_tenth(5 * 19 * 23), "bf16", 8, 81)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()


def _clusters(layer):
    torch.cuda.synchronize()
    g = lambda t: t.cpu().numpy()
    return dict(centroids=g(layer.q_centroids), assign=g(layer.assign), perm=g(layer.perm),
                counts=g(layer.counts), k_centroids=g(layer.k_centroids),
                codes=g(layer.codes).view(np.uint32), status=int(layer.status.item()))


def _same(a, b, keys):
    # bitwise: the fp32 centroids as well as the integer results
    for key in keys:
        assert np.array_equal(a[key].view(np.uint8), b[key].view(np.uint8)), key


def test_warm_start_continues_the_cold_run():
    cfg = MID
    x = inputs.generate(cfg)
    q, k, _ = G.to_device(x)
    iq, ik = torch.from_numpy(x.init_q).cuda(), torch.from_numpy(x.init_k).cuda()
    layer = G.make_layer(cfg, materialize=False)
    layer.cluster_queries(q, iq, iters=2)
    layer.cluster_keys(k, ik, iters=2)
    layer.cluster_queries(q, warm=True, iters=3)
    layer.cluster_keys(k, warm=True, iters=3)
    warm = _clusters(layer)
    cold_layer = G.make_layer(cfg, materialize=False)
    cold_layer.cluster_queries(q, iq, iters=5)
    cold_layer.cluster_keys(k, ik, iters=5)
    cold = _clusters(cold_layer)
    assert warm["status"] == 0 and cold["status"] == 0
    _same(warm, cold, ("centroids", "assign", "perm", "counts", "k_centroids", "codes"))


def test_warm_start_next_step_matches_oracle():
    """Step t clusters cold; step t + 1 (inputs perturbed by a small noise,
    re-rounded to bf16) warm-starts from step t's centroids, on the GPU and
    in the oracle from the same centroids."""
    cfg = MID
    x = inputs.generate(cfg)
    layer = G.make_layer(cfg, materialize=False)
    q, k, _ = G.to_device(x)
    layer.cluster_queries(q, torch.from_numpy(x.init_q).cuda())
    layer.cluster_keys(k, torch.from_numpy(x.init_k).cuda())
    prev = _clusters(layer)
    rng = np.random.default_rng(5)
    for a, bits in ((x.q, x.q_bits), (x.k, x.k_bits)):
        a += (0.05 * rng.standard_normal(a.shape)).astype(np.float32)
        bits[...] = inputs.bf16_bits(a)
        a[...] = inputs.bf16_widen(bits)
    q2, k2, _ = G.to_device(x)
    layer.cluster_queries(q2, warm=True)
    layer.cluster_keys(k2, warm=True)
    gpu = _clusters(layer)
    assert gpu["status"] == 0
    ref_q = oracle.cluster_queries_from(x.q, cfg.c_q, cfg.iters, prev["centroids"])
    ref_k = oracle.cluster_key_subspaces_from(x.k, cfg.ranges, (cfg.c_m,) * 3, cfg.iters,
                                              prev["k_centroids"])
    assert np.array_equal(gpu["assign"], ref_q["assign"])
    assert np.array_equal(gpu["perm"], ref_q["perm"])
    assert np.array_equal(gpu["centroids"].view(np.uint32), ref_q["centroids"].view(np.uint32))
    assert np.array_equal(gpu["codes"], ref_k["codes"])
    assert np.array_equal(gpu["k_centroids"].view(np.uint32),
                          ref_k["centroids"].view(np.uint32))
    moved = float(np.abs(gpu["centroids"] - prev["centroids"]).max())
    G.say(f"[warm] next step: centroids moved by at most {moved:.3e}; bit-exact vs oracle")
