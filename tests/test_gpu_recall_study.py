"""The matched-recall study (App. C, Fig. 9) and attention recall against
density (Fig. 2) end to end on the GPU, against the oracle: the SCOPE and
full-dimensional proxies bit for bit (the oracle's clusterings and lookup
sums), the block-wise proxy within fp32 rounding of the oracle's fp64
block means, and the retention, oracle recall and attention recall that the
study computes from each proxy equal to the oracle's protocol functions on
the same score rows."""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle  # noqa: E402
from paper_2608_12780_amd import inputs  # noqa: E402

import gpu_harness as G  # noqa: E402

MID = inputs.LayerConfig("recall_mid", 2, (5, 19, 23), 128, (16, 56, 56), 24, 20,
                         3, 0.9, inputs.ceil_tenth(5 * 19 * 23), "bf16", 8, 77)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()


def test_recall_study_against_oracle():
    import bench
    cfg, heads, c_q, c_m, block, sample = MID, 2, 24, 20, 16, 48
    everything = [np.arange(cfg.d, dtype=np.int32)]
    sig = 1.0 / math.sqrt(cfg.d)
    for hd in bench.recall_study_rows(cfg, heads, c_q, c_m, block, sample):
        h, x = hd["head"], hd["x"]
        cl = hd["clusters"].cpu().numpy()
        G.say(f"[recall] head {h}: {sample} queries in {len(set(cl.tolist()))} clusters")
        qr = oracle.cluster_queries(x.q[h:h + 1], c_q, cfg.iters, x.init_q[h:h + 1])
        kr = oracle.cluster_key_subspaces(x.k[h:h + 1], cfg.ranges, (c_m,) * 3, cfg.iters,
                                          hd["init3"][h:h + 1])
        S = oracle.proxy_scores(oracle.tables(qr["centroids"], kr["centroids"], cfg.ranges,
                                              (c_m,) * 3), kr["codes"], cfg.d, (c_m,) * 3)[0]
        kf = oracle.cluster_key_partition(x.k[h:h + 1], everything, (c_m,), cfg.iters,
                                          hd["init1"][h:h + 1])
        Sf = oracle.proxy_scores_partition(
            oracle.tables_partition(qr["centroids"], kf["centroids"], everything, (c_m,)),
            kf["codes"], cfg.d, (c_m,))[0]
        got = {name: pr.cpu().numpy() for name, pr in hd["proxies"].items()}
        assert np.array_equal(got["scope_subspaces"].view(np.uint32), S[cl].view(np.uint32))
        assert np.array_equal(got["full_dim_clusters"].view(np.uint32), Sf[cl].view(np.uint32))
        blocks = oracle.block_proxy(qr["centroids"][0][cl], x.k[h], block, sig)
        assert np.allclose(got["blocks"], blocks, rtol=1e-5, atol=1e-5)
        exact = hd["exact"].cpu().numpy()
        p_exact = hd["p_exact"].cpu().numpy().astype(np.float64)
        for name, pr in hd["proxies"].items():
            ret, rec = bench.matched_retention(hd["exact"], pr)
            o_ret, o_rec = oracle.matched_retention(exact, got[name])
            # the same kept-key and oracle-hit counts (the quotients may differ
            # in their last bit between the GPU's and the host's division)
            n, kt = exact.shape[1], -(-exact.shape[1] // 10)
            assert np.array_equal(np.rint(ret.cpu().numpy() * n), np.rint(o_ret * n)), name
            assert np.array_equal(np.rint(rec.cpu().numpy() * kt), np.rint(o_rec * kt)), name
            for dens in (0.05, 0.2, 0.5):
                m = bench.recall_at_density(hd["p_exact"], pr, dens).cpu().numpy()
                assert np.allclose(m, oracle.recall_at_density(p_exact, got[name], dens),
                                   rtol=1e-5, atol=1e-6), (name, dens)
            G.say(f"[recall] head {h} {name}: retention {o_ret.mean():.3f}, "
                  f"oracle recall {o_rec.mean():.3f}")
