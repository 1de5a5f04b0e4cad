"""The recall measures of bench.py's studies (CPU only), checked by brute
force on small hand-made rows."""
import math
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def brute_retention(exact, proxy, top_frac, target):
    N = len(exact)
    kt = math.ceil(top_frac * N)
    oracle = set(sorted(range(N), key=lambda j: (-exact[j], j))[:kt])
    need = math.ceil(target * kt)
    for s in sorted(set(proxy), reverse=True):     # whole groups, best first
        kept = {j for j in range(N) if proxy[j] >= s}
        if len(kept & oracle) >= need:
            return len(kept) / N, len(kept & oracle) / kt
    raise AssertionError("unreachable")


@pytest.mark.parametrize("seed", range(30))
def test_matched_retention_brute_force(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(10, 60))
    exact = rng.standard_normal((3, N))
    groups = int(rng.integers(1, N + 1))
    proxy = rng.standard_normal((3, groups))[:, rng.integers(0, groups, N)]
    if seed % 3 == 0:
        proxy = exact.copy()                        # a perfect proxy
    frac, target = [(0.1, 0.958), (0.3, 0.5), (0.5, 1.0)][seed % 3]
    ret, rec = bench.matched_retention(torch.tensor(exact), torch.tensor(proxy), frac, target)
    for r in range(3):
        want = brute_retention(exact[r].tolist(), proxy[r].tolist(), frac, target)
        assert ret[r].item() == pytest.approx(want[0]) and rec[r].item() == pytest.approx(want[1])
    if seed % 3 == 0:   # exact order: exactly the first ceil(target * kt) oracle keys
        kt = math.ceil(frac * N)
        assert np.allclose(ret.numpy(), math.ceil(target * kt) / N)


def test_recall_at_density():
    p = torch.tensor([[0.5, 0.1, 0.3, 0.1]])
    proxy = torch.tensor([[0.0, 2.0, 1.0, 2.0]])
    # two keys by proxy order: indices 1 and 3 (tie, lower index first)
    assert bench.recall_at_density(p, proxy, 0.5).item() == pytest.approx(0.2)
    assert bench.recall_at_density(p, proxy, 0.75).item() == pytest.approx(0.5)
    assert bench.recall_at_density(p, proxy, 1.0).item() == pytest.approx(1.0)
