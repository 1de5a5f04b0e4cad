"""The sparse attention's work list (Eq. 11 cut into blocks), read back
through scope_debug_attention_items.

Output parity cannot see a chunk that runs twice (the second block writes the
same rows), so these tests check the list itself: every query chunk of every
cluster appears exactly once with its cluster's key count, two chunks share a
block only if they fit its 8 waves, used slots come before empty ones, and
up to 2,048 slots per head the used slots run in non-increasing estimated
cost with each cluster's full chunks adjacent.  The cost estimate restated
here is the work-list kernel's: key tiles of 64 times 171 (5-8 waves) or 118
(1-4 waves) per tile, times 1.15 for a block running two chunks (196, 135).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from paper_2608_12780_amd import binding as B  # noqa: E402

import gpu_harness as G  # noqa: E402

CHUNK = 256


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def expected_chunks(counts, keys):
    n = int(sum(counts))
    keys = [min(max(int(k), 0), n) for k in keys]
    out = []
    for c, (nc, kc) in enumerate(zip(counts, keys)):
        full, rem = divmod(int(nc), CHUNK)
        out += [(c, q * CHUNK, CHUNK, int(kc)) for q in range(full)]
        if rem:
            out.append((c, full * CHUNK, rem, int(kc)))
    return sorted(out)


def slot_cost(a, b):
    waves = -(-a[2] // 32) + (-(-b[2] // 32) if b[2] > 0 else 0)
    tiles = max(-(-a[3] // 64), -(-b[3] // 64) if b[2] > 0 else 0)
    paired = b[2] > 0
    per = (196 if paired else 171) if waves > 4 else (135 if paired else 118)
    return tiles * per


def run(counts_per_head, keys_per_head, pair, sorted_list):
    H, c_q = len(counts_per_head), len(counts_per_head[0])
    n = int(sum(counts_per_head[0]))
    assert all(int(sum(c)) == n for c in counts_per_head)
    offsets = np.zeros((H, c_q + 1), np.int32)
    for h in range(H):
        offsets[h, 1:] = np.cumsum(counts_per_head[h])
    sel = np.asarray(keys_per_head, np.int32)
    G.say(f"[worklist] heads={H} n={n} c_q={c_q} pair={pair} sorted={sorted_list}")
    items = B.scope_debug_attention_items(
        H, n, c_q, torch.from_numpy(offsets).cuda(), torch.from_numpy(sel).cuda(), pair=pair)
    torch.cuda.synchronize()
    items = items.cpu().numpy()
    S = items.shape[1]
    assert S == -(-n // CHUNK) + c_q
    for h in range(H):
        got, used_done = [], False
        prev_cost = None
        where = {}
        for s in range(S):
            a, b = tuple(int(v) for v in items[h, s, 0]), tuple(int(v) for v in items[h, s, 1])
            if a[2] <= 0:
                assert b[2] <= 0, (h, s, a, b)
                used_done = True
                continue
            assert not used_done, f"head {h}: used slot {s} after an empty one"
            if not pair:
                assert b[2] <= 0, (h, s, a, b)
            if b[2] > 0:
                assert -(-a[2] // 32) + -(-b[2] // 32) <= 8, (h, s, a, b)
            for e in (a, b):
                if e[2] > 0:
                    got.append(e)
                    if e[2] == CHUNK:
                        where.setdefault(e[0], []).append(s)
            if sorted_list:
                cost = slot_cost(a, b)
                assert prev_cost is None or cost <= prev_cost, (h, s, prev_cost, cost)
                prev_cost = cost
        assert sorted(got) == expected_chunks(counts_per_head[h], keys_per_head[h]), h
        if sorted_list:
            for c, slots in where.items():
                assert slots == list(range(slots[0], slots[0] + len(slots))), (h, c, slots)


def test_work_list_covers_every_chunk_once_in_cost_order():
    rng = np.random.default_rng(11)
    # remainders of every width (1-255 rows), whole chunks, several chunks
    sizes = np.concatenate([np.arange(1, 256, 7), [256, 512, 300, 480, 700, 1000, 767]])
    H, c_q = 3, 120
    base = rng.choice(sizes, size=c_q).astype(np.int64)
    counts = [rng.permutation(base) for _ in range(H)]
    keys = [rng.integers(1, 20000, size=c_q) for _ in range(H)]
    keys[1][:40] = 5000   # equal key counts: ties keep a cluster's chunks adjacent
    run(counts, keys, pair=True, sorted_list=True)
    run(counts, keys, pair=False, sorted_list=True)


def test_work_list_with_one_cluster_and_with_one_row_clusters():
    run([[4096]], [[4096]], pair=True, sorted_list=True)
    run([[1] * 64], [list(range(1, 65))], pair=True, sorted_list=True)


def test_work_list_above_the_sorting_limit_keeps_its_build_order():
    # more than 2,048 slots per head: the list is not reordered, and above
    # 2,048 clusters remainders are not paired either
    rng = np.random.default_rng(12)
    for c_q in (2040, 2100):
        counts = np.full(c_q, 4)
        counts[: c_q // 3] = 300
        counts[-1] += 8192   # one large cluster
        keys = rng.integers(1, 5000, size=c_q)
        run([counts], [keys], pair=True, sorted_list=False)
