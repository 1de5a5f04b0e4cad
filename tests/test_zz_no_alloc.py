"""The no-allocation attention entry point through the C ABI: its output
must equal the workspace entry point's, bit for bit (the same kernels on the
same work list), on two calls in a row, the second with a smaller problem
whose work list is shorter than the one the first call left in the fixed
array; both are also checked against the oracle's attention."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle  # noqa: E402
from paper_2608_12780_amd import binding as B  # noqa: E402
from paper_2608_12780_amd import inputs  # noqa: E402

import gpu_harness as G  # noqa: E402

FIRST = inputs.LayerConfig("noalloc_a", 3, (5, 19, 23), 128, (16, 56, 56), 32, 16,
                           3, 0.9, inputs.ceil_tenth(5 * 19 * 23), "bf16", 8, 91)
SECOND = inputs.LayerConfig("noalloc_b", 1, (3, 9, 14), 128, (44, 42, 42), 8, 8,
                            3, 0.8, inputs.ceil_tenth(3 * 9 * 14), "bf16", 8, 92)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    oracle.lib()


def _case(cfg):
    G.say(f"[noalloc] {cfg.name}: heads={cfg.heads} n={cfg.n} c_q={cfg.c_q}")
    x = inputs.generate(cfg)
    layer = G.make_layer(cfg, materialize=False)
    gpu = G.run_gpu(layer, x)
    q, k, v = G.to_device(x)
    out = torch.full_like(layer.out, float("nan"))
    B.scope_sparse_attention_noalloc(layer.shape, q, k, v, cfg.c_q, layer.offsets,
                                     layer.perm, layer.sel_counts, layer.sel_idx, 0.0, out)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert np.array_equal(got, gpu["out"])
    qr, kr, vr = (G.bf16_round(a) for a in (x.q, x.k, x.v))
    att = oracle.attention(qr, kr, vr, gpu["offsets"], gpu["perm"], gpu["sel_counts"],
                           gpu["sel_idx"])
    mx, mr = G.assert_attention_close(got, att)
    G.say(f"[noalloc] {cfg.name}: identical to the workspace call; max-abs {mx:.3e}")


def test_noalloc_attention_equals_workspace_call_twice():
    _case(FIRST)
    _case(SECOND)


def test_noalloc_rejects_problems_beyond_its_work_list():
    # 24 heads x (ceil(2^22 / 256) + 1024) work items exceed the fixed list
    shape = B.make_shape(24, 1 << 22, 128, B.BF16, ((0, 16, 72), (16, 56, 56)))
    t = torch.empty(16, dtype=torch.bfloat16, device="cuda")
    i = torch.empty(16, dtype=torch.int32, device="cuda")
    st = B.lib().scope_sparse_attention_noalloc(
        B.ctypes.byref(shape), t.data_ptr(), t.data_ptr(), t.data_ptr(), 1024,
        i.data_ptr(), i.data_ptr(), i.data_ptr(), i.data_ptr(), 0.0, t.data_ptr(), None)
    assert st == 5 and "no-allocation" in B.status_string(st)
