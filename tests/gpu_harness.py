"""Shared helpers of the GPU tests: run the library on generated inputs and
compare with the oracle.  Imported only by tests marked `gpu`."""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
from paper_2608_12780_amd import binding as B
from paper_2608_12780_amd import inputs
from paper_2608_12780_amd.layer import DenseAttention, ScopeLayer, ScopePartitionLayer

# Attention tolerance (bf16 matrix products, fp32 softmax): max |o - ref| and
# sum |o - ref| / sum |ref| over the compared elements.
MAX_ABS = 2e-2
MEAN_REL = 1e-2


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(x: inputs.LayerInputs, device="cuda"):
    """Q, K, V on the GPU in the workload's storage dtype."""
    if x.cfg.dtype == "bf16":
        conv = lambda b: torch.from_numpy(b.view(np.int16)).to(device).view(torch.bfloat16)
        return conv(x.q_bits), conv(x.k_bits), conv(x.v_bits)
    return (torch.from_numpy(x.q).to(device), torch.from_numpy(x.k).to(device),
            torch.from_numpy(x.v).to(device))


def bf16_round(a: np.ndarray) -> np.ndarray:
    return inputs.bf16_widen(inputs.bf16_bits(a))


def make_layer(cfg: inputs.LayerConfig, heads=None, materialize=True, **over):
    a = dict(heads=cfg.heads if heads is None else heads, n=cfg.n, d=cfg.d,
             ranges=cfg.ranges, c_q=cfg.c_q, c_m=(cfg.c_m,) * 3, iters=cfg.iters,
             rho=cfg.rho, k_fix=cfg.k_fix, dtype=cfg.dtype,
             materialize_scores=materialize)
    a.update(over)
    return ScopeLayer(**a)


def make_partition_layer(cfg: inputs.LayerConfig, sets, c_m, heads=None,
                         materialize=True):
    return ScopePartitionLayer(cfg.heads if heads is None else heads, cfg.n, cfg.d,
                               sets, cfg.c_q, c_m, cfg.iters, cfg.rho, cfg.k_fix,
                               cfg.dtype, materialize_scores=materialize)


def run_gpu(layer: ScopeLayer, x: inputs.LayerInputs, use_scores=False, policy="online",
            init_k=None):
    q, k, v = to_device(x)
    iq = torch.from_numpy(x.init_q).cuda()
    ik = torch.from_numpy(x.init_k if init_k is None else init_k).cuda()
    layer.cluster_queries(q, iq)
    layer.cluster_keys(k, ik)
    layer.proxy_scores()
    layer.select(use_scores=use_scores, policy=policy)
    layer.attend(q, k, v)
    torch.cuda.synchronize()
    g = lambda t: None if t is None else t.cpu().numpy()
    return dict(centroids=g(layer.q_centroids), assign=g(layer.assign),
                counts=g(layer.counts), offsets=g(layer.offsets),
                perm=g(layer.perm), k_centroids=g(layer.k_centroids),
                codes=_codes(g(layer.codes)), tables=g(layer.tables),
                scores=g(layer.scores), base=g(layer.base_counts),
                topp=g(layer.topp_counts), k_head=g(layer.k_head),
                sel_counts=g(layer.sel_counts), sel_idx=g(layer.sel_idx),
                out=layer.out.float().cpu().numpy(), status=int(layer.status.item()))


def _codes(c):
    # packed composite codes (int32 storage) or uint16 planes (int16 storage)
    return c.view(np.uint16) if c.dtype == np.int16 else c.view(np.uint32)


def oracle_all(x: inputs.LayerInputs, c_q, c_m, iters, rho, k_fix, policy="online"):
    return oracle.layer(x.q, x.k, x.v, x.cfg.ranges, c_q, c_m, iters, x.init_q,
                        x.init_k, rho, k_fix, policy)


def assert_same_selection(gpu, ref_sel):
    assert np.array_equal(gpu["base"], ref_sel["base_counts"])
    assert np.array_equal(gpu["topp"], ref_sel["topp"])
    assert np.array_equal(gpu["k_head"], ref_sel["k_head"])
    assert np.array_equal(gpu["sel_counts"], ref_sel["sel_counts"])
    H, C, _ = ref_sel["sel_idx"].shape
    for h in range(H):
        for c in range(C):
            r = int(ref_sel["sel_counts"][h, c])
            assert np.array_equal(gpu["sel_idx"][h, c, :r], ref_sel["sel_idx"][h, c, :r]), (h, c)


def attention_error(out, ref):
    diff = np.abs(out.astype(np.float64) - ref.astype(np.float64))
    return float(diff.max()), float(diff.sum() / max(np.abs(ref).sum(), 1e-30))


def assert_attention_close(out, ref):
    mx, mr = attention_error(out, ref)
    assert mx <= MAX_ABS and mr <= MEAN_REL, (mx, mr)
    return mx, mr


def select_from_codes(tables_np, codes_np, counts_np, d, c_m, rho, k_fix):
    """scope_select on given tables and packed codes (logits fused from the
    LUT), against the oracle's selection on the oracle's proxy logits."""
    H, C, _ = tables_np.shape
    n = codes_np.shape[1]
    shape = B.make_shape(H, n, d, B.BF16, ((0, d // 4, d // 2), (d // 4, d // 4, d // 2)))
    dev = "cuda"
    tables = torch.from_numpy(tables_np).to(dev)
    codes = torch.from_numpy(codes_np.view(np.int32)).to(dev)
    counts = torch.from_numpy(counts_np).to(dev)
    i32 = dict(dtype=torch.int32, device=dev)
    base = torch.empty(H, C, **i32)
    topp = torch.empty(H, C, **i32)
    kh = torch.empty(H, **i32)
    sc = torch.empty(H, C, **i32)
    idx = torch.empty(H, C, n, **i32)
    ws = B.alloc_workspace(shape, C, c_m, dev)
    B.scope_select(shape, C, c_m, None, tables, codes, counts, rho, k_fix, base, topp,
                   kh, sc, idx, ws)
    torch.cuda.synchronize()
    gpu = dict(base=base.cpu().numpy(), topp=topp.cpu().numpy(), k_head=kh.cpu().numpy(),
               sel_counts=sc.cpu().numpy(), sel_idx=idx.cpu().numpy())
    ref = oracle.select(oracle.proxy_scores(tables_np, codes_np, d, c_m), counts_np, rho, k_fix)
    assert_same_selection(gpu, ref)
    return gpu
