"""Benchmark of the SCOPE attention layer on one MI355X.

One step = the whole layer (query clustering, key-subspace clustering, score
tables, selection, sparse attention: the five C-ABI calls for every head) on
one batch of synthetic post-RoPE Q/K/V already resident in HBM.  The default
workload is the HunyuanVideo-720p-like layer (24 heads, 33x45x80 = 118800
tokens, d = 128, RoPE split 16/56/56, C_q = 256, C_m = 128, 10 iterations,
rho = 0.9, k_fix = ceil(0.1 N)).

Prints ONE JSON line on stdout; progress goes to stderr.

Summaries of saved JSON lines (any machine):
  python3 bench.py --lines-summary workloads|rho "<command>" line1.json line2.json ...

Traffic measurement (two counter passes, then a summary on any machine):
  rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'attn_kernel|copy' -d F -o run \
      --output-format csv -- python3 bench.py --traffic-probe
  rocprofv3 --pmc WRITE_SIZE --kernel-include-regex 'attn_kernel|copy' -d W -o run \
      --output-format csv -- python3 bench.py --traffic-probe
  python3 bench.py --traffic-summary F/run_counter_collection.csv W/run_counter_collection.csv
The probe runs the layer once, a plain 1 GiB device copy (the calibration:
its counters are scaled to the bytes it is known to move) and one launch of
the sparse attention.
  value          effective TFLOP/s = dense attention flops 4 N^2 d H / layer time
  ms_per_step    layer latency
  roofline       the sparse-attention kernel against the bf16 MFMA peak
                 (algorithmic flops 4 d sum_c n_c r_c per launch); traffic =
                 its HBM bytes per launch from the committed counter summary,
                 null when the kernel source changed since it was taken
  cpu_baseline   the CPU oracle on a bounded sample of one head, extrapolated
  dense_*        the same GPU's dense attention: the library's dense mode and
                 torch's scaled_dot_product_attention (flash backend)
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
HBM_PEAK_GBS = 8000.0
CALIB_BYTES = 1 << 30              # calibration copy: reads and writes this much
ATTN_SRC = os.path.join(ROOT, "paper_2608_12780_amd", "csrc", "attention.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_kernel_hy720_hbm_traffic.txt")

WORKLOAD_NAMES = {
    "hy720": "HunyuanVideo-720p-like",
    "wan720": "Wan2.2-720p-like",
    "wan480": "Wan2.2-480p-like",
    "stress": "HunyuanVideo-720p-like selection stress",
    "tiny": "Tiny",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def dense_flops(cfg):
    return 4.0 * cfg.n * cfg.n * cfg.d * cfg.heads


def time_events(torch, fn, reps, stream):
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    s.record(stream)
    for _ in range(reps):
        fn()
    e.record(stream)
    e.synchronize()
    return s.elapsed_time(e) / reps


def sdpa_ms(torch, q, k, v, reps):
    """torch's fused SDPA on the same bf16 tensors (flash, else efficient)."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    F = torch.nn.functional
    qb, kb, vb = (t.unsqueeze(0) for t in (q, k, v))
    for backend in (SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION):
        try:
            with sdpa_kernel(backend):
                F.scaled_dot_product_attention(qb, kb, vb)
                torch.cuda.synchronize()
                ms = time_events(torch, lambda: F.scaled_dot_product_attention(qb, kb, vb),
                                 reps, torch.cuda.current_stream())
            return ms, backend.name
        except RuntimeError as exc:  # backend not available for this shape
            log(f"sdpa {backend.name} unavailable: {exc}")
    return None, None


ATTN_ROWS = 16384  # query rows of the CPU baseline's attention sample


def cpu_baseline(cfg, x, layer_np):
    """The oracle on one head of the workload, timed on this host's cores.

    Sample (about 12-20 s of CPU work at 720p): head 0 with every stage run
    in full (all k-means iterations, tables, logits, selection of every
    cluster) except attention, which runs for a seeded uniform sample of
    ATTN_ROWS query rows (each row's cost follows its cluster's key count,
    so the sample is unbiased) and is scaled to all rows; the per-head sum
    is scaled to all heads."""
    import oracle
    oracle.lib()
    cm = (cfg.c_m,) * 3
    q, k, v = x.q[:1], x.k[:1], x.v[:1]
    t = {}
    s = time.perf_counter()
    qr = oracle.cluster_queries(q, cfg.c_q, cfg.iters, x.init_q[:1])
    t["query_kmeans"] = time.perf_counter() - s
    s = time.perf_counter()
    kr = oracle.cluster_key_subspaces(k, cfg.ranges, cm, cfg.iters, x.init_k[:1])
    t["key_kmeans"] = time.perf_counter() - s
    s = time.perf_counter()
    P = oracle.tables(qr["centroids"], kr["centroids"], cfg.ranges, cm)
    S = oracle.proxy_scores(P, kr["codes"], cfg.d, cm)
    t["scores"] = time.perf_counter() - s
    s = time.perf_counter()
    sel = oracle.select(S, qr["counts"], cfg.rho, cfg.k_fix)
    t["select"] = time.perf_counter() - s
    del S
    rows = min(ATTN_ROWS, cfg.n)
    mask = np.zeros((1, cfg.n), np.uint8)
    mask[0, np.random.default_rng(0).choice(cfg.n, rows, replace=False)] = 1
    s = time.perf_counter()
    oracle.attention(q, k, v, qr["offsets"], qr["perm"], sel["sel_counts"],
                     sel["sel_idx"], row_mask=mask)
    t_attn = time.perf_counter() - s
    t["attention"] = t_attn * cfg.n / rows
    measured = sum(t.values()) - t["attention"] + t_attn
    per_head = sum(t.values())
    layer_s = per_head * cfg.heads
    return {
        "value": dense_flops(cfg) / layer_s / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "layer_s_extrapolated": layer_s,
        "per_head_stage_s": {k_: round(v_, 3) for k_, v_ in t.items()},
        "measured_s": round(measured, 2),
        "sample": (f"head 0 of {cfg.heads}, every stage in full (query and key "
                   f"k-means, {cfg.iters} iterations each, tables, logits, selection "
                   f"of all {cfg.c_q} clusters) except attention: {rows} of {cfg.n} "
                   f"query rows (seeded uniform sample), scaled to all rows; "
                   f"x{cfg.heads} heads"),
    }


def stage_bytes(cfg, sel_total):
    """Algorithmic HBM bytes per stage of one layer: every input read once
    per pass over it, every output written once (int32 indices, bf16 or fp32
    rows).  sel_total = sum over heads and clusters of r_c."""
    H, N, d, it = cfg.heads, cfg.n, cfg.d, cfg.iters
    e = 2 if cfg.dtype == "bf16" else 4
    rows = H * N * d * e
    i32 = H * N * 4
    return {
        # per iteration: assignment reads Q and writes g; the update reads Q
        # and g; the grouping of the last assignment reads g, writes perm
        "cluster_queries": it * (2 * rows + 2 * i32) + 2 * i32,
        # per iteration: three assignments read K's channel ranges (K once)
        # and write three label arrays, the update reads K and the labels;
        # the final assignment, then the packing into codes
        "cluster_key_subspaces": it * (2 * rows + 6 * i32) + rows + 3 * i32 + 4 * i32,
        # centroids in, tables out (a few MB)
        "proxy_scores": H * (cfg.c_q * d + 3 * cfg.c_m * d // 3 + cfg.c_q * 3 * cfg.c_m) * 4,
        # codes read once per head, the selected index lists written
        "select": i32 + 4 * sel_total,
    }


def trace_summary(trace_csv, cmd, bench_line=None, config_name="hy720"):
    """Per-kernel table of a rocprofv3 kernel trace with algorithmic bytes
    (or flops) per call for the kernels of the workload's layer."""
    import csv
    import re
    from paper_2608_12780_amd import inputs
    cfg = inputs.CONFIGS[config_name]
    H, N, d = cfg.heads, cfg.n, cfg.d
    e = 2 if cfg.dtype == "bf16" else 4
    dx_of = {128: d, 64: max(cfg.split[1], cfg.split[2]), 16: cfg.split[0]}
    rows = []
    for r in csv.DictReader(open(trace_csv)):
        name = re.sub(r"scope::\(anonymous namespace\)::", "", r["Kernel_Name"])
        name = re.sub(r"^void ", "", name).split("(")[0]
        grid = (int(r["Grid_Size_X"]), int(r["Grid_Size_Y"]), int(r["Grid_Size_Z"]))
        rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), name, grid))
    rows.sort()
    # the layer's own steps come first; the one-GPU-share layer (fewer
    # heads), the dense mode and torch's SDPA follow.  The share run begins
    # with the query initialisation over fewer heads.
    share = max(1, math.ceil(H / 8))
    cut = next((t0 for t0, _, nm, g in rows
                if nm.startswith("km_init_kernel") and g[1] == share and share < H), None)

    def table(sel):
        agg = {}
        for t0, t1, name, g in sel:
            key = (name, f"{g[0]}x{g[1]}x{g[2]}")
            a = agg.setdefault(key, [0, 0.0])
            a[0] += 1
            a[1] += (t1 - t0) / 1e3
        return agg

    def model(name, grid):
        m = re.match(r"km_assign_mfma_kernel<(\d+)>", name)
        if m:
            dx = dx_of.get(int(m.group(1)))
            return None if dx is None else ("B", H * N * (dx * e + 4))
        if name.startswith("km_accum_kernel"):
            gy = int(grid.split("x")[1])
            nsub = 1 if gy > 1 else 3     # queries: two channel windows; keys: one
            return ("B", H * N * (d * e + 4 * nsub))
        return None

    lines = [f"command: {cmd}", "",
             "per (kernel, grid in work-items); durations from the kernel trace;",
             "algorithmic bytes per call: rows read once (+ int32 labels) for the k-means",
             f"assignment and update kernels of the {config_name} layer (8000 GB/s peak)"]
    head = f"{'total ms':>10} {'calls':>6} {'avg us':>11} {'pct':>6} {'GB/s':>8} {'of peak':>8} {'grid':>20}  kernel"
    parts = [("layer steps (warmup + timed)", [r for r in rows if cut is None or r[0] < cut], True),
             (f"then: one GPU's share ({share} heads), the library's dense mode, torch SDPA",
              [r for r in rows if cut is not None and r[0] >= cut], False)]
    for title, sel, with_model in parts:
        if not sel:
            continue
        agg = table(sel)
        tot = sum(v[1] for v in agg.values())
        lines += ["", title, head]
        for (name, grid), (c, dsum) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
            avg = dsum / c
            mdl = model(name, grid) if with_model else None
            gbs = f"{mdl[1] / (avg * 1e-6) / 1e9:8.0f}" if mdl else f"{'':>8}"
            frac = f"{mdl[1] / (avg * 1e-6) / 1e9 / HBM_PEAK_GBS:8.2f}" if mdl else f"{'':>8}"
            lines.append(f"{dsum / 1e3:10.2f} {c:>6} {avg:11.1f} {100 * dsum / tot:6.2f} {gbs} {frac} {grid:>20}  {name}")
    if bench_line:
        lines += ["", "bench.py JSON line of the same run:", bench_line.strip()]
    return "\n".join(lines) + "\n"


def policy_study(config_name="hy720", heads=4):
    """The selection-policy ablation (Fig. 6) on synthetic inputs: the online
    policy at the workload's rho sets a realised density (fraction of query-
    key pairs kept); rho of the fixed-floor and pure Top-p policies is
    bisected to the same density; each policy's attention output is then
    compared with dense attention on the same heads."""
    import torch
    from paper_2608_12780_amd import inputs
    from paper_2608_12780_amd.layer import DenseAttention, ScopeLayer
    cfg = inputs.CONFIGS[config_name]
    x = inputs.generate(cfg.with_(heads=heads))
    dev = torch.device("cuda", 0)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    q, k, v = up(x.q_bits), up(x.k_bits), up(x.v_bits)
    L = ScopeLayer(heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3, cfg.iters,
                   cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev)
    L.cluster_queries(q, torch.from_numpy(x.init_q).to(dev))
    L.cluster_keys(k, torch.from_numpy(x.init_k).to(dev))
    L.proxy_scores()
    dense = DenseAttention(heads, cfg.n, cfg.d, cfg.dtype, dev)
    ref = dense.forward(q, k, v).float()
    torch.cuda.synchronize()
    counts = L.counts.double()

    def density(policy, rho):
        L.select(policy=policy, rho=rho)
        return float((counts * L.sel_counts.double()).sum()) / (heads * float(cfg.n) ** 2)

    target = density("online", cfg.rho)
    rows = []
    for policy in ("online", "fixed", "topp"):
        if policy == "online":
            rho = cfg.rho
        else:
            lo, hi = 1e-4, 1.0
            for _ in range(24):
                mid = 0.5 * (lo + hi)
                if density(policy, mid) < target:
                    lo = mid
                else:
                    hi = mid
            rho = hi
        dens = density(policy, rho)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        L.attend(q, k, v)
        e.record()
        e.synchronize()
        out = L.out.float()
        err = out - ref
        rows.append({"policy": policy, "rho": round(rho, 6), "density": round(dens, 5),
                     "rel_l2_vs_dense": float(err.norm() / ref.norm()),
                     "max_abs_vs_dense": float(err.abs().max()),
                     "attention_ms": round(s.elapsed_time(e), 3),
                     "k_head_mean": float(L.k_head.double().mean())})
        log(f"[policy] {rows[-1]}")
    return {"study": "selection policy at matched density", "workload": WORKLOAD_NAMES.get(cfg.name),
            "heads": heads, "n": cfg.n, "target_density": round(target, 5), "rows": rows}


def partition_study(config_name="hy720", heads=4, c_q=300, c_m=333, reps=2,
                    sample=256):
    """The key-partition ablation (Table 3) on synthetic inputs: every
    partition (full-dimensional, 2, random 3-way, RoPE 3-way, 4 and 8 equal
    ranges) at the paper's C_q = 300 and C_m = 333 per subspace, the same
    rho and k_fix.  Per partition: stage and layer latency (HIP events), the
    realised density, the share of the exact softmax mass each sampled query
    keeps (attention recall), and the output's relative L2 error against
    dense attention on the same heads."""
    import torch
    from paper_2608_12780_amd import inputs
    from paper_2608_12780_amd.layer import DenseAttention, ScopeLayer, ScopePartitionLayer
    cfg = inputs.CONFIGS[config_name].with_(c_q=c_q, c_m=c_m)
    x = inputs.generate(cfg.with_(heads=heads))
    dev = torch.device("cuda", 0)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    q, k, v = up(x.q_bits), up(x.k_bits), up(x.v_bits)
    iq = torch.from_numpy(x.init_q).to(dev)
    dense = DenseAttention(heads, cfg.n, cfg.d, cfg.dtype, dev)
    ref = dense.forward(q, k, v).float()
    torch.cuda.synchronize()
    del dense
    rng = np.random.default_rng(cfg.seed)
    rows_q = torch.from_numpy(rng.choice(cfg.n, size=(heads, sample), replace=False)).to(dev)
    scale = 1.0 / math.sqrt(cfg.d)
    stream = torch.cuda.current_stream()
    names = ["cluster_queries", "cluster_keys", "proxy_scores", "select", "sparse_attention"]

    def measure(layer, init_k, label, M):
        layer.forward(q, k, v, iq, init_k)
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(reps)]
        for i in range(reps):
            layer.forward(q, k, v, iq, init_k, marks=lambda j, i=i: ev[i][j].record(stream))
        torch.cuda.synchronize()
        st = {n_: float(np.mean([ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(reps)]))
              for j, n_ in enumerate(names)}
        total = float(np.mean([ev[i][0].elapsed_time(ev[i][5]) for i in range(reps)]))
        counts = layer.counts.double()
        dens = float((counts * layer.sel_counts.double()).sum()) / (heads * float(cfg.n) ** 2)
        err = layer.out.float() - ref
        # attention recall: softmax mass of each sampled query on its key set
        rec = []
        cl = layer.assign.long()
        for h in range(heads):
            qi = rows_q[h]
            p_ = torch.softmax((q[h, qi].float() @ k[h].float().T) * scale, dim=1)
            c_ = cl[h, qi]
            r_ = layer.sel_counts[h, c_].long()
            idx = layer.sel_idx[h, c_].long()
            keep = torch.arange(cfg.n, device=dev)[None, :] < r_[:, None]
            mass = torch.gather(p_, 1, idx.clamp(0, cfg.n - 1)) * keep
            rec.append(mass.sum(1))
        rec = torch.cat(rec)
        row = {"partition": label, "M": M, "layer_ms": round(total, 3),
               "stages_ms": {n_: round(t_, 3) for n_, t_ in st.items()},
               "density": round(dens, 5), "k_head_mean": float(layer.k_head.double().mean()),
               "attention_recall_mean": round(float(rec.mean()), 5),
               "attention_recall_p5": round(float(torch.quantile(rec, 0.05)), 5),
               "rel_l2_vs_dense": float(err.norm() / ref.norm())}
        log(f"[partition] {row}")
        return row

    rows = []
    for kind in inputs.PARTITIONS:
        sets = inputs.partition_sets(cfg, kind)
        M = len(sets)
        init_k = torch.from_numpy(inputs.partition_init(cfg, M, c_m, heads)).to(dev)
        layer = ScopePartitionLayer(heads, cfg.n, cfg.d, sets, c_q, (c_m,) * M, cfg.iters,
                                    cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev)
        rows.append(measure(layer, init_k, kind, M))
        del layer
        torch.cuda.empty_cache()
    # the same RoPE partition through the three-range calls (packed codes)
    init3 = torch.from_numpy(inputs.partition_init(cfg, 3, c_m, heads)).to(dev)
    layer = ScopeLayer(heads, cfg.n, cfg.d, cfg.ranges, c_q, (c_m,) * 3, cfg.iters, cfg.rho,
                       cfg.k_fix, dtype=cfg.dtype, device=dev)
    rows.append(measure(layer, init3, "3-rope (range calls)", 3))
    return {"study": "key partitions (Table 3 analogue)",
            "workload": WORKLOAD_NAMES.get(cfg.name), "heads": heads, "n": cfg.n,
            "c_q": c_q, "c_m": c_m, "rho": cfg.rho, "k_fix": cfg.k_fix,
            "sampled_queries_per_head": sample, "rows": rows}


def matched_retention(exact, proxy, top_frac=0.1, target=0.958):
    """App. C protocol, per row (one query): the oracle set is the top
    ceil(top_frac N) keys by exact score (ties to the lower index); keys
    are taken in proxy-score order, whole groups of equal proxy score at a
    time, until `target` of the oracle set is held.  Returns the retained
    fraction of all keys and the oracle recall reached, per row."""
    import torch
    from fractions import Fraction
    Q, N = exact.shape
    ceil = lambda f: -((-f.numerator) // f.denominator)
    kt = max(1, ceil(Fraction(str(top_frac)) * N))
    need = max(1, ceil(Fraction(str(target)) * kt))
    order_e = torch.argsort(exact, dim=1, descending=True, stable=True)
    oracle = torch.zeros(exact.shape, dtype=torch.bool, device=exact.device)
    oracle.scatter_(1, order_e[:, :kt], True)
    order_p = torch.argsort(proxy, dim=1, descending=True, stable=True)
    hits = torch.gather(oracle, 1, order_p).to(torch.int32).cumsum(1)
    pos = (hits >= need).to(torch.int8).argmax(1)          # first position reaching it
    s_star = torch.gather(torch.gather(proxy, 1, order_p), 1, pos[:, None])
    kept = proxy >= s_star                                   # the whole tie group
    recall = (kept & oracle).sum(1).double() / kt
    return kept.sum(1).double() / N, recall


def recall_at_density(p_exact, proxy, density):
    """Softmax mass of the exact attention row held by the top
    round(density N) keys in proxy order (ties to the lower index)."""
    import torch
    N = proxy.shape[1]
    k = max(1, int(round(density * N)))
    top = torch.argsort(proxy, dim=1, descending=True, stable=True)[:, :k]
    return torch.gather(p_exact, 1, top).sum(1)


def recall_study_rows(cfg, heads, c_q, c_m, block, sample, dev=None):
    """The three key-side proxies of the matched-recall study on the first
    `heads` heads of workload cfg, each scoring a query by its cluster
    centroid: SCOPE's subspace lookup sum (RoPE t/h/w ranges, c_m centroids
    per subspace), full-dimensional key clusters (c_m centroids; the one-set
    partition) and block means of `block` consecutive tokens.  Per head
    yields the sampled query rows and their exact scores, exact attention
    weights and proxy rows (torch tensors on the GPU)."""
    import torch
    from paper_2608_12780_amd import inputs
    from paper_2608_12780_amd.layer import ScopeLayer, ScopePartitionLayer
    cfg = cfg.with_(c_q=c_q, c_m=c_m)
    x = inputs.generate(cfg.with_(heads=heads))
    dev = dev or torch.device("cuda", 0)
    if cfg.dtype == "bf16":
        up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
        q, k = up(x.q_bits), up(x.k_bits)
    else:
        q, k = torch.from_numpy(x.q).to(dev), torch.from_numpy(x.k).to(dev)
    iq = torch.from_numpy(x.init_q).to(dev)
    sig = 1.0 / math.sqrt(cfg.d)
    init3 = inputs.partition_init(cfg, 3, c_m, heads)
    init1 = inputs.partition_init(cfg, 1, c_m, heads)
    scope = ScopeLayer(heads, cfg.n, cfg.d, cfg.ranges, c_q, (c_m,) * 3, cfg.iters,
                       cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev,
                       materialize_scores=True)
    scope.cluster_queries(q, iq)
    scope.cluster_keys(k, torch.from_numpy(init3).to(dev))
    scope.proxy_scores()
    full = ScopePartitionLayer(heads, cfg.n, cfg.d, inputs.partition_sets(cfg, "1"), c_q,
                               (c_m,), cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype,
                               device=dev, materialize_scores=True)
    full.cluster_queries(q, iq)
    full.cluster_keys(k, torch.from_numpy(init1).to(dev))
    full.proxy_scores()
    torch.cuda.synchronize()
    assert torch.equal(scope.assign, full.assign)   # same query clusters
    rng = np.random.default_rng(cfg.seed + 7)
    nb = (cfg.n + block - 1) // block
    for h in range(heads):
        kf = k[h].float()
        pad = torch.zeros(nb * block - cfg.n, cfg.d, device=dev)
        cnt = torch.full((nb,), float(block), device=dev)
        cnt[-1] = block - (nb * block - cfg.n)
        kbar = torch.cat([kf, pad]).reshape(nb, block, cfg.d).sum(1) / cnt[:, None]
        qi = torch.from_numpy(rng.choice(cfg.n, sample, replace=False)).to(dev)
        c_ = scope.assign[h, qi].long()
        exact = (q[h, qi].float() @ kf.T) * sig
        qbar = scope.q_centroids[h, c_]
        yield dict(head=h, x=x, init3=init3, init1=init1, qi=qi, clusters=c_, exact=exact,
                   p_exact=torch.softmax(exact, dim=1), qbar=qbar,
                   proxies={"scope_subspaces": scope.scores[h, c_],
                            "full_dim_clusters": full.scores[h, c_],
                            "blocks": ((qbar @ kbar.T) * sig).repeat_interleave(block, dim=1)[:, :cfg.n]})


def recall_study(config_name="hy720", heads=4, c_q=300, c_m=333, block=64, sample=256,
                 densities=(0.05, 0.1, 0.2, 0.3, 0.5)):
    """Matched-recall retention (App. C, Fig. 9) and attention recall against
    density (Fig. 2) of three key-side proxies that all score a query by its
    cluster centroid: SCOPE's subspace lookup sum (RoPE t/h/w, C_m per
    subspace), full-dimensional key clusters (C_m centroids) and block means
    of `block` consecutive tokens.  Exact scores of sampled queries come
    from their own rows of Q K^T."""
    import torch
    from paper_2608_12780_amd import inputs
    cfg = inputs.CONFIGS[config_name]
    rows = {"scope_subspaces": [], "full_dim_clusters": [], "blocks": []}
    dens = {name: {str(dd): [] for dd in densities} for name in rows}
    for hd in recall_study_rows(cfg, heads, c_q, c_m, block, sample):
        for name, pr in hd["proxies"].items():
            ret, rec = matched_retention(hd["exact"], pr)
            rows[name].append(torch.stack([ret, rec], 1))
            for dd in densities:
                dens[name][str(dd)].append(recall_at_density(hd["p_exact"], pr, dd))
    out = []
    for name in rows:
        r = torch.cat(rows[name])
        row = {"proxy": name, "retention_mean": round(float(r[:, 0].mean()), 4),
               "retention_median": round(float(r[:, 0].median()), 4),
               "oracle_recall_mean": round(float(r[:, 1].mean()), 4),
               "attention_recall_at_density": {dd: round(float(torch.cat(v_).mean()), 4)
                                               for dd, v_ in dens[name].items()}}
        log(f"[recall] {row}")
        out.append(row)
    return {"study": "matched oracle recall and attention recall vs density (App. C, Fig. 2)",
            "workload": WORKLOAD_NAMES.get(cfg.name), "heads": heads, "n": cfg.n,
            "c_q": c_q, "c_m": c_m, "block_tokens": block, "oracle_top_fraction": 0.1,
            "target_oracle_recall": 0.958, "sampled_queries_per_head": sample, "rows": out}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def source_digest():
    import hashlib
    with open(ATTN_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def committed_traffic(config_name):
    """HBM bytes per attention launch from the committed summary, if it was
    taken on this workload with the current kernel source."""
    try:
        kv = dict(l.split(": ", 1) for l in open(TRAFFIC_FILE).read().splitlines()
                  if ": " in l and not l.startswith(" "))
    except OSError:
        return None
    if kv.get("attention_source_sha256") != source_digest() or kv.get("config") != config_name:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def traffic_summary(fetch_csv, write_csv, config_name="hy720"):
    """Scales FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the attention
    kernel by what the same counters read for the calibration copy."""
    import csv

    def per_dispatch(path):
        d = {}
        for r in csv.DictReader(open(path)):
            key = r["Dispatch_Id"]
            e = d.setdefault(key, {"name": r["Kernel_Name"], "v": 0.0,
                                   "dur": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
            e["v"] += float(r["Counter_Value"])
        return list(d.values())

    out = {}
    for tag, path in (("fetch", fetch_csv), ("write", write_csv)):
        rows = per_dispatch(path)
        # the device-to-device copy runs as the runtime's blit kernel
        copies = [e for e in rows if "copy" in e["name"].lower()]
        attn = [e for e in rows if "attn_kernel" in e["name"]]
        if not copies or not attn:
            raise SystemExit(f"{path}: calibration copy or attention dispatch missing")
        cal = max(copies, key=lambda e: e["dur"])
        factor = (CALIB_BYTES / 1024.0) / cal["v"]
        a = attn[-1]
        out[tag] = dict(copy_kib=cal["v"], factor=factor, attn_kib=a["v"],
                        attn_bytes=a["v"] * 1024.0 * factor)
    total = out["fetch"]["attn_bytes"] + out["write"]["attn_bytes"]
    lines = [
        f"config: {config_name}",
        f"attention_source_sha256: {source_digest()}",
        f"hbm_bytes_per_launch: {total:.6e}",
        f"fetch_bytes_per_launch: {out['fetch']['attn_bytes']:.6e}",
        f"write_bytes_per_launch: {out['write']['attn_bytes']:.6e}",
        "",
        "commands (cd /tmp && export TMPDIR=/tmp, then from the repository root):",
        "  rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'attn_kernel|copy' -d F -o run "
        "--output-format csv -- python3 bench.py --traffic-probe",
        "  rocprofv3 --pmc WRITE_SIZE --kernel-include-regex 'attn_kernel|copy' -d W -o run "
        "--output-format csv -- python3 bench.py --traffic-probe",
        "  python3 bench.py --traffic-summary F/run_counter_collection.csv "
        "W/run_counter_collection.csv",
        f"  calibration: one device copy of {CALIB_BYTES} bytes read + written;",
        f"  FETCH_SIZE copy {out['fetch']['copy_kib']:.1f} KiB -> factor {out['fetch']['factor']:.4f};",
        f"  WRITE_SIZE copy {out['write']['copy_kib']:.1f} KiB -> factor {out['write']['factor']:.4f};",
        f"  attention launch: FETCH_SIZE {out['fetch']['attn_kib']:.1f} KiB, "
        f"WRITE_SIZE {out['write']['attn_kib']:.1f} KiB (raw).",
    ]
    return "\n".join(lines) + "\n"


def traffic_probe():
    import torch
    from paper_2608_12780_amd import inputs
    from paper_2608_12780_amd.layer import ScopeLayer
    cfg = inputs.CONFIGS["hy720"]
    x = inputs.generate(cfg)
    dev = torch.device("cuda", 0)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    q, k, v = up(x.q_bits), up(x.k_bits), up(x.v_bits)
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev)
    layer.forward(q, k, v, torch.from_numpy(x.init_q).to(dev),
                  torch.from_numpy(x.init_k).to(dev))
    torch.cuda.synchronize()
    log("[probe] layer done")
    src = torch.ones(CALIB_BYTES // 2, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    log("[probe] calibration copy done")
    layer.attend(q, k, v)
    torch.cuda.synchronize()
    log("[probe] attention done")


def measured_peaks(torch, dev=None, reps=5):
    """Achievable roofs on this GPU, measured with the library's diagnostic
    kernels: a 1 GiB device copy (HBM GB/s counting read + write bytes) and
    a loop of independent bf16 32x32x16 matrix products from registers."""
    from paper_2608_12780_amd import binding as B
    dev = dev or torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    B.scope_debug_copy(src, dst)
    torch.cuda.synchronize()
    c_ms = time_events(torch, lambda: B.scope_debug_copy(src, dst), reps, stream)
    del src, dst
    blocks, iters = 2048, 4096
    out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    B.scope_debug_mfma_loop(out, blocks, 64)
    torch.cuda.synchronize()
    m_ms = time_events(torch, lambda: B.scope_debug_mfma_loop(out, blocks, iters), reps, stream)
    flops = blocks * 4 * 8 * 32768.0 * iters
    return {"hbm_copy_gbs": round(2 * CALIB_BYTES / (c_ms * 1e-3) / 1e9, 1),
            "mfma_bf16_tflops": round(flops / (m_ms * 1e-3) / 1e12, 1),
            "copy_ms": round(c_ms, 4), "mfma_loop_ms": round(m_ms, 4)}


def counters_probe():
    """The program profiled by the counter passes: the measured-peak kernels
    once (their counters calibrate the others), then the HunyuanVideo-720p-like
    layer twice (the first run warms up)."""
    import torch
    from paper_2608_12780_amd import inputs
    from paper_2608_12780_amd.layer import ScopeLayer
    dev = torch.device("cuda", 0)
    peaks = measured_peaks(torch, dev, reps=1)
    log(f"[counters] peaks {peaks}")
    cfg = inputs.CONFIGS["hy720"]
    x = inputs.generate(cfg)
    up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
    q, k, v = up(x.q_bits), up(x.k_bits), up(x.v_bits)
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev)
    iq, ik = torch.from_numpy(x.init_q).to(dev), torch.from_numpy(x.init_k).to(dev)
    for i in range(2):
        layer.forward(q, k, v, iq, ik)
        torch.cuda.synchronize()
        log(f"[counters] layer run {i + 1}/2 done")
    counts = layer.counts.cpu().numpy().astype(np.float64)
    selc = layer.sel_counts.cpu().numpy().astype(np.float64)
    print(json.dumps({"attention_algorithmic_flops": 4.0 * cfg.d * float((counts * selc).sum()),
                      "selected_total": float(selc.sum()), "peaks": peaks}), flush=True)


COUNTER_PASSES = [
    "SQ_CYCLES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_VALU_MFMA_COEXEC_CYCLES "
    "SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_MFMA SQ_INSTS_VALU GRBM_GUI_ACTIVE",
    "SQ_INSTS_LDS SQ_WAIT_INST_LDS SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_VALU_TRANS_F32 "
    "SQ_WAIT_INST_ANY SQ_WAIT_ANY SQ_ACTIVE_INST_VALU",
    "FETCH_SIZE GRBM_GUI_ACTIVE",
    "WRITE_SIZE TCC_HIT_sum TCC_MISS_sum",
    "SQ_INSTS_SALU SQ_INSTS_VMEM SQ_INSTS_SMEM SQ_ACTIVE_INST_LDS SQ_ACTIVE_INST_MISC SQ_WAVES "
    "SQ_INSTS_VALU_FMA_F32 SQ_INSTS_VALU_MUL_F32 TA_BUSY_avr TA_BUSY_max GRBM_GUI_ACTIVE",
]
COUNTER_REGEX = "attn_kernel|km_assign|km_accum|select_base|select_final|code_parts_kernel|peak_"
# MI355X: 8 XCDs x 4 shader engines x 8 CUs x 4 SIMDs
XCDS, SIMDS_PER_SE = 8, 32


def _short_kernel(name):
    import re
    name = re.sub(r"scope::\(anonymous namespace\)::", "", name)
    name = re.sub(r"^void ", "", name)
    name = re.sub(r"\(.*$", "", name)
    return name


def counter_summary(csvs, cmd):
    """Per-kernel table of the counter passes (rocprofv3 --pmc CSVs): MFMA and
    VALU activity, LDS behaviour, HBM traffic (scaled by the calibration copy)
    and occupancy from each kernel's resources.  Counters are summed over
    every SIMD/SE/channel of the GPU by rocprofv3; SQ_CYCLES (per SIMD) is the
    denominator of per-SIMD busy fractions."""
    import csv
    import collections
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    res = {}
    for path in csvs:
        per = collections.defaultdict(lambda: collections.defaultdict(float))
        meta = {}
        for r in csv.DictReader(open(path)):
            key = (_short_kernel(r["Kernel_Name"]), r["Dispatch_Id"])
            per[key][r["Counter_Name"]] += float(r["Counter_Value"])
            meta[key] = r
        for (kname, _), cv in per.items():
            m = meta[(kname, _)]
            for c, v in cv.items():
                agg[kname][c].append(v)
            agg[kname]["_dur_us"].append((int(m["End_Timestamp"]) - int(m["Start_Timestamp"])) / 1e3)
            res[kname] = dict(vgpr=int(m.get("VGPR_Count") or m.get("Arch_VGPR_Count") or 0),
                              agpr=int(m.get("Accum_VGPR_Count") or 0),
                              lds=int(m.get("LDS_Block_Size") or 0),
                              wg=int(m.get("Workgroup_Size") or 0),
                              sgpr=int(m.get("SGPR_Count") or 0))
    mean = {k: {c: float(np.mean(v)) for c, v in d.items()} for k, d in agg.items()}

    def occupancy(r):
        # the trace's VGPR_Count is half the allocated count on this GPU
        # (granules of 8 registers read as granules of 4): the compiler
        # reports 190 VGPRs for attn_kernel_dma, the trace 96
        regs = max(2 * r["vgpr"] + r["agpr"], 1)
        by_regs = 512 // (((regs + 7) // 8) * 8)
        waves_per_block = max(1, (r["wg"] + 63) // 64)
        by_lds = (160 * 1024 // r["lds"]) * waves_per_block / 4.0 if r["lds"] else 8
        return min(8, by_regs, by_lds)

    cal = mean.get("peak_copy_kernel", {})
    f_fac = (CALIB_BYTES / 1024.0) / cal["FETCH_SIZE"] if cal.get("FETCH_SIZE") else None
    w_fac = (CALIB_BYTES / 1024.0) / cal["WRITE_SIZE"] if cal.get("WRITE_SIZE") else None
    lines = [f"command: {cmd}", "",
             "rocprofv3 --pmc passes (each its own run):"]
    lines += [f"  {p}" for p in COUNTER_PASSES]
    lines += ["",
              "per kernel, averaged over its dispatches:",
              "  dur       kernel duration under counter collection (us)",
              "  GHz       GRBM_GUI_ACTIVE / 8 XCDs / duration: the shader clock during the kernel",
              "  mfma%     SQ_VALU_MFMA_BUSY_CYCLES / (SQ_CYCLES * 32 SIMDs per shader engine):",
              "            the matrix pipe's busy fraction, over all 1024 SIMDs",
              "  valu%     4 * SQ_ACTIVE_INST_VALU / the same SIMD cycles (wave time on VALU issue)",
              "  coexec%   SQ_VALU_MFMA_COEXEC_CYCLES / SQ_VALU_MFMA_BUSY_CYCLES (a VALU op issued",
              "            while the matrix pipe was busy)",
              "  bf16 TF   SQ_INSTS_VALU_MFMA_MOPS_BF16 * 512 / dur (performed, padding included)",
              "  valu/mfma SQ_INSTS_VALU / SQ_INSTS_MFMA (SQ_INSTS_VALU counts MFMAs too)",
              "  ldsw%     SQ_WAIT_INST_LDS * 4 / SQ_WAVE_CYCLES*4 (wave time waiting to issue LDS)",
              "  bank%     SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE",
              "  wait%     SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES (waiting on a dependency)",
              "  fetch/write GB  FETCH_SIZE, WRITE_SIZE scaled by the calibration copy of "
              f"{CALIB_BYTES} bytes",
              "  GB/s      (fetch + write bytes) / duration",
              "  TA busy%  TA_BUSY_avr / (GRBM_GUI_ACTIVE / 8): the address unit of buffer loads",
              "  vgpr      VGPR_Count as the trace reports it (half the allocated registers)",
              "  occ       waves per SIMD the kernel's registers and LDS allow", ""]
    if f_fac:
        lines.append(f"calibration copy: FETCH_SIZE factor {f_fac:.4f}, WRITE_SIZE factor "
                     f"{(w_fac or float('nan')):.4f}")
    pk = mean.get("peak_mfma_kernel")
    if pk and pk.get("SQ_CYCLES"):
        lines.append(f"MFMA loop: mfma% {100 * pk['SQ_VALU_MFMA_BUSY_CYCLES'] / (pk['SQ_CYCLES'] * SIMDS_PER_SE):.1f}, "
                     f"clock {pk['GRBM_GUI_ACTIVE'] / XCDS / (pk['_dur_us'] * 1e3):.2f} GHz, "
                     f"bf16 {pk['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * 512 / (pk['_dur_us'] * 1e-6) / 1e12:.0f} TFLOP/s "
                     "(the measured matrix roof)")
    lines += ["", f"{'kernel':<44} {'calls':>5} {'dur us':>9} {'GHz':>5} {'mfma%':>6} {'coexec%':>7} "
              f"{'valu%':>6} {'bf16 TF':>8} {'valu/mfma':>9} {'ldsw%':>6} {'bank%':>6} {'wait%':>6} "
              f"{'fetch GB':>9} {'write GB':>9} {'GB/s':>6} {'TA busy%':>8} {'vgpr':>5} {'agpr':>5} "
              f"{'lds KB':>6} {'occ':>4}"]
    for kname in sorted(mean, key=lambda k: -mean[k]["_dur_us"] * len(agg[k]["_dur_us"])):
        m, r = mean[kname], res[kname]
        g = lambda c: m.get(c)
        def pct(a, b):
            return f"{100 * a / b:.1f}" if a is not None and b else "-"
        # SQ_CYCLES counts each of the SE_INSTANCES shader engines once; the
        # MFMA busy and VALU activity counts cover every SIMD of the GPU
        simd_cycles = g("SQ_CYCLES") * SIMDS_PER_SE if g("SQ_CYCLES") else None
        mf = pct(g("SQ_VALU_MFMA_BUSY_CYCLES"), simd_cycles)
        va = pct(4 * g("SQ_ACTIVE_INST_VALU") if g("SQ_ACTIVE_INST_VALU") else None, simd_cycles)
        ghz = (f"{g('GRBM_GUI_ACTIVE') / XCDS / (m['_dur_us'] * 1e3):.2f}"
               if g("GRBM_GUI_ACTIVE") else "-")
        co = pct(g("SQ_VALU_MFMA_COEXEC_CYCLES"), g("SQ_VALU_MFMA_BUSY_CYCLES"))
        tf = (f"{g('SQ_INSTS_VALU_MFMA_MOPS_BF16') * 512 / (m['_dur_us'] * 1e-6) / 1e12:.0f}"
              if g("SQ_INSTS_VALU_MFMA_MOPS_BF16") else "-")
        vm = f"{g('SQ_INSTS_VALU') / g('SQ_INSTS_MFMA'):.1f}" if g("SQ_INSTS_MFMA") else "-"
        lw = pct(g("SQ_WAIT_INST_LDS"), g("SQ_WAVE_CYCLES"))
        bk = pct(g("SQ_LDS_BANK_CONFLICT"), g("SQ_LDS_IDX_ACTIVE"))
        wt = pct(g("SQ_WAIT_INST_ANY"), g("SQ_WAVE_CYCLES"))
        fe = f"{g('FETCH_SIZE') * 1024 * f_fac / 1e9:.3f}" if g("FETCH_SIZE") is not None and f_fac else "-"
        wr = f"{g('WRITE_SIZE') * 1024 * w_fac / 1e9:.3f}" if g("WRITE_SIZE") is not None and w_fac else "-"
        ta = (f"{g('TA_BUSY_avr') / (g('GRBM_GUI_ACTIVE') / XCDS) * 100:.1f}"
              if g("TA_BUSY_avr") and g("GRBM_GUI_ACTIVE") else "-")
        hbm = ((g("FETCH_SIZE") * f_fac + g("WRITE_SIZE") * w_fac) * 1024 / (m["_dur_us"] * 1e-6) / 1e9
               if g("FETCH_SIZE") is not None and g("WRITE_SIZE") is not None and f_fac and w_fac else None)
        hb = f"{hbm:.0f}" if hbm is not None else "-"
        lines.append(f"{kname[:44]:<44} {len(agg[kname]['_dur_us']):>5} {m['_dur_us']:>9.1f} {ghz:>5} {mf:>6} "
                     f"{co:>7} {va:>6} {tf:>8} {vm:>9} {lw:>6} {bk:>6} {wt:>6} {fe:>9} {wr:>9} {hb:>6} {ta:>8} "
                     f"{r['vgpr']:>5} {r['agpr']:>5} {r['lds'] / 1024:>6.1f} {occupancy(r):>4.1f}")
    lines += ["", "raw means per dispatch:"]
    for kname in sorted(mean):
        lines.append(f"  {kname}: " + ", ".join(f"{c}={v:.6g}" for c, v in sorted(mean[kname].items())))
    return "\n".join(lines) + "\n"


def lines_summary(kind, paths, cmd):
    """Table of bench.py JSON lines (one per file): kind "workloads" (one
    line per workload) or "rho" (one line per rho of a workload)."""
    recs = []
    for p in paths:
        line = [l for l in open(p).read().splitlines() if l.startswith("{")][-1]
        recs.append(json.loads(line))
    out = [f"command: {cmd}", ""]
    if kind == "workloads":
        out += ["the whole layer (5 calls, every head) per workload, HIP-event time;",
                "SDPA = torch scaled_dot_product_attention (flash backend) on the same Q/K/V, same GPU", "",
                f"{'workload':>26} {'heads':>5} {'N':>7} {'layer ms':>9} {'eff TFLOP/s':>11} "
                f"{'q-kmeans':>8} {'k-kmeans':>8} {'select':>7} {'attn ms':>8} {'attn MFMA':>9} "
                f"{'kept':>6} {'SDPA ms':>8} {'speedup':>7}"]
        for r in recs:
            c, st = r["config"], r["stages_ms"]
            sd = r.get("sdpa_ms")
            sp = r.get("speedup_vs_sdpa")
            out.append(f"{c['workload']:>26} {c['heads']:>5} {c['n']:>7} {r['ms_per_step']:>9.2f} "
                       f"{r['value']:>11.1f} {st['cluster_queries']:>8.2f} "
                       f"{st['cluster_key_subspaces']:>8.2f} {st['select']:>7.2f} "
                       f"{st['sparse_attention']:>8.2f} {100 * r['roofline']['frac']:>8.1f}% "
                       f"{r['retained_fraction']:>6.3f} "
                       f"{(f'{sd:8.1f}' if sd is not None else f'{chr(45):>8}')} "
                       f"{(f'{sp:6.2f}x' if sp is not None else f'{chr(45):>7}')}")
    else:
        c = recs[0]["config"]
        out += [f"workload: {c['workload']} ({c['heads']} heads, N = {c['n']}, d = {c['d']}); "
                "event timings in ms", "",
                f"{'rho':>5} {'layer':>8} {'q-kmeans':>9} {'k-kmeans':>9} {'tables':>7} {'select':>7} "
                f"{'attention':>10} {'attn TF/s':>10} {'retained':>9} {'k_head':>8} {'floor binds':>12}"]
        for r in sorted(recs, key=lambda r: r["config"]["rho"]):
            st = r["stages_ms"]
            out.append(f"{r['config']['rho']:>5} {r['ms_per_step']:>8.2f} {st['cluster_queries']:>9.2f} "
                       f"{st['cluster_key_subspaces']:>9.2f} {st['proxy_scores']:>7.2f} {st['select']:>7.2f} "
                       f"{st['sparse_attention']:>10.2f} {r['roofline']['achieved']:>10.1f} "
                       f"{r['retained_fraction']:>9.3f} {r['k_head_mean']:>8.0f} "
                       f"{r['floor_bound_fraction']:>12.3f}")
    out += ["", "JSON lines:"] + [json.dumps(r) for r in recs]
    return "\n".join(out) + "\n"


def main():
    if len(sys.argv) >= 2 and sys.argv[1] == "--lines-summary":
        # --lines-summary workloads|rho "COMMAND" FILE...
        sys.stdout.write(lines_summary(sys.argv[2], sys.argv[4:], sys.argv[3]))
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--traffic-summary":
        sys.stdout.write(traffic_summary(sys.argv[2], sys.argv[3]))
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--traffic-probe":
        traffic_probe()
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--counters":
        counters_probe()
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--counter-summary":
        # --counter-summary "COMMAND" CSV...
        sys.stdout.write(counter_summary(sys.argv[3:], sys.argv[2]))
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--peaks":
        import torch
        print(json.dumps(measured_peaks(torch)), flush=True)
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--recall-study":
        print(json.dumps(recall_study()), flush=True)
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--partition-study":
        print(json.dumps(partition_study()), flush=True)
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--policy-study":
        print(json.dumps(policy_study()), flush=True)
        return
    if len(sys.argv) >= 2 and sys.argv[1] == "--trace-summary":
        # --trace-summary TRACE_CSV "COMMAND" [BENCH_LOG]
        line = None
        if len(sys.argv) > 4:
            line = [l for l in open(sys.argv[4]).read().splitlines() if l.startswith("{")][-1]
        sys.stdout.write(trace_summary(sys.argv[2], sys.argv[3], line))
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="hy720")
    ap.add_argument("--rho", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the layer "
              "shards by head with no communication inside it, so a multi-GPU "
              "figure would be the one-GPU figure times the GPU count.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_12780_amd import inputs
    from paper_2608_12780_amd.layer import DenseAttention, ScopeLayer

    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        sys.exit(1)
    cfg = inputs.CONFIGS[args.config]
    if args.rho is not None:
        cfg = cfg.with_(rho=args.rho)
    log(f"[bench] generating {cfg.name}: heads={cfg.heads} n={cfg.n} d={cfg.d}")
    t0 = time.perf_counter()
    x = inputs.generate(cfg)
    log(f"[bench] inputs ready in {time.perf_counter() - t0:.1f}s")
    dev = torch.device("cuda", 0)
    if cfg.dtype == "bf16":
        up = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
        q, k, v = up(x.q_bits), up(x.k_bits), up(x.v_bits)
    else:
        q, k, v = (torch.from_numpy(a).to(dev) for a in (x.q, x.k, x.v))
    iq = torch.from_numpy(x.init_q).to(dev)
    ik = torch.from_numpy(x.init_k).to(dev)
    layer = ScopeLayer(cfg.heads, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                       cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev)
    stream = torch.cuda.current_stream()
    nstage = 5
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(nstage + 1)]
          for _ in range(args.steps)]

    for i in range(args.warmup):
        layer.forward(q, k, v, iq, ik)
        torch.cuda.synchronize()
        log(f"[bench] warmup step {i + 1}/{args.warmup} done")

    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        layer.forward(q, k, v, iq, ik, marks=lambda j, i=i: ev[i][j].record(stream))
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_start) * 1e3 / args.steps
    stage_names = ["cluster_queries", "cluster_key_subspaces", "proxy_scores",
                   "select", "sparse_attention"]
    stage_ms = {n_: float(np.mean([ev[i][j].elapsed_time(ev[i][j + 1])
                                   for i in range(args.steps)]))
                for j, n_ in enumerate(stage_names)}
    layer_ms = float(np.mean([ev[i][0].elapsed_time(ev[i][nstage])
                              for i in range(args.steps)]))
    log(f"[bench] timed {args.steps} steps: {layer_ms:.2f} ms/layer (wall {wall_ms:.2f})")

    counts = layer.counts.cpu().numpy().astype(np.float64)
    selc = layer.sel_counts.cpu().numpy().astype(np.float64)
    pairs = float((counts * selc).sum())
    attn_flops = 4.0 * cfg.d * pairs
    attn_ms = stage_ms["sparse_attention"]
    achieved = attn_flops / (attn_ms * 1e-3) / 1e12
    retained = pairs / (cfg.heads * float(cfg.n) * cfg.n)
    khead = layer.k_head.cpu().numpy()
    sbytes = stage_bytes(cfg, float(selc.sum()))
    topp = layer.topp_counts.cpu().numpy().astype(np.float64)
    floor_bound = float((topp < cfg.k_fix).mean())

    result = {
        "metric": "SCOPE layer latency (ms) and effective TFLOP/s vs dense attention, 720p; % MFMA peak",
        "value": round(dense_flops(cfg) / (layer_ms * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(layer_ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": WORKLOAD_NAMES.get(cfg.name, cfg.name),
            "heads": cfg.heads, "grid": list(cfg.grid), "n": cfg.n, "d": cfg.d,
            "rope_split": list(cfg.split), "c_q": cfg.c_q, "c_m": cfg.c_m,
            "iters": cfg.iters, "rho": cfg.rho, "k_fix": cfg.k_fix,
        },
        "roofline": {
            "kernel": "sparse_attention",
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": committed_traffic(cfg.name),
            "algorithmic_flops_per_launch": attn_flops,
        },
        "stages_ms": {k_: round(v_, 3) for k_, v_ in stage_ms.items()},
        "hbm": {k_: {"bytes": b_, "gbs": round(b_ / (stage_ms[k_] * 1e-3) / 1e9, 1),
                     "frac": round(b_ / (stage_ms[k_] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
                for k_, b_ in sbytes.items()},
        "wall_ms_per_step": round(wall_ms, 3),
        "retained_fraction": round(retained, 4),
        "k_head_mean": float(khead.mean()),
        "floor_bound_fraction": round(floor_bound, 4),
    }

    # the same roofs measured on this GPU (copy bandwidth, MFMA loop)
    peaks = measured_peaks(torch, dev)
    result["measured_peaks"] = peaks
    result["roofline"]["measured_peak"] = peaks["mfma_bf16_tflops"]
    result["roofline"]["frac_of_measured"] = round(achieved / peaks["mfma_bf16_tflops"], 4)
    for k_, h_ in result["hbm"].items():
        h_["frac_of_measured"] = round(h_["gbs"] / peaks["hbm_copy_gbs"], 4)
    log(f"[bench] measured peaks: {peaks}")

    # one GPU's share of an 8-GPU node when the layer is sharded by head
    share = max(1, math.ceil(cfg.heads / 8))
    if share < cfg.heads:
        sub = ScopeLayer(share, cfg.n, cfg.d, cfg.ranges, cfg.c_q, (cfg.c_m,) * 3,
                         cfg.iters, cfg.rho, cfg.k_fix, dtype=cfg.dtype, device=dev)
        qs, ks, vs = q[:share].contiguous(), k[:share].contiguous(), v[:share].contiguous()
        iqs, iks = iq[:share].contiguous(), ik[:share].contiguous()
        sub.forward(qs, ks, vs, iqs, iks)
        torch.cuda.synchronize()
        sh_ms = time_events(torch, lambda: sub.forward(qs, ks, vs, iqs, iks), 3, stream)
        result["one_gpu_share"] = {"heads": share, "of_heads": cfg.heads, "gpus": 8,
                                   "ms_per_step": round(sh_ms, 3)}
        log(f"[bench] one GPU's share ({share} of {cfg.heads} heads): {sh_ms:.2f} ms")
        del sub

    if not args.no_dense:
        dense = DenseAttention(cfg.heads, cfg.n, cfg.d, cfg.dtype, dev)
        dense.forward(q, k, v)
        torch.cuda.synchronize()
        d_ms = time_events(torch, lambda: dense.forward(q, k, v), 2, stream)
        result["dense_mode_ms"] = round(d_ms, 3)
        result["speedup_vs_dense_mode"] = round(d_ms / layer_ms, 3)
        result["dense_mode_tflops"] = round(dense_flops(cfg) / (d_ms * 1e-3) / 1e12, 2)
        log(f"[bench] library dense mode: {d_ms:.2f} ms")
        del dense
        s_ms, backend = sdpa_ms(torch, q, k, v, 2)
        result["sdpa_ms"] = None if s_ms is None else round(s_ms, 3)
        result["sdpa_backend"] = backend
        if s_ms is not None:
            result["speedup_vs_sdpa"] = round(s_ms / layer_ms, 3)
            log(f"[bench] torch sdpa ({backend}): {s_ms:.2f} ms")

    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(cfg, x, None)
        log(f"[bench] cpu baseline: {result['cpu_baseline']['layer_s_extrapolated']:.1f} s/layer")

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
