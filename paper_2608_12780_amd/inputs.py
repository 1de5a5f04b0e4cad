"""Seeded synthetic inputs for the SCOPE attention layer.

This module only *generates data*: it holds none of the layer's arithmetic
(no clustering, scoring, selection or attention).  It is shared by the test
suite, the benchmark and the oracle harness, and it is the single source of
every random number the layer consumes (the k-means initial rows are drawn
here and passed in as inputs).

Workload recipe (post-3D-RoPE queries/keys of a video DiT head, Sec. 3.1):
  * tokens live on a latent grid (T, H, W), token index i = (t*H + h)*W + w;
  * R spatially smooth fields f_r over the grid (sums of three random cosine
    waves with per-axis frequencies in {0,1,2}), standardised over the grid;
  * per head a shared direction c_h ~ N(0, I_d) and basis B_h ~ N(0,1)^{R x d};
    Q_pre = 0.8 (c_h + F B_h)/sqrt(1+R) + 0.6 eps_Q, K_pre likewise with eps_K,
    V ~ N(0, 1);
  * 3D RoPE on Q_pre and K_pre: each axis (t, h, w) owns a contiguous channel
    range (Sec. 3.3: the rotary transforms of the three coordinates act on
    disjoint channel ranges), rotated as interleaved pairs with angle
    pos_axis * 10000^(-2i/d_axis);
  * optional per-head temperature tau_h ~ logU[0.25, 4] on Q (stress case);
  * storage: fp32 (Tiny) or bf16 with round-to-nearest-even.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import math
import os

import numpy as np


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """One workload: shapes, clustering sizes and selection knobs."""
    name: str
    heads: int
    grid: tuple            # (T, H, W) latent grid
    d: int                 # head dimension
    split: tuple           # channel lengths of the (t, h, w) RoPE ranges
    c_q: int               # query clusters
    c_m: int               # centroids per key subspace (same for T, H, W)
    iters: int             # Lloyd iterations
    rho: float             # Top-p threshold
    k_fix: int             # fixed Top-k floor, ceil(alpha * N)
    dtype: str             # "f32" or "bf16"
    fields: int            # number of smooth fields R
    seed: int
    stress: bool = False   # per-head temperature on Q

    @property
    def n(self) -> int:
        t, h, w = self.grid
        return t * h * w

    @property
    def ranges(self):
        off = [0, self.split[0], self.split[0] + self.split[1]]
        return tuple(off), tuple(self.split)

    def with_(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


def ceil_tenth(n: int) -> int:
    """k_fix for alpha = 0.1, computed in integers: ceil(n / 10)."""
    return (n + 9) // 10


CONFIGS = {
    "tiny": LayerConfig("tiny", 2, (4, 8, 8), 64, (16, 24, 24), 8, 8, 5, 0.9,
                        16, "f32", 4, 1),
    "wan480": LayerConfig("wan480", 40, (21, 30, 52), 128, (44, 42, 42), 128, 64,
                          10, 0.9, ceil_tenth(21 * 30 * 52), "bf16", 8, 2),
    "wan720": LayerConfig("wan720", 40, (21, 45, 80), 128, (44, 42, 42), 256, 128,
                          10, 0.9, ceil_tenth(21 * 45 * 80), "bf16", 8, 3),
    "hy720": LayerConfig("hy720", 24, (33, 45, 80), 128, (16, 56, 56), 256, 128,
                         10, 0.9, ceil_tenth(33 * 45 * 80), "bf16", 8, 4),
    "stress": LayerConfig("stress", 24, (33, 45, 80), 128, (16, 56, 56), 256, 128,
                          10, 0.9, ceil_tenth(33 * 45 * 80), "bf16", 8, 5,
                          stress=True),
}


PARTITIONS = ("1", "2", "3-random", "3-rope", "4", "8")


def partition_sets(cfg: LayerConfig, kind: str, seed: int = 0):
    """Channel sets I_1..I_M of the key-partition ablation (Table 3), each
    ascending: "1" all channels (full-dimensional clustering); "2", "4",
    "8" equal contiguous ranges; "3-rope" the t/h/w RoPE ranges of the
    workload; "3-random" a seeded random split of the channels into sets of
    the RoPE range sizes."""
    d = cfg.d
    if kind == "3-rope":
        off, ln = cfg.ranges
        return [np.arange(o, o + l, dtype=np.int32) for o, l in zip(off, ln)]
    if kind == "3-random":
        perm = np.random.default_rng([cfg.seed, 1009, seed]).permutation(d)
        cuts = np.cumsum(cfg.split)[:-1]
        return [np.sort(x).astype(np.int32) for x in np.split(perm, cuts)]
    m = int(kind)
    if m < 1 or d % m:
        raise ValueError(f"cannot split {d} channels into {m} equal ranges")
    return [np.arange(i * d // m, (i + 1) * d // m, dtype=np.int32) for i in range(m)]


def partition_init(cfg: LayerConfig, M: int, c_m: int, heads: int | None = None,
                   head_offset: int = 0, seed: int = 0) -> np.ndarray:
    """Seeded k-means starting rows for M key subspaces: [heads][M][c_m]."""
    nh = cfg.heads if heads is None else heads
    out = np.empty((nh, M, c_m), np.int32)
    for hi in range(nh):
        rng = np.random.default_rng([cfg.seed, 2003, seed, head_offset + hi])
        for m in range(M):
            out[hi, m] = init_rows(rng, cfg.n, c_m)
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bits -> the exactly equal fp32 values."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _grid_coords(grid):
    t, h, w = grid
    tt, hh, ww = np.meshgrid(np.arange(t), np.arange(h), np.arange(w),
                             indexing="ij")
    return tt.reshape(-1), hh.reshape(-1), ww.reshape(-1)


def _rope_tables(cfg: LayerConfig):
    """cos/sin per token and channel pair, for the three axis ranges."""
    coords = _grid_coords(cfg.grid)
    (offs, lens) = cfg.ranges
    cos = np.empty((cfg.n, cfg.d // 2), np.float32)
    sin = np.empty((cfg.n, cfg.d // 2), np.float32)
    for axis in range(3):
        dm = lens[axis]
        pairs = dm // 2
        freq = 10000.0 ** (-2.0 * np.arange(pairs) / dm)
        ang = coords[axis][:, None].astype(np.float64) * freq[None, :]
        p0 = offs[axis] // 2
        cos[:, p0:p0 + pairs] = np.cos(ang)
        sin[:, p0:p0 + pairs] = np.sin(ang)
    return cos, sin


def _apply_rope(x: np.ndarray, cos, sin) -> np.ndarray:
    x0 = x[:, 0::2]
    x1 = x[:, 1::2]
    out = np.empty(x.shape, np.float32)
    out[:, 0::2] = x0 * cos - x1 * sin
    out[:, 1::2] = x0 * sin + x1 * cos
    return out


def _fields(rng, cfg: LayerConfig, coords):
    t, h, w = cfg.grid
    tt, hh, ww = coords
    out = np.empty((cfg.n, cfg.fields), np.float64)
    for r in range(cfg.fields):
        amp = rng.standard_normal(3)
        kap = rng.integers(0, 3, size=(3, 3))
        phi = rng.uniform(0.0, 2.0 * math.pi, size=3)
        f = np.zeros(cfg.n, np.float64)
        for a in range(3):
            arg = 2.0 * math.pi * (kap[a, 0] * tt / t + kap[a, 1] * hh / h
                                   + kap[a, 2] * ww / w) + phi[a]
            f += amp[a] * np.cos(arg)
        f -= f.mean()
        sd = f.std()
        out[:, r] = f / sd if sd > 1e-9 else 0.0
    return out


def init_rows(rng, n: int, c: int) -> np.ndarray:
    """Distinct seeded k-means starting rows."""
    return np.sort(rng.choice(n, size=c, replace=False)).astype(np.int32)


def default_init_rows(n: int, c: int) -> np.ndarray:
    """The library's default starting rows: floor((2r+1) n / (2c))."""
    r = np.arange(c, dtype=np.int64)
    return ((2 * r + 1) * n // (2 * c)).astype(np.int32)


@dataclasses.dataclass
class LayerInputs:
    cfg: LayerConfig
    q: np.ndarray          # fp32 [heads][n][d]  (bf16-exact for bf16 configs)
    k: np.ndarray
    v: np.ndarray
    q_bits: np.ndarray | None   # uint16 bf16 bits, or None for fp32 configs
    k_bits: np.ndarray | None
    v_bits: np.ndarray | None
    init_q: np.ndarray     # int32 [heads][c_q]
    init_k: np.ndarray     # int32 [heads][3][c_m]
    tau: np.ndarray        # fp64 [heads] temperature applied to Q (1 if none)


def generate(cfg: LayerConfig, heads: int | None = None,
             head_offset: int = 0, threads: int | None = None) -> LayerInputs:
    """Generate heads [head_offset, head_offset + heads) of a workload.

    Each head has its own child stream of SeedSequence(cfg.seed), so a
    subset of heads is identical to the same heads of the full layer, and
    heads are generated in parallel threads with identical results.
    """
    nh = cfg.heads if heads is None else heads
    children = np.random.SeedSequence(cfg.seed).spawn(cfg.heads)
    coords = _grid_coords(cfg.grid)
    cos, sin = _rope_tables(cfg)
    n, d, R = cfg.n, cfg.d, cfg.fields
    q = np.empty((nh, n, d), np.float32)
    k = np.empty((nh, n, d), np.float32)
    v = np.empty((nh, n, d), np.float32)
    init_q = np.empty((nh, cfg.c_q), np.int32)
    init_k = np.empty((nh, 3, cfg.c_m), np.int32)
    tau = np.ones(nh, np.float64)
    def one(hi):
        rng = np.random.default_rng(children[head_offset + hi])
        F = _fields(rng, cfg, coords)
        c_h = rng.standard_normal(d)
        B_h = rng.standard_normal((R, d))
        shared = ((c_h[None, :] + F @ B_h) * (0.8 / math.sqrt(1.0 + R))
                  ).astype(np.float32)
        eq = rng.standard_normal((n, d), dtype=np.float32)
        ek = rng.standard_normal((n, d), dtype=np.float32)
        vv = rng.standard_normal((n, d), dtype=np.float32)
        t_h = math.exp(rng.uniform(math.log(0.25), math.log(4.0)))
        eq *= np.float32(0.6)
        ek *= np.float32(0.6)
        qh = _apply_rope(shared + eq, cos, sin)
        if cfg.stress:
            tau[hi] = t_h
            qh *= np.float32(t_h)
        q[hi] = qh
        k[hi] = _apply_rope(shared + ek, cos, sin)
        v[hi] = vv
        init_q[hi] = init_rows(rng, n, cfg.c_q)
        for m in range(3):
            init_k[hi, m] = init_rows(rng, n, cfg.c_m)
        if cfg.dtype == "bf16":
            qb[hi], kb[hi], vb[hi] = bf16_bits(q[hi]), bf16_bits(k[hi]), bf16_bits(v[hi])
            q[hi], k[hi], v[hi] = bf16_widen(qb[hi]), bf16_widen(kb[hi]), bf16_widen(vb[hi])

    if cfg.dtype == "bf16":
        qb = np.empty((nh, n, d), np.uint16)
        kb = np.empty((nh, n, d), np.uint16)
        vb = np.empty((nh, n, d), np.uint16)
    else:
        qb = kb = vb = None
    workers = max(1, min(nh, threads or os.cpu_count() or 1, 16))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        list(ex.map(one, range(nh)))
    return LayerInputs(cfg, q, k, v, qb, kb, vb, init_q, init_k, tau)
