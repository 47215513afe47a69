"""Seeded synthetic inputs for forced-weight subset evaluation.

This module only draws random numbers and lays them out in the row-major
shapes the library takes; it computes nothing that the method computes (no
logits, weights, sums or selections).  Both the GPU path and the CPU oracle
consume exactly the arrays produced here.

Layout (all contiguous, row-major):
  q     [H][G][d]   query rows, G rows per key/value unit
  k, v  [H][n][d]   keys and values of each unit
  scale [H]         float32 logit scale per unit
  bias  [n]         float32 additive logit bias shared by all rows, or None
For dtype "bf16" the arrays hold raw bfloat16 bit patterns (uint16); for
"f32" they hold float32.  ``as_f64`` widens either exactly.

Stream convention: every unit (a (layer, kv-head) cell, or a block of rows for
the one-row-per-unit workloads) draws from its own PCG64 stream seeded with
``SeedSequence([workload_id, seed, unit_index])``; within a stream the draw
order is q, k, v, then any extras.  bf16 values are drawn in float32 and
rounded to nearest-even.

The five workloads mirror the shapes the paper measures on (five model
families, grouped-query heads, sinks, outlier key channels, heavy hitters,
per-head temperature) — synthetic stand-ins, since no captured rows, model
weights or corpora are used.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Optional, Sequence, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"


# ----------------------------------------------------------------------------
# bfloat16 storage helpers (input preparation, not method arithmetic)
# ----------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest-even) and return the uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    t = b >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += b
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen uint16 bfloat16 bits to float32 (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


@dataclass
class Rows:
    """One batch of attention rows in the layout the C ABI takes."""

    dtype: str
    q: np.ndarray
    k: np.ndarray
    v: Optional[np.ndarray]
    scale: np.ndarray
    bias: Optional[np.ndarray] = None

    @property
    def H(self) -> int:
        return int(self.q.shape[0])

    @property
    def G(self) -> int:
        return int(self.q.shape[1])

    @property
    def n(self) -> int:
        return int(self.k.shape[1])

    @property
    def d(self) -> int:
        return int(self.q.shape[2])

    def as_f64(self, name: str) -> np.ndarray:
        a = getattr(self, name)
        if a is None:
            return None
        if self.dtype == BF16 and a.dtype == np.uint16:
            return bf16_to_f32(a).astype(np.float64)
        return np.asarray(a, dtype=np.float64)

    def unit(self, h: int) -> "Rows":
        """The rows of one unit as a batch of its own (H = 1)."""
        return Rows(self.dtype, self.q[h:h + 1], self.k[h:h + 1],
                    None if self.v is None else self.v[h:h + 1],
                    self.scale[h:h + 1], self.bias)


@dataclass
class Workload:
    name: str
    rows: Rows
    ks: Sequence[int] = ()
    k: int = 0
    max_iters: int = 0
    heads_per_layer: int = 1
    floor: int = 0
    budget: int = 0
    recipe: str = ""
    meta: dict = field(default_factory=dict)


def _draw(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    return bf16_bits(x) if dtype == BF16 else x


def _pool(n_units: int):
    return ThreadPoolExecutor(max_workers=max(1, min(16, n_units)))


# ----------------------------------------------------------------------------
# Generic recipes
# ----------------------------------------------------------------------------
def sink_rows(wid: int, seed: int, H: int, G: int, n: int, d: int, dtype: str,
              sink: float = 4.0, outlier_channels: Sequence[int] = (),
              outlier_scale: float = 8.0, heavy_hitters: int = 0,
              heavy_scale: float = 3.0, with_v: bool = True) -> Rows:
    """q, k, v iid N(0,1); optional sink logit on key 0, outlier key channels
    and heavy-hitter keys (whole key rows scaled before bf16 rounding)."""
    q = np.empty((H, G, d), np.uint16 if dtype == BF16 else np.float32)
    k = np.empty((H, n, d), q.dtype)
    v = np.empty((H, n, d), q.dtype) if with_v else None
    hh = np.zeros((H, heavy_hitters), np.int64)
    ch = np.asarray(outlier_channels, np.int64)

    def one(h):
        rng = _rng(wid, seed, h)
        q[h] = _draw(rng, (G, d), dtype)
        kk = rng.standard_normal((n, d), dtype=np.float32)
        if ch.size:
            kk[:, ch] *= np.float32(outlier_scale)
        if heavy_hitters:
            pos = rng.choice(np.arange(1, n), size=heavy_hitters, replace=False)
            hh[h] = np.sort(pos)
            kk[pos] *= np.float32(heavy_scale)
        k[h] = bf16_bits(kk) if dtype == BF16 else kk
        if with_v:
            v[h] = _draw(rng, (n, d), dtype)

    with _pool(H) as ex:
        list(ex.map(one, range(H)))
    bias = None
    if sink:
        bias = np.zeros(n, np.float32)
        bias[0] = np.float32(sink)
    scale = np.full(H, 1.0 / math.sqrt(d), np.float32)
    rows = Rows(dtype, q, k, v, scale, bias)
    rows.heavy_hitters = hh  # type: ignore[attr-defined]
    return rows


def shifted_key_rows(wid: int, seed: int, R: int, n: int, d: int,
                     shift: float = 1.5, block: int = 1024) -> Rows:
    """One row per unit, fp32: q, v ~ N(0,1); k_j = z_j + shift*u with z_j iid
    N(0,1) and u a unit vector drawn once per row (a shared row direction)."""
    q = np.empty((R, 1, d), np.float32)
    k = np.empty((R, n, d), np.float32)
    v = np.empty((R, n, d), np.float32)
    nb = (R + block - 1) // block

    def one(b):
        lo, hi = b * block, min(R, (b + 1) * block)
        m = hi - lo
        rng = _rng(wid, seed, b)
        q[lo:hi] = rng.standard_normal((m, 1, d), dtype=np.float32)
        z = rng.standard_normal((m, n, d), dtype=np.float32)
        u = rng.standard_normal((m, d), dtype=np.float32)
        u /= np.linalg.norm(u, axis=1, keepdims=True).astype(np.float32)
        z += np.float32(shift) * u[:, None, :]
        k[lo:hi] = z
        v[lo:hi] = rng.standard_normal((m, n, d), dtype=np.float32)

    with _pool(nb) as ex:
        list(ex.map(one, range(nb)))
    return Rows(F32, q, k, v, np.full(R, 1.0 / math.sqrt(d), np.float32), None)


def window_rows(wid: int, seed: int, H: int, G: int, n: int, d: int,
                dtype: str = BF16, t_lo: float = 0.5, t_hi: float = 2.0,
                with_v: bool = True, first: int = 0) -> Rows:
    """Observation-window queries per cell with a per-cell temperature
    T ~ U[t_lo, t_hi]; scale = 1/(sqrt(d)*T) (T < 1 sharpens the head).
    Cells first .. first + H - 1 of the seeded sequence (each cell has its own
    stream, so any cell can be drawn alone)."""
    q = np.empty((H, G, d), np.uint16 if dtype == BF16 else np.float32)
    k = np.empty((H, n, d), q.dtype)
    v = np.empty((H, n, d), q.dtype) if with_v else None
    temp = np.empty(H, np.float64)

    def one(h):
        rng = _rng(wid, seed, first + h)
        temp[h] = rng.uniform(t_lo, t_hi)
        q[h] = _draw(rng, (G, d), dtype)
        k[h] = _draw(rng, (n, d), dtype)
        if with_v:
            v[h] = _draw(rng, (n, d), dtype)

    with _pool(H) as ex:
        list(ex.map(one, range(H)))
    scale = (1.0 / (math.sqrt(d) * temp)).astype(np.float32)
    rows = Rows(dtype, q, k, v, scale, None)
    rows.temperature = temp  # type: ignore[attr-defined]
    return rows


def outlier_channels(seed: int, d: int, count: int = 4, wid: int = 2) -> np.ndarray:
    """The fixed outlier key channels: drawn once per workload seed."""
    rng = _rng(wid, seed, 1 << 30)
    return np.sort(rng.choice(d, size=count, replace=False))


# ----------------------------------------------------------------------------
# The five workloads at full size, and scaled-down shapes for tests
# ----------------------------------------------------------------------------
def tiny_exhaustive(seed: int = 0, rows: int = 256, n: int = 16, d: int = 64,
                    k: int = 4) -> Workload:
    """256 rows, n = 16 keys, d = 64, fp32 N(0,1), +4 logit on key 0, k = 4."""
    r = sink_rows(1, seed, rows, 1, n, d, F32, sink=4.0)
    return Workload("tiny_exhaustive_n16_k4", r, ks=(k,), k=k, max_iters=64,
                    recipe="q,k,v iid N(0,1) fp32; bias[0]=+4; scale 1/sqrt(d)")


def streaming_topk(seed: int = 0, layers: int = 32, kv_heads: int = 8,
                   q_per_kv: int = 4, rows_per_q: int = 64, n: int = 4096,
                   d: int = 128, ks: Sequence[int] = (128, 512, 1024)) -> Workload:
    """GQA model shape: layers x kv_heads units, q_per_kv*rows_per_q rows per
    unit, bf16 N(0,1), 4 outlier key channels x8, +4 logit on key 0."""
    ch = outlier_channels(seed, d)
    r = sink_rows(2, seed, layers * kv_heads, q_per_kv * rows_per_q, n, d, BF16,
                  sink=4.0, outlier_channels=ch)
    return Workload(f"streaming_topk_L{layers}_kv{kv_heads}_n{n}", r, ks=tuple(ks),
                    k=max(ks), heads_per_layer=kv_heads,
                    recipe="bf16 N(0,1); k channels %s x8; bias[0]=+4" % list(ch),
                    meta={"outlier_channels": ch.tolist()})


def exhaustive_rows(seed: int = 0, rows: int = 168_192, n: int = 24, d: int = 128,
                    k: int = 6) -> Workload:
    """One row per unit, n = 24 candidates, d = 128, fp32; keys share a row
    direction of scale 1.5; no bias; k = 6."""
    r = shifted_key_rows(3, seed, rows, n, d, shift=1.5)
    return Workload(f"exhaustive_R{rows}_n{n}_k{k}", r, ks=(k,), k=k,
                    recipe="fp32; k_j = z_j + 1.5*u_row; q,v N(0,1); scale 1/sqrt(d)")


def swap_long_rows(seed: int = 0, kv_heads: int = 8, q_per_kv: int = 4,
                   rows_per_q: int = 32, n: int = 32768, d: int = 128,
                   k: int = 1024, max_iters: int = 64, heavy: int = 16) -> Workload:
    """8 kv units x 128 rows, n = 32768, bf16 N(0,1), +4 logit on key 0, 16
    heavy-hitter keys x3 per unit; k = 1024; at most 64 swaps."""
    r = sink_rows(4, seed, kv_heads, q_per_kv * rows_per_q, n, d, BF16, sink=4.0,
                  heavy_hitters=heavy, heavy_scale=3.0)
    return Workload(f"swap_kv{kv_heads}_n{n}_k{k}", r, ks=(k,), k=k,
                    max_iters=max_iters, heads_per_layer=kv_heads,
                    recipe="bf16 N(0,1); bias[0]=+4; %d heavy keys x3" % heavy)


def pool_rows(seed: int = 0, layers: int = 32, kv_heads: int = 8, q_per_kv: int = 4,
              rows_per_q: int = 6, n: int = 4096, d: int = 128,
              budgets: Sequence[Tuple[int, int]] = ((4, 24), (8, 12), (16, 6), (32, 4)),
              max_swaps: int = 64) -> Workload:
    """Candidate-set search at the enumeration protocol's shape: layers x
    kv_heads units of q_per_kv x rows_per_q sampled rows (six per query head),
    n keys, bf16 N(0,1) with 4 outlier key channels x8 and +4 logit on key 0
    (the streaming recipe, drawn independently); budgets s with their extra
    keys beyond the top-mass set; at most max_swaps balancing swaps."""
    ch = outlier_channels(seed, d, wid=6)
    r = sink_rows(6, seed, layers * kv_heads, q_per_kv * rows_per_q, n, d, BF16,
                  sink=4.0, outlier_channels=ch)
    return Workload(f"pool_L{layers}_kv{kv_heads}_r{q_per_kv * rows_per_q}_n{n}", r,
                    ks=tuple(b for b, _ in budgets), max_iters=max_swaps,
                    heads_per_layer=kv_heads,
                    recipe="bf16 N(0,1); k channels %s x8; bias[0]=+4; (s, extra) %s"
                    % (list(ch), list(budgets)),
                    meta={"budgets": [tuple(b) for b in budgets], "outlier_channels": ch.tolist()})


def curve_ragged(seed: int = 0, layers: int = 32, kv_heads: int = 8, window: int = 64,
                 n: int = 131072, d: int = 128, budget_frac: float = 0.10,
                 floor: int = 32) -> Workload:
    """32 x 8 cells, n = 131072, bf16 K/V N(0,1), 64 window queries, per-cell
    temperature U[0.5, 2]; global 10 % budget with a 32-position floor."""
    H = layers * kv_heads
    r = window_rows(5, seed, H, window, n, d, BF16)
    budget = int(math.floor(budget_frac * H * n))
    return Workload(f"curve_ragged_L{layers}_kv{kv_heads}_n{n}", r, heads_per_layer=kv_heads,
                    floor=floor, budget=budget,
                    recipe="bf16 N(0,1); window %d; T~U[0.5,2]; budget floor(%.2f*H*n)"
                    % (window, budget_frac))


def hardness_instance(w: Sequence[int]) -> dict:
    """The reduction instance sigma(m, w) of the hardness proof: d = 1, the m
    integers as points, uniform masses, budget m/2.  Returned in attention
    form: q = 0 gives uniform weights."""
    w = np.asarray(w, np.float32)
    m = w.size
    return dict(q=np.zeros((1, 1, 1), np.float32), k=np.zeros((1, m, 1), np.float32),
                v=w.reshape(1, m, 1).copy(), k_budget=m // 2)
