"""Seeded synthetic inputs for the SparseSpec-L decode hot path.

This module only draws and lays out input tensors. It holds none of the
method's arithmetic (no attention, no scores, no selection), so both the HIP
path and the CPU oracle may consume what it produces.

Every tensor is drawn in fp32 from ``numpy.random.default_rng(seed)`` (PCG64)
in a fixed order -- context lengths, speculation lengths, the structure draws
(planted positions, rank permutations), verify queries, K and V (one
(sequence, KV head) slice after another, ``max_ctx`` rows each), draft
queries -- the structure is applied to K in fp32, and every value is rounded
to bfloat16 (round to nearest, ties to even).
Tensors are returned as ``uint16`` bf16 bit patterns:

* ``q``        ``[batch][max_q][n_q_heads][head_dim]``: the k+1 verify rows of
  each sequence; rows ``j >= q_len[b]`` are zero.
* ``k``, ``v`` ``[batch][n_kv_heads][max_ctx][head_dim]`` (head-major dense
  cache); rows ``i >= ctx_len[b]`` are zero.
* ``q_draft``  ``[batch][n_q_heads][head_dim]``: one draft-step query.

``ctx_len[b]`` already counts the ``q_len[b]`` verify rows appended to the
cache (bottom-right aligned causal verify block).

The five named workloads follow the attention shapes and context lengths the
paper evaluates (Llama-3.1-8B-like 32/8 heads, a 70B-like 64/8 layer, contexts
16K-131K, speculation lengths 2-10); they stand in for the long-context
benchmarks (LongBench v2, InfiniteBench, RULER) the paper measures on, which
are not reproduced here.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional, Sequence

import numpy as np

try:
    # Large fresh arrays are faulted in far faster without numpy's huge-page
    # advice on some hosts; the values drawn are unaffected.
    from numpy._core.multiarray import _set_madvise_hugepage
    _set_madvise_hugepage(False)
except Exception:  # pragma: no cover - older/newer numpy layouts
    pass

HEAD_DIM = 128
DEFAULT_WINDOW = 16        # Sec. 3.2: aggregation window W
DEFAULT_K_SINK = 4         # reading: the paper gives no value
DEFAULT_K_RECENT = 32      # reading: the paper gives no value


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bits.

    Uses torch's CPU conversion (same rounding as the integer recipe
    ``(u + 0x7FFF + ((u >> 16) & 1)) >> 16`` on the fp32 bit pattern ``u``,
    which the tests check) because it is much faster on large arrays.
    """
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Workload:
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    max_ctx: int
    max_q: int
    ctx_len: np.ndarray          # int32 [batch]
    q_len: np.ndarray            # int32 [batch]
    q: np.ndarray                # uint16 [batch][max_q][Hq][d]
    k: np.ndarray                # uint16 [batch][Hkv][max_ctx][d]
    v: np.ndarray                # uint16 [batch][Hkv][max_ctx][d]
    q_draft: np.ndarray          # uint16 [batch][Hq][d]
    sm_scale: float
    window: int
    k_sink: int
    k_recent: int
    budget: int
    structure: Dict[str, object] = dataclasses.field(default_factory=dict)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def k_mid(self) -> int:
        return self.budget - self.k_sink - self.k_recent

    def kv_bytes(self) -> int:
        """K+V bytes actually holding context rows (sum over sequences)."""
        return int(2 * self.n_kv_heads * self.head_dim * 2 * int(self.ctx_len.sum()))

    def describe(self) -> str:
        return (f"{self.name}: batch={self.batch} Hq={self.n_q_heads} Hkv={self.n_kv_heads} "
                f"d={self.head_dim} ctx={list(map(int, self.ctx_len))} "
                f"q={list(map(int, self.q_len))} B={self.budget}")


def _normal(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def generate(seed: int, *, name: str, batch: int, n_q_heads: int, n_kv_heads: int,
             ctx_len: Optional[Sequence[int]] = None, q_len: Optional[Sequence[int]] = None,
             ctx_range: Optional[tuple] = None, k_range: Optional[tuple] = None,
             head_dim: int = HEAD_DIM, budget: int = 256, max_ctx: Optional[int] = None,
             max_q: Optional[int] = None, window: int = DEFAULT_WINDOW,
             k_sink: int = DEFAULT_K_SINK, k_recent: int = DEFAULT_K_RECENT,
             heavy_hitters: int = 0, heavy_scale: float = 4.0,
             zipf_s: Optional[float] = None) -> Workload:
    """Draw one workload.

    ``ctx_len``/``q_len`` fix the per-sequence lengths; ``ctx_range``/``k_range``
    (inclusive bounds) draw them instead (context length, then speculation
    length k with q_len = k + 1).
    """
    rng = np.random.default_rng(seed)
    if ctx_len is None:
        lo, hi = ctx_range
        ctx = rng.integers(lo, hi, size=batch, endpoint=True).astype(np.int32)
    else:
        ctx = np.asarray(ctx_len, dtype=np.int32).reshape(batch)
    if q_len is None:
        lo, hi = k_range
        ql = (rng.integers(lo, hi, size=batch, endpoint=True) + 1).astype(np.int32)
    else:
        ql = np.asarray(q_len, dtype=np.int32).reshape(batch)
    if max_ctx is None:
        max_ctx = int(ctx.max())
    if max_q is None:
        max_q = int(ql.max())
    hq, hkv, d = n_q_heads, n_kv_heads, head_dim
    g = hq // hkv
    sm_scale = 1.0 / math.sqrt(d)

    # Structure draws come first so that K can be drawn, shaped and rounded one
    # (sequence, KV head) slice at a time.
    structure: Dict[str, object] = {}
    heavy = None
    if heavy_hitters > 0:
        # Planted high-norm key rows at seeded distinct positions of the span
        # that top-B selection ranks (after the sink, before the recent tail).
        heavy = np.zeros((batch, hkv, heavy_hitters), dtype=np.int64)
        for b in range(batch):
            lo, hi = k_sink, int(ctx[b]) - k_recent
            for c in range(hkv):
                heavy[b, c] = np.sort(rng.choice(hi - lo, size=heavy_hitters, replace=False) + lo)
        structure["heavy_positions"] = heavy
    ranks = None
    if zipf_s is not None:
        # Power-law attention profile: a seeded random rank per position.
        ranks = np.zeros((batch, hkv, max_ctx), dtype=np.int64)
        for b in range(batch):
            for c in range(hkv):
                ranks[b, c, :ctx[b]] = rng.permutation(int(ctx[b])) + 1
        structure["zipf_ranks"] = ranks
        structure["zipf_s"] = zipf_s

    q = _normal(rng, (batch, max_q, hq, d))
    for b in range(batch):
        q[b, ql[b]:] = 0.0
    q_bits = f32_to_bf16_bits(q)
    del q
    qf = bf16_bits_to_f32(q_bits)

    k_bits = np.empty((batch, hkv, max_ctx, d), dtype=np.uint16)
    v_bits = np.empty((batch, hkv, max_ctx, d), dtype=np.uint16)
    buf = np.empty((max_ctx, d), dtype=np.float32)
    for b in range(batch):
        T = int(ctx[b])
        for c in range(hkv):
            rng.standard_normal(out=buf, dtype=np.float32)
            if heavy is not None:
                buf[heavy[b, c]] *= np.float32(heavy_scale)
            if ranks is not None:
                # shift keys along the mean verify-query direction u so that the
                # logit of that mean query moves by -s * ln(rank)
                rows = qf[b, :ql[b], c * g:(c + 1) * g, :].reshape(-1, d).astype(np.float64)
                qbar = rows.mean(axis=0)
                nrm = float(np.linalg.norm(qbar))
                u = qbar / nrm
                bias = -zipf_s * np.log(ranks[b, c, :T].astype(np.float64))
                shift = (bias / (sm_scale * nrm))[:, None] * u[None, :]
                buf[:T] = (buf[:T].astype(np.float64) + shift).astype(np.float32)
            buf[T:] = 0.0
            k_bits[b, c] = f32_to_bf16_bits(buf)
    for b in range(batch):
        T = int(ctx[b])
        for c in range(hkv):
            rng.standard_normal(out=buf, dtype=np.float32)
            buf[T:] = 0.0
            v_bits[b, c] = f32_to_bf16_bits(buf)
    qd_bits = f32_to_bf16_bits(_normal(rng, (batch, hq, d)))

    return Workload(name=name, batch=batch, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                    max_ctx=int(max_ctx), max_q=int(max_q), ctx_len=ctx, q_len=ql,
                    q=q_bits, k=k_bits, v=v_bits, q_draft=qd_bits, sm_scale=sm_scale,
                    window=window, k_sink=k_sink, k_recent=k_recent, budget=budget,
                    structure=structure)


# The five named workloads (seed = workload number).
CONFIGS = {
    1: dict(name="tiny-8x2-T4K", batch=1, n_q_heads=8, n_kv_heads=2,
            ctx_len=[4096], q_len=[5], budget=256),
    2: dict(name="llama8b-T32K", batch=1, n_q_heads=32, n_kv_heads=8,
            ctx_len=[32768], q_len=[7], budget=2048, heavy_hitters=4),
    3: dict(name="llama8b-b8-ragged", batch=8, n_q_heads=32, n_kv_heads=8,
            ctx_range=(16384, 65536), k_range=(2, 10), budget=4096, max_ctx=65536),
    4: dict(name="llama8b-T131K-zipf", batch=1, n_q_heads=32, n_kv_heads=8,
            ctx_len=[131072], q_len=[9], budget=4096, zipf_s=1.1),
    5: dict(name="70b-b4-T64K", batch=4, n_q_heads=64, n_kv_heads=8,
            ctx_len=[65536] * 4, q_len=[6] * 4, budget=4096),
}


def make_config(n: int) -> Workload:
    """Workload number ``n`` (1..5), drawn with seed ``n``."""
    return generate(n, **CONFIGS[n])


def config_description(n: int) -> Dict[str, object]:
    c = dict(CONFIGS[n])
    return c
