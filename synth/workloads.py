"""The synthetic workloads the compression pass is tested and measured on.

Each entry describes a cache (shape, patch grid, fill, key/value statistics,
seed) and the compression request (budget, recent-frame window, TaR share).
Shapes follow 7B- and 72B-class video MLLMs: 196 tokens per frame is a 14x14
patch grid (LLaVA-style), 256 tokens per frame a 16x16 grid.
"""
from __future__ import annotations

from dataclasses import dataclass, field

from . import BF16, F32, RhoSpec


@dataclass(frozen=True)
class Workload:
    name: str
    streams: int
    layers: int
    kv_heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    n_tokens: int          # valid rows when the pass runs (the memory cap)
    budget: int            # rows kept per (stream, layer, head)
    recent_frames: int
    alphas: tuple          # TaR shares exercised (the first is the timed one)
    dtype: int
    seeds: tuple           # one seed per stream
    rho_specs: tuple       # one RhoSpec per stream
    value_sigma: tuple = (0.5,)
    cv_tau: tuple | None = None
    stream_frames: int = 0  # >0: frames arrive one at a time and the pass fires at the cap
    note: str = ""

    @property
    def p(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def capacity(self) -> int:
        return self.n_tokens

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == BF16 else 4

    def algorithmic_bytes(self) -> int:
        """K and V read once to score, then every kept row read and written
        once to compact: B*L*H*D*E*(2n + 4C)."""
        return (self.streams * self.layers * self.kv_heads * self.head_dim * self.elem_bytes
                * (2 * self.n_tokens + 4 * self.budget))


_U099 = RhoSpec(0.0, 0.99)

TINY = Workload(
    name="tiny-fp32", streams=1, layers=1, kv_heads=2, head_dim=64, grid_h=4, grid_w=4,
    n_tokens=128, budget=64, recent_frames=1, alphas=(0.5,), dtype=F32, seeds=(0,), rho_specs=(_U099,),
    note="1 layer, 2 KV heads, 8 frames of a 4x4 grid, 128 -> 64 rows")

SEVEN_B = Workload(
    name="7b-class-28L", streams=1, layers=28, kv_heads=4, head_dim=128, grid_h=14, grid_w=14,
    n_tokens=6272, budget=3136, recent_frames=4, alphas=(0.5,), dtype=BF16, seeds=(1,), rho_specs=(_U099,),
    note="28 layers, 4 KV heads, 32 frames of 14x14, 6272 -> 3136 rows")

STREAMING = Workload(
    name="streaming-16x16", streams=1, layers=28, kv_heads=4, head_dim=128, grid_h=16, grid_w=16,
    n_tokens=12288, budget=6144, recent_frames=4, alphas=(0.5,), dtype=BF16, seeds=(2,),
    rho_specs=(RhoSpec(0.0, 0.9, static_frac=0.2, static_rho=0.999),), stream_frames=512,
    note="512 frames of 16x16 arrive one at a time; at 12288 rows the cache is compressed to 6144")

SEVENTY_B = Workload(
    name="72b-class-80L", streams=1, layers=80, kv_heads=8, head_dim=128, grid_h=14, grid_w=14,
    n_tokens=32768, budget=16384, recent_frames=8, alphas=(0.5,), dtype=BF16, seeds=(3,),
    rho_specs=(_U099,), note="80 layers, 8 KV heads, 167 frames of 14x14 plus a 36-row partial frame")

BATCHED = Workload(
    name="batched-16x7b", streams=16, layers=28, kv_heads=4, head_dim=128, grid_h=14, grid_w=14,
    n_tokens=6272, budget=3136, recent_frames=4, alphas=(0.5, 1.0, 0.0), dtype=BF16,
    seeds=tuple(100 + s for s in range(16)),
    rho_specs=tuple(_U099 if s % 2 == 0 else RhoSpec(0.0, 0.99, static_frac=0.5, static_rho=0.999)
                    for s in range(16)),
    note="16 independent 7B-class streams in one launch; TaR shares 0.5, 1, 0")

POOL = Workload(
    name="pool-7b-shape", streams=1, layers=28, kv_heads=4, head_dim=128, grid_h=14, grid_w=14,
    n_tokens=6272, budget=3136, recent_frames=4, alphas=(0.5,), dtype=BF16, seeds=(7,), rho_specs=(_U099,),
    value_sigma=(0.1, 0.35, 0.55, 1.0), cv_tau=(0.3, 0.5, 0.7),
    note="7B-class shape with per-layer value spread cycling so every pooling size 7/5/3/1 occurs")

ONE_LAYER = Workload(
    name="7b-class-1L", streams=1, layers=1, kv_heads=4, head_dim=128, grid_h=14, grid_w=14,
    n_tokens=6272, budget=3136, recent_frames=4, alphas=(0.5,), dtype=BF16, seeds=(1,), rho_specs=(_U099,),
    note="one layer of the 7B-class cache (4 KV heads, 6272 -> 3136 rows): the latency of a single-layer pass")

ALL = (TINY, SEVEN_B, STREAMING, SEVENTY_B, BATCHED)
BY_NAME = {w.name: w for w in ALL + (POOL, ONE_LAYER)}
