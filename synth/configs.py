"""Named synthetic workloads for the Rift hot path.

Each workload fixes the shapes, value distributions and pruning settings of one
scene-query.  The shapes follow the paper: 336x336 px tiles that a LLaVA-1.5
vision encoder turns into 576 tokens each (Sec. 1 and Sec. 2.3, Stage 2), an
8x8 = 64-tile walkthrough scene (App. B, Step 1), a ~400-tile 6700x6700 px
scene (Sec. 1), and a LLaMA-7B-shaped decoder (LLaVA-1.5-7B, Sec. 3 Setup).

This module only describes workloads; it computes nothing of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Tuple


@dataclass(frozen=True)
class ModelShape:
    d: int            # hidden size
    n_heads: int
    head_dim: int
    ffn: int          # SwiGLU inner size
    n_layers: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    weight_std: float = 0.02


@dataclass(frozen=True)
class Workload:
    name: str
    cid: int                  # workload number, feeds the seed
    dtype: str                # "f32" or "bf16": storage type of every input
    n_tiles: int
    n_v: int                  # vision tokens per tile
    n_bg: int                 # background phrases M (Eq. 1)
    n_templates: int          # caption templates averaged into t
    planted_tiles: Tuple[int, ...] | int   # explicit tile ids, or a count chosen by seed
    planted_frac: Tuple[float, float]      # fraction of a planted tile's tokens, U[lo, hi]
    planted_alpha: float      # amplitude of the query-aligned component
    keep_count: int           # keep top-K tiles (0 = threshold mode)
    tau: float                # threshold on the min-max normalised score
    levels: Tuple[int, ...]   # token budgets, descending
    tier_num: Tuple[int, ...] # tier fractions (numerators over tier_den) for all but the last level
    tier_den: int
    n_sys: int
    n_qry: int
    model: ModelShape = field(default_factory=lambda: ModelShape(4096, 32, 128, 11008, 1))

    @property
    def seed_base(self) -> int:
        # "RIFT" in ASCII, offset by the workload number
        return 0x52494654 + self.cid


LLAMA7B_1 = ModelShape(d=4096, n_heads=32, head_dim=128, ffn=11008, n_layers=1)
LLAMA7B_32 = ModelShape(d=4096, n_heads=32, head_dim=128, ffn=11008, n_layers=32)

WORKLOADS = {
    # 4 tiles, d = 256, fp32; tile 1 carries +0.5 t on 20% of its tokens.
    "tiny": Workload(
        name="tiny", cid=1, dtype="f32", n_tiles=4, n_v=576, n_bg=15, n_templates=5,
        planted_tiles=(1,), planted_frac=(0.2, 0.2), planted_alpha=0.5,
        keep_count=2, tau=0.37, levels=(64,), tier_num=(), tier_den=16,
        n_sys=8, n_qry=16,
        model=ModelShape(d=256, n_heads=4, head_dim=64, ffn=688, n_layers=1)),
    # One tile, no pruning: the exhaustive per-tile prompt of 35 + 576 + 32 tokens.
    "one_tile": Workload(
        name="one_tile", cid=2, dtype="bf16", n_tiles=1, n_v=576, n_bg=15, n_templates=5,
        planted_tiles=(), planted_frac=(0.0, 0.0), planted_alpha=0.0,
        keep_count=1, tau=0.37, levels=(576,), tier_num=(), tier_den=16,
        n_sys=35, n_qry=32, model=LLAMA7B_1),
    # 8x8 walkthrough-shaped scene, 6 planted tiles, keep 16, elastic budgets.
    "scene8": Workload(
        name="scene8", cid=3, dtype="bf16", n_tiles=64, n_v=576, n_bg=15, n_templates=5,
        planted_tiles=6, planted_frac=(0.10, 0.30), planted_alpha=2.0,
        keep_count=16, tau=0.37, levels=(576, 288, 144, 64), tier_num=(1, 3, 4), tier_den=16,
        n_sys=35, n_qry=32, model=LLAMA7B_1),
    # 20x20 = 400-tile scene, 5% planted, keep 25%, elastic budgets, 1 layer.
    "scene20": Workload(
        name="scene20", cid=4, dtype="bf16", n_tiles=400, n_v=576, n_bg=15, n_templates=5,
        planted_tiles=20, planted_frac=(0.10, 0.30), planted_alpha=2.0,
        keep_count=100, tau=0.37, levels=(576, 288, 144, 64), tier_num=(1, 3, 4), tier_den=16,
        n_sys=35, n_qry=32, model=LLAMA7B_1),
    # The same 400-tile scene through the full 32-layer decoder stack.
    # (cid 4 again: it is the very same scene and the same per-layer weights.)
    "scene20_l32": Workload(
        name="scene20_l32", cid=4, dtype="bf16", n_tiles=400, n_v=576, n_bg=15, n_templates=5,
        planted_tiles=20, planted_frac=(0.10, 0.30), planted_alpha=2.0,
        keep_count=100, tau=0.37, levels=(576, 288, 144, 64), tier_num=(1, 3, 4), tier_den=16,
        n_sys=35, n_qry=32, model=LLAMA7B_32),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]
