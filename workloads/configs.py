"""Seeded synthetic workload definitions for the aTTT update step.

The paper's runs use agent trajectories (ALFWorld, SWE-bench Lite) and Qwen3.5 /
Gemma-3 models, none of which are available here. These five configurations stand
in for them: the token streams reproduce the repetition regimes the paper
describes (mean novelty 0.42-0.58 under cadence K, Table "tab:cadence"; self-text
repetition above 80% in stuck runs, Sec. 4 drift analysis), and the dense shapes
are Llama-8B / Qwen-14B style LM heads and q/k/v/o projections.

This module holds only sizes and distribution parameters. It contains none of the
method's arithmetic.
"""
from dataclasses import dataclass, field
from typing import List, Tuple


@dataclass(frozen=True)
class Projection:
    name: str
    d_in: int
    d_out: int
    x_group: str  # projections with the same group share one input matrix X


@dataclass(frozen=True)
class Config:
    key: str            # short id, "c1" .. "c5"
    name: str           # descriptive workload name
    seed: int
    episodes: int       # E: independent episodes processed in one call
    update_len: int     # L: tokens of the new update text x_k per episode
    prior_updates: int  # number of previous updates forming H^tok per episode
    prior_len: int      # tokens per previous update
    id_dist: str        # "uniform" or "zipf"
    zipf_s: float
    id_range: int       # token ids drawn from [0, id_range)
    copy_frac: float    # target fraction of update tokens copied from earlier updates
    span: Tuple[int, int]  # copied span lengths, uniform in [lo, hi]
    n: int              # n-gram size
    w_min: float        # weight floor
    d: int              # hidden size
    vocab: int          # LM-head rows V
    dtype: str          # "f32" or "bf16"
    rank: int
    alpha: float
    projections: Tuple[Projection, ...]
    lora_b_zero: bool   # B = 0 (standard LoRA init, dA == 0)

    @property
    def rows(self) -> int:
        return self.episodes * self.update_len

    @property
    def history_per_episode(self) -> int:
        return self.prior_updates * self.prior_len

    @property
    def scale(self) -> float:
        return self.alpha / self.rank


def _qkvo(d, kv):
    return (Projection("q", d, d, "x_qkv"), Projection("k", d, kv, "x_qkv"),
            Projection("v", d, kv, "x_qkv"), Projection("o", d, d, "x_o"))


CONFIGS = {
    "c1": Config("c1", "tiny_fp32_L512_d256_V4096", 1001, 1, 512, 4, 512, "uniform", 0.0,
                 4096, 0.40, (4, 32), 4, 0.05, 256, 4096, "f32", 8, 16.0,
                 (Projection("proj", 256, 256, "x"),), True),
    "c2": Config("c2", "small_bf16_L2048_d2048_V32000", 1002, 1, 2048, 8, 2048, "uniform", 0.0,
                 32000, 0.30, (4, 32), 3, 0.05, 2048, 32000, "bf16", 16, 16.0,
                 _qkvo(2048, 512), False),
    "c3": Config("c3", "llama8b_bf16_L8192_d4096_V128256", 1003, 1, 8192, 32, 4096, "zipf", 1.1,
                 128256, 0.35, (4, 32), 4, 0.05, 4096, 128256, "bf16", 16, 16.0,
                 _qkvo(4096, 1024), False),
    "c4": Config("c4", "qwen14b_long_bf16_L32768_d5120_V151936", 1004, 1, 32768, 64, 8192, "zipf",
                 1.1, 151936, 0.50, (8, 256), 4, 0.05, 5120, 151936, "bf16", 32, 16.0,
                 _qkvo(5120, 1024), False),
    "c5": Config("c5", "stuck16_bf16_E16_L4096_d4096_V128256", 1005, 16, 4096, 128, 4096, "zipf",
                 1.1, 128256, 0.90, (4, 32), 3, 0.05, 4096, 128256, "bf16", 16, 16.0,
                 _qkvo(4096, 1024), False),
}


def get(key: str) -> Config:
    return CONFIGS[key]
