"""Seeded synthetic inputs (token streams, LM-head and LoRA tensors) for the aTTT update step."""
from .configs import CONFIGS, Config, Projection, get
from .gen import Dense, Workload, bf16_bits, bf16_to_f32, pack_episodes, random_dense

__all__ = ["CONFIGS", "Config", "Projection", "get", "Dense", "Workload", "bf16_bits",
           "bf16_to_f32", "pack_episodes", "random_dense"]
