"""Seed derivation shared by every generator (counter-based, no global state)."""
from __future__ import annotations

import numpy as np

_MASK = (1 << 64) - 1
BASE = 0x50534300


def splitmix64(x: int) -> int:
    """SplitMix64 finaliser (Steele, Lea, Flood 2014)."""
    x = (x + 0x9E3779B97F4A7C15) & _MASK
    z = x
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def seed_for(cfg: int, step: int, b: int, salt: int = 0) -> int:
    return splitmix64((BASE + cfg) ^ (step << 20) ^ b ^ (salt << 48))


def rng_for(cfg: int, step: int = 0, b: int = 0, salt: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_for(cfg, step, b, salt)))
