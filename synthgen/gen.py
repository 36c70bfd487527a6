"""Seeded generation of weights and per-input data for a SearchConfig.

Streams: numpy Generator(PCG64) seeded with SeedSequence(cfg.seed); child 0
draws the weights (W_h, E, W_out, W_kv in that order), and per-input data come
from SeedSequence(input_seed) children: child 0 draws h0 rows (row-major, so
the first N' inputs are the same for every N >= N'), child 1 draws lengths.

Distributions (the synthetic Elman decoder h' = tanh(W_h h + E[y]),
z = W_out h): W_h, E, W_out, W_kv ~ N(0, 1/d) in float32; h0 ~ N(0, 1)^d.
bf16 workloads store weights and h0 rounded to bf16 (round-to-nearest-even);
`*_bits` hold the uint16 patterns and the float32 arrays hold the same values
exactly. L_x: uniform integers in [lo, hi], or lognormal(mu, sigma) rounded
half-to-even then clipped to [lo, hi]; max_len: fixed, or floor(1.2 L_x + 10)
evaluated exactly in integers.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from .configs import INPUT_SEED_OVERRIDE, CONFIGS, SearchConfig


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Workload:
    cfg: SearchConfig
    W_h: np.ndarray                  # float32 [d, d]  (bf16-exact for bf16 configs)
    E: np.ndarray                    # float32 [V, d]
    W_out: np.ndarray                # float32 [V, d]
    W_kv: Optional[np.ndarray]       # float32 [L, 2, d, d] or None
    h0: np.ndarray                   # float32 [N, d]
    Lx: np.ndarray                   # int32 [N]
    max_len: np.ndarray              # int32 [N]

    @property
    def is_bf16(self) -> bool:
        return self.cfg.dtype == "bf16"

    def storage(self, name: str) -> np.ndarray:
        """Array in its storage dtype: float32, or uint16 bf16 bit patterns."""
        a = getattr(self, name)
        if a is None:
            return None
        return f32_to_bf16_bits(a) if self.is_bf16 else np.ascontiguousarray(a)


def _draw_lengths(cfg: SearchConfig, rng: np.random.Generator, N: int):
    if cfg.lengths == "uniform":
        Lx = rng.integers(cfg.len_lo, cfg.len_hi, size=N, endpoint=True)
    elif cfg.lengths == "lognormal":
        raw = rng.lognormal(cfg.mu, cfg.sigma, size=N)
        Lx = np.clip(np.rint(raw), cfg.len_lo, cfg.len_hi)
    else:
        raise ValueError(cfg.lengths)
    Lx = Lx.astype(np.int64)
    if cfg.max_len is not None:
        ml = np.full(N, cfg.max_len, dtype=np.int64)
    else:
        ml = (12 * Lx + 100) // 10
    return Lx.astype(np.int32), ml.astype(np.int32)


def _normal(rng, shape, scale):
    a = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        a *= np.float32(scale)
    return a


def make_workload(cfg: SearchConfig, N: Optional[int] = None,
                  weights_only: bool = False) -> Workload:
    """Generate the workload of `cfg` (first N inputs if N is given)."""
    N = cfg.N if N is None else N
    d, V = cfg.d, cfg.V
    scale = float(1.0 / np.sqrt(d))
    wrng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed).spawn(1)[0]))
    W_h = _normal(wrng, (d, d), scale)
    E = _normal(wrng, (V, d), scale)
    W_out = _normal(wrng, (V, d), scale)
    W_kv = _normal(wrng, (cfg.kv_layers, 2, d, d), scale) if cfg.kv_layers else None

    cfg_id = next((i for i, c in CONFIGS.items() if c.seed == cfg.seed), None)
    in_seed = INPUT_SEED_OVERRIDE.get(cfg_id, cfg.seed)
    ss_h, ss_len = np.random.SeedSequence(in_seed).spawn(3)[1:]
    if weights_only:
        h0 = np.zeros((0, d), np.float32)
        Lx = np.zeros(0, np.int32)
        ml = np.zeros(0, np.int32)
    else:
        h0 = _normal(np.random.Generator(np.random.PCG64(ss_h)), (N, d), 1.0)
        Lx, ml = _draw_lengths(cfg, np.random.Generator(np.random.PCG64(ss_len)), N)

    if cfg.dtype == "bf16":
        rt = lambda a: None if a is None else bf16_bits_to_f32(f32_to_bf16_bits(a))
        W_h, E, W_out, W_kv, h0 = rt(W_h), rt(E), rt(W_out), rt(W_kv), rt(h0)
    elif cfg.dtype != "f32":
        raise ValueError(cfg.dtype)
    return Workload(cfg, W_h, E, W_out, W_kv, h0, Lx, ml)
