"""The synthetic decoding workloads (five, plus config 5 with self-attention).

Each config fixes the shape of a synthetic Elman decoder (state size d,
vocabulary |V| with token 0 = EOS = start symbol), its storage dtype, the
per-input length distribution, and the search hyperparameters of the paper's
method: batch size n, beam width k, refill threshold eps (Alg. 1), relative
score threshold delta and max candidates per node M (Sec. 4, pruning
heuristics H).

Workload shapes stand in for the paper's MT (newstest, k=5/50) and parsing
(ATIS/PTB, n=k=10, M=3) regimes; no dataset item is used.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class SearchConfig:
    name: str
    N: int                 # number of inputs
    n: int                 # batch size (beams resident at once)
    k: int                 # beam width
    V: int                 # vocabulary size, token 0 is EOS (and the start symbol)
    d: int                 # decoder state size
    dtype: str             # "f32" or "bf16" storage of weights and states
    eps: float             # refill threshold, Alg. 1
    delta: float           # relative score threshold (nats), math.inf = off
    M: int                 # max kept children per parent (M = k: off)
    beta: float            # EOS bias slope: z[0] += beta * (t - L_x)
    lengths: str           # "uniform" or "lognormal"
    len_lo: int            # uniform lower bound / lognormal clip lower bound
    len_hi: int            # uniform upper bound / lognormal clip upper bound
    max_len: Optional[int] # fixed max length, or None for floor(1.2 L_x + 10)
    kv_layers: int = 0     # per-candidate KV-like state (layers x {K,V} x t x d)
    attn: bool = False     # the projection reads h plus the self-attention read-out over the KV rows
    seed: int = 0
    mu: float = 3.2        # lognormal location
    sigma: float = 0.5     # lognormal scale

    @property
    def max_len_cap(self) -> int:
        """Largest max_len any input of this config can have."""
        if self.max_len is not None:
            return self.max_len
        return (12 * self.len_hi + 100) // 10

    @property
    def R_max(self) -> int:
        return self.n * self.k

    def with_(self, **kw) -> "SearchConfig":
        return dataclasses.replace(self, **kw)


def _cfg(i, **kw):
    return SearchConfig(seed=1000 + i, **kw)


CONFIGS = {
    # Tiny sanity case: small enough for the oracle to run whole.
    1: _cfg(1, name="tiny", N=64, n=8, k=4, V=1000, d=64, dtype="f32", eps=0.25,
            delta=1.5, M=4, beta=0.5, lengths="uniform", len_lo=4, len_hi=20,
            max_len=32),
    # Parsing-shaped: many inputs, small model, M = 3 (paper's parsing runs).
    2: _cfg(2, name="parse", N=16384, n=1024, k=5, V=256, d=256, dtype="f32",
            eps=0.25, delta=2.0, M=3, beta=0.5, lengths="uniform", len_lo=5,
            len_hi=60, max_len=128),
    # MT-shaped fp32, the headline workload: k = 5, |V| = 32000.
    3: _cfg(3, name="mt_f32", N=4096, n=128, k=5, V=32000, d=1024, dtype="f32",
            eps=0.25, delta=1.5, M=5, beta=1.0, lengths="lognormal", len_lo=3,
            len_hi=200, max_len=None),
    # MT-shaped bf16, wide beams; eps is swept over {1/8, 1/4, 1/2}.
    4: _cfg(4, name="mt_bf16_wide", N=8192, n=512, k=10, V=32000, d=1024,
            dtype="bf16", eps=0.25, delta=1.5, M=4, beta=1.0,
            lengths="lognormal", len_lo=3, len_hi=200, max_len=None),
    # Transformer-state reorder stress: config 4 inputs plus a per-candidate
    # KV-like state of 6 layers x {K,V} x t x d bf16 rows.
    5: _cfg(5, name="kv_reorder", N=8192, n=256, k=5, V=64000, d=1024,
            dtype="bf16", eps=0.25, delta=1.5, M=4, beta=1.0,
            lengths="lognormal", len_lo=3, len_hi=200, max_len=None,
            kv_layers=6),
}
# Length-dependent decoder step: config 5 (same weights and inputs) whose
# projection input adds each layer's attention over the candidate's KV rows,
# so a step's cost grows with the output position.
CONFIGS[6] = CONFIGS[5].with_(name="kv_attn", attn=True)
# Config 5 reuses config 4's per-input stream (same h0 / L_x / max_len).
INPUT_SEED_OVERRIDE = {5: CONFIGS[4].seed}

EPS_SWEEP_CFG4: Tuple[float, ...] = (0.125, 0.25, 0.5)


def get_config(i: int) -> SearchConfig:
    return CONFIGS[i]


def scaled(i: int, N: Optional[int] = None, n: Optional[int] = None,
           V: Optional[int] = None, d: Optional[int] = None,
           len_hi: Optional[int] = None, **kw) -> SearchConfig:
    """A reduced copy of config i for tests the oracle must finish quickly."""
    c = CONFIGS[i]
    upd = {}
    for key, val in (("N", N), ("n", n), ("V", V), ("d", d), ("len_hi", len_hi)):
        if val is not None:
            upd[key] = val
    upd.update(kw)
    return c.with_(**upd)

