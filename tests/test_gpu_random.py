"""Seeded random small configurations against the oracle: beam width,
batch size, vocabulary (including |V| = k and lists short enough for the
completion path), state size, dtype, EOS bias, threshold, per-parent limit,
lengths, scheduler, refill threshold and pool drawn per case."""
import math

import numpy as np
import pytest

from synthgen import make_workload, scaled
from tests.gpu_util import check_parity

pytestmark = pytest.mark.gpu

SCHEDS = ["var_stream", "var_batch", "var_fifo", "var_cap", "fixed", "fixed_stream", "fixed_fairseq",
          "fixed_fairseq_stream"]


def random_case(seed):
    """(config, scheduler, eps, pool) of case `seed`."""
    rng = np.random.default_rng(7000 + seed)
    bf16 = rng.random() < 0.35
    sched = SCHEDS[int(rng.integers(len(SCHEDS)))]
    k = int(rng.integers(1, 16 if "fairseq" in sched else 17))
    n = int(rng.integers(1, 17))
    V = int(rng.choice([k, k + 1, 50, 300, 1000, 3000, 9000]))
    d = int(rng.choice([128, 256] if bf16 else [64, 128, 256]))
    delta = float(rng.choice([0.5, 1.5, 3.0, math.inf]))
    M = int(rng.integers(1, k + 1))
    beta = float(rng.choice([0.0, 0.5, 1.0, 2.0]))
    len_hi = int(rng.integers(3, 25))
    cfg = scaled(4 if bf16 else 1, N=int(rng.integers(4, 33)), n=n, V=V, d=d, k=k, M=M, delta=delta, beta=beta,
                 lengths="uniform", len_lo=2, len_hi=len_hi, max_len=None, seed=50000 + seed)
    eps = float(rng.choice([0.0, 0.25, 0.5])) if sched in ("var_stream", "var_fifo", "var_cap", "fixed_stream",
                                                            "fixed_fairseq_stream") else None
    pool = int(rng.integers(n, 3 * n + 1)) if sched == "var_cap" else None
    return cfg, sched, eps, pool


@pytest.mark.parametrize("seed", range(16))
def test_random_config(gpu, seed):
    cfg, sched, eps, pool = random_case(seed)
    wl = make_workload(cfg)
    print(f"[case {seed}] {sched} eps={eps} pool={pool} N={cfg.N} n={cfg.n} k={cfg.k} V={cfg.V} d={cfg.d} "
          f"{cfg.dtype} delta={cfg.delta} M={cfg.M} beta={cfg.beta} len_hi={cfg.len_hi}", flush=True)
    check_parity(wl, sched, eps=eps, pool=pool)
