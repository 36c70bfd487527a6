"""GPU-vs-oracle comparison (test infrastructure; see oracle/__init__).

Per input: the token sequences, statuses and the order of the finalized
hypotheses Y[i] must be identical, and every score must agree with the
oracle's within `score_tol`. An input whose hypotheses differ is excused only
when the oracle logged a decision margin (score gap between two ranked
candidates, or between a candidate and the relative-threshold boundary) below
`tie_tol` at some step of that input: such a decision can legitimately go
either way under rounding, and everything after it may differ. A score error
on identical hypotheses is never excused: a near tie changes which tokens are
kept, not the score of a given token path.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np


@dataclasses.dataclass
class Report:
    n_inputs: int = 0
    n_exact: int = 0
    n_excused: int = 0
    n_tie_inputs: int = 0
    max_score_err: float = 0.0
    excused: List[int] = dataclasses.field(default_factory=list)
    failures: List[str] = dataclasses.field(default_factory=list)

    @property
    def ok(self) -> bool:
        return not self.failures

    def summary(self) -> str:
        return (f"inputs={self.n_inputs} exact={self.n_exact} excused={self.n_excused} "
                f"tie_inputs={self.n_tie_inputs} max_score_err={self.max_score_err:.3g} "
                f"failures={len(self.failures)}")


def compare(oracle_hyps: Sequence, oracle_min_margin: Sequence[float],
            gpu_hyps: Sequence, inputs: Optional[Sequence[int]] = None,
            score_tol: float = 1e-4, tie_tol: float = 1e-4) -> Report:
    """oracle_hyps[j] / gpu_hyps[j]: list of (tokens, score, status) (or
    objects with those attributes) for the j-th compared input; `inputs`
    gives their ids for messages."""
    rep = Report()
    ids = list(range(len(oracle_hyps))) if inputs is None else list(inputs)
    for j, i in enumerate(ids):
        rep.n_inputs += 1
        o = [_t(h) for h in oracle_hyps[j]]
        g = [_t(h) for h in gpu_hyps[j]]
        tie = oracle_min_margin[j] < tie_tol
        rep.n_tie_inputs += int(tie)
        same = len(o) == len(g) and all(a[0] == b[0] and a[2] == b[2] for a, b in zip(o, g))
        if same:
            err = max((abs(a[1] - b[1]) for a, b in zip(o, g)), default=0.0)
            rep.max_score_err = max(rep.max_score_err, err)
            if err <= score_tol:
                rep.n_exact += 1
                continue
            rep.failures.append(f"input {i}: score error {err:.3g} > {score_tol}")
            continue
        if tie:
            rep.n_excused += 1
            rep.excused.append(i)
            continue
        rep.failures.append(f"input {i}: hypotheses differ (min margin "
                            f"{oracle_min_margin[j]:.3g}); oracle={o[:2]} gpu={g[:2]}")
    return rep


def _t(h):
    if isinstance(h, tuple):
        return (tuple(int(x) for x in h[0]), float(h[1]), int(h[2]))
    return (tuple(int(x) for x in h.tokens), float(h.score), int(h.status))
