"""One beam-search step for one input, fp64 (test infrastructure).

Follows Sec. 2 (beam search over the k|V| one-token expansions of a beam,
EOS termination; terminated candidates only get no-op expansions, Fig. 1
caption), Sec. 4 (heuristics H: relative threshold delta and max candidates M
per parent) and App. A.1 (terminated candidates stay on the beam and are
output only once nothing active is ranked above them; they may fall off).

Readings taken where the paper is silent (listed with the design notes):
  * ranking key: (-score, parent rank in the current beam, token), a no-op
    expansion of a terminated candidate has token -1;
  * delta: drop x iff x.score < best.score - delta, best = top of the full
    beam, possibly a terminated candidate (App. A.3);
  * M: walking the full beam in rank order, drop an expansion whose parent
    already has M kept expansions (no replacement; no-ops are exempt);
  * a child with token EOS is terminated (EOS); else a child emitted at
    t == max_len is terminated (MAXLEN); else it stays active;
  * the beam ends when no survivor is active; the survivors, in rank order,
    are its outputs Y[i].
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

ACTIVE, EOS, MAXLEN = 1, 2, 3
NOOP_TOKEN = -1


@dataclasses.dataclass
class Cand:
    """A candidate y_ij: its tokens (start symbol excluded), cumulative
    log-probability, status, and decoder state (row of the state table)."""
    score: float
    tokens: Tuple[int, ...]
    status: int
    h: Optional[np.ndarray]     # state after consuming tokens (None once terminated)
    y: int                      # last token (0 = start symbol for a fresh beam)


@dataclasses.dataclass
class StepResult:
    beam: List[Cand]            # the pruned beam H(B^{t+1}) in rank order
    ended: bool                 # no active survivor: beam is finished
    margin: float               # smallest score gap among this step's decisions
    full: List[tuple]           # the full beam B' as (score, parent, token)


def rank_key(e):
    """Ranking key of an expansion (score, parent rank, token): higher score
    first, then lower parent rank, then lower token (a no-op has -1)."""
    return (-e[0], e[1], e[2])


def _top_children(lp_row: np.ndarray, keep: int) -> np.ndarray:
    """Indices of every token whose lp is >= the keep-th largest lp (ties
    included, so that the exact key order can be applied afterwards)."""
    V = lp_row.shape[0]
    if keep >= V:
        return np.arange(V)
    thr = np.partition(lp_row, V - keep)[V - keep]
    return np.nonzero(lp_row >= thr)[0]


def beam_step(beam: List[Cand], lp: dict, h_new: dict, t: int, max_len: int,
              k: int, delta: float, M: int, eos: int = 0) -> StepResult:
    """Advance one beam by one step.

    beam  : current beam in rank order (rank = list position)
    lp    : {rank: log-prob row [V]} for every active candidate
    h_new : {rank: state after this expansion} for every active candidate
    t     : 1-based index of the token being emitted (this beam's step + 1)
    """
    # Expansion set (Sec. 2): V children per active candidate, one no-op per
    # terminated candidate. Only each parent's best k+1 children can reach
    # the top k+1 overall, which is all the ranking and its margin need.
    pool = []
    for j, c in enumerate(beam):
        if c.status == ACTIVE:
            row = lp[j]
            for w in _top_children(row, k + 1):
                pool.append((c.score + float(row[w]), j, int(w)))
        else:
            pool.append((c.score, j, NOOP_TOKEN))
    pool.sort(key=rank_key)
    full = pool[:k]

    # Margins of every ranking decision: adjacent pairs inside the full beam
    # and the k-th vs (k+1)-th; the threshold boundary is added below. An
    # exact tie is decided by parent rank and token, not by the scores, so it
    # is no decision margin.
    margin = np.inf
    for a, b in zip(pool[:k], pool[1:k + 1]):
        if a[0] != b[0]:
            margin = min(margin, a[0] - b[0])

    # Heuristics H (Sec. 4): relative threshold delta, then max M per parent.
    ref = full[0][0]
    kept = []
    per_parent = {}
    for e in full:
        score, j, w = e
        if np.isfinite(delta):
            margin = min(margin, abs(score - (ref - delta)))
            if score < ref - delta:
                continue
        if w != NOOP_TOKEN:
            if per_parent.get(j, 0) >= M:
                continue
            per_parent[j] = per_parent.get(j, 0) + 1
        kept.append(e)

    new_beam = []
    for score, j, w in kept:
        p = beam[j]
        if w == NOOP_TOKEN:
            new_beam.append(Cand(score, p.tokens, p.status, None, p.y))
            continue
        if w == eos:
            st = EOS
        elif t == max_len:
            st = MAXLEN
        else:
            st = ACTIVE
        new_beam.append(Cand(score, p.tokens + (w,), st,
                             h_new[j] if st == ACTIVE else None, w))
    ended = not any(c.status == ACTIVE for c in new_beam)
    return StepResult(new_beam, ended, float(margin), full)


@dataclasses.dataclass
class FairseqStepResult:
    beam: List[Cand]            # the next beam: active candidates only, rank order
    outputs: List[Cand]         # candidates finalized at this step, in rank order
    margin: float


def beam_step_fairseq(beam: List[Cand], lp: dict, h_new: dict, t: int, max_len: int,
                      k: int, n_out: int, eos: int = 0) -> FairseqStepResult:
    """One step under the Fixed-Fairseq finalization rule (App. A.1, the
    implementation difference to Fairseq): a terminated candidate that
    enters the full beam B' (the best k expansions) is added to the list of
    final outputs at once, instead of staying on the beam where it could be
    displaced later. The beam itself keeps k active candidates: the first k
    active expansions in rank order. Fixed width: no threshold, no M.

    beam  : active candidates in rank order; n_out: outputs collected so far.
    Outputs beyond k in total are not taken.
    """
    pool = []
    for j, c in enumerate(beam):
        row = lp[j]
        # Each parent has one EOS child at most, so its best k+1 children
        # cover both B' and the first k active children.
        for w in _top_children(row, k + 1):
            pool.append((c.score + float(row[w]), j, int(w)))
    pool.sort(key=rank_key)
    # Decisions: membership and order of B' and of the first k active
    # children all lie within the first 2k + 1 ranks.
    margin = np.inf
    head = pool[:2 * k + 1]
    for a, b in zip(head, head[1:]):
        if a[0] != b[0]:   # an exact tie is decided by parent rank and token
            margin = min(margin, a[0] - b[0])

    def terminated(w):
        return w == eos or t == max_len

    outputs = []
    for score, j, w in pool[:k]:
        if terminated(w) and n_out + len(outputs) < k:
            p = beam[j]
            outputs.append(Cand(score, p.tokens + (w,), EOS if w == eos else MAXLEN, None, w))
    new_beam = []
    for score, j, w in pool:
        if len(new_beam) == k:
            break
        if terminated(w):
            continue
        p = beam[j]
        new_beam.append(Cand(score, p.tokens + (w,), ACTIVE, h_new[j], w))
    return FairseqStepResult(new_beam, outputs, float(margin))
