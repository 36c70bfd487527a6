"""Alg. 1 (Var-Stream) and its settings Fixed / Var-Batch, fp64 (test
infrastructure; see oracle/__init__).

Decode(X, E, D, n, eps, k, H) (Sec. 3, Alg. 1):
  c = first unadmitted input; beams B; outputs Y
  while inputs remain or B is non-empty:
      if inputs remain and |B| <= eps * n:
          encode and admit m new inputs (fresh beams holding the start symbol)
      select the beams with minimal l_t (steps taken)
      expand every candidate of the selected beams with D; update each
      selected beam (top-k, H, finalization); a beam whose candidates are
      all terminated is finished and its candidates become Y[i]
      remove finished beams

Readings (listed with the design notes): the refill admits
m = min(n - |B|, inputs left), i.e. it refills the batch to n (Sec. 3: the
initial batch is n and a refill restores size n); inputs are admitted in
index order; Var-Batch is eps = 0 (refill only when the batch is empty) and
Fixed is eps = 0, delta = inf, M = k (App. A.1: Fixed-Ours is eps = 0).

Capacity-constrained streaming (Sec. 3, last paragraph; Sec. 4.2 and 4.3,
a limit of n*k expanded candidates per timestep): up to `pool` >= n beams
are cached; the refill test and amount use the pool size in place of n; at
each timestep the live beams, ordered by (l_t, admission order), are taken
while their active candidates total at most n*k rows (the first beam that
would exceed the limit ends the selection).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from .beam import ACTIVE, Cand, beam_step, beam_step_fairseq


@dataclasses.dataclass
class Hyp:
    tokens: tuple
    score: float
    status: int


@dataclasses.dataclass
class SearchResult:
    hyps: List[List[Hyp]]               # Y[i], rank order
    finalize_step: np.ndarray           # global timestep at which input i finished
    steps_taken: np.ndarray             # l_t of input i's beam when it finished
    min_margin: np.ndarray              # smallest decision margin over input i's steps
    margins: List[List[float]]          # per input, per own step: min margin of that step
    widths: List[List[int]]             # per input, per own step: rows expanded
    timesteps: int = 0
    expansions: int = 0
    noops: int = 0
    refills: int = 0
    admitted: int = 0
    positions: int = 0                  # output positions t of the expanded rows, summed
    rows_per_step: List[int] = dataclasses.field(default_factory=list)

    @property
    def n_hyps(self) -> int:
        return sum(len(y) for y in self.hyps)

    def stats(self) -> dict:
        return dict(timesteps=self.timesteps, expansions=self.expansions,
                    noops=self.noops, refills=self.refills,
                    admitted=self.admitted, hyps=self.n_hyps)


@dataclasses.dataclass
class _Beam:
    input: int
    steps: int
    cands: List[Cand]
    outputs: List[Cand] = dataclasses.field(default_factory=list)   # Fixed-Fairseq rule only


def decode(decoder, h0: np.ndarray, Lx: Sequence[int], max_len: Sequence[int],
           n: int, eps: float, k: int, delta: float = math.inf,
           M: Optional[int] = None, on_step: Optional[Callable] = None,
           select: str = "min_steps", rule: str = "paper",
           pool: Optional[int] = None) -> SearchResult:
    """Run Alg. 1 over inputs 0..N-1 (h0[i] is e_i = E(x_i)).

    `decoder` needs initial_state(h0_row) and expand(h_prev, y, t, Lx) ->
    (h, lp) as in oracle.decoder.ElmanDecoder (tests substitute scripted
    decoders). `on_step(timestep, selected_inputs, rows)` observes the
    schedule. `select` is Alg. 1's beam selection, "min_steps" (the beams
    with minimal l_t), or "fifo" for Var-Str-FIFO (App. A, alternative
    method analysis: beams up to the batch capacity n, starting from the
    one with maximal l_t), or "capacity" (the capacity-constrained
    selection above; `pool` beams are cached, default n). `rule` is the
    finalization rule: "paper"
    (App. A.1: terminated candidates stay on the beam) or "fairseq"
    (App. A.1's Fixed-Fairseq: they are output at once; fixed width, so
    delta and M are not applied); a beam under the Fairseq rule finishes
    with k outputs, kept in the order they were finalized.
    """
    if select not in ("min_steps", "fifo", "capacity"):
        raise ValueError(select)
    if rule not in ("paper", "fairseq"):
        raise ValueError(rule)
    N = len(Lx)
    M = k if M is None else int(M)
    P = n if pool is None else int(pool)
    if not (k >= 1 and n >= 1 and 0.0 <= eps < 1.0 and 1 <= M <= k and P >= n):
        raise ValueError("invalid search parameters")
    if P != n and select != "capacity":
        raise ValueError("a beam pool larger than n needs the capacity selection")
    res = SearchResult(hyps=[None] * N, finalize_step=np.zeros(N, np.int64),
                       steps_taken=np.zeros(N, np.int64),
                       min_margin=np.full(N, np.inf),
                       margins=[[] for _ in range(N)], widths=[[] for _ in range(N)])
    c = 0
    live: List[_Beam] = []
    while c < N or live:
        if c < N and len(live) <= eps * P:
            m = min(P - len(live), N - c)
            for i in range(c, c + m):
                st = decoder.initial_state(h0[i])
                live.append(_Beam(i, 0, [Cand(0.0, (), ACTIVE, st, 0)]))
            c += m
            res.refills += 1
            res.admitted += m
        lmin = min(b.steps for b in live)
        if select == "fifo":
            # At most n beams are live, so the capacity-n prefix of the
            # beams ordered by decreasing l_t is every live beam.
            sel = sorted(live, key=lambda b: -b.steps)[:n]
        elif select == "capacity":
            sel, used = [], 0
            for b in sorted(live, key=lambda b: (b.steps, b.input)):
                width = sum(1 for cand in b.cands if cand.status == ACTIVE)
                if used + width > n * k:
                    break
                sel.append(b)
                used += width
        else:
            sel = [b for b in live if b.steps == lmin]

        # One batched decoder call over every active candidate of the
        # selected beams (the inner loops of Alg. 1).
        rows = [(bi, j) for bi, b in enumerate(sel)
                for j, cand in enumerate(b.cands) if cand.status == ACTIVE]
        h_prev = [sel[bi].cands[j].h for bi, j in rows]
        y = np.array([sel[bi].cands[j].y for bi, j in rows])
        t = np.array([sel[bi].steps + 1 for bi, _ in rows])
        lx = np.array([Lx[sel[bi].input] for bi, _ in rows])
        h_new, lp = decoder.expand(h_prev, y, t, lx)
        res.timesteps += 1
        res.expansions += len(rows)
        res.positions += int(t.sum())
        res.rows_per_step.append(len(rows))
        if on_step is not None:
            on_step(res.timesteps, [b.input for b in sel], len(rows))

        per_beam_lp: Dict[int, dict] = {}
        per_beam_h: Dict[int, dict] = {}
        for r, (bi, j) in enumerate(rows):
            per_beam_lp.setdefault(bi, {})[j] = lp[r]
            per_beam_h.setdefault(bi, {})[j] = h_new[r]
        finished = []
        for bi, b in enumerate(sel):
            res.noops += sum(1 for cand in b.cands if cand.status != ACTIVE)
            res.widths[b.input].append(sum(1 for cand in b.cands if cand.status == ACTIVE))
            if rule == "fairseq":
                fo = beam_step_fairseq(b.cands, per_beam_lp.get(bi, {}), per_beam_h.get(bi, {}),
                                       b.steps + 1, int(max_len[b.input]), k, len(b.outputs))
                b.outputs += fo.outputs
                b.cands = fo.beam
                margin = fo.margin
                ended = len(b.outputs) >= k or not fo.beam
                final = b.outputs
            else:
                out = beam_step(b.cands, per_beam_lp.get(bi, {}), per_beam_h.get(bi, {}),
                                b.steps + 1, int(max_len[b.input]), k, delta, M)
                b.cands = out.beam
                margin = out.margin
                ended = out.ended
                final = out.beam
            res.margins[b.input].append(margin)
            res.min_margin[b.input] = min(res.min_margin[b.input], margin)
            b.steps += 1
            if ended:
                res.hyps[b.input] = [Hyp(cd.tokens, cd.score, cd.status) for cd in final]
                res.finalize_step[b.input] = res.timesteps
                res.steps_taken[b.input] = b.steps
                finished.append(b)
        if finished:
            done = set(id(b) for b in finished)
            live = [b for b in live if id(b) not in done]
    return res


def decode_workload(wl, n=None, eps=None, k=None, delta=None, M=None, sched="var_stream",
                    inputs: Optional[Sequence[int]] = None, decoder=None,
                    pool: Optional[int] = None) -> SearchResult:
    """Convenience wrapper: decode (a subset of) a synthgen Workload with its
    config's parameters; `sched` picks Fixed / Fixed-Stream / Fixed-Fairseq /
    Var-Batch / Var-Stream / Var-Str-FIFO ("var_fifo") / capacity-constrained
    Var-Stream ("var_cap", `pool` cached beams, default 2n)."""
    from .decoder import decoder_for_workload
    c = wl.cfg
    dec = decoder or decoder_for_workload(wl)
    n = c.n if n is None else n
    k = c.k if k is None else k
    eps = c.eps if eps is None else eps
    delta = c.delta if delta is None else delta
    M = c.M if M is None else M
    rule = "paper"
    if sched == "fixed":
        eps, delta, M = 0.0, math.inf, k
    elif sched == "fixed_stream":          # App. A.1 / Table 3: Fixed with streaming refill
        delta, M = math.inf, k
    elif sched == "fixed_fairseq":         # App. A.1: Fairseq's finalization rule
        eps, delta, M, rule = 0.0, math.inf, k, "fairseq"
    elif sched == "fixed_fairseq_stream":  # the same rule with the streaming refill
        delta, M, rule = math.inf, k, "fairseq"
    elif sched == "var_batch":
        eps = 0.0
    elif sched not in ("var_stream", "var_fifo", "var_cap"):
        raise ValueError(sched)
    select = {"var_fifo": "fifo", "var_cap": "capacity"}.get(sched, "min_steps")
    if sched == "var_cap":
        pool = 2 * n if pool is None else pool
    elif pool is not None:
        raise ValueError("pool applies to var_cap only")
    idx = np.arange(len(wl.Lx)) if inputs is None else np.asarray(inputs)
    return decode(dec, wl.h0[idx], wl.Lx[idx], wl.max_len[idx], n, eps, k, delta, M,
                  select=select, rule=rule, pool=pool)
