"""Pins of the oracle's decision-margin log (CPU).

Every GPU/oracle mismatch that the parity rule excuses rests on the margin
the oracle logs per step: the smallest score gap among the ranking decisions
of the step. For the paper's rule (Sec. 2 top-k ranking of the k|V|
expansions, Sec. 4 heuristics) those decisions are the order of adjacent
members of the full beam B', the cut between its k-th and (k+1)-th ranked
expansion, and each member's distance to the relative-threshold boundary
best - delta. Under the Fixed-Fairseq rule (App. A.1) the outputs and the
next beam are both drawn from the first 2k+1 ranks, so the margin covers
the adjacent pairs there. An exact tie is decided by the ranking key
(parent rank, token), not by the scores, and is no margin.

Each case below is worked out by hand from scripted log-probabilities
(probabilities chosen so that a single, known decision carries the smallest
gap), and the expected margin is written as the log-ratio of the two
probabilities involved.
"""
import math

import numpy as np
import pytest

from oracle.beam import ACTIVE, EOS, Cand, beam_step, beam_step_fairseq
from oracle.search import decode
from tests.scripted import PrefixDecoder

INF = math.inf


def _root(score=0.0):
    return Cand(score, (), ACTIVE, np.zeros(1), 0)


def _lp(p):
    return np.log(np.asarray(p, np.float64))


def _step(beam, rows, k, delta=INF, M=None, t=1, max_len=10):
    lp = {j: _lp(p) for j, p in rows.items()}
    h = {j: np.zeros(1) for j in rows}
    return beam_step(beam, lp, h, t, max_len, k, delta, k if M is None else M)


def test_margin_kth_versus_next():
    # One parent, k = 3: full beam .5, .25, .13; the next expansion is .12.
    # Adjacent gaps ln 2 = .693 and ln(.25/.13) = .654; the cut between the
    # 3rd and 4th ranked expansion, ln(.13/.12) = .080, is the smallest.
    r = _step([_root()], {0: [0.5, 0.25, 0.13, 0.12]}, k=3)
    assert r.margin == pytest.approx(math.log(0.13 / 0.12), abs=1e-12)


def test_margin_adjacent_ranks():
    # k = 3: full beam .4, .38, .12, next .1. Gaps ln(.4/.38) = .051,
    # ln(.38/.12) = 1.15, cut ln(.12/.1) = .182: the order of the two best
    # (which fixes their parent ranks at the next step) is the closest call.
    r = _step([_root()], {0: [0.4, 0.38, 0.12, 0.1]}, k=3)
    assert r.margin == pytest.approx(math.log(0.4 / 0.38), abs=1e-12)


def test_margin_with_noop_and_two_parents():
    # Rank 0: a terminated candidate (score ln .5, carried by a no-op);
    # rank 1: active, score ln .3, children .3 x (.2, .5, .3) = .06 (EOS),
    # .15, .09. k = 2: full beam = no-op .5, child .15; next .09.
    # Gaps: ln(.5/.15) = 1.20 and the cut ln(.15/.09) = ln(5/3) = .511.
    beam = [Cand(math.log(0.5), (0,), EOS, None, 0), Cand(math.log(0.3), (1,), ACTIVE, np.zeros(1), 1)]
    r = _step(beam, {1: [0.2, 0.5, 0.3]}, k=2, t=2)
    assert [e[2] for e in r.full] == [-1, 1]
    assert r.margin == pytest.approx(math.log(0.15 / 0.09), abs=1e-12)


def test_margin_threshold_boundary():
    # delta = 1, k = 3: full beam .5, .2, .19, next .11. Reference ln .5,
    # boundary ln .5 - 1. Distances to it: 1, 1 - ln(.5/.2) = .084 and
    # 1 - ln(.5/.19) = .032; gaps ln(.5/.2) = .92, ln(.2/.19) = .051, cut
    # ln(.19/.11) = .55. The member closest to the boundary decides.
    r = _step([_root()], {0: [0.5, 0.2, 0.19, 0.11]}, k=3, delta=1.0)
    assert r.margin == pytest.approx(1.0 - math.log(0.5 / 0.19), abs=1e-12)
    assert len(r.beam) == 3          # all three lie above the boundary


def test_margin_threshold_boundary_of_a_pruned_member():
    # delta = 1, k = 3: full beam .5, .2, .18, next .1. Distances to the
    # boundary ln .5 - 1: 1, 1 - ln(.5/.2) = .084 (kept) and
    # ln(.5/.18) - 1 = .022 (pruned); gaps ln(.5/.2) = .92, ln(.2/.18) = .105,
    # cut ln(.18/.1) = .59. The pruned member's distance is the margin.
    r = _step([_root()], {0: [0.5, 0.2, 0.18, 0.1]}, k=3, delta=1.0)
    assert len(r.beam) == 2
    assert r.margin == pytest.approx(math.log(0.5 / 0.18) - 1.0, abs=1e-12)


def test_exact_tie_is_no_margin():
    # k = 2: two tokens with equal probability .45 share ranks 0 and 1; the
    # ranking key orders them by token. The only scored decision is the cut
    # ln(.45/.1).
    r = _step([_root()], {0: [0.1, 0.45, 0.45]}, k=2)
    assert [e[2] for e in r.full] == [1, 2]
    assert r.margin == pytest.approx(math.log(0.45 / 0.1), abs=1e-12)


def test_fairseq_margin_window():
    # Fixed-Fairseq rule, k = 2, two active parents with scores ln .6, ln .4.
    # Parent 0 children .6 x (.40, .35, .197, .053) = .24 (EOS), .21, .1182;
    # parent 1 children .4 x (.05, .50, .30, .15) = .20, .12, .06 (and EOS
    # .02). Ranked: .24, .21, .20, .12, .1182, .06. The first 2k+1 = 5 ranks
    # give the gaps ln(.24/.21) = .134, ln(.21/.20) = .049, ln(.2/.12) = .51,
    # ln(.12/.1182) = .0151; the last is the smallest, and the gap to the
    # 6th rank (ln(.1182/.06) = .68) lies outside the window.
    beam = [Cand(math.log(0.6), (1,), ACTIVE, np.zeros(1), 1), Cand(math.log(0.4), (2,), ACTIVE, np.zeros(1), 2)]
    lp = {0: _lp([0.40, 0.35, 0.197, 0.053]), 1: _lp([0.05, 0.50, 0.30, 0.15])}
    h = {0: np.zeros(1), 1: np.zeros(1)}
    r = beam_step_fairseq(beam, lp, h, t=2, max_len=10, k=2, n_out=0)
    assert [c.tokens for c in r.outputs] == [(1, 0)]
    assert [c.tokens for c in r.beam] == [(1, 1), (2, 1)]
    assert r.margin == pytest.approx(math.log(0.4 * 0.3 / (0.6 * 0.197)), abs=1e-12)


def test_search_keeps_the_smallest_margin_of_an_input():
    # A scripted two-step search (k = 2, no threshold): step 1 ranks .5 / .3
    # with cut .2, i.e. gaps ln(5/3) = .51 and ln(3/2) = .41; step 2 expands
    # [1] (.5) into .5 x (.1, .46, .44) and [2] (.3) into .3 x (.6, .2, .2),
    # i.e. .23, .22, .18 (EOS), ...: gaps ln(.23/.22) = .044 (adjacent) and
    # cut ln(.22/.18) = .20. Step 3 is max_len. The per-step log and the
    # input's minimum must both show the step-2 gap.
    table = {(): [0.2, 0.5, 0.3], (1,): [0.1, 0.46, 0.44], (2,): [0.6, 0.2, 0.2],
             (1, 1): [0.7, 0.2, 0.1], (1, 2): [0.5, 0.3, 0.2]}
    dec = PrefixDecoder(table, V=3)
    res = decode(dec, np.zeros((1, 1)), [5], [3], n=1, eps=0.0, k=2)
    m = res.margins[0]
    assert m[0] == pytest.approx(math.log(0.3 / 0.2), abs=1e-12)
    assert m[1] == pytest.approx(math.log(0.23 / 0.22), abs=1e-12)
    assert res.min_margin[0] == pytest.approx(math.log(0.23 / 0.22), abs=1e-12)
    assert res.min_margin[0] == min(m)
