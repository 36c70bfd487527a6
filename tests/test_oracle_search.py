"""Pins of the oracle's search and scheduler (Sec. 2, Sec. 3 / Alg. 1,
Sec. 4 heuristics, App. A) against brute force, greedy search, hand-derived
scripted cases and the paper's invariants."""
import json
import math
import os

import numpy as np
import pytest

from oracle import brute
from oracle.beam import EOS, MAXLEN
from oracle.decoder import ElmanDecoder
from oracle.search import decode, decode_workload
from synthgen import get_config, make_workload, scaled
from tests.scripted import LengthDecoder, PrefixDecoder

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_model(V, d, seed, bf16=False, beta=0.5):
    rng = np.random.default_rng(seed)
    W_h = rng.standard_normal((d, d)) / math.sqrt(d)
    E = rng.standard_normal((V, d)) / math.sqrt(d)
    W_out = rng.standard_normal((V, d)) * 1.5 / math.sqrt(d)
    return W_h, E, W_out, beta, bf16


@pytest.mark.parametrize("V,max_len,seed,bf16", [(2, 5, 0, False), (3, 4, 1, False),
                                                  (4, 5, 2, False), (3, 5, 3, True)])
def test_exhaustive_beam_returns_every_complete_output_sorted(V, max_len, seed, bf16):
    # With k >= number of complete outputs and no pruning, no candidate is
    # ever dropped, so Y must be every complete output in score order (Sec. 2).
    d = 4
    model = tiny_model(V, d, seed, bf16)
    rng = np.random.default_rng(100 + seed)
    h0 = rng.standard_normal((1, d))
    Lx = [2]
    allseq = brute.enumerate_complete(*model, h0[0], Lx[0], max_len)
    dec = ElmanDecoder(*model)
    k = len(allseq)
    res = decode(dec, h0, Lx, [max_len], n=1, eps=0.0, k=k)
    got = [(h.tokens, h.score, h.status) for h in res.hyps[0]]
    want = sorted(allseq, key=lambda e: -e[1])
    assert len(got) == len(want)
    for g, w in zip(got, want):
        assert g[0] == w[0] and g[2] == w[2]
        assert abs(g[1] - w[1]) < 1e-12


@pytest.mark.parametrize("seed", range(4))
def test_k1_is_greedy(seed):
    # k = 1: the beam keeps the single best expansion each step, which is the
    # greedy argmax chain of Sec. 2 (pruning cannot remove the top candidate).
    V, d = 9, 6
    model = tiny_model(V, d, seed, beta=0.3)
    rng = np.random.default_rng(seed)
    h0 = rng.standard_normal((5, d))
    Lx = [3, 5, 8, 2, 6]
    ml = [10, 12, 6, 9, 15]
    res = decode(ElmanDecoder(*model), h0, Lx, ml, n=2, eps=0.5, k=1, delta=0.7, M=1)
    for i in range(5):
        toks, sc = brute.greedy(*model, h0[i], Lx[i], ml[i])
        assert len(res.hyps[i]) == 1
        assert res.hyps[i][0].tokens == toks
        assert abs(res.hyps[i][0].score - sc) < 1e-12


@pytest.mark.parametrize("sched", ["var_stream", "fixed_fairseq"])
def test_scores_are_teacher_forced_sums(sched):
    # Every output's score is the sum of its per-token log-probabilities
    # (Sec. 2), recomputed token by token from h0.
    wl = make_workload(scaled(1, N=12, V=50, d=16))
    res = decode_workload(wl, sched=sched)
    c = wl.cfg
    for i in range(12):
        for h in res.hyps[i]:
            s = brute.score_tokens(wl.W_h, wl.E, wl.W_out, c.beta, False, wl.h0[i], wl.Lx[i], h.tokens)
            assert abs(s - h.score) < 1e-10


@pytest.mark.parametrize("V,max_len,seed", [(2, 5, 0), (3, 4, 1), (4, 4, 2)])
def test_fairseq_rule_exhaustive(V, max_len, seed):
    # Fixed-Fairseq rule (App. A.1) with k >= the number of complete outputs:
    # every expansion enters the full beam B', so every complete output is
    # finalized (terminated ones at once) and the beam never drops an active
    # prefix; Y is every complete output (in the order finalized).
    d = 4
    model = tiny_model(V, d, seed, False)
    rng = np.random.default_rng(200 + seed)
    h0 = rng.standard_normal((1, d))
    allseq = brute.enumerate_complete(*model, h0[0], 2, max_len)
    res = decode(ElmanDecoder(*model), h0, [2], [max_len], n=1, eps=0.0, k=len(allseq), rule="fairseq")
    got = sorted(((h.tokens, h.score, h.status) for h in res.hyps[0]), key=lambda e: -e[1])
    want = sorted(allseq, key=lambda e: -e[1])
    assert len(got) == len(want)
    for g, w in zip(got, want):
        assert g[0] == w[0] and g[2] == w[2] and abs(g[1] - w[1]) < 1e-12
    # Finalization order: nondecreasing length (outputs of a step come after
    # those of earlier steps).
    lens = [len(h.tokens) for h in res.hyps[0]]
    assert lens == sorted(lens)


@pytest.mark.parametrize("seed", range(3))
def test_fairseq_rule_k1_is_greedy(seed):
    # k = 1: B' is the single best expansion; it is output if terminated,
    # else it is the whole next beam -- the greedy argmax chain (Sec. 2).
    V, d = 9, 6
    model = tiny_model(V, d, seed, beta=0.3)
    rng = np.random.default_rng(seed)
    h0 = rng.standard_normal((4, d))
    Lx, ml = [3, 5, 8, 2], [10, 12, 6, 9]
    res = decode(ElmanDecoder(*model), h0, Lx, ml, n=2, eps=0.5, k=1, rule="fairseq")
    for i in range(4):
        toks, sc = brute.greedy(*model, h0[i], Lx[i], ml[i])
        assert len(res.hyps[i]) == 1
        assert res.hyps[i][0].tokens == toks and abs(res.hyps[i][0].score - sc) < 1e-12


def test_fairseq_rule_streaming_matches_batch():
    # Results are per input (Sec. 3), so streaming the Fixed-Fairseq search
    # returns Fixed-Fairseq's outputs; every input gets k outputs.
    wl = make_workload(scaled(1, N=17, V=40, d=10, len_hi=9))
    a = decode_workload(wl, n=4, sched="fixed_fairseq")
    b = decode(ElmanDecoder.from_workload(wl), wl.h0, wl.Lx, wl.max_len, n=4, eps=0.5,
               k=wl.cfg.k, rule="fairseq")
    _same_outputs(a, b)
    assert a.expansions == b.expansions and a.noops == 0
    assert all(len(y) == wl.cfg.k for y in a.hyps)


def _load_cases():
    with open(os.path.join(GOLDEN, "scripted_beam_cases.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _load_cases(), ids=lambda c: c["name"])
def test_scripted_cases(case):
    table = {tuple(int(x) for x in key.split(",")) if key else (): v
             for key, v in case["table"].items()}
    dec = PrefixDecoder(table, case["V"])
    delta = math.inf if case["delta"] is None else case["delta"]
    res = decode(dec, np.zeros((1, 1)), [0], [case["max_len"]], n=1, eps=0.0,
                 k=case["k"], delta=delta, M=case["M"], rule=case.get("rule", "paper"))
    got = [(list(h.tokens), h.status, h.score) for h in res.hyps[0]]
    assert len(got) == len(case["expect"])
    for g, (toks, st, p) in zip(got, case["expect"]):
        assert g[0] == toks and g[1] == st
        assert abs(g[2] - math.log(p)) < 1e-12


def test_fixed_yields_k_outputs():
    # Fixed-width search yields k finalized candidates per input (Sec. 2).
    wl = make_workload(scaled(1, N=10, V=40, d=16))
    res = decode_workload(wl, sched="fixed")
    assert all(len(y) == wl.cfg.k for y in res.hyps)


def _same_outputs(a, b):
    for ya, yb in zip(a.hyps, b.hyps):
        assert [(h.tokens, h.status) for h in ya] == [(h.tokens, h.status) for h in yb]
        assert all(abs(x.score - y.score) < 1e-9 for x, y in zip(ya, yb))


@pytest.mark.parametrize("cfg_seed,n,eps", [(0, 4, 0.25), (1, 5, 0.5), (2, 3, 1 / 3), (3, 8, 0.125)])
def test_var_stream_matches_var_batch(cfg_seed, n, eps):
    # Sec. 3: Var-Stream is an implementation optimization that exactly
    # matches Var-Batch's outputs; the candidate expansions are equal too
    # (Table 4, Table 5's eps rows).
    cfg = scaled(1, N=21, V=60, d=12, len_hi=9, seed=7000 + cfg_seed, delta=1.2, M=3, k=4)
    wl = make_workload(cfg)
    vb = decode_workload(wl, n=n, sched="var_batch")
    vs = decode_workload(wl, n=n, eps=eps, sched="var_stream")
    _same_outputs(vb, vs)
    assert vb.expansions == vs.expansions
    assert vb.noops == vs.noops
    # Exp/Step never exceeds the batch capacity n k (Table 2).
    assert max(vs.rows_per_step) <= n * cfg.k and max(vb.rows_per_step) <= n * cfg.k


@pytest.mark.parametrize("cfg_seed,n,eps", [(0, 4, 0.25), (2, 3, 1 / 3), (3, 8, 0.5)])
def test_var_fifo_matches_var_batch(cfg_seed, n, eps):
    # App. A (alternative method analysis, Table 4): Var-Str-FIFO changes only
    # which beams are expanded at a timestep, so outputs and the number of
    # expanded candidates equal Var-Batch's.
    cfg = scaled(1, N=21, V=60, d=12, len_hi=9, seed=7000 + cfg_seed, delta=1.2, M=3, k=4)
    wl = make_workload(cfg)
    vb = decode_workload(wl, n=n, sched="var_batch")
    vf = decode_workload(wl, n=n, eps=eps, sched="var_fifo")
    _same_outputs(vb, vf)
    assert vb.expansions == vf.expansions and vb.noops == vf.noops
    assert max(vf.rows_per_step) <= n * cfg.k
    # Refilling only an empty batch keeps every live beam at the same l_t:
    # with eps = 0 the FIFO selection is Var-Batch's schedule step for step.
    v0 = decode_workload(wl, n=n, eps=0.0, sched="var_fifo")
    assert v0.rows_per_step == vb.rows_per_step and list(v0.finalize_step) == list(vb.finalize_step)


def test_fixed_stream_matches_fixed():
    # App. A.1 / Table 3: streaming applied to fixed width (eps > 0) returns
    # what Fixed-Ours (eps = 0) returns.
    wl = make_workload(scaled(1, N=15, V=30, d=10, len_hi=8))
    a = decode_workload(wl, n=4, sched="fixed")
    b = decode(ElmanDecoder.from_workload(wl), wl.h0, wl.Lx, wl.max_len, n=4, eps=0.5,
               k=wl.cfg.k, delta=math.inf, M=wl.cfg.k)
    _same_outputs(a, b)
    assert a.expansions == b.expansions


def _replay(widths, n, eps, fifo=False, pool=None, budget=None):
    """Independent event simulation of Alg. 1's schedule from each input's
    per-step active widths: returns (rows per timestep, finalize timesteps).
    fifo: every live beam steps (Var-Str-FIFO); pool/budget: up to `pool`
    beams cached, and beams step in (l_t, input) order while their widths
    fit in `budget` rows; else the minimal-l_t ones."""
    N = len(widths)
    P = pool or n
    c, live, rows, fin = 0, [], [], [0] * N
    while c < N or live:
        if c < N and len(live) <= eps * P:
            m = min(P - len(live), N - c)
            live += [[i, 0] for i in range(c, c + m)]
            c += m
        lo = min(s for _, s in live)
        if budget is not None:
            sel, used = [], 0
            for b in sorted(live, key=lambda b: (b[1], b[0])):
                if used + widths[b[0]][b[1]] > budget:
                    break
                used += widths[b[0]][b[1]]
                sel.append(b)
        else:
            sel = list(live) if fifo else [b for b in live if b[1] == lo]
        rows.append(sum(widths[i][s] for i, s in sel))
        for b in sel:
            b[1] += 1
            if b[1] == len(widths[b[0]]):
                fin[b[0]] = len(rows)
        live = [b for b in live if b[1] < len(widths[b[0]])]
    return rows, fin


@pytest.mark.parametrize("eps", [0.0, 0.25, 0.5])
def test_schedule_event_replay(eps):
    wl = make_workload(scaled(1, N=30, V=50, d=12, len_hi=12))
    res = decode_workload(wl, n=6, eps=eps)
    rows, fin = _replay(res.widths, 6, eps)
    assert rows == res.rows_per_step
    assert fin == list(res.finalize_step)


@pytest.mark.parametrize("eps", [0.25, 0.5])
def test_fifo_schedule_event_replay(eps):
    wl = make_workload(scaled(1, N=30, V=50, d=12, len_hi=12))
    res = decode_workload(wl, n=6, eps=eps, sched="var_fifo")
    rows, fin = _replay(res.widths, 6, eps, fifo=True)
    assert rows == res.rows_per_step
    assert fin == list(res.finalize_step)


@pytest.mark.parametrize("eps,pool", [(0.25, 12), (0.5, 9), (0.0, 18)])
def test_capacity_schedule_event_replay(eps, pool):
    # Variable widths (delta and M pruning) make the row limit bind at
    # different beams from step to step.
    cfg = scaled(1, N=30, V=50, d=12, len_hi=12, seed=7100, delta=1.2, M=3, k=4)
    wl = make_workload(cfg)
    res = decode_workload(wl, n=6, eps=eps, sched="var_cap", pool=pool)
    rows, fin = _replay(res.widths, 6, eps, pool=pool, budget=6 * cfg.k)
    assert rows == res.rows_per_step
    assert fin == list(res.finalize_step)
    assert max(res.rows_per_step) <= 6 * cfg.k
    assert len(set(w for ws in res.widths for w in ws)) > 2


@pytest.mark.parametrize("cfg_seed,n,eps", [(0, 4, 0.25), (2, 3, 1 / 3), (3, 8, 0.5)])
def test_capacity_pool_of_n_is_fifo(cfg_seed, n, eps):
    # With no more beams cached than n, every live beam fits the n k row
    # limit, so the capacity-constrained selection takes them all: the
    # schedule is Var-Str-FIFO's step for step (App. A), and outputs are
    # Var-Batch's (Sec. 3) for any pool size.
    cfg = scaled(1, N=21, V=60, d=12, len_hi=9, seed=7000 + cfg_seed, delta=1.2, M=3, k=4)
    wl = make_workload(cfg)
    vf = decode_workload(wl, n=n, eps=eps, sched="var_fifo")
    vc = decode_workload(wl, n=n, eps=eps, sched="var_cap", pool=n)
    assert vc.rows_per_step == vf.rows_per_step
    assert list(vc.finalize_step) == list(vf.finalize_step)
    vb = decode_workload(wl, n=n, sched="var_batch")
    for pool in (n, 2 * n, 3 * n + 1):
        v = decode_workload(wl, n=n, eps=eps, sched="var_cap", pool=pool)
        _same_outputs(vb, v)
        assert v.expansions == vb.expansions and v.noops == vb.noops
        assert max(v.rows_per_step) <= n * cfg.k


def test_capacity_schedule():
    with open(os.path.join(GOLDEN, "capacity_schedule.json")) as f:
        g = json.load(f)
    L = g["L"]
    trace = []
    res = decode(LengthDecoder(g["V"]), np.zeros((len(L), 1)), L, [50] * len(L), n=g["n"],
                 eps=g["eps"], k=g["k"], on_step=lambda t, sel, r: trace.append([t, sorted(sel)]),
                 select="capacity", pool=g["pool"])
    assert trace == g["trace"]
    assert res.rows_per_step == g["rows_per_step"]
    assert list(res.finalize_step) == g["finalize_step"]


def test_fig1_schedule():
    with open(os.path.join(GOLDEN, "fig1_schedule.json")) as f:
        g = json.load(f)
    L = g["L"]
    trace = []
    res = decode(LengthDecoder(g["V"]), np.zeros((len(L), 1)), L, [50] * len(L), n=g["n"],
                 eps=g["eps"], k=g["k"], on_step=lambda t, sel, r: trace.append([t, sorted(sel)]))
    assert trace == g["var_stream_trace"]
    assert list(res.finalize_step) == g["var_stream_finalize_step"]
    vb = decode(LengthDecoder(g["V"]), np.zeros((len(L), 1)), L, [50] * len(L), n=g["n"],
                eps=0.0, k=g["k"])
    assert vb.timesteps == g["var_batch_timesteps"]
    assert list(vb.finalize_step) == g["var_batch_finalize_step"]
    assert vb.expansions == res.expansions
    trace = []
    vf = decode(LengthDecoder(g["V"]), np.zeros((len(L), 1)), L, [50] * len(L), n=g["n"],
                eps=g["eps"], k=g["k"], on_step=lambda t, sel, r: trace.append([t, sorted(sel)]),
                select="fifo")
    assert trace == g["var_fifo_trace"]
    assert list(vf.finalize_step) == g["var_fifo_finalize_step"]
    assert vf.expansions == res.expansions
