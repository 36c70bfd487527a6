"""Pins of the oracle's length-dependent decoder step (AttnDecoder: the
projection reads h plus the layer-mean self-attention over the candidate's
KV rows). Each pin reduces the attention to a case with a closed form or to
the plain Elman decoder; the state, KV row and logit pieces it builds on are
pinned in test_oracle_decoder. CPU only."""
import math

import numpy as np
import pytest

from oracle.decoder import AttnDecoder, ElmanDecoder, bf16_round, log_softmax
from oracle.search import decode_workload
from synthgen import make_workload, scaled


def tiny(seed=0, V=40, d=16, L=3, zero_k=False, zero_kv=False):
    rng = np.random.default_rng(seed)
    r = lambda *s: bf16_round(rng.standard_normal(s) / math.sqrt(d))
    W_h, E, W_out = r(d, d), r(V, d), r(V, d) * 1.5
    W_kv = r(L, 2, d, d) * math.sqrt(d) / 2
    if zero_k:
        W_kv[:, 0] = 0.0
    if zero_kv:
        W_kv[:] = 0.0
    return AttnDecoder(W_h, E, W_out, 0.5, True, W_kv), ElmanDecoder(W_h, E, W_out, 0.5, True, W_kv)


def teacher_forced(dec, h0, tokens):
    """States and log-probs along a fixed token path (one candidate)."""
    st = dec.initial_state(h0)
    out = []
    y = 0
    for t, w in enumerate(tokens, start=1):
        (st,), lp = dec.expand([st], [y], [t], [7])
        out.append((st, lp[0]))
        y = w
    return out


def h0_of(seed, d=16):
    return bf16_round(np.random.default_rng(100 + seed).standard_normal(d))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_single_position_reads_its_value_row(seed):
    # At the first step the candidate has one KV row, its own: the softmax
    # over one position is 1, so each layer's read-out is that V row.
    att, el = tiny(seed)
    h0 = h0_of(seed)
    (st, lp), = teacher_forced(att, h0, [3])
    h = el.next_state(h0[None, :], np.array([0]))[0]
    kv = el.kv_row(h)
    x = bf16_round(h + np.mean(kv[:, 1], axis=0))
    want = log_softmax(el.logits(x[None, :], np.array([1]), np.array([7])))[0]
    assert np.max(np.abs(lp - want)) < 1e-12
    assert np.array_equal(st[0], h) and att.kv(st)[0].shape == (3, 1, 16)


@pytest.mark.parametrize("seed", [0, 3])
def test_uniform_scores_average_the_value_rows(seed):
    # K rows of zero give every position the score 0: the read-out of a layer
    # is the plain mean of its V rows.
    att, el = tiny(seed, zero_k=True)
    toks = [5, 9, 2, 11]
    steps = teacher_forced(att, h0_of(seed), toks)
    st, lp = steps[-1]
    h = st[0]
    Vs = np.stack([el.kv_row(s[0])[:, 1] for s, _ in steps])      # [t, L, d]
    x = bf16_round(h + np.mean(np.mean(Vs, axis=0), axis=0))
    want = log_softmax(el.logits(x[None, :], np.array([4]), np.array([7])))[0]
    assert np.max(np.abs(lp - want)) < 1e-12


@pytest.mark.parametrize("seed", [1, 4])
def test_two_positions_logistic_form(seed):
    # With two positions the softmax weight of position 0 is the logistic
    # function of the score difference (K_0 - K_1) . h / sqrt(d).
    att, el = tiny(seed)
    steps = teacher_forced(att, h0_of(seed), [6, 1])
    (s1, _), (s2, lp) = steps
    h = s2[0]
    K, V = att.kv(s2)
    acc = np.zeros(16)
    for l in range(3):
        k0, k1 = K[l, 0], K[l, 1]
        v0, v1 = V[l, 0], V[l, 1]
        g = 1.0 / (1.0 + math.exp(-float((k0 - k1) @ h) / 4.0))      # sqrt(16) = 4
        acc += v1 + g * (v0 - v1)
    x = bf16_round(h + acc / 3)
    want = log_softmax(el.logits(x[None, :], np.array([2]), np.array([7])))[0]
    assert np.max(np.abs(lp - want)) < 1e-12
    # the KV rows are those of the two states, in order
    assert np.array_equal(K[:, 0], el.kv_row(s1[0])[:, 0])


def test_recurrence_reads_h_not_the_attention_input():
    # The next state is tanh(W_h h + E[y]) of the previous h: the attention
    # read-out only feeds the projection.
    att, el = tiny(5)
    h0 = h0_of(5)
    steps = teacher_forced(att, h0, [4, 8, 3])
    h = h0[None, :]
    for (st, _), y in zip(steps, [0, 4, 8]):
        h = el.next_state(h, np.array([y]))
        assert np.array_equal(st[0], h[0])


def test_zero_kv_weights_reduce_to_the_elman_decoder():
    # With W_kv = 0 every K and V row is 0, so x = h and a whole search
    # returns exactly what the Elman decoder's search returns.
    cfg = scaled(6, N=12, n=4, V=50, d=16, len_hi=8, kv_layers=2)
    wl = make_workload(cfg)
    wl.W_kv[:] = 0.0
    a = decode_workload(wl, sched="var_stream")
    b = decode_workload(wl, sched="var_stream", decoder=ElmanDecoder.from_workload(wl))
    for ya, yb in zip(a.hyps, b.hyps):
        assert [(h.tokens, h.score) for h in ya] == [(h.tokens, h.score) for h in yb]


def test_attention_changes_the_search_and_keeps_scheduler_invariance():
    # The read-out matters (outputs differ from the Elman decoder's), and
    # Sec. 3 still holds: Var-Stream, Var-Str-FIFO and the capacity mode
    # return Var-Batch's outputs.
    cfg = scaled(6, N=16, n=4, V=50, d=16, len_hi=8, kv_layers=2)
    wl = make_workload(cfg)
    vb = decode_workload(wl, sched="var_batch")
    el = decode_workload(wl, sched="var_batch", decoder=ElmanDecoder.from_workload(wl))
    assert any([h.tokens for h in ya] != [h.tokens for h in yb] for ya, yb in zip(vb.hyps, el.hyps))
    for sched in ("var_stream", "var_fifo", "var_cap"):
        r = decode_workload(wl, sched=sched)
        assert r.expansions == vb.expansions
        for ya, yb in zip(vb.hyps, r.hyps):
            assert [(h.tokens, h.score) for h in ya] == [(h.tokens, h.score) for h in yb]
