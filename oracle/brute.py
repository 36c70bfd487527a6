"""Exhaustive enumeration and teacher-forced scoring (test infrastructure).

Straight-line per-sequence code, written separately from the batched
decoder, used to pin the search:
  * score_tokens: the cumulative log-likelihood of one output (Sec. 2: the
    score of a candidate is the sum of its per-token log-probabilities),
    recomputed one token at a time from h0;
  * enumerate_complete: every complete output of length <= max_len, i.e.
    every token path that ends in EOS or reaches max_len (Sec. 2: a
    candidate is finalized once it appends EOS or reaches the maximum length);
  * greedy: the argmax chain of Sec. 2 (greedy search).
"""
from __future__ import annotations

import math
from typing import List, Tuple

import numpy as np


class _Scalarized:
    """Per-vector decoder evaluation with math-module reductions."""

    def __init__(self, W_h, E, W_out, beta, bf16_state, eos=0):
        self.W_h = np.asarray(W_h, np.float64)
        self.E = np.asarray(E, np.float64)
        self.W_out = np.asarray(W_out, np.float64)
        self.beta = float(beta)
        self.bf16 = bool(bf16_state)
        self.eos = eos

    def _round_bf16(self, v):
        out = []
        for x in v:
            if x == 0.0:
                out.append(0.0)
                continue
            m, e = math.frexp(x)
            q = math.ldexp(1.0, max(e - 8, -133))
            r = x / q
            fl = math.floor(r)
            frac = r - fl
            if frac > 0.5 or (frac == 0.5 and fl % 2 == 1):
                fl += 1
            out.append(fl * q)
        return np.array(out)

    def step(self, h, y, t, Lx):
        d = h.shape[0]
        pre = np.array([math.fsum(self.W_h[i, j] * h[j] for j in range(d)) + self.E[y, i]
                        for i in range(d)])
        hn = np.array([math.tanh(p) for p in pre])
        if self.bf16:
            hn = self._round_bf16(hn)
        z = [math.fsum(self.W_out[v, j] * hn[j] for j in range(d)) for v in range(self.W_out.shape[0])]
        z[self.eos] += self.beta * (t - Lx)
        mz = max(z)
        lse = mz + math.log(math.fsum(math.exp(a - mz) for a in z))
        return hn, [a - lse for a in z]


def score_tokens(W_h, E, W_out, beta, bf16_state, h0, Lx, tokens) -> float:
    """Teacher-forced cumulative log-probability of `tokens` from h0."""
    dec = _Scalarized(W_h, E, W_out, beta, bf16_state)
    h = np.asarray(h0, np.float64)
    y, total = 0, 0.0
    for t, w in enumerate(tokens, start=1):
        h, lp = dec.step(h, y, t, Lx)
        total += lp[w]
        y = w
    return total


def enumerate_complete(W_h, E, W_out, beta, bf16_state, h0, Lx, max_len,
                       eos=0) -> List[Tuple[Tuple[int, ...], float, int]]:
    """All complete outputs as (tokens, score, status) with status 2 = EOS,
    3 = cut at max_len. Depth-first over every prefix: |V|^t growth, so only
    for tiny V and max_len."""
    dec = _Scalarized(W_h, E, W_out, beta, bf16_state, eos)
    V = dec.W_out.shape[0]
    out = []

    def rec(h, y, prefix, score):
        t = len(prefix) + 1
        hn, lp = dec.step(h, y, t, Lx)
        for w in range(V):
            s = score + lp[w]
            if w == eos:
                out.append((prefix + (w,), s, 2))
            elif t == max_len:
                out.append((prefix + (w,), s, 3))
            else:
                rec(hn, w, prefix + (w,), s)

    rec(np.asarray(h0, np.float64), 0, (), 0.0)
    return out


def greedy(W_h, E, W_out, beta, bf16_state, h0, Lx, max_len, eos=0):
    """Greedy search (Sec. 2): append the argmax token until EOS or max_len.
    Returns (tokens, score)."""
    dec = _Scalarized(W_h, E, W_out, beta, bf16_state, eos)
    h = np.asarray(h0, np.float64)
    y, toks, total = 0, [], 0.0
    for t in range(1, max_len + 1):
        h, lp = dec.step(h, y, t, Lx)
        w = int(np.argmax(lp))
        toks.append(w)
        total += lp[w]
        y = w
        if w == eos:
            break
    return tuple(toks), total
