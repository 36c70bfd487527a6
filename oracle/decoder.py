"""Synthetic Elman decoder, fp64 (test infrastructure; see oracle/__init__).

The paper's decoder D(e_i, y_i) scores the next token of a partial output
(Sec. 2). The synthetic stand-in used here:

    h   = tanh(W_h h_prev + E[y])          y = last token (start symbol = 0)
    h   = bf16_rne(h)                      bf16 workloads only: stored state
    z   = W_out h ;  z[0] += beta (t - L_x)   t = 1-based index of the token
                                              being emitted, in this beam
    lp  = z - logsumexp(z)                 log-softmax (the log-likelihood
                                              increments of Sec. 2)

All arithmetic is float64. Weights arrive as float32 arrays whose values
(bf16-exact for bf16 workloads) are held exactly in float64, so for bf16
workloads the pre-activation W_h h + E[y] is an exact sum of exact products.

AttnDecoder adds a length-dependent step (the decoder self-attention whose
cost grows with the output position, App. A.2 and its Fig. 2): the
candidate's state also holds its KV rows, and the projection reads
x = bf16_rne(h + mean over layers of attention(h; K_l, V_l)).
"""
from __future__ import annotations

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    Rounds directly from float64 (no float32 intermediate, which could round
    twice). A bf16 normal number has 8 significant bits, so for
    x = m * 2^e with m in [0.5, 1) the quantum is 2^(e-8); below bf16's
    smallest normal (2^-126) the quantum is the subnormal step 2^-133.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q_exp = np.maximum(e - 8, -133)
    q = np.ldexp(np.ones_like(x), q_exp)
    return np.rint(x / q) * q   # x / q and * q are exact (powers of two)


def log_softmax(z: np.ndarray) -> np.ndarray:
    """Row-wise z - log(sum(exp(z))), max-shifted (Sec. 2 log-likelihoods)."""
    m = np.max(z, axis=-1, keepdims=True)
    s = np.sum(np.exp(z - m), axis=-1, keepdims=True)
    return z - (m + np.log(s))


class ElmanDecoder:
    """Batched fp64 expansion of candidates (the D calls of Alg. 1)."""

    def __init__(self, W_h, E, W_out, beta: float, bf16_state: bool,
                 W_kv=None, eos: int = 0):
        self.W_h = np.asarray(W_h, dtype=np.float64)
        self.E = np.asarray(E, dtype=np.float64)
        self.W_out = np.asarray(W_out, dtype=np.float64)
        self.W_kv = None if W_kv is None else np.asarray(W_kv, dtype=np.float64)
        self.beta = float(beta)
        self.bf16_state = bool(bf16_state)
        self.eos = int(eos)
        self.V, self.d = self.W_out.shape

    @classmethod
    def from_workload(cls, wl):
        c = wl.cfg
        return cls(wl.W_h, wl.E, wl.W_out, c.beta, c.dtype == "bf16", wl.W_kv)

    def initial_state(self, h0: np.ndarray) -> np.ndarray:
        """e_i = E(x_i): the synthetic encoder is the identity on h0."""
        return np.asarray(h0, dtype=np.float64)

    def next_state(self, h_prev: np.ndarray, y: np.ndarray) -> np.ndarray:
        """h = tanh(W_h h_prev + E[y]) for each row (rows are candidates)."""
        pre = h_prev @ self.W_h.T + self.E[np.asarray(y)]
        h = np.tanh(pre)
        if self.bf16_state:
            h = bf16_round(h)
        return h

    def logits(self, h: np.ndarray, t: np.ndarray, Lx: np.ndarray) -> np.ndarray:
        """z = W_out h with the EOS bias beta (t - L_x) added to token 0."""
        z = h @ self.W_out.T
        z[:, self.eos] += self.beta * (np.asarray(t, np.float64) - np.asarray(Lx, np.float64))
        return z

    def expand(self, h_prev, y, t, Lx, chunk: int = 256):
        """One decoder step for R candidates: returns (h [R,d], lp [R,V])."""
        h_prev = np.asarray(h_prev, dtype=np.float64).reshape(-1, self.d)
        R = h_prev.shape[0]
        h = np.empty((R, self.d))
        lp = np.empty((R, self.V))
        y, t, Lx = np.asarray(y), np.asarray(t), np.asarray(Lx)
        for a in range(0, R, chunk):
            b = min(R, a + chunk)
            h[a:b] = self.next_state(h_prev[a:b], y[a:b])
            lp[a:b] = log_softmax(self.logits(h[a:b], t[a:b], Lx[a:b]))
        return h, lp

    def kv_row(self, h: np.ndarray) -> np.ndarray:
        """Per-candidate KV-like rows appended at each step: [L, 2, d] of
        bf16_rne(h . W_kv[l, j]) (row vector times matrix)."""
        if self.W_kv is None:
            raise ValueError("decoder has no KV state")
        out = np.einsum("i,ljio->ljo", np.asarray(h, np.float64), self.W_kv)
        return bf16_round(out)


class AttnDecoder(ElmanDecoder):
    """Elman decoder whose projection input adds a self-attention read-out
    over the candidate's own KV rows (bf16 workloads with W_kv).

    A candidate's state is (h, chain): chain holds the KV rows [L, 2, d] of
    the states h_s of its first t tokens, bf16_rne(h_s . W_kv[l, j]), as a
    linked list shared with its ancestors (kv() stacks them into K, V of
    shape [L, t, d]). One step, for a candidate emitting token t:
        h     = bf16_rne(tanh(W_h h_prev + E[y]))          as ElmanDecoder
        K, V  += the rows of h                             position t - 1
        a_l   = sum_s softmax_s(K_l[s] . h / sqrt(d)) V_l[s]   s = 0 .. t-1
        x     = bf16_rne(h + (1/L) sum_l a_l)
        z     = W_out x ;  z[0] += beta (t - L_x)
    The next step's recurrence reads h, not x.
    """

    def __init__(self, *a, **kw):
        super().__init__(*a, **kw)
        if self.W_kv is None or not self.bf16_state:
            raise ValueError("attention needs bf16 states and W_kv")
        self.L = self.W_kv.shape[0]

    def initial_state(self, h0):
        return (np.asarray(h0, dtype=np.float64), None)

    def kv(self, state):
        """(K, V), each [L, t, d], of a candidate state, positions in order."""
        rows, chain = [], state[1]
        while chain is not None:
            chain, row = chain
            rows.append(row)
        a = np.stack(rows[::-1]) if rows else np.zeros((0, self.L, 2, self.d))
        return a[:, :, 0].transpose(1, 0, 2), a[:, :, 1].transpose(1, 0, 2)

    def attention(self, h, K, V):
        """(1/L) sum_l a_l for one candidate: h [d], K, V [L, t, d]."""
        out = np.zeros(self.d)
        for l in range(self.L):
            s = K[l] @ h / np.sqrt(self.d)
            w = np.exp(s - np.max(s))
            out += (w / np.sum(w)) @ V[l]
        return out / self.L

    def expand(self, states, y, t, Lx, chunk: int = 256):
        """One step for R candidates: returns (new states, lp [R,V])."""
        R = len(states)
        h = self.next_state(np.stack([st[0] for st in states]), np.asarray(y))
        t, Lx = np.asarray(t), np.asarray(Lx)
        x = np.empty((R, self.d))
        new = []
        for r, (_, chain) in enumerate(states):
            st = (h[r], (chain, self.kv_row(h[r])))      # this step's rows appended
            K, V = self.kv(st)
            if K.shape[1] != t[r]:
                raise ValueError("KV rows do not match the output position")
            x[r] = bf16_round(h[r] + self.attention(h[r], K, V))
            new.append(st)
        lp = np.empty((R, self.V))
        for a in range(0, R, chunk):
            b = min(R, a + chunk)
            lp[a:b] = log_softmax(self.logits(x[a:b], t[a:b], Lx[a:b]))
        return new, lp


def decoder_for_workload(wl):
    """The oracle decoder of a synthgen workload (AttnDecoder when the
    config enables attention)."""
    c = wl.cfg
    cls = AttnDecoder if getattr(c, "attn", False) else ElmanDecoder
    return cls(wl.W_h, wl.E, wl.W_out, c.beta, c.dtype == "bf16", wl.W_kv)
