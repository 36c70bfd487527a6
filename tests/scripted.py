"""Scripted decoders for hand-derived search cases (test helper).

A scripted decoder replaces the synthetic Elman decoder with a table of
next-token probabilities, so the beam mechanics can be checked against
expectations worked out by hand.
"""
import math

import numpy as np


class PrefixDecoder:
    """Next-token probabilities looked up by the emitted prefix.

    table: {prefix tuple: [p(token 0), p(token 1), ...]}. A prefix missing
    from the table falls back to `default` (if given)."""

    def __init__(self, table, V, default=None):
        self.V = V
        self.table = {tuple(k): np.log(np.asarray(v, np.float64)) for k, v in table.items()}
        self.default = None if default is None else np.log(np.asarray(default, np.float64))
        self.ids = {}
        self.prefixes = []

    def _id(self, prefix):
        if prefix not in self.ids:
            self.ids[prefix] = len(self.prefixes)
            self.prefixes.append(prefix)
        return self.ids[prefix]

    def initial_state(self, h0):
        return np.array([-1.0])          # start symbol not consumed yet

    def expand(self, h_prev, y, t, Lx):
        h_prev = np.asarray(h_prev).reshape(-1, 1)
        R = h_prev.shape[0]
        h = np.empty((R, 1))
        lp = np.empty((R, self.V))
        for r in range(R):
            sid = int(h_prev[r, 0])
            prefix = () if sid < 0 else self.prefixes[sid] + (int(y[r]),)
            h[r, 0] = self._id(prefix)
            row = self.table.get(prefix, self.default)
            if row is None:
                raise KeyError(f"no scripted row for prefix {prefix}")
            lp[r] = row
        return h, lp


class LengthDecoder:
    """Every beam ends exactly at its own step L (passed as L_x): before it,
    two non-EOS tokens dominate; at step L, EOS takes almost all mass."""

    def __init__(self, V=3):
        self.V = V
        p = np.full(V, 1e-6)
        p[1], p[2] = 0.6, 0.4 - (V - 2) * 1e-6
        self.run = np.log(p)
        q = np.full(V, 0.01 / (V - 1))
        q[0] = 0.99
        self.stop = np.log(q)

    def initial_state(self, h0):
        return np.zeros(1)

    def expand(self, h_prev, y, t, Lx):
        R = len(y)
        lp = np.where((np.asarray(t) >= np.asarray(Lx))[:, None], self.stop, self.run)
        return np.zeros((R, 1)), lp
