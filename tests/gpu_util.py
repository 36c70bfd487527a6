"""Helpers shared by the GPU tests: run the HIP search on a workload and
compare it with the oracle."""
import math

import numpy as np

from oracle.compare import compare
from oracle.search import decode_workload


def gpu_decode(wl, sched, eps=None, n=None, inputs=None, weights=None, timing=False, pool=None):
    """Run the HIP decoder over (a subset of) a workload; returns
    (per-input hypotheses, stats, decoder)."""
    import torch
    from paper_2010_02164_amd import decoder_for_workload, group_by_input, inputs_to_device
    idx = np.arange(len(wl.Lx)) if inputs is None else np.asarray(inputs)
    dec = decoder_for_workload(wl, sched=sched, eps=eps, n=n, max_inputs=len(idx), weights=weights,
                               pool=pool)
    if timing:
        dec.set_timing(True)
    dec.submit(inputs_to_device(wl, idx), wl.Lx[idx], wl.max_len[idx])
    dec.run()
    hyps = group_by_input(dec.collect(), len(idx))
    st = dec.stats()
    torch.cuda.synchronize()
    return hyps, st, dec


def score_tol(wl):
    return 2e-2 if wl.is_bf16 else 1e-4


def tie_tol(wl):
    """Decision margin below which a mismatching input is excused.

    1e-4 nats covers fp32/bf16 accumulation-order differences of the logits.
    With the attention read-out, the bf16 projection input x can differ by
    one bf16 step in an element where a KV row element did (the KV rows are
    fp32-accumulated bf16 products, at most one bf16 step from the oracle's
    fp64 value): |x_j| < 2 gives a step of at most 2^-7, and |W_out[v, j]|
    stays below 0.14 (4.5 standard deviations of N(0, 1/1024)), so a logit
    moves by at most 1.1e-3 per such element and two candidates' gap by
    2.2e-3. The threshold for attention workloads is 3e-3."""
    return 3e-3 if getattr(wl.cfg, "attn", False) else 1e-4


def check_parity(wl, sched, eps=None, n=None, inputs=None, oracle_res=None, weights=None,
                 require_stats=True, pool=None, max_excused=0):
    """GPU vs oracle on the same inputs; returns the comparison report.

    No input may be excused by the near-tie rule unless the caller allows
    `max_excused` of them (tests that plant ties on purpose)."""
    idx = np.arange(len(wl.Lx)) if inputs is None else np.asarray(inputs)
    o = oracle_res or decode_workload(wl, sched=sched, eps=eps, n=n, inputs=idx, pool=pool)
    g, st, dec = gpu_decode(wl, sched, eps=eps, n=n, inputs=idx, weights=weights, pool=pool)
    dec.close()
    rep = compare(o.hyps, o.min_margin, [[(h.tokens, h.score, h.status) for h in y] for y in g],
                  inputs=idx, score_tol=score_tol(wl), tie_tol=tie_tol(wl))
    print(f"[parity] {wl.cfg.name} {sched} eps={eps} n={n} pool={pool} N={len(idx)}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]
    assert rep.n_excused <= max_excused, (rep.n_excused, rep.excused[:10])
    if require_stats and rep.n_excused == 0:
        for key in ("timesteps", "expansions", "noops", "refills", "admitted", "positions"):
            assert st[key] == getattr(o, key), (key, st[key], getattr(o, key))
        assert st["hyps"] == o.n_hyps
        fin = [y[0].finalize_step for y in g]
        assert fin == list(o.finalize_step)
    return rep, g, st, o


# The oracle setting with a scheduler's outputs (per input, the schedulers of
# one family return the same hypotheses).
ORACLE_FAMILY = {"var_stream": "var_batch", "var_batch": "var_batch", "var_fifo": "var_batch",
                 "var_cap": "var_batch", "fixed": "fixed", "fixed_stream": "fixed",
                 "fixed_fairseq": "fixed_fairseq", "fixed_fairseq_stream": "fixed_fairseq"}


def sampled_parity(wl, g, sample, label, sched="var_stream"):
    """Compare the GPU decode `g` (per-input hypotheses of the whole
    workload) on the inputs `sample` with the oracle decoding just those
    inputs, as one batch of len(sample) beams (an input's result does not
    depend on the beams it shares the batch with, Sec. 3). Nothing may be
    excused."""
    from oracle.compare import compare
    from oracle.search import decode_workload
    sample = [int(i) for i in sample]
    o = decode_workload(wl, sched=ORACLE_FAMILY[sched], inputs=sample, n=len(sample))
    rep = compare(o.hyps, o.min_margin, [[(h.tokens, h.score, h.status) for h in g[i]] for i in sample],
                  inputs=sample, score_tol=score_tol(wl), tie_tol=tie_tol(wl))
    print(f"[parity] {label}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]
    assert rep.n_excused == 0, rep.excused[:10]
    return rep


def length_sample(wl, count, longest=8, seed=0):
    """`count` input ids spread over the length distribution: the `longest`
    inputs by max_len, the rest drawn evenly over the inputs sorted by
    L_x."""
    order = np.argsort(wl.max_len, kind="stable")
    top = order[-longest:]
    rest = order[:-longest]
    pick = rest[np.linspace(0, len(rest) - 1, count - longest).round().astype(int)]
    return sorted(set(top.tolist()) | set(pick.tolist()))
