"""Edge cases of the HIP search against the oracle: no inputs, one beam at
a time, outputs cut at the first token, the smallest vocabulary, the widest
beam, pruning down to one candidate, and decoder reuse (several submits, a
reset, a second run)."""
import numpy as np
import pytest

from synthgen import make_workload, scaled
from tests.gpu_util import check_parity, gpu_decode

pytestmark = pytest.mark.gpu


def test_no_inputs(gpu):
    import torch
    from paper_2010_02164_amd import decoder_for_workload
    wl = make_workload(scaled(1, N=4))
    dec = decoder_for_workload(wl, max_inputs=4)
    dec.run()
    assert dec.collect() == []
    st = dec.stats()
    assert st["timesteps"] == 0 and st["expansions"] == 0 and st["hyps"] == 0
    torch.cuda.synchronize()
    dec.close()


@pytest.mark.parametrize("sched,kw", [("var_stream", {}), ("var_fifo", {}), ("var_cap", dict(pool=3)),
                                      ("fixed_fairseq", {})])
def test_one_beam_at_a_time(gpu, sched, kw):
    wl = make_workload(scaled(1, N=6))
    check_parity(wl, sched, n=1, eps=0.0 if sched == "fixed_fairseq" else 0.5, **kw)


@pytest.mark.parametrize("sched", ["var_stream", "fixed", "fixed_fairseq", "var_cap"])
def test_max_len_one(gpu, sched):
    # Every candidate of the first step is terminated (EOS or max length).
    wl = make_workload(scaled(1, N=16))
    wl.max_len[:] = 1
    rep, g, st, o = check_parity(wl, sched)
    assert all(len(h.tokens) == 1 for y in g for h in y)
    assert st["expansions"] == len(wl.Lx)


def test_vocabulary_of_k_tokens(gpu):
    wl = make_workload(scaled(1, N=16, V=4, k=4, M=4, d=64))
    check_parity(wl, "var_stream")


@pytest.mark.parametrize("sched", ["var_stream", "var_cap"])
def test_widest_beam(gpu, sched):
    wl = make_workload(scaled(1, N=12, n=4, V=600, k=16, M=16, len_hi=10))
    check_parity(wl, sched)


def test_prune_to_one(gpu):
    # A tiny threshold and one child per parent: beams of width one.
    wl = make_workload(scaled(1, N=24, delta=1e-3, M=1))
    check_parity(wl, "var_stream")


def test_reuse_after_reset(gpu):
    import torch
    from paper_2010_02164_amd import decoder_for_workload, group_by_input, inputs_to_device
    wl = make_workload(scaled(1, N=20))
    ref, _, _ = gpu_decode(wl, "var_stream")
    dec = decoder_for_workload(wl, sched="var_stream", max_inputs=20)
    key = lambda ys: [[(h.tokens, h.score, h.status) for h in y] for y in ys]
    for _ in range(2):
        idx = np.arange(20)
        dec.submit(inputs_to_device(wl, idx[:7]), wl.Lx[:7], wl.max_len[:7])
        dec.submit(inputs_to_device(wl, idx[7:]), wl.Lx[7:], wl.max_len[7:])
        dec.run()
        got = group_by_input(dec.collect(), 20)
        assert key(got) == key(ref)
        dec.reset()
    torch.cuda.synchronize()
    dec.close()


def test_caller_ids_are_echoed(gpu):
    import torch
    from paper_2010_02164_amd import decoder_for_workload, inputs_to_device
    wl = make_workload(scaled(1, N=12))
    ref, _, _ = gpu_decode(wl, "var_stream")
    ids = 1000 + 7 * np.arange(12)
    dec = decoder_for_workload(wl, sched="var_stream", max_inputs=12)
    dec.submit(inputs_to_device(wl), wl.Lx, wl.max_len, ids=ids)
    dec.run()
    got = {}
    for h in dec.collect():
        got.setdefault(h.input, []).append((h.tokens, h.score, h.status))
    assert sorted(got) == sorted(ids.tolist())
    for i, y in enumerate(ref):
        assert got[int(ids[i])] == [(h.tokens, h.score, h.status) for h in y]
    torch.cuda.synchronize()
    dec.close()
