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


def test_largest_rows_and_state(gpu):
    # n*k = 65536 rows per step at most (n = 4096, k = 16) with d = 4096: the
    # decode runs to completion and sampled inputs match the oracle decoding
    # them alone (results are per input, Sec. 3).
    from oracle.compare import compare
    from oracle.search import decode_workload
    wl = make_workload(scaled(1, N=4096, n=4096, k=16, M=16, V=512, d=4096, len_lo=3, len_hi=6))
    g, st, dec = gpu_decode(wl, "var_stream")
    dec.close()
    assert st["finished"] == 4096 and st["hyps"] == sum(len(y) for y in g)
    sample = [0, 2047, 4095]
    hy, mm = [], []
    for i in sample:
        o = decode_workload(wl, inputs=[i])
        hy.append(o.hyps[0])
        mm.append(o.min_margin[0])
    rep = compare(hy, mm, [[(h.tokens, h.score, h.status) for h in g[i]] for i in sample], inputs=sample)
    print(f"[parity] n=4096 k=16 d=4096 sampled: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures
    assert rep.n_excused == 0, rep.excused


def test_long_outputs(gpu):
    # Outputs of about 300 tokens (max_len 400): deep backpointer histories.
    wl = make_workload(scaled(1, N=6, n=4, V=64, d=64, len_lo=290, len_hi=310, max_len=400))
    rep, g, st, o = check_parity(wl, "var_stream")
    assert max(len(h.tokens) for y in g for h in y) > 250


def _plant_ties(wl, pairs):
    # Tokens 2j+1 and 2j+2 share their output and embedding rows: their
    # logits are equal, and so are the states and scores of two children
    # that differ only in them, at every later step. Such exact ties are
    # decided by the ranking key alone (parent rank, then token), and the
    # oracle logs them as no decision margin, so these inputs are compared
    # strictly.
    for a in range(1, 2 * pairs, 2):
        wl.W_out[a + 1] = wl.W_out[a]
        wl.E[a + 1] = wl.E[a]


@pytest.mark.parametrize("cfg_i,over,pairs,sched,kw", [
    (1, dict(N=24), 200, "var_stream", {}),
    (1, dict(N=24), 200, "fixed", {}),
    (1, dict(N=24), 200, "fixed_fairseq", {}),
    (1, dict(N=24), 200, "var_cap", dict(pool=16)),
    (4, dict(N=24, n=8, V=4000, d=256, len_hi=20), 600, "var_stream", {}),
])
def test_exact_ties_follow_rank_key(gpu, cfg_i, over, pairs, sched, kw):
    # Small vocabularies: every tile keeps the full key list, so no tile is
    # recomputed and every logit comes from the projection kernel.
    wl = make_workload(scaled(cfg_i, **over))
    _plant_ties(wl, pairs)
    rep, g, st, o = check_parity(wl, sched, max_excused=len(wl.Lx) // 3, **kw)
    tied = sum(1 for y in o.hyps for i in range(len(y)) for j in range(i + 1, len(y)) if y[i].score == y[j].score)
    assert tied > 0                                  # the ties reach the outputs


def test_collect_in_pieces_through_the_c_abi(gpu):
    # sb_collect with buffers too small for everything: each call returns
    # whole inputs (SB_E_TRUNCATED while some remain), the tokens of its
    # hypotheses packed from offset 0 of the caller's buffer; the pieces
    # together equal a single collect of the same decode.
    import ctypes

    import numpy as np
    import torch
    from paper_2010_02164_amd import _native as N
    from paper_2010_02164_amd import decoder_for_workload, inputs_to_device
    wl = make_workload(scaled(1, N=24))
    ref_dec = decoder_for_workload(wl, sched="var_stream")
    ref_dec.submit(inputs_to_device(wl), wl.Lx, wl.max_len)
    ref_dec.run()
    ref = ref_dec.collect()
    ref_dec.close()
    dec = decoder_for_workload(wl, sched="var_stream")
    dec.submit(inputs_to_device(wl), wl.Lx, wl.max_len)
    dec.run()
    L = N.lib()
    got, calls, truncated = [], 0, 0
    while True:
        hyps = (N.SbHyp * 7)()
        toks = np.full(400, -7, np.int32)
        nh, nt = ctypes.c_int64(0), ctypes.c_int64(0)
        st = L.sb_collect(dec.handle, hyps, 7, toks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 400,
                          ctypes.byref(nh), ctypes.byref(nt))
        calls += 1
        assert st in (N.SB_OK, N.SB_E_TRUNCATED)
        truncated += st == N.SB_E_TRUNCATED
        assert nt.value == sum(hyps[i].length for i in range(nh.value))
        assert (toks[nt.value:] == -7).all()          # nothing written past the returned tokens
        for i in range(nh.value):
            h = hyps[i]
            got.append((int(h.input), int(h.rank), tuple(toks[h.tok_offset:h.tok_offset + h.length].tolist()),
                        float(h.score), int(h.status)))
        if st == N.SB_OK or nh.value == 0:
            break
    torch.cuda.synchronize()
    dec.close()
    assert truncated > 0 and calls > 2
    assert got == [(h.input, h.rank, h.tokens, h.score, h.status) for h in ref]
