"""The allocation-free entry point sb_create_noalloc: a decoder over the
library's static device scratch must return exactly what a decoder made by
sb_create returns, on two calls in a row (the second with a smaller input,
over a scratch that still holds the first call's contents), and refuse
shapes beyond the scratch or a second live decoder on the same GPU."""
import numpy as np
import pytest

from oracle.compare import compare
from oracle.search import decode_workload
from synthgen import make_workload, scaled

pytestmark = pytest.mark.gpu


def _run(wl, sched, noalloc):
    import torch
    from paper_2010_02164_amd import decoder_for_workload, group_by_input, inputs_to_device
    dec = decoder_for_workload(wl, sched=sched, noalloc=noalloc)
    assert (dec.workspace is None) == noalloc
    dec.submit(inputs_to_device(wl), wl.Lx, wl.max_len)
    dec.run()
    hyps = group_by_input(dec.collect(), len(wl.Lx))
    st = dec.stats()
    hist = dec.rows_histogram()
    dec.close()
    torch.cuda.synchronize()
    return [[(h.tokens, h.score, h.status, h.finalize_step) for h in y] for y in hyps], st, hist


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_sb_create(gpu, order):
    cases = [
        # bf16 with the exact recurrence's digit buffers and short tile lists, ~12 MiB
        (make_workload(scaled(4, N=48, n=8, V=8320, d=512)), "var_stream"),
        (make_workload(scaled(2, N=1024, n=64)), "var_stream"),   # ~10 MiB of workspace
        (make_workload(scaled(1, N=24, n=4)), "var_fifo"),        # smaller, over the same scratch
    ]
    for wl, sched in cases:
        ref, st_ref, hist_ref = _run(wl, sched, noalloc=False)
        got, st_got, hist_got = _run(wl, sched, noalloc=True)
        assert got == ref                     # same kernels, same arithmetic: bit for bit
        assert st_got == st_ref and hist_got == hist_ref
        o = decode_workload(wl, sched=sched)
        rep = compare(o.hyps, o.min_margin, [[(t, s, u) for t, s, u, _ in y] for y in got],
                      score_tol=2e-2 if wl.is_bf16 else 1e-4)
        print(f"[noalloc] {wl.cfg.name} {sched} N={len(wl.Lx)}: {rep.summary()}", flush=True)
        assert rep.ok and rep.n_excused == 0, rep.failures[:3]
        assert st_got["expansions"] == o.expansions and st_got["timesteps"] == o.timesteps


def test_noalloc_limits(gpu):
    from paper_2010_02164_amd import _native as N
    from paper_2010_02164_amd import decoder_for_workload
    # Beyond the scratch: refused with the sizes in the message.
    big = make_workload(scaled(2, N=16384, n=1024, d=64))
    with pytest.raises(N.StreambeamError) as e:
        decoder_for_workload(big, noalloc=True)
    assert e.value.status == N.SB_E_WORKSPACE and "static scratch" in str(e.value)
    # One live decoder per GPU over the scratch.
    wl = make_workload(scaled(1, N=8, n=2))
    a = decoder_for_workload(wl, noalloc=True)
    with pytest.raises(N.StreambeamError) as e:
        decoder_for_workload(wl, noalloc=True)
    assert e.value.status == N.SB_E_STATE
    a.close()
    b = decoder_for_workload(wl, noalloc=True)
    b.close()
