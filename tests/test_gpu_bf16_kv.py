"""bf16 workloads (config 4 shape) and the per-candidate KV-like state
(config 5 shape): end-to-end parity with the oracle and the KV rows against
a teacher-forced recomputation."""
import numpy as np
import pytest

from oracle.decoder import ElmanDecoder
from synthgen import make_workload, scaled
from synthgen.gen import bf16_bits_to_f32, f32_to_bf16_bits
from tests.gpu_util import check_parity, gpu_decode, length_sample, sampled_parity

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("sched,eps", [("var_batch", None), ("var_stream", 0.125), ("var_stream", 0.5),
                                       ("fixed", None), ("var_fifo", 0.25)])
def test_cfg4_reduced(gpu, sched, eps):
    # |V| = 8320 (65 tiles): the short tile lists of the full vocabulary.
    wl = make_workload(scaled(4, N=48, n=16, V=8320))
    rep, _, _, _ = check_parity(wl, sched, eps=eps)
    # bf16 states are reproduced exactly, so scores match like fp32 ones
    assert rep.max_score_err < 1e-4


@pytest.mark.parametrize("sched", ["fixed", "var_batch", "var_stream", "var_fifo"])
def test_cfg5_reduced_search(gpu, sched):
    wl = make_workload(scaled(5, N=24, n=8, V=8320, len_hi=30))
    check_parity(wl, sched)


@pytest.mark.parametrize("sched,eps", [("var_stream", None), ("var_batch", None), ("fixed", None),
                                       ("var_stream", 0.125)])
def test_cfg4_full_size_sampled(gpu, sched, eps):
    # The full bf16 wide-beam workload: 8192 inputs, n = 512, k = 10 (steps
    # of up to 5 120 rows), |V| = 32000, d = 1024; 48 inputs over the length
    # distribution (the 8 longest included) decoded by the oracle as one
    # batch.
    from synthgen import get_config
    wl = make_workload(get_config(4))
    g, st, dec = gpu_decode(wl, sched, eps=eps)
    counts, width = dec.rows_histogram()
    dec.close()
    assert st["finished"] == len(wl.Lx) and st["hyps"] == sum(len(y) for y in g)
    assert sum(c for i, c in enumerate(counts) if i * width >= 4096) > 0   # full-size steps ran
    sampled_parity(wl, g, length_sample(wl, 48), f"cfg4 full {sched} eps={eps}, 48 sampled", sched)


@pytest.mark.parametrize("sched", ["var_stream", "fixed"])
def test_cfg5_full_size_sampled(gpu, sched):
    # Config 5 at full size: 8192 inputs, n = 256, k = 5, |V| = 64000,
    # d = 1024, KV rows of 6 layers appended every step; 24 inputs over the
    # length distribution (the 8 longest included) decoded by the oracle.
    from synthgen import get_config
    wl = make_workload(get_config(5))
    g, st, dec = gpu_decode(wl, sched)
    dec.close()
    assert st["finished"] == len(wl.Lx) and st["hyps"] == sum(len(y) for y in g)
    sampled_parity(wl, g, length_sample(wl, 24), f"cfg5 full {sched}, 24 sampled", sched)


def _kv_reference(wl, dec_o, i, tokens):
    """KV rows of a candidate of input i with emitted `tokens`: row r is
    bf16(h_r . W_kv) with h_r the state computed at step r (teacher forced)."""
    h = dec_o.initial_state(wl.h0[i])[None, :]
    y = 0
    rows = []
    for t in range(len(tokens)):
        h = dec_o.next_state(h, np.array([y]))
        rows.append(dec_o.kv_row(h[0]))
        y = tokens[t]
    return np.stack(rows, axis=2)   # [L, 2, t, d]


@pytest.mark.parametrize("sched", ["var_stream", "var_fifo"])
def test_cfg5_kv_rows(gpu, sched):
    import torch
    from paper_2010_02164_amd import decoder_for_workload, inputs_to_device
    # n below N: refills put beams at different steps side by side (under
    # Var-Str-FIFO they are expanded in the same timestep).
    wl = make_workload(scaled(5, N=9, n=6, V=6000, len_hi=40))
    c = wl.cfg
    dec = decoder_for_workload(wl, sched=sched, eps=0.5)
    dec.submit(inputs_to_device(wl), wl.Lx, wl.max_len)
    for _ in range(12):
        dec.step(sync=True)
    o = ElmanDecoder.from_workload(wl)
    checked, diff_ulps = 0, []
    for b in range(c.n):
        for r in range(c.k):
            info = dec.debug_slot(b, r, kv_layers=c.kv_layers)
            if info["status"] != 1 or info["kv"] is None:
                continue
            assert len(info["tokens"]) == info["steps"]
            ref = _kv_reference(wl, o, info["input"], info["tokens"])
            got = bf16_bits_to_f32(info["kv"].reshape(-1)).reshape(info["kv"].shape).astype(np.float64)
            assert got.shape == ref.shape
            rb = f32_to_bf16_bits(ref.astype(np.float32).reshape(-1)).astype(np.int32)
            gb = info["kv"].reshape(-1).astype(np.int32)
            # sign-magnitude ulp distance between bf16 codes
            to_ord = lambda x: np.where(x & 0x8000, -(x & 0x7FFF), x & 0x7FFF)
            d = np.abs(to_ord(rb) - to_ord(gb))
            # Near zero a bf16 step is smaller than the fp32 accumulation
            # error (~sqrt(d) 2^-24 |h||w| ~ 1e-6 at d = 1024): there the
            # bound is absolute.
            small = np.abs(got.reshape(-1) - ref.reshape(-1)) <= 4e-6
            d = np.where(small, 0, d)
            diff_ulps.append(d)
            checked += 1
    dec.close()
    assert checked >= 3
    d = np.concatenate(diff_ulps)
    print(f"[kv] slots={checked} rows exact={np.mean(d == 0):.4f} max_ulp={d.max()}", flush=True)
    # fp32-accumulated bf16 products vs the fp64 value: at most one bf16 step
    assert d.max() <= 1
    assert np.mean(d == 0) > 0.99


def test_bf16_schedulers_agree_bitwise_across_tile_shapes(gpu):
    # |V| = 32000 with steps of up to 640 rows: large steps use 256-wide
    # vocabulary tiles, small ones 128-wide tiles of 1 to 8 blocks; a row's
    # sums must not depend on which.
    wl = make_workload(scaled(4, N=96, n=64, V=32000, d=256))
    a, sa, da = gpu_decode(wl, "var_batch")
    counts, width = da.rows_histogram()
    assert sum(c for i, c in enumerate(counts) if i * width >= 384) > 0
    for sched, kw in (("var_stream", {}), ("var_fifo", dict(n=24)), ("var_cap", dict(n=40, pool=80))):
        b, sb, _ = gpu_decode(wl, sched, **kw)
        assert sb["expansions"] == sa["expansions"]
        for ya, yb in zip(a, b):
            assert [(h.tokens, h.score, h.status) for h in ya] == [(h.tokens, h.score, h.status) for h in yb]


def test_cfg4_wide_tiles_parity(gpu):
    wl = make_workload(scaled(4, N=96, n=64, V=32000, d=256))
    check_parity(wl, "var_stream")
