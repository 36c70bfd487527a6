"""Decoder-step kernels (recurrence, projection + log-sum-exp + per-row
top-k, row merge) against the oracle's fp64 decoder on explicit rows."""
import dataclasses

import numpy as np
import pytest

from oracle.decoder import ElmanDecoder
from synthgen import make_workload, scaled

pytestmark = pytest.mark.gpu


def _expand_case(wl, R, seed, h_prev=None):
    import torch
    from paper_2010_02164_amd import decoder_for_workload
    rng = np.random.default_rng(seed)
    c = wl.cfg
    dec = decoder_for_workload(wl, max_inputs=4)
    R = min(R, c.n * c.k)
    if h_prev is None:
        h_prev = np.tanh(rng.standard_normal((R, c.d))).astype(np.float32)
    R = h_prev.shape[0]
    if wl.is_bf16:
        from synthgen.gen import bf16_bits_to_f32, f32_to_bf16_bits
        h_prev = bf16_bits_to_f32(f32_to_bf16_bits(h_prev))
    y = rng.integers(0, c.V, R).astype(np.int32)
    t = rng.integers(1, 40, R).astype(np.int32)
    Lx = rng.integers(3, 40, R).astype(np.int32)
    hp = torch.from_numpy(h_prev).cuda()
    if wl.is_bf16:
        hp = hp.to(torch.bfloat16)
    h_gpu, lse, lp, tok = dec.debug_expand(hp, y, t, Lx)
    h_gpu = h_gpu.float().cpu().numpy()
    dec.close()
    o = ElmanDecoder.from_workload(wl)
    h_ref, lp_ref = o.expand(h_prev.astype(np.float64), y, t, Lx)
    z_ref = None
    return h_prev, y, t, Lx, h_gpu, lse, lp, tok, h_ref, lp_ref


def _check_rows(wl, h_gpu, lp, tok, h_ref, lp_ref, lse):
    k = wl.cfg.k
    if wl.is_bf16:
        assert np.array_equal(h_gpu, h_ref.astype(np.float32)), "bf16 states must be bit-identical"
    else:
        # fp32 accumulation over d products: the rounding error grows like
        # sqrt(d) * 2^-24 * |pre-activation| (|pre| <~ 4), ~8e-6 at d = 1024;
        # the bound allows 8 times that (6.1e-5 at d = 1024).
        tol = 8 * np.sqrt(wl.cfg.d) * 2.0**-24 * 4
        assert np.max(np.abs(h_gpu - h_ref)) < tol
    R = lp.shape[0]
    # log-sum-exp consistency: lp_ref of the GPU's tokens vs the GPU's lp
    for r in range(R):
        ref_row = lp_ref[r]
        kth = np.sort(ref_row)[::-1][:k]
        got = ref_row[tok[r]]
        assert np.all(np.abs(lp[r] - got) < 2e-5), (r, lp[r], got)
        # the GPU's list is a valid top-k: same values as the oracle's best k
        assert np.all(np.abs(np.sort(got)[::-1] - kth) < 2e-5)
        assert np.all(np.diff(lp[r]) <= 1e-12)          # best first
        assert len(set(tok[r].tolist())) == k


@pytest.mark.parametrize("cfg_i,R,over", [
    (1, 32, {}),                                   # V=1000 (ragged last tile), d=64
    (2, 300, {}),                                  # V=256, d=256, R not a tile multiple
    (3, 640, dict(V=8000)),                        # d=1024, k=5
    (1, 7, dict(V=130, k=3, M=3, n=4)),            # tiny ragged vocab, k < 4
])
def test_expand_f32(gpu, cfg_i, R, over):
    wl = make_workload(scaled(cfg_i, N=4, **over))
    _, _, _, _, h_gpu, lse, lp, tok, h_ref, lp_ref = _expand_case(wl, R, 11)
    print(f"[expand] cfg{cfg_i} {over} R={R}", flush=True)
    _check_rows(wl, h_gpu, lp, tok, h_ref, lp_ref, lse)


@pytest.mark.parametrize("over", [dict(V=8000, n=32), dict(V=4160, d=256, n=16, k=16),
                                  dict(V=32000, n=64), dict(V=32128, d=256, n=64)])
def test_expand_bf16(gpu, over):
    # The last two use 256-wide vocabulary tiles (640 rows fill a round of
    # them); 32128 tokens leave the last 256-wide tile half empty.
    wl = make_workload(scaled(4, N=4, **over))
    _, _, _, _, h_gpu, lse, lp, tok, h_ref, lp_ref = _expand_case(wl, 640 if over["V"] >= 32000 else 200, 12)
    print(f"[expand] bf16 {over}", flush=True)
    _check_rows(wl, h_gpu, lp, tok, h_ref, lp_ref, lse)


# The bf16 recurrence sums W_h h exactly from 7-bit digits of the values
# scaled per W_h row and per state row, with the values too small for a
# row's 21-bit window added from per-row lists (a state row whose list
# overflows is scanned, a W_h whose lists overflow keeps the fp64 MFMA sum).
# These cases put such values, zeros, signed zeros, subnormals and large
# entries into W_h and the states; the states must stay bit-identical.
def _bf16(x):
    from synthgen.gen import bf16_bits_to_f32, f32_to_bf16_bits
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(x, np.float32)))


def _tiny(rng, cnt, lo=-40, hi=-16):
    return rng.choice([-1.0, 1.0], cnt) * 2.0 ** rng.uniform(lo, hi, cnt)


def _planted_wh(wl, rng, long_row=0):
    d = wl.cfg.d
    W = wl.W_h.copy()
    for o, cnt in [(0, 1), (1, 5), (2, 12), (40, 3), (1000 % d, 8)]:
        W[o, rng.choice(d, cnt, replace=False)] = _tiny(rng, cnt)
    W[7, 3] = 0.9                      # a large entry widens the row's window
    W[8, :5] = 1e-39                   # bf16 subnormals
    W[9, 10:20] = 0.0
    W[9, 20] = -0.0
    if long_row:
        W[5, rng.choice(d, long_row, replace=False)] = _tiny(rng, long_row)
    return dataclasses.replace(wl, W_h=_bf16(W))


def _planted_states(wl, rng, R):
    d = wl.cfg.d
    h = np.tanh(rng.standard_normal((R, d)))
    for r, cnt in [(0, 3), (1, 40), (5, 15), (6, 16), (33, 2), (70, 100)]:
        h[r, rng.choice(d, cnt, replace=False)] = _tiny(rng, cnt, -30, -14)
    h[2] = 0.0
    h[3, 0] = 6.0
    h[4, :8] = 1e-39 * np.sign(rng.standard_normal(8))
    h[4, 8:12] = -0.0
    h[7] = _tiny(rng, d, -30, -20)     # a row of small values only
    h[64:96] = 0.0                     # a whole tile of zero states
    if R > 1000:
        for r, cnt in [(700, 5), (701, 30), (1090, 15), (1099, 16)]:
            h[r, rng.choice(d, cnt, replace=False)] = _tiny(rng, cnt, -30, -14)
        h[1024:1088] = 0.0             # a whole 64-row tile of zero states
    return _bf16(h)


@pytest.mark.parametrize("long_row,R", [(0, 200), (40, 200), (0, 1100)])
def test_expand_bf16_small_values(gpu, long_row, R):
    # 1 100 rows run the 64 x 64 tiles (a step whose 64-row tiles fill half
    # the grid), 200 the 32 x 32 tiles with the K range split over waves.
    wl = _planted_wh(make_workload(scaled(4, N=4, V=8000, n=128)), np.random.default_rng(21), long_row)
    h_prev = _planted_states(wl, np.random.default_rng(22), R)
    _, _, _, _, h_gpu, lse, lp, tok, h_ref, lp_ref = _expand_case(wl, R, 23, h_prev=h_prev)
    print(f"[expand] bf16 small values long_row={long_row} R={R}", flush=True)
    _check_rows(wl, h_gpu, lp, tok, h_ref, lp_ref, lse)


@pytest.mark.parametrize("long_row", [0, 40])
def test_decode_bf16_small_values(gpu, long_row):
    """Whole decodes with encodings holding small values, zeros and large
    entries (their digits are made at submission) and the planted W_h (with
    a 40-value row list: the whole decode on the fp64 recurrence)."""
    from tests.gpu_util import check_parity
    rng = np.random.default_rng(31)
    wl = _planted_wh(make_workload(scaled(4, N=24, V=8000, n=8)), rng, long_row)
    h0 = wl.h0.copy()
    for i, cnt in [(0, 3), (1, 40), (2, 15), (3, 16)]:
        h0[i, rng.choice(wl.cfg.d, cnt, replace=False)] = _tiny(rng, cnt, -30, -12)
    h0[4] = 0.0
    h0[5, 0] = 60.0
    h0[6, :8] = 1e-39
    wl = dataclasses.replace(wl, h0=_bf16(h0))
    print(f"[parity] bf16 small values long_row={long_row}", flush=True)
    check_parity(wl, "var_stream")
