"""Pins of the oracle's decoder arithmetic against closed forms and special
cases (Sec. 2 synthetic decoder; log-softmax log-likelihoods)."""
import math

import numpy as np
import pytest

from oracle.decoder import ElmanDecoder, bf16_round, log_softmax
from synthgen.gen import bf16_bits_to_f32, f32_to_bf16_bits


def test_bf16_round_known_values():
    # bf16 keeps 8 significant bits: spacing 2^-7 on [1, 2).
    cases = {
        1.0: 1.0,
        1.0 + 2**-8: 1.0,                    # tie -> even (1.0)
        1.0 + 3 * 2**-8: 1.0 + 2**-6,        # tie -> even (1 + 2^-6)
        1.0 + 2**-8 + 2**-30: 1.0 + 2**-7,   # just above the tie
        -0.75: -0.75,
        0.1: 0.10009765625,                  # 0x3DCD
        2.0**-130: 2.0**-130,                # subnormal bf16, exact
        3 * 2.0**-134: 2.0**-132,            # subnormal tie 1.5*2^-133 -> even
    }
    for x, want in cases.items():
        assert bf16_round(np.array([x]))[0] == want, x


def test_bf16_round_matches_bitwise_fp32_path():
    # The generator rounds float32 bit patterns; the oracle rounds float64
    # values. On float32 inputs both define RNE to bf16 and must agree.
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32),
                        (rng.standard_normal(2000) * 1e-38).astype(np.float32)])
    a = bf16_bits_to_f32(f32_to_bf16_bits(x)).astype(np.float64)
    b = bf16_round(x.astype(np.float64))
    assert np.array_equal(a, b)


def test_log_softmax_closed_forms():
    z = np.array([[0.3, -1.2, 2.0, 0.0]])
    lp = log_softmax(z)
    assert abs(math.fsum(np.exp(lp[0])) - 1.0) < 1e-15
    assert np.all(lp <= 0)
    assert np.allclose(log_softmax(z + 1234.5), lp, atol=1e-12)       # shift invariance
    two = log_softmax(np.array([[1.0, 3.0]]))[0]
    assert abs(two[0] - (-math.log1p(math.exp(2.0)))) < 1e-15          # -log(1+e^2)
    assert abs(two[1] - (-math.log1p(math.exp(-2.0)))) < 1e-15


@pytest.mark.parametrize("t,Lx,beta", [(1, 5, 1.0), (9, 5, 1.0), (4, 4, 0.5), (2, 20, 0.5)])
def test_zero_weights_leave_only_eos_bias(t, Lx, beta):
    # W_h = E = 0 -> h = 0 -> z = 0 except z[EOS] = beta (t - L_x).
    V, d = 7, 3
    dec = ElmanDecoder(np.zeros((d, d)), np.zeros((V, d)), np.ones((V, d)), beta, False)
    h, lp = dec.expand(np.ones((1, d)), [3], [t], [Lx])
    b = beta * (t - Lx)
    Z = math.exp(b) + (V - 1)
    assert np.all(h == 0)
    assert abs(lp[0, 0] - (b - math.log(Z))) < 1e-14
    assert np.allclose(lp[0, 1:], -math.log(Z), atol=1e-14)


def test_recurrence_orientation_and_embedding_row():
    # W_h with one non-zero entry W_h[0, 1] = a: (W_h h)[0] = a h[1], (W_h h)[1] = 0.
    # A transposed W_h would put a h[0] into component 1 instead.
    a, x0, x1 = 0.7, -0.4, 1.3
    W_h = np.array([[0.0, a], [0.0, 0.0]])
    E = np.array([[0.0, 0.0], [0.25, -0.5], [0.0, 0.0]])
    dec = ElmanDecoder(W_h, E, np.zeros((3, 2)), 0.0, False)
    h = dec.next_state(np.array([[x0, x1]]), np.array([1]))[0]
    assert abs(h[0] - math.tanh(a * x1 + 0.25)) < 1e-15
    assert abs(h[1] - math.tanh(-0.5)) < 1e-15


def test_output_projection_orientation():
    # W_out[2, 1] = b is the only weight: z[2] = b h[1], every other z is 0
    # (no bias: t = L_x). A transposed W_out could not even be applied (V != d).
    b = 1.5
    W_out = np.zeros((4, 2))
    W_out[2, 1] = b
    dec = ElmanDecoder(np.zeros((2, 2)), np.array([[0.0, 0.3]] * 4), W_out, 1.0, False)
    h, lp = dec.expand(np.zeros((1, 2)), [0], [3], [3])
    hv = math.tanh(0.3)
    Z = math.exp(b * hv) + 3
    assert abs(lp[0, 2] - (b * hv - math.log(Z))) < 1e-14
    assert abs(lp[0, 0] - (-math.log(Z))) < 1e-14


def test_bf16_state_is_representable_and_nearest():
    rng = np.random.default_rng(3)
    d, V = 16, 5
    W_h = rng.standard_normal((d, d)) / 4
    dec = ElmanDecoder(W_h, rng.standard_normal((V, d)) / 4, rng.standard_normal((V, d)), 1.0, True)
    exact = ElmanDecoder(W_h, dec.E, dec.W_out, 1.0, False)
    h0 = rng.standard_normal((3, d))
    hb = dec.next_state(h0, np.array([0, 1, 2]))
    hf = exact.next_state(h0, np.array([0, 1, 2]))
    assert np.array_equal(bf16_round(hb), hb)
    # nearest: the error is at most half a bf16 spacing (2^-8 relative to the
    # leading power of two)
    _, e = np.frexp(hf)
    assert np.all(np.abs(hb - hf) <= np.ldexp(1.0, e - 9) + 0.0)


def test_kv_row_orientation():
    d = 2
    W_kv = np.zeros((1, 2, d, d))
    W_kv[0, 0, 1, 0] = 2.0      # K: out[0] = 2 h[1]
    W_kv[0, 1, 0, 1] = -1.0     # V: out[1] = -h[0]
    dec = ElmanDecoder(np.zeros((d, d)), np.zeros((3, d)), np.zeros((3, d)), 0, True, W_kv)
    kv = dec.kv_row(np.array([0.5, 0.25]))
    assert np.array_equal(kv, np.array([[[0.5, 0.0], [0.0, -0.5]]]))
