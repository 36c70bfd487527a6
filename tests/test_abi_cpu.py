"""The C-ABI library loads, exports every declared symbol and validates its
arguments on the host (no GPU calls)."""
import ctypes
import math

import pytest

from paper_2010_02164_amd import _native as N
from paper_2010_02164_amd.decoder import make_model, make_params, workspace_bytes
from synthgen import CONFIGS


def test_exports_every_declared_symbol(native_lib):
    names = N.header_symbols()
    assert "sb_create" in names and "sb_collect" in names
    for name in names:
        assert hasattr(native_lib, name), name


def _mp(cfg, **over):
    m = make_model(cfg.V, cfg.d, cfg.dtype, cfg.beta, 1, 1, 1, cfg.kv_layers, 1 if cfg.kv_layers else 0,
                   attn=cfg.attn)
    p = make_params(cfg.k, cfg.n, cfg.eps, cfg.delta, cfg.M, "var_stream", cfg.max_len_cap, cfg.N)
    for k, v in over.items():
        setattr(m if hasattr(m, k) else p, k, v)
    return m, p


@pytest.mark.parametrize("i", sorted(CONFIGS))
def test_workspace_sizes(native_lib, i):
    cfg = CONFIGS[i]
    m, p = _mp(cfg)
    assert native_lib.sb_validate(ctypes.byref(m), ctypes.byref(p)) == N.SB_OK
    b = workspace_bytes(m, p)
    assert b > 0 and b % 256 == 0
    # grows with the queue capacity by at least the per-input storage
    p2 = make_params(cfg.k, cfg.n, cfg.eps, cfg.delta, cfg.M, "var_stream", cfg.max_len_cap, 2 * cfg.N)
    assert workspace_bytes(m, p2) >= b + cfg.N * (cfg.d * (2 if cfg.dtype == "bf16" else 4))


@pytest.mark.parametrize("over,code", [
    (dict(k=0), N.SB_E_UNSUPPORTED), (dict(k=17), N.SB_E_UNSUPPORTED),
    (dict(d=48), N.SB_E_UNSUPPORTED), (dict(eps=1.0), N.SB_E_INVALID_ARG),
    (dict(eps=-0.1), N.SB_E_INVALID_ARG), (dict(max_per_node=6), N.SB_E_INVALID_ARG),
    (dict(max_per_node=0), N.SB_E_INVALID_ARG), (dict(delta=0.0), N.SB_E_INVALID_ARG),
    (dict(sched=7), N.SB_E_INVALID_ARG), (dict(max_len_cap=0), N.SB_E_INVALID_ARG),
    (dict(max_inputs=0), N.SB_E_INVALID_ARG), (dict(vocab=3), N.SB_E_INVALID_ARG),
    (dict(n=0), N.SB_E_UNSUPPORTED), (dict(kv_layers=2), N.SB_E_UNSUPPORTED),
    (dict(finalize_rule=2), N.SB_E_INVALID_ARG), (dict(k=16, finalize_rule=1), N.SB_E_UNSUPPORTED),
    (dict(pool=256), N.SB_E_INVALID_ARG), (dict(sched=5, pool=64), N.SB_E_INVALID_ARG),
    (dict(sched=5, pool=4097), N.SB_E_INVALID_ARG), (dict(sched=6), N.SB_E_INVALID_ARG),
])
def test_validate_rejects(native_lib, over, code):
    m, p = _mp(CONFIGS[3], **over)
    assert native_lib.sb_validate(ctypes.byref(m), ctypes.byref(p)) == code
    assert workspace_bytes(m, p) == 0


def test_fairseq_rule_workspace(native_lib):
    # The Fairseq rule keeps 2k backpointers per level (beam + outputs).
    m, p = _mp(CONFIGS[3])
    m2, p2 = _mp(CONFIGS[3], finalize_rule=1)
    c = CONFIGS[3]
    assert native_lib.sb_validate(ctypes.byref(m2), ctypes.byref(p2)) == N.SB_OK
    assert workspace_bytes(m2, p2) >= workspace_bytes(m, p) + c.N * c.max_len_cap * c.k * 4


def test_capacity_pool_workspace(native_lib):
    # Beam and candidate storage scale with the pool of cached beams; the row
    # buffers stay at n*k rows.
    c = CONFIGS[3]
    m, p = _mp(c)
    m2, p2 = _mp(c, sched=N.SB_VAR_CAP, pool=2 * c.n)
    m3, p3 = _mp(c, sched=N.SB_VAR_CAP, pool=0)
    assert native_lib.sb_validate(ctypes.byref(m2), ctypes.byref(p2)) == N.SB_OK
    assert native_lib.sb_validate(ctypes.byref(m3), ctypes.byref(p3)) == N.SB_OK
    assert workspace_bytes(m3, p3) == workspace_bytes(m, p)
    extra = workspace_bytes(m2, p2) - workspace_bytes(m, p)
    slot_state = c.n * c.k * c.d * 4
    assert slot_state <= extra < 2 * slot_state


@pytest.mark.parametrize("over,code", [
    (dict(attn=2), N.SB_E_INVALID_ARG), (dict(d=1536), N.SB_E_UNSUPPORTED),
])
def test_validate_rejects_attention(native_lib, over, code):
    m, p = _mp(CONFIGS[6], **over)
    assert native_lib.sb_validate(ctypes.byref(m), ctypes.byref(p)) == code


def test_attention_needs_kv_state(native_lib):
    m, p = _mp(CONFIGS[4], attn=1)
    assert native_lib.sb_validate(ctypes.byref(m), ctypes.byref(p)) == N.SB_E_INVALID_ARG


def test_attention_workspace(native_lib):
    # The attention read-out adds per expanded candidate one bf16 row and
    # an fp64 row per layer.
    c = CONFIGS[6]
    m5, p5 = _mp(CONFIGS[5])
    m6, p6 = _mp(c)
    assert workspace_bytes(m6, p6) - workspace_bytes(m5, p5) >= c.R_max * c.d * (2 + 8 * c.kv_layers)


def test_delta_inf_is_valid(native_lib):
    m, p = _mp(CONFIGS[1], delta=math.inf)
    assert native_lib.sb_validate(ctypes.byref(m), ctypes.byref(p)) == N.SB_OK


def test_create_rejects_bad_workspace_without_gpu(native_lib):
    m, p = _mp(CONFIGS[1])
    h = ctypes.c_void_p()
    need = workspace_bytes(m, p)
    assert native_lib.sb_create(ctypes.byref(m), ctypes.byref(p), None, need, None, ctypes.byref(h)) == N.SB_E_WORKSPACE
    assert native_lib.sb_create(ctypes.byref(m), ctypes.byref(p), ctypes.c_void_p(0x1000 + 8), need, None,
                                ctypes.byref(h)) == N.SB_E_WORKSPACE
    assert native_lib.sb_create(ctypes.byref(m), ctypes.byref(p), ctypes.c_void_p(0x1000), need - 256, None,
                                ctypes.byref(h)) == N.SB_E_WORKSPACE
    assert h.value is None


def test_status_strings(native_lib):
    for s in range(8):
        assert native_lib.sb_status_string(s)
    assert native_lib.sb_destroy(None) == N.SB_E_INVALID_ARG
