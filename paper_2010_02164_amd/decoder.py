"""Python binding of the streambeam decoder.

PyTorch provides device memory (weights, workspace, h0 staging) and the HIP
stream; every step of the search runs in the HIP library through the C ABI
declared in include/streambeam.h.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

from . import _native as N


@dataclasses.dataclass
class Hypothesis:
    input: int
    rank: int
    tokens: tuple
    score: float
    status: int            # 2 = EOS, 3 = cut at max_len
    finalize_step: int


def _check(status: int, where: str, dec_handle=None):
    if status == N.SB_OK:
        return
    detail = ""
    L = N.lib()
    if dec_handle is not None or where == "sb_create_noalloc":
        # (a failed sb_create_noalloc leaves its text for a NULL decoder)
        msg = L.sb_last_error(dec_handle)
        detail = msg.decode() if msg else ""
    if not detail:
        detail = L.sb_status_string(status).decode()
    raise N.StreambeamError(status, where, detail)


def make_params(k, n, eps, delta, M, sched, max_len_cap, max_inputs, rule=None, pool=None) -> N.SbParams:
    """sched: a scheduler name (N.SCHEDULERS, or N.FAIRSEQ_SCHEDULERS, which
    also select the Fairseq finalization rule) or an sb_sched value. pool:
    beams cached by the capacity-constrained scheduler ("var_cap"; None
    means n)."""
    if isinstance(sched, str) and sched in N.FAIRSEQ_SCHEDULERS:
        code, rule = N.FAIRSEQ_SCHEDULERS[sched], N.SB_RULE_FAIRSEQ
    else:
        code = N.SCHEDULERS[sched] if isinstance(sched, str) else int(sched)
    return N.SbParams(k=int(k), n=int(n), eps=float(eps),
                      delta=float(math.inf if delta is None else delta), max_per_node=int(M),
                      sched=code, max_len_cap=int(max_len_cap), max_inputs=int(max_inputs),
                      finalize_rule=int(N.SB_RULE_PAPER if rule is None else rule),
                      pool=0 if pool is None else int(pool))


def make_model(vocab, d, dtype, beta, W_h=0, E=0, W_out=0, kv_layers=0, W_kv=0, attn=False) -> N.SbModel:
    return N.SbModel(vocab=int(vocab), d=int(d), dtype=N.SB_BF16 if dtype == "bf16" else N.SB_F32,
                     eos_beta=float(beta), W_h=W_h or None, E=E or None, W_out=W_out or None,
                     kv_layers=int(kv_layers), W_kv=W_kv or None, attn=int(bool(attn)))


def workspace_bytes(model: N.SbModel, params: N.SbParams) -> int:
    return int(N.lib().sb_workspace_bytes(ctypes.byref(model), ctypes.byref(params)))


class Decoder:
    """A streambeam decoder over torch-owned device memory.

    Weights are torch tensors on the GPU: float32, or bfloat16 for bf16
    models ([d,d], [V,d], [V,d], optional [L,2,d,d]). They must outlive the
    decoder (the decoder keeps references). With noalloc=True the decoder
    is made by sb_create_noalloc: its workspace is the library's static
    scratch (one such decoder per GPU at a time, workspace at most
    SB_NOALLOC_SCRATCH_BYTES) and no workspace tensor is allocated."""

    def __init__(self, W_h, E, W_out, *, beta: float, k: int, n: int, eps: float = 0.0,
                 delta: Optional[float] = None, M: Optional[int] = None, sched: str = "var_stream",
                 max_len_cap: int = 256, max_inputs: int = 1024, W_kv=None, stream=None,
                 pool: Optional[int] = None, attn: bool = False, noalloc: bool = False):
        import torch
        self.torch = torch
        if not torch.cuda.is_available():
            raise RuntimeError("streambeam needs a ROCm GPU (torch.cuda is not available)")
        self.dtype = "bf16" if W_out.dtype == torch.bfloat16 else "f32"
        want = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        for name, t in (("W_h", W_h), ("E", E), ("W_out", W_out)):
            if t.dtype != want or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous {want} CUDA tensor")
        V, d = W_out.shape
        self.V, self.d, self.k, self.n = V, d, k, n
        self._keep = [W_h, E, W_out, W_kv]
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.model = make_model(V, d, self.dtype, beta, W_h.data_ptr(), E.data_ptr(), W_out.data_ptr(),
                                0 if W_kv is None else W_kv.shape[0],
                                0 if W_kv is None else W_kv.data_ptr(), attn=attn)
        self.params = make_params(k, n, eps, delta, k if M is None else M, sched, max_len_cap, max_inputs,
                                  pool=pool)
        L = N.lib()
        _check(L.sb_validate(ctypes.byref(self.model), ctypes.byref(self.params)), "sb_validate")
        h = ctypes.c_void_p()
        if noalloc:
            self.workspace = None
            _check(L.sb_create_noalloc(ctypes.byref(self.model), ctypes.byref(self.params),
                                       ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)),
                   "sb_create_noalloc")
        else:
            nbytes = workspace_bytes(self.model, self.params)
            self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=W_out.device)
            _check(L.sb_create(ctypes.byref(self.model), ctypes.byref(self.params),
                               ctypes.c_void_p(self.workspace.data_ptr()), nbytes,
                               ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)), "sb_create")
        self.handle = h
        self.n_submitted = 0
        self._h0_keep = []

    # -- lifecycle ------------------------------------------------------------
    def close(self):
        if getattr(self, "handle", None):
            N.lib().sb_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reset(self):
        _check(N.lib().sb_reset(self.handle), "sb_reset", self.handle)
        self.n_submitted = 0
        self._h0_keep = []

    # -- Alg. 1 calls ---------------------------------------------------------
    def submit(self, h0, L_x: Sequence[int], max_len: Sequence[int], ids: Optional[Sequence[int]] = None):
        """Queue inputs: h0 is a device tensor [count, d] of the model dtype;
        ids (optional) are echoed as Hypothesis.input (default: queue
        positions)."""
        torch = self.torch
        want = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        if h0.dtype != want or not h0.is_cuda or h0.dim() != 2 or h0.shape[1] != self.d:
            raise ValueError("h0 must be a CUDA tensor [count, d] of the model dtype")
        h0 = h0.contiguous()
        lx = np.ascontiguousarray(L_x, dtype=np.int32)
        ml = np.ascontiguousarray(max_len, dtype=np.int32)
        cnt = h0.shape[0]
        if lx.shape != (cnt,) or ml.shape != (cnt,):
            raise ValueError("L_x and max_len must have one entry per h0 row")
        idp = None
        if ids is not None:
            idv = np.ascontiguousarray(ids, dtype=np.int64)
            if idv.shape != (cnt,):
                raise ValueError("ids must have one entry per h0 row")
            idp = idv.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
        _check(N.lib().sb_submit(self.handle, cnt, idp, ctypes.c_void_p(h0.data_ptr()),
                                 lx.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                 ml.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))),
               "sb_submit", self.handle)
        self._h0_keep.append(h0)
        self.n_submitted += cnt

    def step(self, sync: bool = True) -> Optional[bool]:
        done = ctypes.c_int32(0)
        _check(N.lib().sb_step(self.handle, ctypes.byref(done) if sync else None), "sb_step", self.handle)
        return bool(done.value) if sync else None

    def run(self):
        _check(N.lib().sb_run(self.handle), "sb_run", self.handle)

    def collect_arrays(self) -> dict:
        """Finalized hypotheses not yet collected, as numpy arrays (no
        per-hypothesis Python objects): `input`, `rank`, `length`, `status`,
        `finalize_step`, `score`, `tok_offset` (one entry per hypothesis, in
        input then rank order) and `tokens` (all token ids back to back;
        hypothesis j holds tokens[tok_offset[j] : tok_offset[j] + length[j]])."""
        L = N.lib()
        cap_h = max(16, self.n_submitted * self.k)
        cap_t = max(64, cap_h * int(self.params.max_len_cap))
        recs, toks = [], []
        base = 0
        while True:
            hyps = np.empty(cap_h, dtype=N.SB_HYP_DTYPE)
            tk = np.empty(cap_t, dtype=np.int32)
            nh, nt = ctypes.c_int64(0), ctypes.c_int64(0)
            st = L.sb_collect(self.handle, hyps.ctypes.data_as(ctypes.POINTER(N.SbHyp)), cap_h,
                              tk.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), cap_t, ctypes.byref(nh),
                              ctypes.byref(nt))
            if st not in (N.SB_OK, N.SB_E_TRUNCATED):
                _check(st, "sb_collect", self.handle)
            h = hyps[:nh.value].copy() if st == N.SB_E_TRUNCATED else hyps[:nh.value]
            h["tok_offset"] += base
            recs.append(h)
            toks.append(tk[:nt.value])
            base += nt.value
            if st == N.SB_OK or nh.value == 0:
                break
        h = recs[0] if len(recs) == 1 else np.concatenate(recs)
        out = {f: h[f] for f in h.dtype.names}
        out["tokens"] = toks[0] if len(toks) == 1 else np.concatenate(toks)
        return out

    def collect(self) -> List[Hypothesis]:
        """Finalized hypotheses not yet collected, as Hypothesis objects."""
        a = self.collect_arrays()
        tokens = a["tokens"].tolist()
        return [Hypothesis(int(i), int(r), tuple(tokens[o:o + n]), float(sc), int(st), int(f))
                for i, r, n, st, f, sc, o in zip(a["input"].tolist(), a["rank"].tolist(), a["length"].tolist(),
                                                 a["status"].tolist(), a["finalize_step"].tolist(),
                                                 a["score"].tolist(), a["tok_offset"].tolist())]

    def stats(self) -> dict:
        s = N.SbStats()
        _check(N.lib().sb_stats(self.handle, ctypes.byref(s)), "sb_stats", self.handle)
        return {f: int(getattr(s, f)) for f, _ in N.SbStats._fields_}

    def rows_histogram(self):
        """(counts[64], bucket width): timesteps by rows expanded."""
        counts = (ctypes.c_int64 * 64)()
        w = ctypes.c_int32(0)
        _check(N.lib().sb_rows_histogram(self.handle, counts, ctypes.byref(w)), "sb_rows_histogram",
               self.handle)
        return [int(c) for c in counts], int(w.value)

    # -- timing ---------------------------------------------------------------
    def set_timing(self, enable: bool):
        _check(N.lib().sb_set_timing(self.handle, int(enable)), "sb_set_timing", self.handle)

    def timing(self):
        ms, n = ctypes.c_double(0), ctypes.c_int64(0)
        _check(N.lib().sb_timing(self.handle, ctypes.byref(ms), ctypes.byref(n)), "sb_timing", self.handle)
        return ms.value, n.value

    # -- test support ---------------------------------------------------------
    def debug_expand(self, h_prev, y, t, L_x):
        """One decoder step on explicit rows: returns (h [R,d] tensor,
        lse [R], top_lp [R,k], top_tok [R,k])."""
        torch = self.torch
        R = h_prev.shape[0]
        h_prev = h_prev.contiguous()
        h_out = torch.empty_like(h_prev)
        y = np.ascontiguousarray(y, np.int32)
        t = np.ascontiguousarray(t, np.int32)
        lx = np.ascontiguousarray(L_x, np.int32)
        lse = np.empty(R, np.float64)
        lp = np.empty((R, self.k), np.float64)
        tok = np.empty((R, self.k), np.int32)
        P = ctypes.POINTER
        _check(N.lib().sb_debug_expand(
            self.handle, R, ctypes.c_void_p(h_prev.data_ptr()), y.ctypes.data_as(P(ctypes.c_int32)),
            t.ctypes.data_as(P(ctypes.c_int32)), lx.ctypes.data_as(P(ctypes.c_int32)),
            ctypes.c_void_p(h_out.data_ptr()), lse.ctypes.data_as(P(ctypes.c_double)),
            lp.ctypes.data_as(P(ctypes.c_double)), tok.ctypes.data_as(P(ctypes.c_int32))),
            "sb_debug_expand", self.handle)
        return h_out, lse, lp, tok

    def debug_slot(self, beam: int, rank: int, kv_layers: int = 0):
        st, sc, inp, steps, nt = (ctypes.c_int32(), ctypes.c_double(), ctypes.c_int64(), ctypes.c_int32(),
                                  ctypes.c_int32())
        cap = int(self.params.max_len_cap)
        toks = np.zeros(cap, np.int32)
        kv_cap = kv_layers * 2 * cap * self.d
        kv = np.zeros(max(kv_cap, 1), np.uint16)
        P = ctypes.POINTER
        _check(N.lib().sb_debug_slot(self.handle, beam, rank, ctypes.byref(st), ctypes.byref(sc),
                                     ctypes.byref(inp), ctypes.byref(steps),
                                     toks.ctypes.data_as(P(ctypes.c_int32)), cap, ctypes.byref(nt),
                                     kv.ctypes.data_as(P(ctypes.c_uint16)) if kv_layers else None,
                                     kv_cap), "sb_debug_slot", self.handle)
        s = steps.value
        kvr = kv[:kv_layers * 2 * s * self.d].reshape(kv_layers, 2, s, self.d) if kv_layers else None
        return dict(status=st.value, score=sc.value, input=inp.value, steps=s,
                    tokens=tuple(toks[:nt.value].tolist()), kv=kvr)


def weights_to_device(wl, device="cuda"):
    """Device tensors of a synthgen Workload's weights in its storage dtype."""
    import torch
    if wl.is_bf16:
        conv = lambda a: torch.from_numpy(a).to(device).to(torch.bfloat16)   # values are bf16-exact
    else:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    W_kv = None if wl.W_kv is None else conv(wl.W_kv).contiguous()
    return conv(wl.W_h).contiguous(), conv(wl.E).contiguous(), conv(wl.W_out).contiguous(), W_kv


def inputs_to_device(wl, idx=None, device="cuda"):
    import torch
    h0 = wl.h0 if idx is None else wl.h0[idx]
    t = torch.from_numpy(np.ascontiguousarray(h0)).to(device)
    return t.to(torch.bfloat16).contiguous() if wl.is_bf16 else t.contiguous()


def decoder_for_workload(wl, sched="var_stream", eps=None, n=None, max_inputs=None, weights=None,
                         **kw) -> Decoder:
    """A decoder for a synthgen workload with its config's parameters; the
    capacity-constrained scheduler caches 2n beams unless `pool` is given."""
    c = wl.cfg
    if sched == "var_cap" and kw.get("pool") is None:
        kw["pool"] = 2 * (c.n if n is None else n)
    kw.setdefault("attn", c.attn)
    W_h, E, W_out, W_kv = weights if weights is not None else weights_to_device(wl)
    return Decoder(W_h, E, W_out, W_kv=W_kv, beta=c.beta, k=c.k, n=c.n if n is None else n,
                   eps=c.eps if eps is None else eps, delta=c.delta, M=c.M, sched=sched,
                   max_len_cap=c.max_len_cap, max_inputs=max_inputs or len(wl.Lx), **kw)


def group_by_input(hyps: List[Hypothesis], n_inputs: int):
    out = [[] for _ in range(n_inputs)]
    for h in hyps:
        out[h.input].append(h)
    for y in out:
        y.sort(key=lambda h: h.rank)
    return out
