"""Benchmark of the streaming beam-search decoder on one MI355X.

A bench "step" is one whole decode of the workload: queue every input
(device-resident encodings), run the search until every beam is finished
(refill, selection, expansion, top-k, pruning, finalization, state reorder,
the rebuild of the output tokens in device memory), then collect every
finalized hypothesis to the host (records and packed tokens, as numpy
arrays). The timed region runs with projection timing on (kernels launched
one by one, HIP events around each projection launch); the same decodes
replayed as captured step graphs are reported as graph_replay_hyps_per_s.

Default workload: the MT-shaped fp32 configuration (N=4096 inputs, n=128,
k=5, |V|=32000, d=1024, Var-Stream eps=1/4, delta=1.5), synthetic.

Prints one JSON line: finalized hypotheses/s (value), candidate
expansions/s, the projection kernel's achieved MFMA rate against the
MI355X peak (timed with HIP events on the decoder's stream), and the fp64
oracle timed on this host's cores on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}   # dense MFMA, MI355X
HBM_PEAK_BPS = 8.0e12                            # MI355X HBM3E


def attainable_proj_seconds(hist, width, d, V, dtype, peak_tflops):
    """Roofline bound of the projection over one decode: per step the larger
    of its MFMA time (2 d |V| flops per row at peak) and the time to stream
    W_out once from HBM; steps taken from the rows histogram at bucket
    midpoints."""
    es = 2 if dtype == "bf16" else 4
    w_bytes = ((V + 127) // 128) * 128 * d * es
    t = 0.0
    for i, c in enumerate(hist):
        if c:
            rows = max(1.0, i * width + (width - 1) / 2.0)
            t += c * max(2.0 * d * V * rows / (peak_tflops * 1e12), w_bytes / HBM_PEAK_BPS)
    return t
# Sources of the projection kernel; measured HBM traffic is reported only
# while they are unchanged since the counters were taken.
PROJ_SOURCES = ["paper_2010_02164_amd/csrc/proj.hip", "paper_2010_02164_amd/csrc/topk.h",
                "paper_2010_02164_amd/csrc/mfma_common.h", "paper_2010_02164_amd/csrc/wave.h",
                "paper_2010_02164_amd/csrc/sb_internal.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_proj_traffic.md")
METRIC = "finalized hyps/sec + expansions/sec (Var-Stream, k=5, |V|=32k), % roofline"


def _workload_desc(cfg, sched, eps, pool=None):
    return (f"{cfg.name}: N={cfg.N} inputs, n={cfg.n}, k={cfg.k}, |V|={cfg.V}, d={cfg.d}, "
            f"{cfg.dtype}, {sched} eps={eps:g}" + (f" pool={pool}" if pool else "")
            + f", delta={cfg.delta:g}, M={cfg.M}, "
            f"L_x {cfg.lengths}[{cfg.len_lo},{cfg.len_hi}]"
            + (f", KV {cfg.kv_layers}x2xtxd" if cfg.kv_layers else ""))


def cpu_baseline(wl, sched, eps, sample, pool=None):
    """The fp64 oracle (as it stands) on the first `sample` inputs."""
    from oracle.search import decode_workload
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 0) for i in threadpool_info()] or [0])
    except Exception:
        threads = 0
    cores = threads or len(os.sched_getaffinity(0))
    try:
        b = np.show_config(mode="dicts").get("Build Dependencies", {}).get("blas", {})
        blas = f"{b.get('name', '?')} {b.get('version', '')}".strip()
    except Exception:
        blas = "unknown"
    idx = np.arange(min(sample, len(wl.Lx)))
    t0 = time.perf_counter()
    r = decode_workload(wl, sched=sched, eps=eps, inputs=idx, pool=pool)
    dt = time.perf_counter() - t0
    return {"value": r.n_hyps / dt, "unit": "hyps/s", "cores": cores, "kind": "oracle",
            "sample": f"first {len(idx)} of {len(wl.Lx)} inputs, same n/k/eps/delta/M/pool, numpy fp64 "
                      f"({dt:.1f} s, {r.expansions} expansions)",
            "expansions_per_s": r.expansions / dt, "seconds": dt, "blas": blas, "blas_threads": threads or None,
            "host_cpus": len(os.sched_getaffinity(0))}


def proj_source_sha256():
    """Hash of the projection kernel's sources with // comments, trailing
    blanks and empty lines removed (a comment edit keeps the measured
    figures valid; any code edit invalidates them)."""
    h = hashlib.sha256()
    for rel in PROJ_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def measured_traffic(workload_key):
    """HBM bytes per projection launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, calibrated against a plain copy), or None when
    that summary is for another workload or an older kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    for block in re.findall(r"```json\n(.*?)\n```", text, re.S):
        rec = json.loads(block)
        if rec.get("workload_key") == workload_key and rec.get("source_sha256") == proj_source_sha256():
            return rec["hbm_bytes_per_launch"]
    return None


def copy_calibration(nbytes, reps=5):
    """A plain device copy of a known size, for scaling the HBM byte counters."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def unfused_reference(cfg_i, rows_list, reps=20):
    """Times the unfused alternative to the fused projection on the same
    shapes: a library GEMM writing the [R, |V|] logits to HBM, then a
    log-softmax and a top-k over them (torch / hipBLASLt). Comparison only;
    the decoder never takes this path."""
    import torch
    from synthgen import get_config, make_workload
    cfg = get_config(cfg_i)
    wl = make_workload(cfg, N=8)
    dt = torch.bfloat16 if wl.is_bf16 else torch.float32
    W = torch.from_numpy(wl.W_out).to("cuda", dtype=dt)
    out = []
    for R in rows_list:
        h = torch.tanh(torch.randn(R, cfg.d, device="cuda")).to(dt)
        def once():
            z = (h @ W.T).float()
            lp = torch.log_softmax(z, dim=1)
            return torch.topk(lp, cfg.k, dim=1)
        for _ in range(3):
            once()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            once()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        out.append({"rows": R, "us": us, "logits_bytes": R * cfg.V * 4,
                    "tflops": 2.0 * cfg.d * cfg.V * R / (us * 1e-6) / 1e12})
    print(json.dumps({"unfused_reference": f"cfg{cfg_i}", "dtype": cfg.dtype, "V": cfg.V, "d": cfg.d,
                      "k": cfg.k, "results": out}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--sched", default="var_stream",
                    choices=["fixed", "fixed_stream", "fixed_fairseq", "fixed_fairseq_stream", "var_batch",
                             "var_stream", "var_fifo", "var_cap"])
    ap.add_argument("--eps", type=float, default=None)
    ap.add_argument("--pool", type=int, default=None,
                    help="beams cached by var_cap (default 2n); rows per step stay <= n*k")
    ap.add_argument("--cpu-sample", type=int, default=512)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sorted", action="store_true",
                    help="submit the inputs by increasing source length L_x (the paper's batching order; "
                         "a secondary setting: L_x nearly fixes the output length here)")
    ap.add_argument("--no-graph-replay", action="store_true",
                    help="skip the extra untimed graph-replay decodes (counter runs)")
    ap.add_argument("--unfused", default=None, metavar="ROWS",
                    help="only time the unfused torch alternative (GEMM + log-softmax + top-k) at these "
                         "comma-separated row counts")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the decoder runs on one GPU; --gpus {args.gpus} is not supported "
              "(inputs are independent: shard them over GPUs, one decoder per GPU)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.unfused:
        unfused_reference(args.config, [int(x) for x in args.unfused.split(",")])
        return

    import torch
    from paper_2010_02164_amd import decoder_for_workload, inputs_to_device, weights_to_device
    from synthgen import get_config, make_workload

    cfg = get_config(args.config)
    eps = cfg.eps if args.eps is None else args.eps
    if args.sched not in ("var_stream", "var_fifo", "fixed_stream", "fixed_fairseq_stream", "var_cap"):
        eps = 0.0
    if args.pool is not None and args.sched != "var_cap":
        ap.error("--pool applies to --sched var_cap only")
    pool = (2 * cfg.n if args.pool is None else args.pool) if args.sched == "var_cap" else None
    wl = make_workload(cfg)
    weights = weights_to_device(wl)
    h0 = inputs_to_device(wl)
    dec = decoder_for_workload(wl, sched=args.sched, eps=eps, weights=weights, pool=pool)
    N = len(wl.Lx)
    order = np.argsort(wl.Lx, kind="stable") if args.sorted else np.arange(N)
    if args.sorted:   # inputs reordered once, before any timing; results keep the original ids
        h0 = h0[torch.from_numpy(order).to(h0.device)].contiguous()
    sub_Lx, sub_ml, sub_ids = wl.Lx[order], wl.max_len[order], order.astype(np.int64)

    collect_s = []

    def run_once():
        dec.reset()
        dec.submit(h0, sub_Lx, sub_ml, ids=sub_ids)
        dec.run()              # returns once the decode is complete on the device
        tc = time.perf_counter()
        out = dec.collect_arrays()
        collect_s.append(time.perf_counter() - tc)
        return out

    for _ in range(args.warmup):
        run_once()
    torch.cuda.synchronize()
    dec.set_timing(True)
    torch.cuda.synchronize()
    collect_s.clear()
    t0 = time.perf_counter()
    run_ends = []
    for _ in range(args.steps):
        got = run_once()
        run_ends.append(time.perf_counter())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    run_ms = np.diff(np.array([t0] + run_ends)) * 1e3
    proj_ms, proj_launches = dec.timing()
    dec.set_timing(False)
    st = dec.stats()            # counters of the last run
    hist, hist_w = dec.rows_histogram()
    assert len(got["input"]) == st["hyps"] and len(np.unique(got["input"])) == N
    collect_mean_s = float(np.mean(collect_s))

    # The same workload replayed as captured step graphs, untimed kernels.
    graph_per_run = None
    if not args.no_graph_replay:
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        for _ in range(args.steps):
            run_once()
        torch.cuda.synchronize()
        graph_per_run = (time.perf_counter() - t2) / args.steps

    per_run = elapsed / args.steps
    hyps_per_s = st["hyps"] / per_run
    exps_per_s = st["expansions"] / per_run
    # Projection: 2 d |V| flops per expansion (algorithmic), every timed run.
    proj_flops = 2.0 * cfg.d * cfg.V * st["expansions"] * args.steps
    achieved = proj_flops / (proj_ms * 1e-3) / 1e12 if proj_ms > 0 else 0.0
    peak = PEAK_TFLOPS[cfg.dtype]
    t_att = attainable_proj_seconds(hist, hist_w, cfg.d, cfg.V, cfg.dtype, peak)
    proj_s_per_decode = proj_ms * 1e-3 / args.steps
    workload_key = f"cfg{args.config} {args.sched} eps={eps:g}" + (f" pool={pool}" if pool else "") + (" sorted" if args.sorted else "")
    out = {
        "metric": METRIC, "value": hyps_per_s, "unit": "hyps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": per_run * 1e3,
        "ms_per_step_std": float(run_ms.std(ddof=1)) if len(run_ms) > 1 else 0.0,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": _workload_desc(cfg, args.sched, eps, pool) + (", inputs sorted by L_x" if args.sorted else ""), "key": workload_key, "inputs": N,
                   "parallelism": "single GPU"},
        "expansions_per_s": exps_per_s,
        "search": {k: st[k] for k in ("timesteps", "expansions", "noops", "refills", "hyps", "positions")},
        "roofline": {"bound": "mfma", "kernel": "k_proj (vocabulary projection + log-sum-exp + top-k)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": measured_traffic(workload_key), "launches": proj_launches,
                     "avg_launch_us": proj_ms * 1e3 / max(proj_launches, 1),
                     "attainable_ms_per_decode": t_att * 1e3,
                     "frac_of_attainable": t_att / proj_s_per_decode if proj_s_per_decode > 0 else None},
        "rows_per_step_hist": {"bucket_width": hist_w,
                               "counts": {str(i * hist_w): c for i, c in enumerate(hist) if c}},
        "projection_share_of_step": (proj_ms * 1e-3) / elapsed if elapsed > 0 else None,
        "graph_replay_hyps_per_s": st["hyps"] / graph_per_run if graph_per_run else None,
        "collect_ms": collect_mean_s * 1e3,
        "decode_only_hyps_per_s": st["hyps"] / (per_run - collect_mean_s),
    }
    dec.close()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.sched, eps, args.cpu_sample, pool)
        out["gpu_over_cpu"] = hyps_per_s / out["cpu_baseline"]["value"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
