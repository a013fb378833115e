"""Benchmark of the E2-TTT chunk update (forward + backward) on one MI355X.

One step = e2ttt_chunk_forward (saving for backward) + e2ttt_chunk_backward
over the 1.3B-model layer shape: B=8, H=16 (d_model 1024 = 16 x 64), T=4096,
MLP fast weight d=64 -> 256 -> 64, chunk 64, bf16 io with fp32 state.  Inputs
are synthetic (seeded recipe of paper_2608_21308_amd.workloads) and resident
in HBM before timing starts.  Prints one JSON line.

Throughput counts tokens (B*T) per second of whole fwd+bwd steps.  The
roofline object reports the dominant kernel: algorithmic FLOP per launch
(GEMM units x 2 C d dh, unpadded, no recompute) over its average launch time
measured with HIP events on the launch stream.  cpu_baseline times the fp64
oracle on a bounded sample of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "chain_bwd_mlp_1p3b_traffic.json")
METRIC = "E²-TTT layer fwd+bwd tokens/s (H=16,d=64,T=4096) + MFMA util %"


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_21308_amd", "csrc")
    for n in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, n), "rb") as fh:
            h.update(n.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def gemm_flop(w, units_per_chunk: int) -> float:
    """units x 2 C d dh per chunk, over all chunks and (batch, head) units."""
    return float(units_per_chunk) * 2.0 * w.d * w.dh * w.T * w.B * w.H


def cpu_baseline(w, seconds_hint: float = 20.0) -> dict:
    """The fp64 oracle (forward + backward) on a bounded sample of units."""
    import numpy as np
    from oracle import oracle
    from paper_2608_21308_amd import workloads as WL
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 1)
    threads = max(1, min(threads, os.cpu_count() or 1))
    n_units = min(threads, w.B * w.H)
    x = WL.make_inputs(w, units=list(range(n_units)))
    t0 = time.perf_counter()
    oracle.forward(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], None, C=w.C,
                   fw=w.fw, dh=w.dh, nthreads=threads)
    oracle.backward(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], None,
                    x["d_out"], C=w.C, fw=w.fw, dh=w.dh, nthreads=threads)
    dt = time.perf_counter() - t0
    # the full workload has B*H units; with units spread over the same threads
    full = dt * (w.B * w.H) / n_units
    return {"value": (w.B * w.T) / full, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "%d of %d (batch, head) units, full T=%d, fwd+bwd, fp64, %.1f s wall; "
                      "scaled by %d/%d" % (n_units, w.B * w.H, w.T, dt, w.B * w.H, n_units)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this size (for counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the chunk update shards over (batch, head) units "
              "with no exchange, so more GPUs are not exercised here", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_21308_amd import e2ttt, workloads as WL

    w = WL.WORKLOADS[3]
    x = WL.make_inputs(w)
    dev = torch.device("cuda:0")
    t = {}
    for n, a in x.items():
        if a is None:
            t[n] = None
            continue
        ten = torch.from_numpy(a).to(dev)
        t[n] = ten.to(torch.bfloat16) if n in ("q", "k", "v", "d_out") else ten
    cfg = e2ttt.Config(w.B, w.H, w.T, w.d, w.dh, w.C, w.fw, e2ttt.DT_BF16)
    ws = e2ttt.alloc_workspace(cfg, True, dev)
    scratch = torch.empty(e2ttt.backward_scratch_bytes(cfg), dtype=torch.uint8, device=dev)
    out = torch.empty_like(t["q"])
    w_out = torch.empty_like(t["w_in"])
    m_out = torch.empty_like(t["w_in"])
    grads = dict(dq=torch.empty_like(t["q"]), dk=torch.empty_like(t["k"]),
                 dv=torch.empty_like(t["v"]), d_eta=torch.empty_like(t["eta"]),
                 d_beta=torch.empty_like(t["beta"]), d_gamma=torch.empty_like(t["gamma"]),
                 d_w_in=torch.empty_like(t["w_in"]), d_m_in=torch.empty_like(t["w_in"]))

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                      None, out=out, w_out=w_out, m_out=m_out, workspace=ws,
                      save_for_backward=True)
        if ev is not None:
            ev[1].record()
        e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                       None, ws, t["d_out"], grads=grads, scratch=scratch)
        if ev is not None:
            ev[2].record()

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print("calibration copy: %d bytes read, %d written" % (n * 4, n * 4), file=sys.stderr)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print("warmup step %d done" % i, file=sys.stderr, flush=True)

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd_ms = [e[0].elapsed_time(e[1]) for e in events]
    bwd_ms = [e[1].elapsed_time(e[2]) for e in events]
    ms_step = wall * 1e3 / args.steps
    tokens = w.B * w.T
    value = tokens / (ms_step / 1e3)

    flop_fwd = gemm_flop(w, 9)      # F1, F2, F5, two F7, two F8, outputs (2)
    flop_bwd = gemm_flop(w, 18)     # output branch 4 + state branch 14
    avg_fwd = sum(fwd_ms) / len(fwd_ms)
    avg_bwd = sum(bwd_ms) / len(bwd_ms)
    dom = "chain_bwd" if avg_bwd >= avg_fwd else "chain_fwd"
    dom_ms = max(avg_bwd, avg_fwd)
    dom_flop = flop_bwd if dom == "chain_bwd" else flop_fwd
    achieved = dom_flop / (dom_ms / 1e3) / 1e12
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as fh:
            tr = json.load(fh)
        if tr.get("source_hash") == source_hash() and tr.get("kernel") == dom:
            traffic = tr.get("bytes_per_launch")
    res = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "T": w.T, "d": w.d, "dh": w.dh,
                   "chunk": w.C, "fast_weight": "gelu_mlp", "pass": "fwd+bwd",
                   "global_batch": w.B, "seq_len": w.T, "parallelism": "none"},
        "mfma_util_pct": 100.0 * (flop_fwd + flop_bwd) / (ms_step / 1e3) / 1e12 /
                         PEAK_BF16_TFLOPS,
        "token_heads_per_s": tokens * w.H / (ms_step / 1e3),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
                     "flop_per_launch": dom_flop, "avg_launch_ms": dom_ms},
        "detail": {"fwd_ms": avg_fwd, "bwd_ms": avg_bwd, "source_hash": source_hash()},
    }
    if args.no_cpu_baseline:
        res["cpu_baseline"] = None
    else:
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
