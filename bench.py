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
PEAK_F32_TFLOPS = 157.3          # MI355X dense fp32 MFMA
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
    # three units per thread: about 10 s of wall time on 16 cores
    n_units = min(3 * threads, w.B * w.H)
    x = WL.make_inputs(w, units=list(range(n_units)))
    t0 = time.perf_counter()
    oracle.forward(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], None, C=w.C,
                   fw=w.fw, dh=w.dh, nthreads=threads)
    oracle.backward(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], None,
                    x["d_out"], C=w.C, fw=w.fw, dh=w.dh, nthreads=threads)
    dt = time.perf_counter() - t0
    # the full workload has B*H units; with units spread over the same threads
    full = dt * (w.B * w.H) / n_units
    # one unit on one thread: the oracle's single-core rate, scaled the same way
    x1 = WL.make_inputs(w, units=[0])
    t1 = time.perf_counter()
    oracle.forward(x1["q"], x1["k"], x1["v"], x1["eta"], x1["beta"], x1["gamma"], x1["w_in"], None,
                   C=w.C, fw=w.fw, dh=w.dh, nthreads=1)
    oracle.backward(x1["q"], x1["k"], x1["v"], x1["eta"], x1["beta"], x1["gamma"], x1["w_in"], None,
                    x1["d_out"], C=w.C, fw=w.fw, dh=w.dh, nthreads=1)
    dt1 = time.perf_counter() - t1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": (w.B * w.T) / full, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "%d of %d (batch, head) units, full T=%d, fwd+bwd, fp64, %.1f s wall; "
                      "scaled by %d/%d" % (n_units, w.B * w.H, w.T, dt, w.B * w.H, n_units),
            "single_thread_value": (w.B * w.T) / (dt1 * w.B * w.H),
            "single_thread_sample": "1 unit on 1 thread, %.1f s, scaled by %d" % (dt1, w.B * w.H),
            "cpu_model": model}


def time_long_chunk(e2ttt, w, t, dev, reps: int = 10) -> dict:
    """Forward (no saving) of the same layer at chunk 64 and at the paper's
    chunk 512 (64-token tiles at the chunk-start weights), and the fwd+bwd
    step at chunk 512: HIP events around back-to-back calls."""
    import torch
    res = {}
    for C in (w.C, 512):
        cfg = e2ttt.Config(w.B, w.H, w.T, w.d, w.dh, C, w.fw, e2ttt.DT_BF16)
        ws = e2ttt.alloc_workspace(cfg, False, dev)
        out = torch.empty_like(t["q"])
        wo, mo = torch.empty_like(t["w_in"]), torch.empty_like(t["w_in"])

        def call():
            e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                          t["w_in"], None, out=out, w_out=wo, m_out=mo, workspace=ws)

        for _ in range(3):
            call()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(reps):
            call()
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / reps
        res["C%d_fwd_ms" % C] = ms
        res["C%d_tokens_per_s" % C] = w.B * w.T / (ms * 1e-3)
    # the training step (forward saving for the backward, then the backward) at
    # chunk 512, as the headline step is timed at the workload's chunk
    cfg = e2ttt.Config(w.B, w.H, w.T, w.d, w.dh, 512, w.fw, e2ttt.DT_BF16)
    ws = e2ttt.alloc_workspace(cfg, True, dev)
    scratch = torch.empty(e2ttt.backward_scratch_bytes(cfg), dtype=torch.uint8, device=dev)
    out = torch.empty_like(t["q"])
    wo, mo = torch.empty_like(t["w_in"]), torch.empty_like(t["w_in"])
    grads = dict(dq=torch.empty_like(t["q"]), dk=torch.empty_like(t["k"]), dv=torch.empty_like(t["v"]),
                 d_eta=torch.empty_like(t["eta"]), d_beta=torch.empty_like(t["beta"]),
                 d_gamma=torch.empty_like(t["gamma"]), d_w_in=torch.empty_like(t["w_in"]),
                 d_m_in=torch.empty_like(t["w_in"]))

    def step():
        e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"], None,
                      out=out, w_out=wo, m_out=mo, workspace=ws, save_for_backward=True)
        e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"], None,
                       ws, t["d_out"], grads=grads, scratch=scratch)

    for _ in range(3):
        step()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        step()
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    res["C512_step_ms"] = ms
    res["C512_step_tokens_per_s"] = w.B * w.T / (ms * 1e-3)
    return res


def time_gates(e2ttt, w, dev, reps: int = 50) -> dict:
    """Gate parameterization kernels (eqs. (12)-(14)) over the same B*H*T
    tokens, outside the timed step: average time of back-to-back calls through
    the C ABI from HIP events, and the HBM rate of their algorithmic bytes (forward reads 3 logits and writes
    3 gates per token, backward reads 6 values and writes 3; fp32)."""
    import ctypes
    import torch
    lib = e2ttt.load()
    n = w.B * w.H * w.T
    g = torch.Generator(device=dev).manual_seed(11)
    le, lb, la, de, db, dg = (torch.randn(n, device=dev, generator=g) for _ in range(6))
    p = ctypes.byref(e2ttt.GateParams())
    o = [torch.empty(n, device=dev) for _ in range(6)]
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    res = {}
    for name, nbytes, call in (
            ("fwd", 24 * n, lambda: lib.e2ttt_gates_forward(p, n, P(le), P(lb), P(la), P(o[0]),
                                                            P(o[1]), P(o[2]), st)),
            ("bwd", 36 * n, lambda: lib.e2ttt_gates_backward(p, n, P(le), P(lb), P(la), P(de),
                                                             P(db), P(dg), P(o[3]), P(o[4]),
                                                             P(o[5]), st))):
        if call() != 0:
            raise RuntimeError("gate %s call failed" % name)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(reps):
            call()
        ev[1].record()
        torch.cuda.synchronize()
        us = ev[0].elapsed_time(ev[1]) * 1e3 / reps
        res[name + "_us"] = us
        res[name + "_GBs"] = nbytes / (us * 1e-6) / 1e9
        res[name + "_hbm_frac"] = res[name + "_GBs"] / PEAK_HBM_GBS
    res["tokens"] = n
    return res


def time_decode(e2ttt, w, x, dev, reps: int = 200) -> dict:
    """Streaming decode over the same units (eq. (6), Table 1): per step every
    unit answers one token with e2ttt_apply at its chunk-start state, and every
    C steps e2ttt_chunk_forward over the C buffered tokens advances the state.
    Both are timed back to back on the stream through the C ABI (HIP events);
    a step's cost is apply + update / C, and a step yields one token for each
    of the B sequences.  The apply kernel is bound by reading the fp32 state
    (P floats per unit) once."""
    import ctypes
    import torch
    lib = e2ttt.load()
    U = w.B * w.H
    cfg1 = e2ttt.Config(w.B, w.H, 1, w.d, w.dh, w.C, w.fw, e2ttt.DT_BF16)
    cfgc = e2ttt.Config(w.B, w.H, w.C, w.d, w.dh, w.C, w.fw, e2ttt.DT_BF16)
    state = torch.from_numpy(x["w_in"]).to(dev)
    q1 = torch.from_numpy(x["q"][:, :, :1].copy()).to(dev).to(torch.bfloat16)
    o1 = torch.empty_like(q1)
    chunk = {n: torch.from_numpy(x[n][:, :, :w.C].copy()).to(dev)
             for n in ("q", "k", "v", "eta", "beta", "gamma")}
    for n in ("q", "k", "v"):
        chunk[n] = chunk[n].to(torch.bfloat16)
    w_next, m_next = torch.empty_like(state), torch.empty_like(state)
    ws = e2ttt.alloc_workspace(cfgc, False, dev)
    oc = torch.empty_like(chunk["q"])
    d1, dc = cfg1.desc(), cfgc.desc()
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())

    def apply():
        return lib.e2ttt_apply(ctypes.byref(d1), P(q1), P(state), P(o1), st)

    def update():
        return lib.e2ttt_chunk_forward(ctypes.byref(dc), P(chunk["q"]), P(chunk["k"]),
                                       P(chunk["v"]), P(chunk["eta"]), P(chunk["beta"]),
                                       P(chunk["gamma"]), P(state), None, P(oc), P(w_next),
                                       P(m_next), P(ws), ws.numel(), 0, st)

    res = {}
    for name, call, n in (("apply", apply, reps), ("update", update, max(1, reps // 10))):
        if call() != 0:
            raise RuntimeError("decode %s call failed" % name)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(n):
            call()
        ev[1].record()
        torch.cuda.synchronize()
        res[name + "_us"] = ev[0].elapsed_time(ev[1]) * 1e3 / n
    state_bytes = U * e2ttt.Config(w.B, w.H, 1, w.d, w.dh, w.C, w.fw).P * 4
    step_us = res["apply_us"] + res["update_us"] / w.C
    res.update(step_us=step_us, tokens_per_s=w.B / (step_us * 1e-6),
               apply_state_GBs=state_bytes / (res["apply_us"] * 1e-6) / 1e9,
               apply_hbm_frac=state_bytes / (res["apply_us"] * 1e-6) / 1e9 / PEAK_HBM_GBS,
               batch=w.B, units=U, chunk=w.C)
    return res


def measure_peaks(dev) -> dict:
    """What this MI355X reaches on the two roofline resources: a dense bf16 GEMM
    (torch.matmul, 8192^3, hipBLASLt) and a device-to-device copy of 1 GiB
    (read + write bytes), each timed with HIP events over back-to-back calls.
    Reported beside the published peaks the roofline fractions use."""
    import torch
    res = {}
    n = 8192
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    c = torch.empty(n, n, device=dev, dtype=torch.bfloat16)
    for _ in range(3):
        torch.matmul(a, b, out=c)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    reps = 20
    ev[0].record()
    for _ in range(reps):
        torch.matmul(a, b, out=c)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    res["bf16_gemm_TFLOPs"] = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    res["bf16_gemm_frac_of_published"] = res["bf16_gemm_TFLOPs"] / PEAK_BF16_TFLOPS
    del a, b, c
    nb = 1 << 30
    src = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        dst.copy_(src)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    res["copy_GBs"] = 2.0 * nb / (ms * 1e-3) / 1e9
    res["copy_frac_of_published"] = res["copy_GBs"] / PEAK_HBM_GBS
    res["shapes"] = "gemm %dx%dx%d bf16 (torch.matmul); copy 1 GiB device to device" % (n, n, n)
    return res


def time_workloads(e2ttt, WL, dev, reps: int = 10) -> dict:
    """The other synthetic workloads at their own shapes (parity-test cases,
    timed here as context), and the paper's own 1.3B throughput shape (head
    dim 128, chunk 512): every pass they include, back to back, HIP events
    around each call; tokens/s counts B*T per forward (+ backward) pass."""
    import torch
    res = {}
    for w in (WL.WORKLOADS[0], WL.WORKLOADS[1], WL.WORKLOADS[2], WL.WORKLOADS[4],
              WL.PAPER_1P3B):
        x = WL.make_inputs(w)
        bf = w.io == "bf16"
        t = {}
        for n, a in x.items():
            if a is None:
                t[n] = None
                continue
            ten = torch.from_numpy(a).to(dev)
            t[n] = ten.to(torch.bfloat16) if (bf and n in ("q", "k", "v", "d_out")) else ten
        cfg = e2ttt.Config(w.B, w.H, w.T, w.d, w.dh, w.C, w.fw,
                           e2ttt.DT_BF16 if bf else e2ttt.DT_F32)
        ws = e2ttt.alloc_workspace(cfg, w.backward, dev)
        out = torch.empty_like(t["q"])
        wo, mo = torch.empty_like(t["w_in"]), torch.empty_like(t["w_in"])
        scratch = (torch.empty(e2ttt.backward_scratch_bytes(cfg), dtype=torch.uint8, device=dev)
                   if w.backward else None)
        grads = None
        if w.backward:
            grads = dict(dq=torch.empty_like(t["q"]), dk=torch.empty_like(t["k"]),
                         dv=torch.empty_like(t["v"]), d_eta=torch.empty_like(t["eta"]),
                         d_beta=torch.empty_like(t["beta"]), d_gamma=torch.empty_like(t["gamma"]),
                         d_w_in=torch.empty_like(t["w_in"]), d_m_in=torch.empty_like(t["w_in"]))

        def step():
            e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                          t["w_in"], None, out=out, w_out=wo, m_out=mo, workspace=ws,
                          save_for_backward=w.backward)
            if w.backward:
                e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                               t["w_in"], None, ws, t["d_out"], grads=grads, scratch=scratch)

        for _ in range(3):
            step()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(reps):
            step()
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / reps
        units = (9 + 18 * w.backward) if w.fw == WL.FW_MLP else (13 + 26 * w.backward)
        flop = float(units) * 2.0 * w.d * w.dh * w.T * w.B * w.H
        peak = PEAK_BF16_TFLOPS if bf else PEAK_F32_TFLOPS
        res[w.name] = {"pass": "fwd+bwd" if w.backward else "fwd", "ms": ms,
                       "tokens_per_s": w.B * w.T / (ms * 1e-3),
                       "mfma_frac": flop / (ms * 1e-3) / 1e12 / peak,
                       "peak_TFLOPs": peak, "units_x_chunks": "%d x %d" % (w.units, w.n_chunks)}
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the headline step (no averaged-rule, gate or decode timings)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this size (for counter calibration)")
    ap.add_argument("--workloads-only", action="store_true",
                    help="time only the other workloads and the paper's 1.3B shape (for a kernel "
                         "trace of their kernels); prints their timings as one JSON object")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the chunk update shards over (batch, head) units "
              "with no exchange, so more GPUs are not exercised here", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_21308_amd import e2ttt, workloads as WL

    if args.workloads_only:
        print(json.dumps({"other_workloads": time_workloads(e2ttt, WL, torch.device("cuda:0")),
                          "source_hash": source_hash()}), flush=True)
        return

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
    if not args.no_extras:
        # the same step under the chunk-averaged rule (ablation baseline): only
        # the scalar kernels differ, so this isolates what the closed form costs
        cfg_main = cfg
        cfg = e2ttt.Config(w.B, w.H, w.T, w.d, w.dh, w.C, w.fw, e2ttt.DT_BF16,
                           e2ttt.FLAG_CHUNK_AVERAGED)
        step()
        torch.cuda.synchronize()
        na = max(1, args.steps // 2)
        ta = time.perf_counter()
        for _ in range(na):
            step()
        torch.cuda.synchronize()
        res["averaged_rule_ms_per_step"] = (time.perf_counter() - ta) * 1e3 / na
        cfg = cfg_main
        res["long_chunk_forward"] = time_long_chunk(e2ttt, w, t, dev)
        res["gates"] = time_gates(e2ttt, w, dev)
        res["decode"] = time_decode(e2ttt, w, x, dev)
        # the same decode loop for one layer at the paper's 1.3B shape (head dim
        # 128, hidden 512, C 512), at the two batch sizes of its decode table
        res["decode_paper_1p3b"] = {}
        for b in (1, 8):
            wp = WL.PAPER_1P3B.with_(B=b)
            res["decode_paper_1p3b"]["B%d" % b] = time_decode(
                e2ttt, wp, WL.make_inputs(wp, with_grads=False), dev)
        res["other_workloads"] = time_workloads(e2ttt, WL, dev)
        res["peaks_measured"] = measure_peaks(dev)
    if args.no_cpu_baseline:
        res["cpu_baseline"] = None
    else:
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
