"""Helpers for the GPU parity tests: move seeded inputs to the device, call the
HIP library through its binding, and measure rel-L2 against the oracle."""
import numpy as np
import torch

from paper_2608_21308_amd import e2ttt

TOL = {"f32": 1e-5, "bf16": 2e-2}


def rel_l2(a, b) -> float:
    if isinstance(a, torch.Tensor):
        a = a.float().cpu().numpy()
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def config_of(w, **over) -> e2ttt.Config:
    kw = dict(B=w.B, H=w.H, T=w.T, d=w.d, dh=w.dh, chunk=w.C, fw=w.fw,
              io=e2ttt.DT_BF16 if w.io == "bf16" else e2ttt.DT_F32)
    kw.update(over)
    return e2ttt.Config(**kw)


def to_dev(x: dict, io: str, dev="cuda") -> dict:
    t = {}
    for n, a in x.items():
        if a is None:
            t[n] = None
            continue
        ten = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        if n in ("q", "k", "v", "d_out") and io == "bf16":
            ten = ten.to(torch.bfloat16)
        t[n] = ten
    return t


def gpu_forward(cfg, t, save=False, m_in=None):
    return e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                         t.get("m_in") if m_in is None else m_in, save_for_backward=save)


def slice_tokens(x: dict, lo: int, hi: int) -> dict:
    y = {}
    for n, a in x.items():
        if a is None or n in ("w_in", "m_in", "d_w_out", "d_m_out"):
            y[n] = a
        else:
            y[n] = np.ascontiguousarray(a[:, :, lo:hi])
    return y


def fp32_sensitivity(fn, x, keys=("q", "k", "v", "w_in", "m_in"), seed=0):
    """rel-L2 change of the oracle outputs fn(x) under a one-ulp (2^-24)
    relative perturbation of the float inputs x[keys]: the intrinsic conditioning of a case
    at fp32 precision."""
    rng = np.random.default_rng(seed)
    ref = fn(x)
    xp = dict(x)
    for k in keys:
        if xp.get(k) is not None:
            xp[k] = x[k] * (1 + 2.0 ** -24 * rng.standard_normal(x[k].shape))
    out = fn(xp)
    return {n: rel_l2(out[n], ref[n]) for n in ref if ref[n] is not None}
