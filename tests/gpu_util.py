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


# ------------------------------------------------------- block-wise maxima
# A whole-tensor rel-L2 dilutes an error confined to a few token rows (one
# wrong row of a 2,048-token unit moves it by about sqrt(1/2048) of that row's
# own error), so every parity check also bounds local errors:
#   * row tensors [B, H, T, d] (outputs, dq, dk, dv): the rel-L2 of every
#     (unit, tile of up to 64 tokens) within BLOCK_FACTOR times the bar, and
#     the error of every single row within TOKEN_FACTOR times the bar;
#   * per-token tensors [B, H, T] (d_eta, d_beta, d_gamma): the error of
#     every single token within TOKEN_FACTOR times the bar;
#   * state tensors [B, H, P]: the rel-L2 of every unit within BLOCK_FACTOR
#     times the bar.
# A row's error is measured against the unit's RMS row norm, so that a row that
# happens to be near zero does not read as a large error, while a wrong,
# shifted or unwritten row (an error the size of the values themselves,
# relative error ~1) fails by a wide margin.  Gate gradients are measured
# against the RMS over all units and get no tile bound: a chunk's gate
# gradients are dominated by a few inner products over the whole state
# (<Wb_C, W_0> and its kin), whose rounding error is set by the size of their
# terms, the same in every unit, while their value can cancel to a small
# fraction of it in one unit's chunk (measured: 1/26 of the other unit's, with
# a 10 % relative error of that chunk's d_gamma).
BLOCK_FACTOR = 2.0
TOKEN_FACTOR = 10.0


def _as64(a):
    if isinstance(a, torch.Tensor):
        a = a.float().cpu().numpy()
    return np.asarray(a, dtype=np.float64)


def block_rel_l2(a, b, block=None) -> float:
    """Largest block rel-L2 between a and the reference b.

    Token tensors [B, H, T] or [B, H, T, d] (block = tokens per block): blocks
    are (unit, consecutive `block` tokens), each measured against its own norm
    floored at the unit's RMS block norm.  State tensors [B, H, P] (block
    None): one block per unit."""
    a, b = _as64(a), _as64(b)
    assert a.shape == b.shape, (a.shape, b.shape)
    U = a.shape[0] * a.shape[1]
    if block is None:
        a2 = a.reshape(U, 1, -1)
        b2 = b.reshape(U, 1, -1)
    else:
        T = a.shape[2]
        nb = (T + block - 1) // block
        pad = nb * block - T
        a2 = a.reshape(U, T, -1)
        b2 = b.reshape(U, T, -1)
        if pad:
            z = np.zeros((U, pad, a2.shape[2]))
            a2 = np.concatenate([a2, z], axis=1)
            b2 = np.concatenate([b2, z], axis=1)
        a2 = a2.reshape(U, nb, -1)
        b2 = b2.reshape(U, nb, -1)
    num = np.sqrt(((a2 - b2) ** 2).sum(axis=2))
    den = np.sqrt((b2 ** 2).sum(axis=2))
    rms = np.sqrt((den ** 2).mean(axis=1, keepdims=True))
    den = np.maximum(den, np.maximum(rms, 1e-300))
    return float((num / den).max())


def token_max_err(a, b, per_unit=True) -> float:
    """Largest error of one token row (or one per-token value) of a token
    tensor [B, H, T(, d)], relative to the RMS row norm of its unit (or of the
    whole tensor when per_unit is False)."""
    a, b = _as64(a), _as64(b)
    U, T = a.shape[0] * a.shape[1], a.shape[2]
    a2 = a.reshape(U, T, -1)
    b2 = b.reshape(U, T, -1)
    num = np.sqrt(((a2 - b2) ** 2).sum(axis=2))
    sq = (b2 ** 2).sum(axis=2)
    rms = np.sqrt(sq.mean(axis=1, keepdims=True) if per_unit else sq.mean())
    return float((num / np.maximum(rms, 1e-300)).max())


def parity_errors(pairs: dict, block) -> dict:
    """Errors of named (got, ref[, kind]) pairs, all to be held to one bar.

    kind "state" for [B, H, P] tensors, else a token tensor ([B, H, T, d]
    rows, or [B, H, T] per-token values).  Returns name -> whole-tensor rel-L2,
    name + "/blk" -> largest tile (or unit) rel-L2 / BLOCK_FACTOR, and name +
    "/tok" -> largest row (token) error / TOKEN_FACTOR, so that checking every
    value against the bar applies the local bounds above."""
    errs = {}
    for n, p in pairs.items():
        got, ref = p[0], p[1]
        kind = p[2] if len(p) > 2 else None
        errs[n] = rel_l2(got, ref)
        if kind == "state":
            errs[n + "/blk"] = block_rel_l2(got, ref, None) / BLOCK_FACTOR
            continue
        rows = np.ndim(ref) == 4
        if rows:
            errs[n + "/blk"] = block_rel_l2(got, ref, block) / BLOCK_FACTOR
        errs[n + "/tok"] = token_max_err(got, ref, per_unit=rows) / TOKEN_FACTOR
    return errs


def tile_of(C: int) -> int:
    """Block length for a chunk length C: the chunk, or 64-token tiles of longer chunks."""
    return min(C, 64)
