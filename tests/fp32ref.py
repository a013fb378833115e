"""A plain float32 evaluation of the chunk update -- test infrastructure only.

It sizes the fp32 bar of the GPU parity tests: the paper's tolerance for fp32
is rel-L2 1e-5, but some fp32 cases are ill-conditioned enough that any fp32
evaluation lands farther than that from the fp64 oracle.  For those cases the
GPU is held to a multiple of what this evaluation reaches on the same inputs
(``fp32_bar``), instead of a factor applied to a perturbation probe.

What it computes is the closed form of Prop. 1 (eqs. (9)-(11)), chunk by
chunk, with correctly rounded float32 operations of PyTorch on the CPU:
  * scalar kernels from their definitions (App. A): suffix products by
    cumulative products, S_t by the reverse recursion S_C = 1,
    S_t = g~_t + beta_{t+1} S_{t+1}; K^W_t = eta_t S_t, K^M_t = eta_t b~_t,
    carries (g~_0, beta_1 S_1, b~_0);
  * sum_t K_t G_t as minus the gradient (torch.autograd) at the chunk-start
    weights of sum_t K_t 1/2 ||f_{W_0}(k_t) - v_t||^2;
  * W_C = g~_0 W_0 + beta_1 S_1 M_0 + sum K^W G,  M_C = b~_0 M_0 + sum K^M G;
  * outputs f_{W_0}(q_t) (eq. (6));
and the backward by torch.autograd through all of it (second order with
create_graph).  The net comes from library routines (tests/torchref.py).  In
float64 it reproduces the oracle (pinned in tests/test_oracle_pins.py), so in
float32 it is the same computation with nothing but fp32 rounding.
"""
from __future__ import annotations

import numpy as np
import torch

from tests import torchref

# The GPU may be this many times as far from the oracle as the plain fp32
# evaluation: twice for the kernel's approximate operations (hardware
# reciprocal, reciprocal square root and exp2, a rational erfc with 1.5e-7
# absolute error: each up to a few ulp against the half ulp of a correctly
# rounded operation), twice for two independent accumulations of rounding
# through the same trajectory.
FP32_FACTOR = 4.0


def scalar_kernels(eta, beta, gamma):
    """K^W, K^M [L] and carries (cw, cm, cb) of one chunk (1-D tensors)."""
    L = eta.shape[0]
    one = torch.ones(1, dtype=eta.dtype)

    def suffix_excl(x):          # x~_t = prod_{i > t} x_i
        if L == 1:
            return one
        return torch.cat([torch.flip(torch.cumprod(torch.flip(x[1:], [0]), 0), [0]), one])

    bt = suffix_excl(beta)
    gt = suffix_excl(gamma) if gamma is not None else torch.ones(L, dtype=eta.dtype)
    S = [None] * L
    S[L - 1] = one[0]
    for t in range(L - 2, -1, -1):
        S[t] = gt[t] + beta[t + 1] * S[t + 1]
    S = torch.stack(S)
    cw = gt[0] * (gamma[0] if gamma is not None else 1.0)
    return eta * S, eta * bt, (cw, beta[0] * S[0], beta[0] * bt[0])


def closed_form_unit(q, k, v, eta, beta, gamma, w_in, m_in, C, d, dh, fw, resln=True, eps=1e-5,
                     ln_a=None, ln_b=None, post_norm=False):
    """One unit over all chunks: (outputs [T, d], W_T, M_T), differentiable;
    ln_a, ln_b: the unit's LayerNorm affine [d], or None; post_norm: the rows
    rescaled to w_in's row norms at every chunk end."""
    T = q.shape[0]
    W = w_in
    M = m_in if m_in is not None else torch.zeros_like(w_in)
    outs = []
    for s0 in range(0, T, C):
        sl = slice(s0, min(T, s0 + C))
        W0, M0 = W, M
        if not W0.requires_grad:
            W0 = W0.detach().requires_grad_(True)
        g = None if gamma is None else gamma[sl]
        kw, km, (cw, cm, cb) = scalar_kernels(eta[sl], beta[sl], g)
        outs.append(torchref.net(W0, q[sl], d, dh, fw, resln, eps, ln_a, ln_b))
        per_tok = 0.5 * ((torchref.net(W0, k[sl], d, dh, fw, resln, eps, ln_a, ln_b) - v[sl]) ** 2
                         ).sum(-1)
        (gw,) = torch.autograd.grad((kw * per_tok).sum(), W0, create_graph=True)
        (gm,) = torch.autograd.grad((km * per_tok).sum(), W0, create_graph=True)
        W = cw * W0 + cm * M0 - gw
        M = cb * M0 - gm
        if post_norm:
            W = torchref.row_normalise(W, w_in, d, dh, fw)
    return torch.cat(outs), W, M


def _t(a, dtype, grad=False):
    if a is None:
        return None
    t = torch.tensor(np.asarray(a), dtype=dtype)
    return t.requires_grad_(True) if grad else t


def forward(x, *, C, fw, dh, flags=0, eps=1e-5, dtype=torch.float32, ln=None):
    """(out [B,H,T,d], w_out, m_out) as float64 numpy, evaluated in `dtype`;
    ln: the LayerNorm affine per head, a pair of [H, d] arrays, or None."""
    B, H, T, d = np.asarray(x["q"]).shape
    resln = not (flags & 1)
    outs, ws, ms = [], [], []
    for b in range(B):
        for h in range(H):
            g = lambda n: None if x.get(n) is None else _t(x[n][b, h], dtype)
            la, lb = (None, None) if ln is None else (_t(ln[0][h], dtype), _t(ln[1][h], dtype))
            o, W, M = closed_form_unit(g("q"), g("k"), g("v"), g("eta"), g("beta"), g("gamma"),
                                       g("w_in"), g("m_in"), C, d, dh, fw, resln, eps, la, lb,
                                       post_norm=bool(flags & 8))
            outs.append(o.detach().double().numpy())
            ws.append(W.detach().double().numpy())
            ms.append(M.detach().double().numpy())
    P = ws[0].shape[-1]
    return (np.stack(outs).reshape(B, H, T, d), np.stack(ws).reshape(B, H, P),
            np.stack(ms).reshape(B, H, P))


def backward(x, *, C, fw, dh, flags=0, eps=1e-5, dtype=torch.float32, ln=None):
    """Gradients of sum<d_out,out> + <d_w_out,w_out> + <d_m_out,m_out>, named as
    the oracle's (dq, dk, dv, d_eta, d_beta, d_gamma, d_w_in, d_m_in, and with
    the affine ln = (a, b) [H, d] also d_ln_a, d_ln_b summed over the batch),
    float64 numpy."""
    B, H, T, d = np.asarray(x["q"]).shape
    resln = not (flags & 1)
    if ln is not None:
        ta = _t(ln[0], dtype, grad=True)
        tb = _t(ln[1], dtype, grad=True)
    names = ("q", "k", "v", "eta", "beta", "gamma", "w_in", "m_in")
    gname = {"q": "dq", "k": "dk", "v": "dv", "eta": "d_eta", "beta": "d_beta",
             "gamma": "d_gamma", "w_in": "d_w_in", "m_in": "d_m_in"}
    res = {}
    for b in range(B):
        for h in range(H):
            leaf = {}
            for n in names:
                if n == "m_in" and x.get("m_in") is None:
                    leaf[n] = torch.zeros(np.asarray(x["w_in"]).shape[-1], dtype=dtype,
                                          requires_grad=True)
                elif x.get(n) is None:
                    leaf[n] = None
                else:
                    leaf[n] = _t(x[n][b, h], dtype, grad=True)
            o, W, M = closed_form_unit(leaf["q"], leaf["k"], leaf["v"], leaf["eta"],
                                       leaf["beta"], leaf["gamma"], leaf["w_in"], leaf["m_in"],
                                       C, d, dh, fw, resln, eps,
                                       None if ln is None else ta[h],
                                       None if ln is None else tb[h],
                                       post_norm=bool(flags & 8))
            loss = (o * _t(x["d_out"][b, h], dtype)).sum()
            if x.get("d_w_out") is not None:
                loss = loss + (W * _t(x["d_w_out"][b, h], dtype)).sum()
            if x.get("d_m_out") is not None:
                loss = loss + (M * _t(x["d_m_out"][b, h], dtype)).sum()
            live = [n for n in names if leaf[n] is not None]
            if ln is not None:
                loss.backward(inputs=[ta, tb], retain_graph=True)
            grads = torch.autograd.grad(loss, [leaf[n] for n in live], allow_unused=True)
            for n, gr in zip(live, grads):
                val = np.zeros(leaf[n].shape) if gr is None else gr.detach().double().numpy()
                res.setdefault(gname[n], []).append(val)
    out = {}
    for n in gname.values():
        if n not in res:
            out[n] = None
            continue
        a = np.stack(res[n])
        out[n] = a.reshape((B, H) + a.shape[1:])
    if ln is not None:
        out["d_ln_a"] = ta.grad.double().numpy()
        out["d_ln_b"] = tb.grad.double().numpy()
    return out


def fp32_bar(err32: dict, tol: float = 1e-5) -> dict:
    """Per-check fp32 bar: the plain tolerance, or FP32_FACTOR times what the
    float32 evaluation itself reaches on the same check where that is larger.
    err32 holds the float32 evaluation's errors under the same names as the
    GPU's (gpu_util.parity_errors: whole tensors and their local maxima)."""
    return {n: max(tol, FP32_FACTOR * e) for n, e in err32.items()}
