"""fp64 oracle of the chunk-averaged update rule -- TEST INFRASTRUCTURE ONLY.

The ablation baseline of Sec. 5 (Tables 4 and 5): the per-token momentum and
decay factors of a chunk are collapsed to chunk-level means, after the
chunk-level momentum of LaCT in eqs. (4)-(5).  For chunk r with start state
(W_0, M_0) and tokens t = 1..L:
    G   = -grad_W sum_t eta_t 1/2 ||f_{W_0}(k_t) - v_t||^2          (4)
    M_C = mean(beta) M_0 + G,   W_C = mean(gamma) W_0 + M_C          (5)
    o_t = f_{W_0}(q_t)                                               (6)
(gamma absent: mean(gamma) = 1, which is eqs. (4)-(5) as printed).  The net f
is the Sec. 4 fast-weight net assembled from torch library routines (exact
erf GELU, SiLU, LayerNorm without affine, biased variance); G is taken by
torch.autograd of the weighted summed loss exactly as eq. (4) writes it, and
the backward is torch.autograd through the whole chunk loop (second order
through autograd.grad(create_graph=True)).  CPU, float64.  Only the tests,
and nothing of the HIP package, may use this module.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def _mats(W, d, dh, fw):
    """Unpack one unit's P parameters (W x rule): MLP W1[dh][d], W2[d][dh];
    SwiGLU Wg[dh][d], Wu[dh][d], Wd[d][dh]."""
    if fw == 0:
        return W[: dh * d].reshape(dh, d), W[dh * d:].reshape(d, dh)
    return (W[: dh * d].reshape(dh, d), W[dh * d: 2 * dh * d].reshape(dh, d),
            W[2 * dh * d:].reshape(d, dh))


def net(W, x, d, dh, fw, resln=True, eps=1e-5):
    """f_W(x) for rows x[n, d] (Sec. 4): x + LN(W2 GELU(W1 x)) or
    x + LN(Wd (SiLU(Wg x) * Wu x)); the bare net without resln."""
    if fw == 0:
        W1, W2 = _mats(W, d, dh, fw)
        y = F.gelu(x @ W1.T) @ W2.T
    else:
        Wg, Wu, Wd = _mats(W, d, dh, fw)
        y = (F.silu(x @ Wg.T) * (x @ Wu.T)) @ Wd.T
    return x + F.layer_norm(y, (d,), eps=eps) if resln else y


def _unit(q, k, v, eta, beta, gamma, w_in, m_in, C, d, dh, fw, resln, eps, train=True):
    """One (batch, head) unit: (out [T, d], W_T, M_T); differentiable end to
    end with train, else each chunk starts from detached values."""
    T = q.shape[0]
    W = w_in
    M = torch.zeros_like(w_in) if m_in is None else m_in
    outs = []
    for s0 in range(0, T, C):
        s1 = min(T, s0 + C)
        if train and W.requires_grad:
            W0 = W
        else:
            W0 = W.detach().requires_grad_(True)
            M = M.detach()
        outs.append(net(W0, q[s0:s1], d, dh, fw, resln, eps))                       # (6)
        r = net(W0, k[s0:s1], d, dh, fw, resln, eps) - v[s0:s1]
        loss = (eta[s0:s1] * 0.5 * (r * r).sum(dim=1)).sum()
        (g,) = torch.autograd.grad(loss, W0, create_graph=True)
        G = -g                                                                        # (4)
        b_bar = beta[s0:s1].mean()
        g_bar = gamma[s0:s1].mean() if gamma is not None else 1.0
        M = b_bar * M + G                                                             # (5)
        W = g_bar * W0 + M
    return torch.cat(outs), W, M


def _t(a, grad=False):
    if a is None:
        return None
    return torch.tensor(np.asarray(a, dtype=np.float64), requires_grad=grad)


def forward(q, k, v, eta, beta, gamma, w_in, m_in, *, C, fw, dh, flags=0, eps=1e-5):
    """Returns (out [B,H,T,d], w_out [B,H,P], m_out [B,H,P]) in float64.
    flags bit 0: the bare net (no residual LayerNorm)."""
    B, H, T, d = np.shape(q)
    out = np.zeros((B, H, T, d))
    P = np.shape(w_in)[-1]
    wo, mo = np.zeros((B, H, P)), np.zeros((B, H, P))
    for b in range(B):
        for h in range(H):
            o, W, M = _unit(_t(q[b, h]), _t(k[b, h]), _t(v[b, h]), _t(eta[b, h]),
                            _t(beta[b, h]), None if gamma is None else _t(gamma[b, h]),
                            _t(w_in[b, h]), None if m_in is None else _t(m_in[b, h]),
                            C, d, dh, fw, not (flags & 1), eps, train=False)
            out[b, h], wo[b, h], mo[b, h] = o.detach().numpy(), W.detach().numpy(), M.detach().numpy()
    return out, wo, mo


def backward(q, k, v, eta, beta, gamma, w_in, m_in, d_out, d_w_out=None, d_m_out=None, *, C, fw,
             dh, flags=0, eps=1e-5):
    """Gradients of sum<d_out, out> + <d_w_out, w_out> + <d_m_out, m_out> with
    respect to every input, as a dict (dq, dk, dv, d_eta, d_beta, d_gamma,
    d_w_in, d_m_in) of float64 arrays (d_gamma None without gamma)."""
    B, H, T, d = np.shape(q)
    P = np.shape(w_in)[-1]
    names = ("q", "k", "v", "eta", "beta", "gamma", "w_in", "m_in")
    res = {("d" + n if len(n) == 1 else "d_" + n): None for n in names}
    shapes = {"q": (B, H, T, d), "k": (B, H, T, d), "v": (B, H, T, d), "eta": (B, H, T),
              "beta": (B, H, T), "gamma": (B, H, T), "w_in": (B, H, P), "m_in": (B, H, P)}
    for n in names:
        if n != "gamma" or gamma is not None:
            res["d" + n if len(n) == 1 else "d_" + n] = np.zeros(shapes[n])
    for b in range(B):
        for h in range(H):
            src = dict(q=q, k=k, v=v, eta=eta, beta=beta, gamma=gamma, w_in=w_in)
            x = {n: None if a is None else _t(a[b, h], grad=True) for n, a in src.items()}
            x["m_in"] = _t(np.zeros(P) if m_in is None else m_in[b, h], grad=True)
            o, W, M = _unit(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"],
                            x["m_in"], C, d, dh, fw, not (flags & 1), eps)
            J = (_t(d_out[b, h]) * o).sum()
            if d_w_out is not None:
                J = J + (_t(d_w_out[b, h]) * W).sum()
            if d_m_out is not None:
                J = J + (_t(d_m_out[b, h]) * M).sum()
            J.backward()
            for n in names:
                key = "d" + n if len(n) == 1 else "d_" + n
                if x[n] is not None and res[key] is not None:
                    res[key][b, h] = x[n].grad.numpy() if x[n].grad is not None else 0.0
    return res
