"""Independent fp64 PyTorch check of the oracle -- test infrastructure only.

The fast-weight net is assembled from library routines (``F.gelu`` with its
exact erf form, ``F.silu``, ``F.layer_norm`` without affine) and every
derivative comes from ``torch.autograd``; nothing here repeats the oracle's
hand-written gradient code.
"""
import torch
import torch.nn.functional as F


def split(W, d, dh, fw):
    if fw == 0:
        return W[: dh * d].reshape(dh, d), W[dh * d:].reshape(d, dh)
    return (W[: dh * d].reshape(dh, d), W[dh * d: 2 * dh * d].reshape(dh, d),
            W[2 * dh * d:].reshape(d, dh))


def net(W, x, d, dh, fw, resln=True, eps=1e-5, ln_a=None, ln_b=None):
    """f_W(x) for x [..., d] (paper Sec. 4, fast-weight network); ln_a, ln_b:
    the LayerNorm's elementwise affine (weight, bias), or None."""
    if fw == 0:
        W1, W2 = split(W, d, dh, fw)
        y = F.gelu(x @ W1.T) @ W2.T
    else:
        Wg, Wu, Wd = split(W, d, dh, fw)
        y = (F.silu(x @ Wg.T) * (x @ Wu.T)) @ Wd.T
    if not resln:
        return y
    return x + F.layer_norm(y, (d,), weight=ln_a, bias=ln_b, eps=eps)


def neg_grad(W, k, v, d, dh, fw, resln=True, eps=1e-5, create_graph=False):
    """-grad_W of 1/2 ||f_W(k) - v||^2 for a single token, via autograd."""
    if not W.requires_grad:
        W = W.detach().requires_grad_(True)
    L = 0.5 * ((net(W, k, d, dh, fw, resln, eps) - v) ** 2).sum()
    (g,) = torch.autograd.grad(L, W, create_graph=create_graph)
    return -g


def row_normalise(W, W_init, d, dh, fw):
    """Every row of every matrix (over its input dimension) rescaled to the
    norm of the same row of W_init, via torch.linalg.vector_norm (rows of norm
    zero are left as they are)."""
    out = []
    for Wm, Im in zip(split(W, d, dh, fw), split(W_init, d, dh, fw)):
        n = torch.linalg.vector_norm(Wm, dim=1, keepdim=True)
        t = torch.linalg.vector_norm(Im, dim=1, keepdim=True)
        safe = torch.where(n > 0, n, torch.ones_like(n))
        out.append(torch.where(n > 0, Wm * (t / safe), Wm).reshape(-1))
    return torch.cat(out)


def chunked_forward(q, k, v, eta, beta, gamma, w_in, m_in, C, d, dh, fw, resln=True, eps=1e-5,
                    ln_a=None, ln_b=None, post_norm=False):
    """One unit: token recurrence with gradients at chunk-start weights
    (paper eq. (7)), outputs f_{W_0}(q_t); differentiable end to end.
    post_norm: rows renormalised to w_in's row norms at every chunk end."""
    T = q.shape[0]
    W = w_in
    M = m_in if m_in is not None else torch.zeros_like(w_in)
    outs = []
    for s0 in range(0, T, C):
        W0 = W
        idx = range(s0, min(T, s0 + C))
        for t in idx:
            outs.append(net(W0, q[t], d, dh, fw, resln, eps, ln_a, ln_b))
        for t in idx:
            L = 0.5 * ((net(W0, k[t], d, dh, fw, resln, eps, ln_a, ln_b) - v[t]) ** 2).sum()
            (g,) = torch.autograd.grad(L, W0, create_graph=True)
            M = beta[t] * M + eta[t] * (-g)
            g_t = gamma[t] if gamma is not None else 1.0
            W = g_t * W + M
        if post_norm:
            W = row_normalise(W, w_in, d, dh, fw)
    return torch.stack(outs), W, M
