"""fp64 oracle of the gate parameterization -- TEST INFRASTRUCTURE ONLY.

Sec. 4 ("Input-Dependent Dynamics"), eqs. (12)-(14): per token, from the
logits of the three linear heads,
    eta   = eta_base * sigmoid(l_eta)                              (12)
    beta  = sigmoid(l_beta) ** (1 / tau)                           (13)
    alpha = alpha_base * sigmoid(l_alpha),  gamma = 1 - eta alpha  (14)
and the reverse-mode derivative of those three maps (chain rule, written out
below).  Plain numpy in float64; only the tests may import this module, and it
imports nothing from the HIP library's package.
"""
from __future__ import annotations

import numpy as np


def _sigmoid(x):
    """1 / (1 + exp(-x)), evaluated as exp(x) / (1 + exp(x)) for x < 0 so that
    neither branch overflows or cancels."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def forward(l_eta, l_beta, l_alpha=None, *, eta_base=0.01, alpha_base=0.1, tau=32.0):
    """(eta, beta, gamma); gamma is None without l_alpha (gamma = 1)."""
    eta = eta_base * _sigmoid(l_eta)
    beta = _sigmoid(l_beta) ** (1.0 / tau)
    gamma = None
    if l_alpha is not None:
        alpha = alpha_base * _sigmoid(l_alpha)
        gamma = 1.0 - eta * alpha
    return eta, beta, gamma


def backward(l_eta, l_beta, l_alpha, d_eta, d_beta, d_gamma, *, eta_base=0.01, alpha_base=0.1,
             tau=32.0):
    """Gradients of the logits: (d_l_eta, d_l_beta, d_l_alpha).

    The sigmoid's derivative is s (1 - s) with 1 - sigmoid(x) = sigmoid(-x);
    the second factor is evaluated as sigmoid(-x), since 1 - s cancels for
    large x (at x = 30 the difference would keep only three digits)."""
    l_eta = np.asarray(l_eta, dtype=np.float64)
    l_beta = np.asarray(l_beta, dtype=np.float64)
    s_e = _sigmoid(l_eta)
    s_b = _sigmoid(l_beta)
    eta = eta_base * s_e
    beta = s_b ** (1.0 / tau)
    d_eta_total = np.asarray(d_eta, dtype=np.float64)
    d_l_alpha = None
    if l_alpha is not None:
        l_alpha = np.asarray(l_alpha, dtype=np.float64)
        s_a = _sigmoid(l_alpha)
        alpha = alpha_base * s_a
        d_gamma = np.asarray(d_gamma, dtype=np.float64)
        d_eta_total = d_eta_total - alpha * d_gamma          # d gamma / d eta = -alpha
        d_alpha = -eta * d_gamma                              # d gamma / d alpha = -eta
        d_l_alpha = d_alpha * alpha_base * s_a * _sigmoid(-l_alpha)
    d_l_eta = d_eta_total * eta_base * s_e * _sigmoid(-l_eta)
    # beta = s_b^(1/tau): d beta / d l = (1/tau) s_b^(1/tau - 1) s_b (1 - s_b)
    d_l_beta = np.asarray(d_beta, dtype=np.float64) * beta * _sigmoid(-l_beta) / tau
    return d_l_eta, d_l_beta, d_l_alpha
