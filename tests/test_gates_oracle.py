"""Pins of the fp64 gate oracle (Sec. 4, eqs. (12)-(14)) against closed forms,
limits, torch autograd of the forward maps, and finite differences."""
import math

import numpy as np
import pytest
import torch

from oracle import gates

P = dict(eta_base=0.01, alpha_base=0.1, tau=32.0)


def test_closed_form_at_exact_sigmoid_values():
    # sigmoid(0) = 1/2, sigmoid(ln 3) = 3/4, sigmoid(-ln 3) = 1/4
    l = np.array([0.0, math.log(3.0), -math.log(3.0)])
    eta, beta, gamma = gates.forward(l, l, l[::-1].copy(), **P)
    np.testing.assert_allclose(eta, [0.005, 0.0075, 0.0025], rtol=1e-15)
    np.testing.assert_allclose(beta, [0.5 ** (1 / 32), 0.75 ** (1 / 32), 0.25 ** (1 / 32)], rtol=1e-15)
    alpha = np.array([0.025, 0.075, 0.05])   # 0.1 sigmoid(-ln 3, ln 3, 0)
    np.testing.assert_allclose(gamma, 1.0 - eta * alpha, rtol=1e-15)


def test_limits_and_bounds():
    big = np.array([-60.0, 60.0])
    eta, beta, gamma = gates.forward(big, big, big, **P)
    np.testing.assert_allclose(eta, [0.0, 0.01], atol=1e-20)
    # beta = sigmoid(l)^(1/tau) stays far from 0 even at l = -60 (tau = 32)
    np.testing.assert_allclose(beta, [math.exp(-(60.0 + math.log1p(math.exp(-60.0))) / 32.0), 1.0],
                               rtol=1e-12)
    np.testing.assert_allclose(gamma, [1.0, 1.0 - 0.01 * 0.1], atol=1e-15)
    x = np.linspace(-20, 20, 401)
    eta, beta, gamma = gates.forward(x, x, x, **P)
    assert np.all(np.diff(eta) > 0) and np.all(np.diff(beta) >= 0) and np.all(np.diff(gamma) <= 0)
    assert np.all((eta > 0) & (eta < 0.01)) and np.all((beta > 0) & (beta <= 1))
    assert np.all((gamma >= 1 - 0.01 * 0.1) & (gamma <= 1))


def test_beta_forgetting_rate_is_softplus():
    # -log beta = -log(sigmoid(l)) / tau = log1p(exp(-l)) / tau (to fp64 resolution of beta)
    x = np.linspace(-30, 30, 121)
    _, beta, _ = gates.forward(x, x, None, **P)
    np.testing.assert_allclose(-np.log(beta) * 32.0, np.log1p(np.exp(-x)), rtol=1e-12, atol=1e-13)


def torch_forward(le, lb, la, eta_base, alpha_base, tau):
    eta = eta_base * torch.sigmoid(le)
    beta = torch.sigmoid(lb) ** (1.0 / tau)
    gamma = None if la is None else 1.0 - eta * (alpha_base * torch.sigmoid(la))
    return eta, beta, gamma


@pytest.mark.parametrize("with_alpha", [True, False])
@pytest.mark.parametrize("p", [P, dict(eta_base=0.3, alpha_base=0.7, tau=3.0)])
def test_backward_against_autograd(with_alpha, p):
    rng = np.random.default_rng(5)
    n = 257
    le, lb, la = (rng.normal(0, 4, n) for _ in range(3))
    de, db, dg = (rng.normal(0, 1, n) for _ in range(3))
    if not with_alpha:
        la = dg = None
    got = gates.backward(le, lb, la, de, db, dg, **p)
    T = [None if a is None else torch.tensor(a, dtype=torch.float64, requires_grad=True)
         for a in (le, lb, la)]
    outs = torch_forward(*T, p["eta_base"], p["alpha_base"], p["tau"])
    loss = (outs[0] * torch.tensor(de)).sum() + (outs[1] * torch.tensor(db)).sum()
    if with_alpha:
        loss = loss + (outs[2] * torch.tensor(dg)).sum()
    loss.backward()
    for g, t in zip(got, T):
        if t is None:
            assert g is None
            continue
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-12, atol=1e-15)


def test_backward_against_finite_differences():
    rng = np.random.default_rng(9)
    n = 64
    le, lb, la = (rng.normal(0, 2, n) for _ in range(3))
    de, db, dg = (rng.normal(0, 1, n) for _ in range(3))
    got = gates.backward(le, lb, la, de, db, dg, **P)

    def loss(le_, lb_, la_):
        e, b, g = gates.forward(le_, lb_, la_, **P)
        return np.sum(e * de) + np.sum(b * db) + np.sum(g * dg)

    h = 1e-5
    for which in range(3):
        args = [le, lb, la]
        fd = np.empty(n)
        for i in range(n):
            ap = [a.copy() for a in args]
            am = [a.copy() for a in args]
            ap[which][i] += h
            am[which][i] -= h
            fd[i] = (loss(*ap) - loss(*am)) / (2 * h)
        np.testing.assert_allclose(got[which], fd, rtol=1e-5, atol=1e-10)


def test_backward_at_saturated_logits():
    # sigmoid'(x) = exp(-x) / (1 + exp(-x))^2 = exp(x) / (1 + exp(x))^2: at
    # |x| = 30 and 80 the gradients keep full fp64 relative accuracy
    x = np.array([30.0, -30.0, 80.0, -80.0])
    one = np.ones(4)
    d = np.exp(-np.abs(x)) / (1.0 + np.exp(-np.abs(x))) ** 2
    ge, gb, ga = gates.backward(x, x, x, one, one, one, **P)
    s = 1.0 / (1.0 + np.exp(-x))
    np.testing.assert_allclose(ge, (1.0 - 0.1 * s) * 0.01 * d, rtol=1e-13)
    np.testing.assert_allclose(ga, -0.01 * s * 0.1 * d, rtol=1e-13)
    # d beta / d l = beta (1 - sigmoid(l)) / tau, 1 - sigmoid(l) = 1 / (1 + exp(l))
    np.testing.assert_allclose(gb, s ** (1 / 32) / (1.0 + np.exp(x)) / 32, rtol=1e-13)
