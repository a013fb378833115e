"""Pins of the fp64 chunk-averaged-rule oracle (oracle/averaged.py; Sec. 5,
Tables 4 and 5, eqs. (4)-(6) with mean factors) against the E2-TTT oracle at
C = 1, the C++ oracle's per-token gradients, hand assembly of the chunk-level
recurrence, and finite differences."""
import numpy as np
import pytest

from oracle import averaged as A
from oracle import oracle as E

NETS = [(0, 0), (1, 0), (0, 1)]   # (fw, flags): MLP, SwiGLU, bare MLP


def problem(T, d, dh, fw, seed, with_gamma=True, m_in=True):
    rng = np.random.default_rng(seed)
    P = (2 if fw == 0 else 3) * d * dh
    return dict(q=rng.standard_normal((1, 1, T, d)), k=rng.standard_normal((1, 1, T, d)),
                v=rng.standard_normal((1, 1, T, d)), eta=rng.uniform(0.05, 0.4, (1, 1, T)),
                beta=rng.uniform(0.3, 1.0, (1, 1, T)),
                gamma=rng.uniform(0.8, 1.0, (1, 1, T)) if with_gamma else None,
                w_in=0.3 * rng.standard_normal((1, 1, P)),
                m_in=0.05 * rng.standard_normal((1, 1, P)) if m_in else None)


@pytest.mark.parametrize("fw,flags", NETS)
def test_chunk_size_one_is_the_token_rule(fw, flags):
    """At C = 1 the means are the token's own factors: the rule is the
    token-wise recurrence of eq. (7), which the C++ oracle computes at C = 1
    (forward and backward, independent code)."""
    d, dh, T = 4, 6, 7
    x = problem(T, d, dh, fw, 11 + fw + 2 * flags)
    got = A.forward(**x, C=1, fw=fw, dh=dh, flags=flags)
    want = E.forward(**x, C=1, fw=fw, dh=dh, flags=flags)
    for g, w in zip(got, want):
        np.testing.assert_allclose(g, w, rtol=1e-10, atol=1e-12)
    rng = np.random.default_rng(3)
    dO = rng.standard_normal(x["q"].shape)
    dw = rng.standard_normal(x["w_in"].shape)
    dm = rng.standard_normal(x["w_in"].shape)
    ga = A.backward(**x, d_out=dO, d_w_out=dw, d_m_out=dm, C=1, fw=fw, dh=dh, flags=flags)
    ge = E.backward(**x, d_out=dO, d_w_out=dw, d_m_out=dm, C=1, fw=fw, dh=dh, flags=flags)
    for n in ga:
        np.testing.assert_allclose(ga[n], ge[n], rtol=1e-9, atol=1e-11, err_msg=n)


@pytest.mark.parametrize("fw,flags", NETS)
def test_chunk_gradient_is_the_weighted_sum_of_token_gradients(fw, flags):
    """Eq. (4): from a zero momentum, M_C is the gradient of the eta-weighted
    summed loss, i.e. sum_t eta_t G_t with G_t from the C++ oracle."""
    d, dh, T = 4, 6, 5
    x = problem(T, d, dh, fw, 21 + fw, m_in=False)
    _, wo, mo = A.forward(**x, C=T, fw=fw, dh=dh, flags=flags)
    G = E.neg_grad(x["w_in"][0, 0], x["k"][0, 0], x["v"][0, 0], fw=fw, dh=dh, flags=flags)
    want = (x["eta"][0, 0][:, None] * G).sum(axis=0)
    np.testing.assert_allclose(mo[0, 0], want, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(wo[0, 0], x["gamma"][0, 0].mean() * x["w_in"][0, 0] + want,
                               rtol=1e-11, atol=1e-13)


def test_chunk_means_and_ragged_tail():
    """Two chunks (4 + 3 tokens), assembled by hand from per-token gradients of
    the C++ oracle: M = mean(beta) M + sum eta G(W_0), W = mean(gamma) W_0 + M,
    outputs at each chunk's start state."""
    d, dh, T, C, fw = 4, 6, 7, 4, 0
    x = problem(T, d, dh, fw, 31)
    out, wo, mo = A.forward(**x, C=C, fw=fw, dh=dh)
    W, M = x["w_in"][0, 0], x["m_in"][0, 0]
    want_out = []
    for s0 in (0, 4):
        sl = slice(s0, min(T, s0 + C))
        want_out.append(E.net(W, x["q"][0, 0][sl], fw=fw, dh=dh))
        G = E.neg_grad(W, x["k"][0, 0][sl], x["v"][0, 0][sl], fw=fw, dh=dh)
        M = x["beta"][0, 0][sl].mean() * M + (x["eta"][0, 0][sl][:, None] * G).sum(axis=0)
        W = x["gamma"][0, 0][sl].mean() * W + M
    np.testing.assert_allclose(out[0, 0], np.concatenate(want_out), rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(wo[0, 0], W, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(mo[0, 0], M, rtol=1e-11, atol=1e-13)


def test_no_gamma_is_unit_decay():
    d, dh, T = 4, 6, 6
    x = problem(T, d, dh, 0, 41)
    y = dict(x, gamma=np.ones_like(x["gamma"]))
    x["gamma"] = None
    for a, b in zip(A.forward(**x, C=4, fw=0, dh=dh), A.forward(**y, C=4, fw=0, dh=dh)):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("fw,flags", NETS)
def test_backward_finite_differences(fw, flags):
    d, dh, T, C = 3, 5, 6, 4
    x = problem(T, d, dh, fw, 51 + fw + 2 * flags)
    rng = np.random.default_rng(8)
    dO = rng.standard_normal(x["q"].shape)
    dw = rng.standard_normal(x["w_in"].shape)
    dm = rng.standard_normal(x["w_in"].shape)
    g = A.backward(**x, d_out=dO, d_w_out=dw, d_m_out=dm, C=C, fw=fw, dh=dh, flags=flags)

    def J(y):
        o, W, M = A.forward(**y, C=C, fw=fw, dh=dh, flags=flags)
        return (dO * o).sum() + (dw * W).sum() + (dm * M).sum()

    # fourth-order central differences along a random direction (error ~h^4:
    # the LayerNorm makes the fifth derivative large, hence the small step)
    h = 2e-5
    for n, gn in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("eta", "d_eta"), ("beta", "d_beta"),
                  ("gamma", "d_gamma"), ("w_in", "d_w_in"), ("m_in", "d_m_in")):
        dx = rng.standard_normal(x[n].shape)
        Js = [J(dict(x, **{n: x[n] + s * h * dx})) for s in (2, 1, -1, -2)]
        fd = (-Js[0] + 8 * Js[1] - 8 * Js[2] + Js[3]) / (12 * h)
        np.testing.assert_allclose((g[gn] * dx).sum(), fd, rtol=1e-7, atol=1e-9, err_msg=n)
