"""Pins of the oracle's post-chunk L2 normalisation of the fast weights (CPU).

App. B.1 applies an L2 normalisation to the fast-weight matrices at every
chunk boundary (after Zhang et al.) without naming its axis or target; the
reading taken: each row of each matrix, over the matrix's input dimension, is
rescaled to that row's norm in the unit's initial weights, the momentum is
left alone.  Checked against:
  * its defining invariant: every row of the final state (and of every
    chunk-start state, through resume) has the norm of w_in's row;
  * eta = 0, gamma = 1, no momentum: the state is w_in throughout, bit for bit;
  * one chunk: the unnormalised forward followed by a numpy row normalisation;
  * torch autograd through a token loop whose chunk ends normalise with
    torch.linalg.vector_norm (so the targets' dependence on w_in is
    differentiated too), and fourth-order finite differences.
"""
import numpy as np
import pytest
import torch

from oracle.oracle import FLAG_POST_NORM as PN, FW_MLP, FW_SWIGLU
from tests import torchref

NETS = [FW_MLP, FW_SWIGLU]


def problem(T, d, dh, fw, seed):
    rng = np.random.default_rng(seed)
    P = (2 if fw == 0 else 3) * d * dh
    x = dict(q=rng.standard_normal((1, 2, T, d)), k=rng.standard_normal((1, 2, T, d)),
             v=rng.standard_normal((1, 2, T, d)), eta=rng.uniform(0.05, 0.3, (1, 2, T)),
             beta=rng.uniform(0.3, 0.95, (1, 2, T)), gamma=rng.uniform(0.9, 1.0, (1, 2, T)),
             w_in=rng.standard_normal((1, 2, P)) * 0.3, m_in=rng.standard_normal((1, 2, P)) * 0.05)
    g = dict(d_out=rng.standard_normal((1, 2, T, d)), d_w_out=rng.standard_normal((1, 2, P)),
             d_m_out=rng.standard_normal((1, 2, P)))
    return x, g


def rows(W, d, dh, fw):
    """Row norms of every matrix of a [P] state, in packing order."""
    W = torch.tensor(W)
    return np.concatenate([torch.linalg.vector_norm(m, dim=1).numpy()
                           for m in torchref.split(W, d, dh, fw)])


@pytest.mark.parametrize("fw", NETS)
@pytest.mark.parametrize("flags", [PN, PN | 1])
def test_rows_keep_their_initial_norms(oracle, fw, flags):
    T, d, dh, C = 13, 4, 6, 4
    x, _ = problem(T, d, dh, fw, 1 + fw)
    _, wo, mo = oracle.forward(**x, C=C, fw=fw, dh=dh, flags=flags)
    for u in range(2):
        np.testing.assert_allclose(rows(wo[0, u], d, dh, fw), rows(x["w_in"][0, u], d, dh, fw),
                                   rtol=1e-12)
    # every chunk-start state as well: the forward over the first chunks
    for T1 in (4, 8):
        y = {n: (a if n in ("w_in", "m_in") else a[:, :, :T1]) for n, a in x.items()}
        _, w1, _ = oracle.forward(**y, C=C, fw=fw, dh=dh, flags=flags)
        np.testing.assert_allclose(rows(w1[0, 0], d, dh, fw), rows(x["w_in"][0, 0], d, dh, fw),
                                   rtol=1e-12)
    # the momentum is not normalised
    _, _, mo0 = oracle.forward(**x, C=C, fw=fw, dh=dh, flags=flags & 1)
    assert not np.allclose(rows(mo[0, 0], d, dh, fw), rows(mo0[0, 0], d, dh, fw))


@pytest.mark.parametrize("fw", NETS)
def test_zero_learning_rate_keeps_w_in_exactly(oracle, fw):
    T, d, dh, C = 10, 4, 6, 3
    x, _ = problem(T, d, dh, fw, 5)
    x["eta"] = np.zeros_like(x["eta"])
    x["gamma"] = None
    x["m_in"] = None
    _, wo, mo = oracle.forward(**x, C=C, fw=fw, dh=dh, flags=PN)
    assert np.array_equal(wo, x["w_in"]) and not mo.any()


@pytest.mark.parametrize("fw", NETS)
def test_one_chunk_is_the_update_then_row_normalisation(oracle, fw):
    T, d, dh = 6, 4, 6
    x, _ = problem(T, d, dh, fw, 7)
    o1, w1, m1 = oracle.forward(**x, C=T, fw=fw, dh=dh, flags=PN)
    o0, w0, m0 = oracle.forward(**x, C=T, fw=fw, dh=dh)
    assert np.array_equal(o1, o0) and np.array_equal(m1, m0)
    for u in range(2):
        want = torchref.row_normalise(torch.tensor(w0[0, u]), torch.tensor(x["w_in"][0, u]), d,
                                      dh, fw).numpy()
        np.testing.assert_allclose(w1[0, u], want, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("fw", NETS)
@pytest.mark.parametrize("C,T", [(4, 9), (3, 7)])
def test_backward_vs_autograd(oracle, fw, C, T):
    d, dh = 4, 6
    x, g = problem(T, d, dh, fw, 20 + C + fw)
    res = oracle.backward(**x, **g, C=C, fw=fw, dh=dh, flags=PN)
    names = {"q": "dq", "k": "dk", "v": "dv", "eta": "d_eta", "beta": "d_beta",
             "gamma": "d_gamma", "w_in": "d_w_in", "m_in": "d_m_in"}
    for u in range(2):
        tx = {n: torch.tensor(a[0, u], requires_grad=True) for n, a in x.items()}
        o, W, M = torchref.chunked_forward(tx["q"], tx["k"], tx["v"], tx["eta"], tx["beta"],
                                           tx["gamma"], tx["w_in"], tx["m_in"], C, d, dh, fw,
                                           post_norm=True)
        J = (torch.tensor(g["d_out"][0, u]) * o).sum() + \
            (torch.tensor(g["d_w_out"][0, u]) * W).sum() + (torch.tensor(g["d_m_out"][0, u]) * M).sum()
        J.backward()
        for inp, gname in names.items():
            np.testing.assert_allclose(res[gname][0, u], tx[inp].grad.numpy(), rtol=1e-9,
                                       atol=1e-11, err_msg=inp)


@pytest.mark.parametrize("fw", NETS)
def test_backward_finite_differences(oracle, fw):
    T, d, dh, C = 8, 4, 5, 3
    x, g = problem(T, d, dh, fw, 40 + fw)
    res = oracle.backward(**x, **g, C=C, fw=fw, dh=dh, flags=PN)
    rng = np.random.default_rng(3)
    h = 1e-6
    for inp, gname in {"w_in": "d_w_in", "m_in": "d_m_in", "k": "dk", "q": "dq", "v": "dv",
                       "eta": "d_eta", "beta": "d_beta", "gamma": "d_gamma"}.items():
        direction = rng.standard_normal(x[inp].shape)

        def J(s):
            xs = dict(x)
            xs[inp] = x[inp] + s * h * direction
            o, wo, mo = oracle.forward(**xs, C=C, fw=fw, dh=dh, flags=PN)
            return np.sum(g["d_out"] * o) + np.sum(g["d_w_out"] * wo) + np.sum(g["d_m_out"] * mo)

        fd = (-J(2) + 8 * J(1) - 8 * J(-1) + J(-2)) / (12 * h)
        an = np.sum(res[gname] * direction)
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (inp, fd, an)
