"""Pins of the oracle's learnable LayerNorm affine (CPU).

The fast-weight net of Sec. 4 ends in a LayerNorm; with its elementwise affine
(a weight a and a bias b per head, slow weights shared by the batch) the net
is f(x) = x + a * LN(y) + b.  The oracle's affine is checked against:
  * the identity affine (a = 1, b = 0): exactly the net without affine,
    forward and backward, bit for bit;
  * torch autograd through a differentiable token loop whose net is built from
    F.layer_norm(weight=a, bias=b) (second order via create_graph), with two
    batch entries per head so that the per-head gradients sum over the batch;
  * fourth-order central finite differences of every gradient, a and b
    included.
"""
import numpy as np
import pytest
import torch

from oracle.oracle import FW_MLP, FW_SWIGLU
from tests import torchref

NETS = [FW_MLP, FW_SWIGLU]


def problem(B, H, T, d, dh, fw, seed):
    rng = np.random.default_rng(seed)
    P = (2 if fw == 0 else 3) * d * dh
    x = dict(q=rng.standard_normal((B, H, T, d)), k=rng.standard_normal((B, H, T, d)),
             v=rng.standard_normal((B, H, T, d)), eta=rng.uniform(0.01, 0.1, (B, H, T)),
             beta=rng.uniform(0.3, 0.95, (B, H, T)), gamma=rng.uniform(0.9, 1.0, (B, H, T)),
             w_in=rng.standard_normal((B, H, P)) * 0.3,
             m_in=rng.standard_normal((B, H, P)) * 0.05)
    ln = dict(ln_a=1.0 + 0.3 * rng.standard_normal((H, d)), ln_b=0.2 * rng.standard_normal((H, d)))
    g = dict(d_out=rng.standard_normal((B, H, T, d)), d_w_out=rng.standard_normal((B, H, P)),
             d_m_out=rng.standard_normal((B, H, P)))
    return x, ln, g


@pytest.mark.parametrize("fw", NETS)
def test_identity_affine_is_the_plain_net(oracle, fw):
    B, H, T, d, dh, C = 1, 2, 9, 4, 6, 4
    x, _, g = problem(B, H, T, d, dh, fw, 10 + fw)
    one, zero = np.ones((H, d)), np.zeros((H, d))
    a = oracle.forward(**x, C=C, fw=fw, dh=dh)
    b = oracle.forward(**x, C=C, fw=fw, dh=dh, ln_a=one, ln_b=zero)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
    ga = oracle.backward(**x, **g, C=C, fw=fw, dh=dh)
    gb = oracle.backward(**x, **g, C=C, fw=fw, dh=dh, ln_a=one, ln_b=zero)
    for n, r in ga.items():
        assert (r is None and gb[n] is None) or np.array_equal(r, gb[n]), n


@pytest.mark.parametrize("fw", NETS)
@pytest.mark.parametrize("C,T", [(4, 8), (3, 7)])
def test_affine_forward_and_backward_vs_autograd(oracle, fw, C, T):
    B, H, d, dh = 2, 2, 4, 6
    x, ln, g = problem(B, H, T, d, dh, fw, 100 + C + 10 * fw)
    out, wo, mo = oracle.forward(**x, C=C, fw=fw, dh=dh, **ln)
    res = oracle.backward(**x, **g, C=C, fw=fw, dh=dh, **ln)
    ta = torch.tensor(ln["ln_a"], requires_grad=True)
    tb = torch.tensor(ln["ln_b"], requires_grad=True)
    names = {"q": "dq", "k": "dk", "v": "dv", "eta": "d_eta", "beta": "d_beta",
             "gamma": "d_gamma", "w_in": "d_w_in", "m_in": "d_m_in"}
    for bi in range(B):
        for h in range(H):
            tx = {n: torch.tensor(a[bi, h], requires_grad=True) for n, a in x.items()}
            o, W, M = torchref.chunked_forward(tx["q"], tx["k"], tx["v"], tx["eta"], tx["beta"],
                                               tx["gamma"], tx["w_in"], tx["m_in"], C, d, dh, fw,
                                               ln_a=ta[h], ln_b=tb[h])
            np.testing.assert_allclose(out[bi, h], o.detach().numpy(), rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(wo[bi, h], W.detach().numpy(), rtol=1e-12, atol=1e-12)
            J = (torch.tensor(g["d_out"][bi, h]) * o).sum() + \
                (torch.tensor(g["d_w_out"][bi, h]) * W).sum() + \
                (torch.tensor(g["d_m_out"][bi, h]) * M).sum()
            J.backward()
            for inp, gname in names.items():
                np.testing.assert_allclose(res[gname][bi, h], tx[inp].grad.numpy(), rtol=1e-9,
                                           atol=1e-11, err_msg=inp)
    # a and b accumulated their gradients over both batch entries of each head
    np.testing.assert_allclose(res["d_ln_a"], ta.grad.numpy(), rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(res["d_ln_b"], tb.grad.numpy(), rtol=1e-9, atol=1e-11)


@pytest.mark.parametrize("fw", NETS)
def test_affine_backward_finite_differences(oracle, fw):
    B, H, T, d, dh, C = 2, 1, 7, 4, 5, 3
    x, ln, g = problem(B, H, T, d, dh, fw, 300 + fw)
    res = oracle.backward(**x, **g, C=C, fw=fw, dh=dh, **ln)
    rng = np.random.default_rng(7)
    h = 1e-6
    inputs = dict(x, **ln)
    names = {"ln_a": "d_ln_a", "ln_b": "d_ln_b", "k": "dk", "v": "dv", "w_in": "d_w_in",
             "q": "dq", "eta": "d_eta"}
    for inp, gname in names.items():
        direction = rng.standard_normal(inputs[inp].shape)

        def J(s):
            xs = dict(inputs)
            xs[inp] = inputs[inp] + s * h * direction
            o, wo, mo = oracle.forward(**{n: xs[n] for n in x}, C=C, fw=fw, dh=dh,
                                       ln_a=xs["ln_a"], ln_b=xs["ln_b"])
            return np.sum(g["d_out"] * o) + np.sum(g["d_w_out"] * wo) + np.sum(g["d_m_out"] * mo)

        fd = (-J(2) + 8 * J(1) - 8 * J(-1) + J(-2)) / (12 * h)
        an = np.sum(res[gname] * direction)
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (inp, fd, an)


def test_affine_needs_the_layer_norm(oracle):
    x, ln, _ = problem(1, 1, 4, 4, 6, FW_MLP, 1)
    with pytest.raises(ValueError):
        oracle.forward(**x, C=4, fw=FW_MLP, dh=6, flags=1, **ln)
