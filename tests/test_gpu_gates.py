"""GPU parity of the gate parameterization (Sec. 4, eqs. (12)-(14)) and its
backward against the fp64 oracle (oracle/gates.py).

The kernels are elementwise fp32; the bar is a relative error per element of
a few fp32 ulp: max relative error 2e-6 on the gates (beta and gamma sit near
1, where an fp32 value resolves 1 - beta only to 2^-24 absolute; the chunk
kernels take beta and gamma themselves) and 1e-5 on the logit gradients, which
multiply up to five rounded factors (relative to the gradient's magnitude
without cancellation where a difference enters).
"""
import numpy as np
import pytest
import torch

from oracle import gates as gref
from paper_2608_21308_amd import e2ttt

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    e2ttt.load()


def logits(n, seed, scale=3.0):
    rng = np.random.default_rng(seed)
    out = [rng.normal(0, scale, n).astype(np.float32) for _ in range(3)]
    if n >= 8:   # extremes and exact zeros
        for a in out:
            a[:8] = [0.0, -0.0, 30.0, -30.0, 88.0, -88.0, 1e-3, -1e-3]
    return out


def maxrel(a, b, floor):
    a = a.double().cpu().numpy()
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), floor))) if b.size else 0.0


@pytest.mark.parametrize("n", [1, 7, 256, 1000, 524288 + 13])
@pytest.mark.parametrize("with_alpha", [True, False])
@pytest.mark.parametrize("params", [dict(eta_base=0.01, alpha_base=0.1, tau=32.0),
                                    dict(eta_base=0.5, alpha_base=1.0, tau=1.0)])
def test_gates_forward_backward(n, with_alpha, params):
    le, lb, la = logits(n, 100 + n)
    rng = np.random.default_rng(7 + n)
    de, db, dg = (rng.normal(0, 1, n).astype(np.float32) for _ in range(3))
    if not with_alpha:
        la = dg = None
    p = e2ttt.GateParams(**params)
    dev = lambda a: None if a is None else torch.from_numpy(a).cuda()
    eta, beta, gamma = e2ttt.gates_forward(p, dev(le), dev(lb), dev(la))
    g_e, g_b, g_a = e2ttt.gates_backward(p, dev(le), dev(lb), dev(la), dev(de), dev(db), dev(dg))
    torch.cuda.synchronize()
    f64 = lambda a: None if a is None else a.astype(np.float64)
    r_eta, r_beta, r_gamma = gref.forward(f64(le), f64(lb), f64(la), **params)
    r_ge, r_gb, r_ga = gref.backward(f64(le), f64(lb), f64(la), f64(de), f64(db), f64(dg), **params)
    print("gates n=%d alpha=%s" % (n, with_alpha), flush=True)
    # a few fp32 ulp of each value (beta and gamma near 1: a few 2^-24 absolute)
    assert maxrel(eta, r_eta, 1e-30) <= 2e-6
    assert maxrel(beta, r_beta, 1e-30) <= 2e-6
    if with_alpha:
        assert maxrel(gamma, r_gamma, 1e-30) <= 2e-6
        assert maxrel(g_a, r_ga, 1e-30 + 1e-6 * np.max(np.abs(r_ga))) <= 1e-5
    else:
        assert gamma is None and g_a is None
    # d l_eta = (d_eta - alpha d_gamma) eta_base s (1 - s): the difference can
    # cancel, so its error is measured against the same sum taken in absolute
    # values, which the oracle gives for d_eta = |d_eta|, d_gamma = -|d_gamma|
    ab = lambda a: None if a is None else np.abs(f64(a))
    s_ge, s_gb, _ = gref.backward(f64(le), f64(lb), f64(la), ab(de), ab(db),
                                  None if dg is None else -ab(dg), **params)
    assert maxrel(g_e, r_ge, s_ge + 1e-30) <= 1e-5
    assert maxrel(g_b, r_gb, s_gb + 1e-30) <= 1e-5


def test_gates_empty_is_a_no_op():
    p = e2ttt.GateParams()
    z = torch.empty(0, device="cuda")
    eta, beta, gamma = e2ttt.gates_forward(p, z, z, z)
    assert eta.numel() == 0 and beta.numel() == 0 and gamma.numel() == 0


def test_gates_feed_the_chunk_update():
    """Gates formed by the kernel drive e2ttt_chunk_forward to the oracle's
    result with the oracle's gates, within the chain's own sensitivity to
    one-ulp gate changes (the kernel's gates differ from the exact ones by a
    few fp32 ulp)."""
    from oracle import oracle
    from paper_2608_21308_amd import workloads as WL
    from tests.gpu_util import config_of, fp32_sensitivity, rel_l2, to_dev
    w = WL.WORKLOADS[0].with_(B=1, H=2, T=64, C=16)
    x = WL.make_inputs(w)
    le, lb, la = logits(w.B * w.H * w.T, 5, scale=1.5)
    shape = (w.B, w.H, w.T)
    r_eta, r_beta, r_gamma = gref.forward(*(a.astype(np.float64) for a in (le, lb, la)))
    x = dict(x, eta=r_eta.reshape(shape), beta=r_beta.reshape(shape), gamma=r_gamma.reshape(shape))

    def ref(y):
        o, wo_, mo_ = oracle.forward(y["q"], y["k"], y["v"], y["eta"], y["beta"], y["gamma"],
                                     y["w_in"], None, C=w.C, fw=w.fw, dh=w.dh)
        return {"out": o, "w_out": wo_, "m_out": mo_}

    want = ref(x)
    sens = fp32_sensitivity(ref, x, keys=("eta", "beta", "gamma"))
    p = e2ttt.GateParams()
    eta, beta, gamma = e2ttt.gates_forward(p, *(torch.from_numpy(a).cuda() for a in (le, lb, la)))
    t = to_dev(x, w.io)
    t.update(eta=eta.reshape(shape), beta=beta.reshape(shape), gamma=gamma.reshape(shape))
    out, wo, mo, _ = e2ttt.forward(config_of(w), t["q"], t["k"], t["v"], t["eta"], t["beta"],
                                   t["gamma"], t["w_in"], None)
    got = {"out": out, "w_out": wo, "m_out": mo}
    errs = {n: rel_l2(got[n], want[n]) for n in want}
    print("gates -> chunk", {k: "%.2e" % v for k, v in errs.items()},
          "sens", {k: "%.1e" % v for k, v in sens.items()}, flush=True)
    for n in errs:
        assert errs[n] <= max(1e-5, 10 * sens[n]), n


def test_gates_and_chunk_update_through_autograd():
    """Logits -> GatesFunction -> E2TTTFunction -> loss, differentiated by
    torch autograd: the logit gradients equal the oracle's chain backward
    (d_eta, d_beta, d_gamma) mapped through the gate oracle's backward (fp32
    path, within the chain's 1e-5 bar)."""
    from oracle import oracle
    from paper_2608_21308_amd import workloads as WL
    from tests.gpu_util import config_of, rel_l2, to_dev
    w = WL.WORKLOADS[0].with_(B=1, H=2, T=40, C=16, backward=True)
    x = WL.make_inputs(w)
    le, lb, la = (a.reshape(w.B, w.H, w.T) for a in logits(w.B * w.H * w.T, 9, scale=1.5))
    r_eta, r_beta, r_gamma = gref.forward(*(a.astype(np.float64) for a in (le, lb, la)))
    rg = oracle.backward(x["q"], x["k"], x["v"], r_eta, r_beta, r_gamma, x["w_in"], None,
                         x["d_out"], C=w.C, fw=w.fw, dh=w.dh)
    want = gref.backward(*(a.astype(np.float64) for a in (le, lb, la)), rg["d_eta"],
                         rg["d_beta"], rg["d_gamma"])
    t = to_dev(x, w.io)
    L = [torch.from_numpy(a).cuda().requires_grad_(True) for a in (le, lb, la)]
    eta, beta, gamma = e2ttt.GatesFunction.apply(e2ttt.GateParams(), *L)
    out, wo, mo = e2ttt.E2TTTFunction.apply(config_of(w), t["q"], t["k"], t["v"], eta, beta,
                                            gamma, t["w_in"], None)
    (out * t["d_out"]).sum().backward()
    errs = [rel_l2(l.grad, r) for l, r in zip(L, want)]
    print("autograd logits", ["%.2e" % e for e in errs], flush=True)
    assert all(e <= 1e-5 for e in errs), errs
