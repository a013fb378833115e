"""GPU parity of the chunk-averaged update rule (E2TTT_FLAG_CHUNK_AVERAGED;
the ablation baseline of Sec. 5, eqs. (4)-(6) with mean momentum and decay)
against its fp64 oracle (oracle/averaged.py).

The rule changes only the scalar kernels (K^W = K^M = eta, carries from the
chunk means); the chain kernels are the ones the closed form runs.  Bars as
for the closed form: rel-L2 1e-5 for fp32 io, 2e-2 for bf16 io, on outputs,
state deltas and every gradient; the coefficients themselves: K^W and K^M
equal eta bit for bit, the means within a few fp32 roundings.
"""
import numpy as np
import pytest
import torch

from oracle import averaged as A
from paper_2608_21308_amd import e2ttt, workloads as WL
from tests.gpu_util import TOL, config_of, parity_errors, tile_of, to_dev

pytestmark = pytest.mark.gpu

AVG = e2ttt.FLAG_CHUNK_AVERAGED
GRADS = ("dq", "dk", "dv", "d_eta", "d_beta", "d_gamma", "d_w_in", "d_m_in")


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    e2ttt.load()


@pytest.mark.parametrize("T,C", [(64, 64), (100, 16), (37, 7), (5, 1)])
@pytest.mark.parametrize("with_gamma", [True, False])
def test_averaged_coefficients(T, C, with_gamma):
    w = WL.WORKLOADS[0].with_(B=2, H=3, T=T, C=C)
    x = WL.make_inputs(w, with_grads=False)
    if not with_gamma:
        x["gamma"] = None
    cfg = config_of(w, flags=AVG)
    t = to_dev(x, w.io)
    kw, km, carry = e2ttt.chunk_coeffs(cfg, t["eta"], t["beta"], t["gamma"])
    torch.cuda.synchronize()
    assert torch.equal(kw, t["eta"]) and torch.equal(km, t["eta"])
    carry = carry.cpu().numpy().astype(np.float64)
    NC = cfg.n_chunks
    for r in range(NC):
        sl = slice(r * C, min(T, (r + 1) * C))
        b_bar = x["beta"][:, :, sl].astype(np.float64).mean(axis=2)
        g_bar = (x["gamma"][:, :, sl].astype(np.float64).mean(axis=2) if with_gamma
                 else np.ones_like(b_bar))
        for col, want in ((0, g_bar), (1, b_bar), (2, b_bar)):
            np.testing.assert_allclose(carry[:, :, r, col], want, rtol=1e-6)


def run_gpu(w, x, flags):
    cfg = config_of(w, flags=flags)
    t = to_dev(x, w.io)
    out, wo, mo, ws = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                    t["w_in"], t.get("m_in"), save_for_backward=True)
    g = e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                       t.get("m_in"), ws, t["d_out"], t.get("d_w_out"), t.get("d_m_out"))
    torch.cuda.synchronize()
    return dict(out=out, w_out=wo, m_out=mo, **g)


def run_oracle(w, x, flags):
    args = (x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], x.get("m_in"))
    kw = dict(C=w.C, fw=w.fw, dh=w.dh, flags=flags & e2ttt.FLAG_NO_RESIDUAL_LN)
    out, wo, mo = A.forward(*args, **kw)
    g = A.backward(*args, x["d_out"], x.get("d_w_out"), x.get("d_m_out"), **kw)
    return dict(out=out, w_out=wo, m_out=mo, **g)


def compare(w, x, flags, what):
    got = run_gpu(w, x, flags | AVG)
    ref = run_oracle(w, x, flags)
    pairs = {}
    for n, r in ref.items():
        if r is None:
            assert got[n] is None, n
            continue
        a = got[n].float().cpu().numpy()
        if n == "w_out":      # the state moves little: compare its change
            pairs[n] = (a - x["w_in"], r - x["w_in"], "state")
        elif n in ("m_out", "d_w_in", "d_m_in"):
            pairs[n] = (a, r, "state")
        else:
            pairs[n] = (a, r)
    errs = parity_errors(pairs, tile_of(w.C))
    tol = TOL[w.io]
    print(what, {k: "%.2e" % v for k, v in errs.items()}, flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, "%s rel-L2 above %g: %s" % (what, tol, bad)


def with_state(x, seed, m_scale):
    rng = np.random.default_rng(seed)
    x = dict(x)
    x["m_in"] = (m_scale * rng.standard_normal(x["w_in"].shape)).astype(np.float32)
    x["d_w_out"] = rng.standard_normal(x["w_in"].shape).astype(np.float32)
    x["d_m_out"] = rng.standard_normal(x["w_in"].shape).astype(np.float32)
    return x


@pytest.mark.parametrize("fw", [WL.FW_MLP, WL.FW_SWIGLU])
@pytest.mark.parametrize("T,C,flags", [(40, 16, 0), (37, 7, 0), (48, 16, 1)])
def test_averaged_rule_fp32(fw, T, C, flags):
    w = WL.WORKLOADS[0].with_(fw=fw, B=2, H=2, T=T, C=C, backward=True, seed=900 + T + C)
    x = with_state(WL.make_inputs(w), T, 1e-3)
    compare(w, x, flags, "avg fp32 fw=%d T=%d C=%d flags=%d" % (fw, T, C, flags))


def test_averaged_rule_fp32_without_gamma():
    w = WL.WORKLOADS[0].with_(B=1, H=2, T=40, C=16, backward=True, seed=950)
    x = WL.make_inputs(w)
    x["gamma"] = None
    compare(w, x, 0, "avg fp32 gamma=None")


@pytest.mark.parametrize("fw,dh", [(WL.FW_MLP, 256), (WL.FW_MLP, 64), (WL.FW_SWIGLU, 172)])
def test_averaged_rule_bf16(fw, dh):
    w = WL.WORKLOADS[1].with_(fw=fw, B=1, H=2, T=150, C=64, dh=dh, backward=True, seed=960 + dh)
    x = with_state(WL.make_inputs(w), dh, 1e-2)
    compare(w, x, 0, "avg bf16 fw=%d dh=%d" % (fw, dh))
