"""GPU parity of the learnable LayerNorm affine (E2TTT_FLAG_LN_AFFINE):
f(x) = x + a * LN(y) + b with a, b per head, through the forward, the
backward (every input gradient plus those of a and b, summed over the batch)
and the net evaluation, against the fp64 oracle.

Bars as everywhere: rel-L2 2e-2 for bf16 io with the local maxima of
gpu_util.parity_errors; for fp32 io 1e-5, widened only where the float32
evaluation of tests/fp32ref.py (which carries the same affine) is itself
farther from the oracle.  The affine's gradients are [H, d] per-head tensors,
checked per head like a unit's state.  Affine draws: a = 1 + 0.3 N(0, 1),
b = 0.2 N(0, 1) per head and column.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2608_21308_amd import e2ttt, workloads as WL
from tests import fp32ref
from tests.gpu_util import TOL, config_of, parity_errors, tile_of, to_dev

pytestmark = pytest.mark.gpu

AFF = e2ttt.FLAG_LN_AFFINE
GRADS = ("dq", "dk", "dv", "d_eta", "d_beta", "d_gamma", "d_w_in", "d_m_in")


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    e2ttt.load()


def affine(H, d, seed):
    rng = np.random.default_rng(seed)
    return ((1.0 + 0.3 * rng.standard_normal((H, d))).astype(np.float32),
            (0.2 * rng.standard_normal((H, d))).astype(np.float32))


def with_state(x, seed, m_scale):
    rng = np.random.default_rng(seed)
    x = dict(x)
    x["m_in"] = (m_scale * rng.standard_normal(x["w_in"].shape)).astype(np.float32)
    x["d_w_out"] = rng.standard_normal(x["w_in"].shape).astype(np.float32)
    x["d_m_out"] = rng.standard_normal(x["w_in"].shape).astype(np.float32)
    return x


def run_gpu(w, x, ln, backward):
    cfg = config_of(w, flags=AFF)
    t = to_dev(x, w.io)
    la = torch.from_numpy(ln[0]).cuda()
    lb = torch.from_numpy(ln[1]).cuda()
    out, wo, mo, ws = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                    t["w_in"], t.get("m_in"), save_for_backward=backward,
                                    ln_weight=la, ln_bias=lb)
    res = dict(out=out, w_out=wo, m_out=mo)
    if backward:
        res.update(e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                  t["w_in"], t.get("m_in"), ws, t["d_out"], t.get("d_w_out"),
                                  t.get("d_m_out"), ln_weight=la, ln_bias=lb))
    torch.cuda.synchronize()
    return {n: None if v is None else v.float().cpu().numpy() for n, v in res.items()}


def run_oracle(w, x, ln, backward):
    args = (x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], x.get("m_in"))
    out, wo, mo = oracle.forward(*args, C=w.C, fw=w.fw, dh=w.dh, ln_a=ln[0], ln_b=ln[1])
    res = dict(out=out, w_out=wo, m_out=mo)
    if backward:
        res.update(oracle.backward(*args, x["d_out"], x.get("d_w_out"), x.get("d_m_out"), C=w.C,
                                   fw=w.fw, dh=w.dh, ln_a=ln[0], ln_b=ln[1]))
        res["d_ln_weight"] = res.pop("d_ln_a")
        res["d_ln_bias"] = res.pop("d_ln_b")
    return res


def errors(got, ref, x, C):
    pairs = {}
    for n, r in ref.items():
        if r is None:
            assert got.get(n) is None, n
            continue
        a = got[n]
        if n == "w_out":
            pairs[n] = (a - x["w_in"], r - x["w_in"], "state")
        elif n in ("m_out", "d_w_in", "d_m_in"):
            pairs[n] = (a, r, "state")
        elif n in ("d_ln_weight", "d_ln_bias"):
            pairs[n] = (a[None], r[None], "state")        # one block per head
        else:
            pairs[n] = (a, r)
    return parity_errors(pairs, tile_of(C))


def check(errs, bound, what):
    print(what, {k: "%.2e" % v for k, v in errs.items()}, flush=True)
    bad = {n: (e, bound[n] if isinstance(bound, dict) else bound) for n, e in errs.items()
           if not e <= (bound[n] if isinstance(bound, dict) else bound)}
    assert not bad, what + ": %s" % bad


# ------------------------------------------------------------------ fp32
@pytest.mark.parametrize("fw", [WL.FW_MLP, WL.FW_SWIGLU])
@pytest.mark.parametrize("T,C,dh", [(40, 16, 64), (23, 7, 50), (150, 65, 64)])
def test_affine_fp32(fw, T, C, dh):
    w = WL.WORKLOADS[0].with_(fw=fw, B=2, H=2, T=T, C=C, dh=dh, backward=True, seed=4000 + T + dh)
    x = with_state(WL.make_inputs(w), T, 1e-3)
    ln = affine(w.H, w.d, T)
    got = run_gpu(w, x, ln, True)
    ref = run_oracle(w, x, ln, True)
    errs = errors(got, ref, x, C)
    f32 = dict(zip(("out", "w_out", "m_out"), fp32ref.forward(x, C=C, fw=fw, dh=dh, ln=ln)))
    g32 = fp32ref.backward(x, C=C, fw=fw, dh=dh, ln=ln)
    f32.update(g32)
    f32["d_ln_weight"] = f32.pop("d_ln_a")
    f32["d_ln_bias"] = f32.pop("d_ln_b")
    check(errs, fp32ref.fp32_bar(errors(f32, ref, x, C)),
          "affine fp32 fw=%d T=%d C=%d dh=%d" % (fw, T, C, dh))


# ------------------------------------------------------------------ bf16
@pytest.mark.parametrize("fw,d,dh,T,C", [
    (WL.FW_MLP, 64, 64, 200, 64),        # one workgroup per unit
    (WL.FW_MLP, 64, 256, 200, 64),       # two (the headline net)
    (WL.FW_SWIGLU, 64, 172, 130, 64),    # three
    (WL.FW_MLP, 64, 256, 600, 512),      # chunks of eight tiles
    (WL.FW_MLP, 128, 256, 130, 64),      # head dim 128 on four workgroups
])
def test_affine_bf16(fw, d, dh, T, C):
    base = WL.WORKLOADS[1] if d == 64 else WL.PAPER_1P3B
    w = base.with_(fw=fw, B=2, H=2, T=T, C=C, dh=dh, backward=True, seed=4100 + T + dh)
    x = with_state(WL.make_inputs(w), T, 1e-2)
    ln = affine(w.H, w.d, dh)
    ref = run_oracle(w, x, ln, True)
    errs = errors(run_gpu(w, x, ln, True), ref, x, C)
    what = "affine bf16 fw=%d d=%d dh=%d T=%d C=%d" % (fw, d, dh, T, C)
    if fw == WL.FW_SWIGLU:
        # SwiGLU with the residual LayerNorm is ill-conditioned over several
        # chunks (its trajectories are chaotic under these inputs): the bar is
        # widened by the case's own conditioning, as in the chunk-window tests,
        # to twice the oracle's change when its initial state is rounded to
        # bf16 once (measured here: dq 2.6e-2 with the affine, 1.8e-3 without)
        xb = dict(x, w_in=WL.round_bf16(x["w_in"]), m_in=WL.round_bf16(x["m_in"]))
        sens = errors(run_oracle(w, xb, ln, True), ref, x, C)
        bound = {n: max(TOL["bf16"], 2 * sens[n.split("/")[0]]) for n in errs}
        print(what, "bf16-state sensitivity", {k: "%.1e" % v for k, v in sens.items()
                                               if "/" not in k}, flush=True)
        check(errs, bound, what)
    else:
        check(errs, TOL["bf16"], what)


def test_affine_identity_equals_plain_path():
    # a = 1, b = 0: the affine path computes what the plain path does (every
    # product with a is by 1, every sum with b adds 0), on the headline net; the
    # two branches are compiled with different fused multiply-adds, so they
    # agree to rounding (measured: w_out differs in 519 of 131,072 values, by at
    # most 7.9e-6 absolute), not bit for bit
    w = WL.WORKLOADS[1].with_(B=2, H=2, T=130, dh=256, backward=True, seed=4200)
    x = WL.make_inputs(w)
    ln = (np.ones((w.H, w.d), np.float32), np.zeros((w.H, w.d), np.float32))
    got = run_gpu(w, x, ln, True)
    cfg = config_of(w)
    t = to_dev(x, "bf16")
    out, wo, mo, ws = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                    t["w_in"], None, save_for_backward=True)
    g = e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                       None, ws, t["d_out"])
    torch.cuda.synchronize()
    plain = dict(out=out, w_out=wo, m_out=mo, **g)
    for n in ("out", "w_out", "m_out") + GRADS:
        b = plain[n].float().cpu().numpy()
        e = float(np.linalg.norm(got[n] - b) / np.linalg.norm(b))
        assert e <= 1e-4, (n, e)


def test_affine_apply_and_decode_bf16():
    # the net evaluation with the affine (decode), d = 64 and d = 128
    for w in (WL.WORKLOADS[1].with_(B=2, H=3, T=13, dh=256),
              WL.PAPER_1P3B.with_(fw=WL.FW_SWIGLU, B=2, H=3, T=5, dh=344)):
        x = WL.make_inputs(w, with_grads=False)
        ln = affine(w.H, w.d, 7)
        cfg = config_of(w, flags=AFF)
        t = to_dev(x, "bf16")
        got = e2ttt.apply(cfg, t["q"], t["w_in"], ln_weight=torch.from_numpy(ln[0]).cuda(),
                          ln_bias=torch.from_numpy(ln[1]).cuda()).float().cpu().numpy()
        ref = np.stack([np.stack([oracle.net(x["w_in"][b, h], x["q"][b, h], fw=w.fw, dh=w.dh,
                                             ln_a=ln[0][h], ln_b=ln[1][h])
                                  for h in range(w.H)]) for b in range(w.B)])
        e = np.abs(got - ref)
        ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7)
        bound = ulp + 1e-6 * (np.abs(x["q"]) + np.abs(ref) + 1.0)
        assert np.all(e <= bound), float(np.max(e / bound))
