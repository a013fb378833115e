"""The float32 reference that sizes the fp32 bars (tests/fp32ref.py) computes
the same thing as the oracle: evaluated in float64 it reproduces the oracle's
token recurrence (Prop. 1) to round-off, forward and backward, for both nets,
ragged chunks, with and without the decay gate, with the bare net, and with
the post-chunk normalisation of the fast weights (flag 8)."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2608_21308_amd import workloads as WL
from tests import fp32ref
from tests.gpu_util import rel_l2


@pytest.mark.parametrize("fw", [WL.FW_MLP, WL.FW_SWIGLU])
@pytest.mark.parametrize("T,C,flags,gamma", [(40, 16, 0, True), (23, 7, 0, False),
                                             (30, 30, 1, True), (5, 1, 0, True),
                                             (40, 16, 8, True), (23, 7, 9, False)])
def test_fp64_closed_form_equals_the_oracle(fw, T, C, flags, gamma):
    w = WL.WORKLOADS[0].with_(fw=fw, B=1, H=2, T=T, C=C, dh=24, backward=True, seed=40 + T)
    x = WL.make_inputs(w)
    rng = np.random.default_rng(T)
    if not gamma:
        x["gamma"] = None
    x["m_in"] = (1e-2 * rng.standard_normal(x["w_in"].shape)).astype(np.float32)
    x["d_w_out"] = rng.standard_normal(x["w_in"].shape).astype(np.float32)
    x["d_m_out"] = rng.standard_normal(x["w_in"].shape).astype(np.float32)
    args = (x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], x["m_in"])
    ro = oracle.forward(*args, C=C, fw=fw, dh=w.dh, flags=flags)
    fo = fp32ref.forward(x, C=C, fw=fw, dh=w.dh, flags=flags, dtype=torch.float64)
    for a, b in zip(fo, ro):
        assert rel_l2(a, b) < 1e-12
    rb = oracle.backward(*args, x["d_out"], x["d_w_out"], x["d_m_out"], C=C, fw=fw, dh=w.dh,
                         flags=flags)
    fb = fp32ref.backward(x, C=C, fw=fw, dh=w.dh, flags=flags, dtype=torch.float64)
    for n, r in rb.items():
        if r is None:
            assert fb[n] is None
            continue
        assert rel_l2(fb[n], r) < 1e-12, n


def test_fp32_evaluation_is_fp32_accurate():
    # in float32 it lands within a few float32 roundings of the oracle on a
    # well-conditioned case (so that FP32_FACTOR times its error is a bar that
    # a correct fp32 kernel can meet)
    w = WL.WORKLOADS[0].with_(B=1, H=2, T=64, C=16, backward=False, seed=9)
    x = WL.make_inputs(w)
    ro = oracle.forward(x["q"], x["k"], x["v"], x["eta"], x["beta"], x["gamma"], x["w_in"], None,
                        C=w.C, fw=w.fw, dh=w.dh)
    fo = fp32ref.forward(x, C=w.C, fw=w.fw, dh=w.dh)
    errs = [rel_l2(a, b) for a, b in zip(fo, ro)]
    assert all(1e-9 < e < 1e-5 for e in errs), errs


@pytest.mark.parametrize("fw", [WL.FW_MLP, WL.FW_SWIGLU])
def test_fp64_closed_form_with_affine_equals_the_oracle(fw):
    from tests.test_ln_affine_oracle import problem
    x, ln, g = problem(2, 2, 9, 4, 6, fw, 21 + fw)
    pair = (ln["ln_a"], ln["ln_b"])
    for a, b in zip(fp32ref.forward(x, C=4, fw=fw, dh=6, dtype=torch.float64, ln=pair),
                    oracle.forward(**x, C=4, fw=fw, dh=6, **ln)):
        assert rel_l2(a, b) < 1e-12
    ref = oracle.backward(**x, **g, C=4, fw=fw, dh=6, **ln)
    got = fp32ref.backward(dict(x, **g), C=4, fw=fw, dh=6, dtype=torch.float64, ln=pair)
    for n, r in ref.items():
        assert rel_l2(got[n], r) < 1e-12, n
