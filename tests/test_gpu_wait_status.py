"""The bounded waits between the workgroups of a unit report an expiry.

Units whose net is split over several workgroups swap partial sums through
global memory and wait for each other with a bounded poll; a wait that gives
up marks a status word, poisons the group so that every rank stops waiting,
and lets the grid drain.  e2ttt_wait_status reads that word.  Here the host
makes the waits give up by setting their limit to zero (E2TTT_WAIT_LIMIT_US=0,
read at every call): every kernel still runs to its end, nothing faults, the
status reports the expiry, and the next call with the normal limit is correct
again.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2608_21308_amd import e2ttt, workloads as WL
from tests.gpu_util import TOL, config_of, parity_errors, tile_of, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    e2ttt.load()


def fwd_bwd(cfg, t, scratch):
    out, wo, mo, ws = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                    t["w_in"], None, save_for_backward=True)
    g = e2ttt.backward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                       None, ws, t["d_out"], scratch=scratch)
    return out, wo, mo, ws, g


# GELU MLP dh 256 on two workgroups per unit; SwiGLU dh 172 on three
@pytest.mark.parametrize("fw,dh", [(WL.FW_MLP, 256), (WL.FW_SWIGLU, 172)])
def test_expired_waits_are_reported(fw, dh, monkeypatch):
    # the status word as a caller reads it after asynchronous calls (without
    # E2TTT_DEBUG_SYNC, which makes the call itself report the expiry: below)
    monkeypatch.delenv("E2TTT_DEBUG_SYNC", raising=False)
    w = WL.WORKLOADS[3].with_(fw=fw, dh=dh, B=8, H=16, T=512, seed=3300 + dh)
    x = WL.make_inputs(w)
    cfg = config_of(w)
    t = to_dev(x, "bf16")
    scratch = torch.empty(e2ttt.backward_scratch_bytes(cfg), dtype=torch.uint8, device="cuda")
    # normal limit: no expiry
    _, _, _, ws, _ = fwd_bwd(cfg, t, scratch)
    assert e2ttt.wait_status(cfg, workspace=ws, scratch=scratch) == 0
    # zero limit: every wait gives up at once
    monkeypatch.setenv("E2TTT_WAIT_LIMIT_US", "0")
    _, _, _, ws0, _ = fwd_bwd(cfg, t, scratch)
    st_f = e2ttt.wait_status(cfg, workspace=ws0)
    st_b = e2ttt.wait_status(cfg, scratch=scratch)
    torch.cuda.synchronize()
    print("zero wait limit: forward status %d, backward status %d" % (st_f, st_b), flush=True)
    assert st_f == 6 and st_b == 6
    # the normal limit again: status clear, results right (sampled units)
    monkeypatch.delenv("E2TTT_WAIT_LIMIT_US")
    out, wo, mo, ws1, g = fwd_bwd(cfg, t, scratch)
    assert e2ttt.wait_status(cfg, workspace=ws1, scratch=scratch) == 0
    units = [0, 127]
    xs = WL.make_inputs(w, units=units)
    ro, rw, rm = oracle.forward(xs["q"], xs["k"], xs["v"], xs["eta"], xs["beta"], xs["gamma"],
                                xs["w_in"], None, C=w.C, fw=fw, dh=dh)
    flat = lambda a: a.reshape((w.B * w.H,) + a.shape[2:])[units][None]
    errs = parity_errors({"out": (flat(out), ro), "w_out": (flat(wo), rw, "state"),
                          "m_out": (flat(mo), rm, "state")}, tile_of(w.C))
    print("after the expiry", {k: "%.2e" % v for k, v in errs.items()}, flush=True)
    if fw == WL.FW_MLP:   # (the SwiGLU + LN trajectory is chaotic over 8 chunks)
        assert all(e <= TOL["bf16"] for e in errs.values()), errs
    assert torch.isfinite(out.float()).all()


def test_debug_sync_reports_the_expiry_from_the_call(monkeypatch):
    # with E2TTT_DEBUG_SYNC=1 every call waits for its kernels and returns the
    # status word itself: an expired wait is the call's E2TTT_ERR_DEVICE (6)
    w = WL.WORKLOADS[3].with_(B=2, H=4, T=256, seed=3400)
    x = WL.make_inputs(w)
    cfg = config_of(w)
    t = to_dev(x, "bf16")
    monkeypatch.setenv("E2TTT_DEBUG_SYNC", "1")
    out, _, _, _ = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                 t["w_in"], None)
    assert torch.isfinite(out.float()).all()
    monkeypatch.setenv("E2TTT_WAIT_LIMIT_US", "0")
    with pytest.raises(e2ttt.E2TTTError) as err:
        e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"], None)
    assert err.value.status == 6
    torch.cuda.synchronize()


def test_single_workgroup_units_have_no_waits():
    w = WL.WORKLOADS[1].with_(B=1, H=2, T=128, dh=64)
    cfg = config_of(w)
    t = to_dev(WL.make_inputs(w, with_grads=False), "bf16")
    _, _, _, ws = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"],
                                t["w_in"], None)
    assert e2ttt.wait_status(cfg, workspace=ws) == 0
