"""e2ttt_chunk_forward_static: the forward on the library's own workspace,
for callers that cannot allocate.  Its outputs must equal those of
e2ttt_chunk_forward on a caller-owned workspace bit for bit (same kernels,
same inputs), on consecutive calls that reuse the array, the second with a
smaller input; a descriptor too large for the array is refused before any
launch."""
import numpy as np
import pytest
import torch

from paper_2608_21308_amd import e2ttt, workloads as WL
from tests.gpu_util import config_of, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    e2ttt.load()


def both(w, m_scale=0.0):
    x = WL.make_inputs(w, with_grads=False)
    cfg = config_of(w)
    t = to_dev(x, w.io)
    m_in = None
    if m_scale:
        m_in = torch.from_numpy((m_scale * np.random.default_rng(1).standard_normal(
            x["w_in"].shape)).astype(np.float32)).cuda()
    ref = e2ttt.forward(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                        m_in)[:3]
    got = tuple(torch.full_like(r, float("nan")) for r in ref)
    e2ttt.forward_static(cfg, t["q"], t["k"], t["v"], t["eta"], t["beta"], t["gamma"], t["w_in"],
                         m_in, *got)
    torch.cuda.synchronize()
    return got, ref


def test_static_workspace_forward_equals_the_workspace_forward():
    # the headline layer shape (two workgroups per unit), then a smaller
    # SwiGLU shape on three workgroups per unit and a ragged fp32 one, all
    # on the same array
    cases = [WL.WORKLOADS[3],
             WL.WORKLOADS[2].with_(B=1, H=3, T=200),
             WL.WORKLOADS[0].with_(B=1, H=2, T=75, C=7)]
    for i, w in enumerate(cases):
        assert e2ttt.workspace_bytes(config_of(w), False) <= e2ttt.STATIC_WORKSPACE_BYTES
        got, ref = both(w, m_scale=1e-3 if i else 0.0)
        for n, a, b in zip(("out", "w_out", "m_out"), got, ref):
            assert torch.equal(a, b), (w.name, n)
        print("static workspace forward == workspace forward:", w.name, w.B, w.H, w.T, flush=True)


def test_static_workspace_forward_refuses_what_does_not_fit():
    w = WL.WORKLOADS[3].with_(B=64, T=8192)     # about 0.6 GB of workspace
    cfg = config_of(w)
    assert e2ttt.workspace_bytes(cfg, False) > e2ttt.STATIC_WORKSPACE_BYTES
    small = WL.WORKLOADS[3].with_(B=1, H=1, T=64)
    t = to_dev(WL.make_inputs(small, with_grads=False), "bf16")
    # validation fails before any pointer is used; the tensors only fill the slots
    lib = e2ttt.load()
    d = cfg.desc()
    p = lambda x: None if x is None else x.data_ptr()
    st = lib.e2ttt_chunk_forward_static(
        __import__("ctypes").byref(d), p(t["q"]), p(t["k"]), p(t["v"]), p(t["eta"]),
        p(t["beta"]), p(t["gamma"]), p(t["w_in"]), None, p(t["q"]), p(t["w_in"]), p(t["w_in"]),
        None)
    assert st == 4
