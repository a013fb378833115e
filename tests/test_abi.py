"""C ABI checks that run without a GPU: the library loads, exports every entry
point of include/e2ttt.h, sizes workspaces, and rejects bad arguments before
launching anything (no call here reaches a kernel)."""
import ctypes
import os
import re

import pytest

from paper_2608_21308_amd import e2ttt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return e2ttt.load()


def header_functions():
    src = open(os.path.join(ROOT, "include", "e2ttt.h")).read()
    return sorted(set(re.findall(r"\b(e2ttt_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_function(lib):
    names = header_functions()
    assert set(names) == set(e2ttt.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def desc(**kw):
    base = dict(B=2, H=4, T=2048, d=64, dh=256, chunk=64, fw=0, io=1, flags=0, ln_eps=1e-5)
    base.update(kw)
    return e2ttt.Desc(**base)


def test_sizes(lib):
    d = desc()
    assert lib.e2ttt_param_count(ctypes.byref(d)) == 2 * 64 * 256
    ws0 = lib.e2ttt_workspace_bytes(ctypes.byref(d), 0)
    ws1 = lib.e2ttt_workspace_bytes(ctypes.byref(d), 1)
    # per-token K^W, K^M and per-chunk carries; plus bf16 W and M checkpoints per chunk
    assert ws0 >= 2 * 8 * 2048 * 4 + 8 * 32 * 3 * 4
    assert ws1 >= ws0 + 8 * 32 * 2 * 2 * (2 * 64 * 256)
    assert lib.e2ttt_backward_scratch_bytes(ctypes.byref(d)) >= ws0
    d = desc(fw=1, dh=172)
    assert lib.e2ttt_param_count(ctypes.byref(d)) == 3 * 64 * 172


def test_post_norm_sizes(lib):
    # E2TTT_FLAG_POST_NORM (8): the workspace adds the target norms, the
    # exchange rows, one more checkpoint block per unit (the final state) and,
    # when saving, the norms before each chunk end's normalisation; the
    # backward scratch adds what flows into the targets and its exchange rows
    for kw in (dict(), dict(fw=1, dh=172), dict(d=128, dh=512), dict(io=0, d=16, dh=64)):
        d0, d8 = desc(**kw), desc(flags=8, **kw)
        U, T, C = d0.B * d0.H, d0.T, d0.chunk
        NC = (T + C - 1) // C
        R = (1 if d0.fw == 0 else 2) * d0.dh + d0.d
        ws0 = lib.e2ttt_workspace_bytes(ctypes.byref(d0), 1)
        ws8 = lib.e2ttt_workspace_bytes(ctypes.byref(d8), 1)
        assert ws8 >= ws0 + U * R * 4 + U * NC * R * 4, kw
        assert lib.e2ttt_workspace_bytes(ctypes.byref(d8), 0) >= \
            lib.e2ttt_workspace_bytes(ctypes.byref(d0), 0) + U * R * 4, kw
        assert lib.e2ttt_backward_scratch_bytes(ctypes.byref(d8)) >= \
            lib.e2ttt_backward_scratch_bytes(ctypes.byref(d0)) + U * R * 4, kw
        assert lib.e2ttt_param_count(ctypes.byref(d8)) == lib.e2ttt_param_count(ctypes.byref(d0))


@pytest.mark.parametrize("kw,status", [
    (dict(T=0), 2), (dict(B=-1), 2), (dict(chunk=0), 2), (dict(ln_eps=0.0), 2),
    (dict(chunk=513), 3), (dict(fw=2), 3), (dict(io=7), 3), (dict(flags=16), 3),
    (dict(flags=5), 2),
    (dict(d=32), 3), (dict(d=16), 3), (dict(dh=300), 3), (dict(fw=1, dh=200), 3),
    (dict(io=0, d=64), 3), (dict(io=0, d=16, dh=200), 3)])
def test_bad_descriptors(lib, kw, status):
    d = desc(**kw)
    assert lib.e2ttt_param_count(ctypes.byref(d)) == 0
    assert lib.e2ttt_workspace_bytes(ctypes.byref(d), 1) == 0
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    st = lib.e2ttt_chunk_forward(ctypes.byref(d), *([fake] * 12), 1 << 40, 0, None)
    assert st == status
    st = lib.e2ttt_chunk_backward(ctypes.byref(d), *([fake] * 9), 1 << 40, *([fake] * 12),
                                  1 << 40, None)
    assert st == status
    assert lib.e2ttt_apply(ctypes.byref(d), fake, fake, fake, None) == status


def test_null_and_workspace_errors(lib):
    d = desc()
    fake = ctypes.c_void_p(16)
    args = [fake] * 12
    assert lib.e2ttt_chunk_forward(None, *args, 1 << 40, 0, None) == 1
    for i in (0, 1, 2, 3, 4, 6, 8, 9, 10, 11):    # q k v eta beta w_in out w_out m_out workspace
        a = list(args)
        a[i] = None
        assert lib.e2ttt_chunk_forward(ctypes.byref(d), *a, 1 << 40, 0, None) == 1, i
    # gamma (5) and m_in (7) are optional: with a too-small workspace the call
    # gets past the pointer checks and stops at the size check
    a = list(args)
    a[5] = None
    a[7] = None
    ws = lib.e2ttt_workspace_bytes(ctypes.byref(d), 1)
    assert lib.e2ttt_chunk_forward(ctypes.byref(d), *a, ws - 1, 1, None) == 4
    # a workspace without checkpoints is too small for save_for_backward
    ws0 = lib.e2ttt_workspace_bytes(ctypes.byref(d), 0)
    assert lib.e2ttt_chunk_forward(ctypes.byref(d), *args, ws0, 1, None) == 4
    # state outputs aliasing the inputs are refused when saving for backward
    a = list(args)
    a[9] = a[6] = ctypes.c_void_p(32)
    assert lib.e2ttt_chunk_forward(ctypes.byref(d), *a, 1 << 40, 1, None) == 2
    # token tensors and buffers are moved as 16-byte vectors: misaligned ones are refused
    for i in (0, 1, 2, 8, 11):    # q k v out workspace
        a = list(args)
        a[i] = ctypes.c_void_p(18)
        assert lib.e2ttt_chunk_forward(ctypes.byref(d), *a, 1 << 40, 0, None) == 2, i
    # backward: d_gamma must be given iff gamma is
    bargs = [fake] * 9 + [1 << 40] + [fake] * 12 + [1 << 40, None]
    for i in (0, 1, 2, 8, 10, 13, 14, 15, 21):   # q k v workspace d_out dq dk dv scratch
        b = list(bargs)
        b[i] = ctypes.c_void_p(24)
        assert lib.e2ttt_chunk_backward(ctypes.byref(d), *b) == 2, i
    b = list(bargs)
    b[5] = None
    assert lib.e2ttt_chunk_backward(ctypes.byref(d), *b) == 2
    b = list(bargs)
    b[9] = ws - 1
    assert lib.e2ttt_chunk_backward(ctypes.byref(d), *b) == 4
    sc = lib.e2ttt_backward_scratch_bytes(ctypes.byref(d))
    b = list(bargs)
    b[-2] = sc - 1
    assert lib.e2ttt_chunk_backward(ctypes.byref(d), *b) == 4


def test_ln_affine_pointer_rules(lib):
    # E2TTT_FLAG_LN_AFFINE (4): the *_ln entry points need ln_weight / ln_bias
    # (and the backward their gradients); the plain ones have none to give;
    # without the flag the affine pointers must be NULL; ln arrays 16-byte aligned
    fake = ctypes.c_void_p(16)
    da = desc(flags=4)
    d0 = desc()
    args = [fake] * 12
    assert lib.e2ttt_chunk_forward(ctypes.byref(da), *args, 1 << 40, 0, None) == 1
    assert lib.e2ttt_chunk_forward_ln(ctypes.byref(da), None, fake, *args, 1 << 40, 0, None) == 1
    assert lib.e2ttt_chunk_forward_ln(ctypes.byref(d0), fake, fake, *args, 1 << 40, 0, None) == 2
    assert lib.e2ttt_chunk_forward_ln(ctypes.byref(da), ctypes.c_void_p(20), fake, *args,
                                      1 << 40, 0, None) == 2
    def bargs(dlw, dlb):   # ..., d_m_in, d_ln_weight, d_ln_bias, scratch, scratch_bytes, stream
        return [fake] * 9 + [1 << 40] + [fake] * 11 + [dlw, dlb, fake, 1 << 40, None]
    assert lib.e2ttt_chunk_backward_ln(ctypes.byref(da), fake, fake, *bargs(None, fake)) == 1
    assert lib.e2ttt_chunk_backward_ln(ctypes.byref(d0), None, None, *bargs(fake, None)) == 2
    assert lib.e2ttt_apply_ln(ctypes.byref(da), fake, None, fake, fake, fake, None) == 1
    assert lib.e2ttt_apply(ctypes.byref(da), fake, fake, fake, None) == 1
    # the scratch of an affine backward also holds the written rows and partial sums
    sa = lib.e2ttt_backward_scratch_bytes(ctypes.byref(da))
    s0 = lib.e2ttt_backward_scratch_bytes(ctypes.byref(d0))
    assert sa >= s0 + 2 * 4 * 2048 * 64 * 4


def test_status_strings(lib):
    seen = set()
    for s in range(7):
        txt = lib.e2ttt_status_str(s)
        assert txt and txt != b"unknown status"
        seen.add(txt)
    assert len(seen) == 7
    assert lib.e2ttt_status_str(7) == b"unknown status"


def test_split_workspace_sizes(lib):
    # the dh = 256 MLP runs two workgroups per unit: the workspace grows by the
    # exchange slots and sync words, the backward scratch by per-rank partials
    d = desc(B=8, H=16, T=4096)
    U, T, NC = 128, 4096, 64
    ws = lib.e2ttt_workspace_bytes(ctypes.byref(d), 0)
    ws_save = lib.e2ttt_workspace_bytes(ctypes.byref(d), 1)
    sc = lib.e2ttt_backward_scratch_bytes(ctypes.byref(d))
    tok = U * T * 4
    # forward slots per rank: two Y_K parities and one Y_Q, fp32 [C][d] each
    assert ws >= 2 * tok + U * NC * 3 * 4 + 128 * 2 * 3 * 64 * 64 * 4
    # checkpoints of W and M (bf16, both ranks) plus Z and 1/sigma of both passes
    assert ws_save - ws >= U * NC * 2 * 2 * 64 * 256 * 2 + 2 * (tok * 64 + tok)
    # backward slots per rank: two parities of the fp32 dYh partial and of the
    # bf16 dk, dq partials
    assert sc >= 2 * (2 * tok + U * NC * 3 * 4) + 128 * 2 * 2 * (64 * 64 * 4 + 2 * 64 * 64 * 2)


def test_gate_argument_errors(lib):
    """e2ttt_gates_forward / _backward validate everything before launching."""
    p = e2ttt.GateParams()
    f = ctypes.c_void_p(16)   # never dereferenced
    fwd, bwd = lib.e2ttt_gates_forward, lib.e2ttt_gates_backward
    assert fwd(None, 8, f, f, f, f, f, f, None) == 1
    assert fwd(ctypes.byref(p), -1, f, f, f, f, f, f, None) == 2
    assert fwd(ctypes.byref(p), 0, None, None, None, None, None, None, None) == 0   # no-op
    for i in range(4):                               # l_eta, l_beta, eta, beta
        a = [f, f, f, f, f, f]
        a[[0, 1, 3, 4][i]] = None
        assert fwd(ctypes.byref(p), 8, *a, None) == 1, i
    assert fwd(ctypes.byref(p), 8, f, f, None, f, f, f, None) == 1       # gamma without l_alpha
    assert fwd(ctypes.byref(p), 8, f, f, f, f, f, None, None) == 1       # l_alpha without gamma
    for bad in (e2ttt.GateParams(tau=0.0), e2ttt.GateParams(eta_base=-1.0),
                e2ttt.GateParams(alpha_base=float("nan")), e2ttt.GateParams(tau=float("inf"))):
        assert fwd(ctypes.byref(bad), 8, f, f, f, f, f, f, None) == 2
    b = [f] * 9
    assert bwd(None, 8, *b, None) == 1
    assert bwd(ctypes.byref(p), -3, *b, None) == 2
    for i in (0, 1, 3, 4, 6, 7):                     # l_eta l_beta d_eta d_beta d_l_eta d_l_beta
        a = list(b)
        a[i] = None
        assert bwd(ctypes.byref(p), 8, *a, None) == 1, i
    for i in (2, 5, 8):                              # the alpha side is all or nothing
        a = list(b)
        a[i] = None
        assert bwd(ctypes.byref(p), 8, *a, None) == 1, i


def test_binding_rejects_host_and_misshaped_tensors():
    """The Python binding refuses host tensors, wrong dtypes and wrong element
    counts before it reaches the library (a host pointer handed to a kernel
    would fault the GPU)."""
    import torch
    cfg = e2ttt.Config(1, 2, 32, 16, 64, 16, e2ttt.FW_MLP, e2ttt.DT_F32)
    io = torch.zeros(1, 2, 32, 16)
    g = torch.zeros(1, 2, 32)
    st = torch.zeros(1, 2, cfg.P)
    with pytest.raises(ValueError, match="device tensor"):
        e2ttt.forward(cfg, io, io, io, g, g, g, st, None)
    with pytest.raises(ValueError, match="device tensor"):
        e2ttt.backward(cfg, io, io, io, g, g, g, st, None, torch.zeros(8, dtype=torch.uint8), io)
    with pytest.raises(ValueError, match="device tensor"):
        e2ttt.chunk_coeffs(cfg, g, g, g)
    with pytest.raises(ValueError, match="device tensor"):
        e2ttt.gates_forward(e2ttt.GateParams(), g, g, g)
    with pytest.raises(ValueError, match="device tensor"):
        e2ttt.gates_backward(e2ttt.GateParams(), g, g, g, g, g, g)
    # element type and count by role, checked before the device
    for kw in (dict(q=io.to(torch.bfloat16)), dict(k=io[..., :8].contiguous()),
               dict(eta=io), dict(w_in=g), dict(d_w_in=st.double()),
               dict(workspace=torch.zeros(4))):
        with pytest.raises(ValueError, match="expected"):
            e2ttt._check_tensors(cfg, **kw)
    with pytest.raises(ValueError, match="contiguous"):
        e2ttt._check_tensors(cfg, q=torch.zeros(1, 2, 16, 32).transpose(2, 3))
    with pytest.raises(ValueError, match="device tensor"):
        e2ttt._check_tensors(cfg, q=io, eta=g, w_in=st, workspace=torch.zeros(4, dtype=torch.uint8))


def test_apply_argument_errors(lib):
    d = desc()
    f = ctypes.c_void_p(256)   # never dereferenced
    assert lib.e2ttt_apply(None, f, f, f, None) == 1
    for i in range(3):
        a = [f, f, f]
        a[i] = None
        assert lib.e2ttt_apply(ctypes.byref(d), *a, None) == 1, i
    # the state is read as float4: a pointer that is not 16-byte aligned is refused
    assert lib.e2ttt_apply(ctypes.byref(d), f, ctypes.c_void_p(260), f, None) == 2


def test_long_chunks(lib):
    """Chunks of 65..512 tokens run on every variant, forward and backward;
    above 512 the call is refused before any launch."""
    f = ctypes.c_void_p(16)   # never dereferenced
    for kw in (dict(chunk=128), dict(chunk=512), dict(io=0, d=16, dh=64, chunk=200)):
        d = desc(**kw)
        assert lib.e2ttt_param_count(ctypes.byref(d)) > 0
        ws0 = lib.e2ttt_workspace_bytes(ctypes.byref(d), 0)
        ws1 = lib.e2ttt_workspace_bytes(ctypes.byref(d), 1)
        assert 0 < ws0 < ws1
        short = desc(**dict(kw, chunk=64))
        # the backward scratch adds two fp32 copies of each workgroup's state share
        assert (lib.e2ttt_backward_scratch_bytes(ctypes.byref(d)) >
                lib.e2ttt_backward_scratch_bytes(ctypes.byref(short)))
    # SwiGLU on bf16: the forward workspace also holds every workgroup's copy
    # of W_0 (fp32) for the chunk's later tiles
    d = desc(fw=1, dh=172, chunk=512)
    short = desc(fw=1, dh=172, chunk=64)
    assert (lib.e2ttt_workspace_bytes(ctypes.byref(d), 0) >
            lib.e2ttt_workspace_bytes(ctypes.byref(short), 0) + 3 * 64 * 64 * 4)
    assert lib.e2ttt_backward_scratch_bytes(ctypes.byref(d)) > 0
    d = desc(fw=1, dh=172, chunk=513)
    assert lib.e2ttt_workspace_bytes(ctypes.byref(d), 0) == 0
    assert lib.e2ttt_backward_scratch_bytes(ctypes.byref(d)) == 0
    assert lib.e2ttt_chunk_forward(ctypes.byref(d), *([f] * 12), 1 << 40, 0, None) == 3
    assert lib.e2ttt_chunk_backward(ctypes.byref(d), *([f] * 9), 1 << 40, *([f] * 12),
                                    1 << 40, None) == 3
