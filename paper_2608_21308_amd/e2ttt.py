"""ctypes binding of libe2ttt.so (the HIP implementation, C ABI in include/e2ttt.h).

Argument marshalling only: tensors are passed as device pointers together with
the current HIP stream; every step of the computation runs in the library's
kernels.  PyTorch provides device memory and streams.  Importing this module
on a machine without the built library raises immediately.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libe2ttt.so")

FW_MLP = 0
FW_SWIGLU = 1
DT_F32 = 0
DT_BF16 = 1
FLAG_NO_RESIDUAL_LN = 1
FLAG_CHUNK_AVERAGED = 2
FLAG_LN_AFFINE = 4
FLAG_POST_NORM = 8       # post-chunk L2 normalisation of the fast-weight rows (App. B.1)

STATUS = {0: "ok", 1: "null argument", 2: "bad shape", 3: "unsupported",
          4: "workspace too small", 5: "HIP error", 6: "device-side wait expired"}

# Every entry point the header declares (checked by the CPU test-suite).
EXPORTS = ("e2ttt_param_count", "e2ttt_workspace_bytes", "e2ttt_backward_scratch_bytes",
           "e2ttt_chunk_forward", "e2ttt_chunk_backward", "e2ttt_chunk_coeffs",
           "e2ttt_apply", "e2ttt_gates_forward", "e2ttt_gates_backward", "e2ttt_wait_status",
           "e2ttt_chunk_forward_static", "e2ttt_chunk_forward_ln", "e2ttt_chunk_backward_ln",
           "e2ttt_apply_ln", "e2ttt_status_str")


class E2TTTError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, STATUS.get(status, "?"), status))


class Desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("T", ctypes.c_int32),
                ("d", ctypes.c_int32), ("dh", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("fw", ctypes.c_int32), ("io", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("ln_eps", ctypes.c_float)]


class GateParams(ctypes.Structure):
    """e2ttt_gate_params (the paper's defaults, App. B.1)."""
    _fields_ = [("eta_base", ctypes.c_float), ("alpha_base", ctypes.c_float),
                ("tau", ctypes.c_float)]

    def __init__(self, eta_base=0.01, alpha_base=0.1, tau=32.0):
        super().__init__(eta_base, alpha_base, tau)


_lib = None


def load():
    """Load the in-tree HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libe2ttt.so is not built (run __graft_entry__.build() or "
                          "python paper_2608_21308_amd/build_lib.py)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz, i = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    dp = ctypes.POINTER(Desc)
    lib.e2ttt_param_count.argtypes = [dp]
    lib.e2ttt_param_count.restype = sz
    lib.e2ttt_workspace_bytes.argtypes = [dp, i]
    lib.e2ttt_workspace_bytes.restype = sz
    lib.e2ttt_backward_scratch_bytes.argtypes = [dp]
    lib.e2ttt_backward_scratch_bytes.restype = sz
    lib.e2ttt_chunk_forward.argtypes = [dp] + [vp] * 12 + [sz, i, vp]
    lib.e2ttt_chunk_forward.restype = i
    lib.e2ttt_chunk_backward.argtypes = [dp] + [vp] * 9 + [sz] + [vp] * 12 + [sz, vp]
    lib.e2ttt_chunk_backward.restype = i
    lib.e2ttt_chunk_coeffs.argtypes = [dp] + [vp] * 7
    lib.e2ttt_chunk_coeffs.restype = i
    lib.e2ttt_apply.argtypes = [dp] + [vp] * 4
    lib.e2ttt_apply.restype = i
    gp = ctypes.POINTER(GateParams)
    lib.e2ttt_gates_forward.argtypes = [gp, ctypes.c_int64] + [vp] * 7
    lib.e2ttt_gates_forward.restype = i
    lib.e2ttt_gates_backward.argtypes = [gp, ctypes.c_int64] + [vp] * 10
    lib.e2ttt_gates_backward.restype = i
    lib.e2ttt_wait_status.argtypes = [dp, vp, vp, vp]
    lib.e2ttt_wait_status.restype = i
    lib.e2ttt_chunk_forward_static.argtypes = [dp] + [vp] * 12
    lib.e2ttt_chunk_forward_static.restype = i
    lib.e2ttt_chunk_forward_ln.argtypes = [dp] + [vp] * 14 + [sz, i, vp]
    lib.e2ttt_chunk_forward_ln.restype = i
    lib.e2ttt_chunk_backward_ln.argtypes = [dp] + [vp] * 11 + [sz] + [vp] * 14 + [sz, vp]
    lib.e2ttt_chunk_backward_ln.restype = i
    lib.e2ttt_apply_ln.argtypes = [dp] + [vp] * 6
    lib.e2ttt_apply_ln.restype = i
    lib.e2ttt_status_str.argtypes = [i]
    lib.e2ttt_status_str.restype = ctypes.c_char_p
    _lib = lib
    return lib


@dataclass(frozen=True)
class Config:
    B: int
    H: int
    T: int
    d: int
    dh: int
    chunk: int
    fw: int = FW_MLP
    io: int = DT_BF16
    flags: int = 0
    ln_eps: float = 1e-5

    def desc(self) -> Desc:
        return Desc(self.B, self.H, self.T, self.d, self.dh, self.chunk, self.fw, self.io,
                    self.flags, self.ln_eps)

    @property
    def P(self) -> int:
        return (2 if self.fw == FW_MLP else 3) * self.d * self.dh

    @property
    def n_chunks(self) -> int:
        return (self.T + self.chunk - 1) // self.chunk

    @property
    def torch_io(self):
        return torch.bfloat16 if self.io == DT_BF16 else torch.float32


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(st: int, where: str):
    if st != 0:
        raise E2TTTError(st, where)


_IO = ("q", "k", "v", "out", "d_out", "dq", "dk", "dv")
_GATE = ("eta", "beta", "gamma", "d_eta", "d_beta", "d_gamma", "kw", "km")
_STATE = ("w_in", "m_in", "w_out", "m_out", "d_w_in", "d_m_in", "d_w_out", "d_m_out")
_HEAD = ("ln_weight", "ln_bias", "d_ln_weight", "d_ln_bias")


def _check_tensors(cfg: Config, **ts):
    """Host-side guard before any launch: every tensor the library will read or
    write is a contiguous device tensor on the device of the first one, with
    the element type and element count the header gives for its role.  The
    library itself checks only sizes it is handed (workspace, scratch)."""
    dev = None
    n_tok = cfg.B * cfg.H * cfg.T
    for name, t in ts.items():
        if t is None:
            continue
        if not isinstance(t, torch.Tensor) or not t.is_contiguous():
            raise ValueError("%s must be a contiguous tensor" % name)
        if name in _IO:
            want = (cfg.torch_io, n_tok * cfg.d)
        elif name in _GATE:
            want = (torch.float32, n_tok)
        elif name in _STATE:
            want = (torch.float32, cfg.B * cfg.H * cfg.P)
        elif name in _HEAD:
            want = (torch.float32, cfg.H * cfg.d)
        else:                       # workspace, scratch: byte buffers
            want = (torch.uint8, t.numel())
        if t.dtype != want[0] or t.numel() != want[1]:
            raise ValueError("%s: expected %d elements of %s, got %d of %s"
                             % (name, want[1], want[0], t.numel(), t.dtype))
        if t.device.type != "cuda":
            raise ValueError("%s must be a device tensor" % name)
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("%s is on %s, expected %s" % (name, t.device, dev))


def workspace_bytes(cfg: Config, save_for_backward: bool) -> int:
    d = cfg.desc()
    return int(load().e2ttt_workspace_bytes(ctypes.byref(d), int(bool(save_for_backward))))


def backward_scratch_bytes(cfg: Config) -> int:
    d = cfg.desc()
    return int(load().e2ttt_backward_scratch_bytes(ctypes.byref(d)))


def alloc_workspace(cfg: Config, save_for_backward: bool, device="cuda"):
    n = workspace_bytes(cfg, save_for_backward)
    if n == 0:
        raise E2TTTError(3, "e2ttt_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def forward(cfg: Config, q, k, v, eta, beta, gamma, w_in, m_in=None, *, out=None, w_out=None,
            m_out=None, workspace=None, save_for_backward=False, ln_weight=None, ln_bias=None):
    """Runs e2ttt_chunk_forward (e2ttt_chunk_forward_ln with the LayerNorm affine
    ln_weight, ln_bias [H, d]) on the current stream; returns (out, w_out, m_out, workspace)."""
    _check_tensors(cfg, q=q, k=k, v=v, eta=eta, beta=beta, gamma=gamma, w_in=w_in, m_in=m_in,
                   out=out, w_out=w_out, m_out=m_out, workspace=workspace, ln_weight=ln_weight,
                   ln_bias=ln_bias)
    lib = load()
    dev = q.device
    if out is None:
        out = torch.empty_like(q)
    if w_out is None:
        w_out = torch.empty_like(w_in)
    if m_out is None:
        m_out = torch.empty_like(w_in)
    if workspace is None:
        workspace = alloc_workspace(cfg, save_for_backward, dev)
    d = cfg.desc()
    st = lib.e2ttt_chunk_forward_ln(ctypes.byref(d), _ptr(ln_weight), _ptr(ln_bias), _ptr(q),
                                    _ptr(k), _ptr(v), _ptr(eta), _ptr(beta), _ptr(gamma),
                                    _ptr(w_in), _ptr(m_in), _ptr(out), _ptr(w_out), _ptr(m_out),
                                    _ptr(workspace), workspace.numel(),
                                    int(bool(save_for_backward)), _stream())
    _check(st, "e2ttt_chunk_forward")
    return out, w_out, m_out, workspace


# Bytes of the library-owned workspace of e2ttt_chunk_forward_static.
STATIC_WORKSPACE_BYTES = 64 << 20


def forward_static(cfg: Config, q, k, v, eta, beta, gamma, w_in, m_in, out, w_out, m_out):
    """Runs e2ttt_chunk_forward_static (no save for the backward) on the current
    stream into the caller's out, w_out, m_out; allocates nothing."""
    for name, t in (("out", out), ("w_out", w_out), ("m_out", m_out)):
        if t is None:
            raise ValueError("%s must be given: this entry point allocates nothing" % name)
    _check_tensors(cfg, q=q, k=k, v=v, eta=eta, beta=beta, gamma=gamma, w_in=w_in, m_in=m_in,
                   out=out, w_out=w_out, m_out=m_out)
    d = cfg.desc()
    st = load().e2ttt_chunk_forward_static(ctypes.byref(d), _ptr(q), _ptr(k), _ptr(v), _ptr(eta),
                                           _ptr(beta), _ptr(gamma), _ptr(w_in), _ptr(m_in),
                                           _ptr(out), _ptr(w_out), _ptr(m_out), _stream())
    _check(st, "e2ttt_chunk_forward_static")
    return out, w_out, m_out


def backward(cfg: Config, q, k, v, eta, beta, gamma, w_in, m_in, workspace, d_out, d_w_out=None,
             d_m_out=None, *, grads=None, scratch=None, ln_weight=None, ln_bias=None):
    """Runs e2ttt_chunk_backward (e2ttt_chunk_backward_ln with the LayerNorm affine);
    returns a dict of gradients (dq, dk, dv, d_eta, d_beta, d_gamma, d_w_in, d_m_in, and
    d_ln_weight, d_ln_bias [H, d] with the affine)."""
    _check_tensors(cfg, q=q, k=k, v=v, eta=eta, beta=beta, gamma=gamma, w_in=w_in, m_in=m_in,
                   workspace=workspace, d_out=d_out, d_w_out=d_w_out, d_m_out=d_m_out,
                   scratch=scratch, ln_weight=ln_weight, ln_bias=ln_bias, **(grads or {}))
    lib = load()
    dev = q.device
    if grads is None:
        grads = dict(dq=torch.empty_like(q), dk=torch.empty_like(k), dv=torch.empty_like(v),
                     d_eta=torch.empty_like(eta), d_beta=torch.empty_like(beta),
                     d_gamma=None if gamma is None else torch.empty_like(gamma),
                     d_w_in=torch.empty_like(w_in), d_m_in=torch.empty_like(w_in))
        if ln_weight is not None:
            grads["d_ln_weight"] = torch.empty_like(ln_weight)
            grads["d_ln_bias"] = torch.empty_like(ln_weight)
    if scratch is None:
        scratch = torch.empty(backward_scratch_bytes(cfg), dtype=torch.uint8, device=dev)
    d = cfg.desc()
    g = grads
    st = lib.e2ttt_chunk_backward_ln(
        ctypes.byref(d), _ptr(ln_weight), _ptr(ln_bias), _ptr(q), _ptr(k), _ptr(v), _ptr(eta),
        _ptr(beta), _ptr(gamma), _ptr(w_in), _ptr(m_in), _ptr(workspace), workspace.numel(),
        _ptr(d_out), _ptr(d_w_out), _ptr(d_m_out), _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]),
        _ptr(g["d_eta"]), _ptr(g["d_beta"]), _ptr(g["d_gamma"]), _ptr(g["d_w_in"]),
        _ptr(g["d_m_in"]), _ptr(g.get("d_ln_weight")), _ptr(g.get("d_ln_bias")), _ptr(scratch),
        scratch.numel(), _stream())
    _check(st, "e2ttt_chunk_backward")
    return grads


def apply(cfg: Config, q, w, out=None, ln_weight=None, ln_bias=None):
    """Runs e2ttt_apply (e2ttt_apply_ln with the LayerNorm affine): out = f_W(q)
    for the cfg.T tokens of q per unit, all at the state w [B,H,P]."""
    _check_tensors(cfg, q=q, w_in=w, out=out, ln_weight=ln_weight, ln_bias=ln_bias)
    lib = load()
    if out is None:
        out = torch.empty_like(q)
    d = cfg.desc()
    st = lib.e2ttt_apply_ln(ctypes.byref(d), _ptr(ln_weight), _ptr(ln_bias), _ptr(q), _ptr(w),
                            _ptr(out), _stream())
    _check(st, "e2ttt_apply")
    return out


def wait_status(cfg: Config, workspace=None, scratch=None) -> int:
    """e2ttt_wait_status: waits for the current stream, then returns the status
    code of the bounded waits of the last forward that used `workspace` and the
    last backward that used `scratch` (0, or 6 when a wait expired)."""
    if workspace is None and scratch is None:
        raise ValueError("give a workspace, a scratch buffer or both")
    _check_tensors(cfg, workspace=workspace, scratch=scratch)
    d = cfg.desc()
    return int(load().e2ttt_wait_status(ctypes.byref(d), _ptr(workspace), _ptr(scratch),
                                        _stream()))


def chunk_coeffs(cfg: Config, eta, beta, gamma):
    """Scalar kernels: (kw [B,H,T], km [B,H,T], carry [B,H,NC,3])."""
    _check_tensors(cfg, eta=eta, beta=beta, gamma=gamma)
    lib = load()
    kw = torch.empty_like(eta)
    km = torch.empty_like(eta)
    carry = torch.empty((cfg.B, cfg.H, cfg.n_chunks, 3), dtype=torch.float32, device=eta.device)
    d = cfg.desc()
    st = lib.e2ttt_chunk_coeffs(ctypes.byref(d), _ptr(eta), _ptr(beta), _ptr(gamma), _ptr(kw),
                                _ptr(km), _ptr(carry), _stream())
    _check(st, "e2ttt_chunk_coeffs")
    return kw, km, carry


def _check_gate_tensors(*ts):
    n = ts[0].numel()
    for t in ts:
        if t is None:
            continue
        if t.dtype != torch.float32 or not t.is_contiguous() or t.numel() != n:
            raise ValueError("gate arrays must be contiguous float32 tensors of one size")
        if t.device.type != "cuda" or t.device != ts[0].device:
            raise ValueError("gate arrays must be device tensors on one GPU")


def gates_forward(params: GateParams, l_eta, l_beta, l_alpha=None, out=None):
    """Gate parameterization, eqs. (12)-(14): (eta, beta, gamma) from the logits
    (gamma None when l_alpha is None).  `out`: optional (eta, beta, gamma)
    tensors to write into."""
    _check_gate_tensors(l_eta, l_beta, l_alpha)
    lib = load()
    if out is None:
        eta = torch.empty_like(l_eta)
        beta = torch.empty_like(l_beta)
        gamma = None if l_alpha is None else torch.empty_like(l_alpha)
    else:
        eta, beta, gamma = out
        _check_gate_tensors(eta, beta, gamma)
        if eta.numel() != l_eta.numel() or (gamma is None) != (l_alpha is None):
            raise ValueError("gate outputs must match the logits")
    st = lib.e2ttt_gates_forward(ctypes.byref(params), l_eta.numel(), _ptr(l_eta), _ptr(l_beta),
                                 _ptr(l_alpha), _ptr(eta), _ptr(beta), _ptr(gamma), _stream())
    _check(st, "e2ttt_gates_forward")
    return eta, beta, gamma


def gates_backward(params: GateParams, l_eta, l_beta, l_alpha, d_eta, d_beta, d_gamma,
                   out=None):
    """Gradients of the logits from the gate gradients: (d_l_eta, d_l_beta,
    d_l_alpha).  `out`: optional tensors of those three to write into."""
    _check_gate_tensors(l_eta, l_beta, l_alpha, d_eta, d_beta, d_gamma)
    lib = load()
    if out is None:
        g_eta = torch.empty_like(l_eta)
        g_beta = torch.empty_like(l_beta)
        g_alpha = None if l_alpha is None else torch.empty_like(l_alpha)
    else:
        g_eta, g_beta, g_alpha = out
        _check_gate_tensors(g_eta, g_beta, g_alpha)
        if g_eta.numel() != l_eta.numel() or (g_alpha is None) != (l_alpha is None):
            raise ValueError("gate gradient outputs must match the logits")
    st = lib.e2ttt_gates_backward(ctypes.byref(params), l_eta.numel(), _ptr(l_eta), _ptr(l_beta),
                                  _ptr(l_alpha), _ptr(d_eta), _ptr(d_beta), _ptr(d_gamma),
                                  _ptr(g_eta), _ptr(g_beta), _ptr(g_alpha), _stream())
    _check(st, "e2ttt_gates_backward")
    return g_eta, g_beta, g_alpha


class E2TTTFunction(torch.autograd.Function):
    """Autograd wrapper: forward saves the workspace, backward calls the library."""

    @staticmethod
    def forward(ctx, cfg, q, k, v, eta, beta, gamma, w_in, m_in):
        out, w_out, m_out, ws = forward(cfg, q, k, v, eta, beta, gamma, w_in, m_in,
                                        save_for_backward=True)
        ctx.cfg = cfg
        ctx.save_for_backward(q, k, v, eta, beta, gamma, w_in, m_in, ws)
        return out, w_out, m_out

    @staticmethod
    def backward(ctx, d_out, d_w_out, d_m_out):
        q, k, v, eta, beta, gamma, w_in, m_in, ws = ctx.saved_tensors
        g = backward(ctx.cfg, q, k, v, eta, beta, gamma, w_in, m_in, ws, d_out.contiguous(),
                     None if d_w_out is None else d_w_out.contiguous(),
                     None if d_m_out is None else d_m_out.contiguous())
        return (None, g["dq"], g["dk"], g["dv"], g["d_eta"], g["d_beta"], g["d_gamma"],
                g["d_w_in"], None if m_in is None else g["d_m_in"])


class GatesFunction(torch.autograd.Function):
    """Autograd wrapper of the gate parameterization (eqs. (12)-(14)): logits
    in, (eta, beta, gamma) out; the backward calls e2ttt_gates_backward.
    gamma is None when l_alpha is None."""

    @staticmethod
    def forward(ctx, params, l_eta, l_beta, l_alpha):
        eta, beta, gamma = gates_forward(params, l_eta, l_beta, l_alpha)
        ctx.params = params
        ctx.save_for_backward(l_eta, l_beta, l_alpha)
        return eta, beta, gamma

    @staticmethod
    def backward(ctx, d_eta, d_beta, d_gamma):
        l_eta, l_beta, l_alpha = ctx.saved_tensors
        zero = lambda ref: torch.zeros_like(ref)
        d_eta = zero(l_eta) if d_eta is None else d_eta.contiguous()
        d_beta = zero(l_beta) if d_beta is None else d_beta.contiguous()
        if l_alpha is not None:
            d_gamma = zero(l_alpha) if d_gamma is None else d_gamma.contiguous()
        else:
            d_gamma = None
        g_eta, g_beta, g_alpha = gates_backward(ctx.params, l_eta, l_beta, l_alpha, d_eta,
                                                d_beta, d_gamma)
        return None, g_eta, g_beta, g_alpha
