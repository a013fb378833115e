"""fp64 CPU oracle for the E2-TTT chunk update -- TEST INFRASTRUCTURE ONLY.

Thin ctypes wrapper around ``e2ttt_oracle.cpp`` (a plain token-by-token loop in
double precision, see the header of that file for what it follows in the paper).
Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  The HIP library never does, and this
module imports nothing from the HIP library's package.

Arrays are numpy float64, C-contiguous:
  q, k, v, out, dq, dk, dv : [B, H, T, d]
  eta, beta, gamma, d_*    : [B, H, T]
  w_in, m_in, w_out, ...   : [B, H, P]   (P = 2 d dh for the MLP, 3 d dh for SwiGLU)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "e2ttt_oracle.cpp")
_LIB = os.path.join(_HERE, "libe2ttt_oracle.so")

FW_MLP = 0
FW_SWIGLU = 1
FLAG_NO_RESIDUAL_LN = 1
FLAG_POST_NORM = 8        # post-chunk L2 normalisation of the fast-weight rows

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["g++", "-std=c++17", "-O2", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
               _SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.c_void_p
        i = ctypes.c_int
        d = ctypes.c_double
        lib.e2ttt_oracle_forward.argtypes = [i, i, i, i, i, i, i, i, d] + [dp] * 13 + [i]
        lib.e2ttt_oracle_forward.restype = i
        lib.e2ttt_oracle_backward.argtypes = [i, i, i, i, i, i, i, i, d] + [dp] * 23 + [i]
        lib.e2ttt_oracle_backward.restype = i
        lib.e2ttt_oracle_chunk_coeffs.argtypes = [i] + [dp] * 6
        lib.e2ttt_oracle_chunk_coeffs.restype = i
        lib.e2ttt_oracle_net.argtypes = [i, i, i, i, d, dp, dp, dp, i, dp, dp]
        lib.e2ttt_oracle_net.restype = i
        lib.e2ttt_oracle_neg_grad.argtypes = [i, i, i, i, d, dp, dp, dp, i, dp, dp, dp]
        lib.e2ttt_oracle_neg_grad.restype = i
        lib.e2ttt_oracle_param_count.argtypes = [i, i, i]
        lib.e2ttt_oracle_param_count.restype = ctypes.c_long
        _lib = lib
    return _lib


def _f64(a):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def param_count(d: int, dh: int, fw: int) -> int:
    return int(_load().e2ttt_oracle_param_count(d, dh, fw))


def default_threads() -> int:
    return max(1, min(os.cpu_count() or 1, int(os.environ.get("E2TTT_ORACLE_THREADS", "64"))))


def forward(q, k, v, eta, beta, gamma, w_in, m_in, *, C, fw, dh, flags=0, eps=1e-5, nthreads=None,
            ln_a=None, ln_b=None):
    """Returns (out [B,H,T,d], w_out [B,H,P], m_out [B,H,P]) in float64.

    ln_a, ln_b: the learnable LayerNorm affine per head, [H, d] (None: a = 1, b = 0)."""
    q, k, v, eta, beta, gamma, w_in, m_in = map(_f64, (q, k, v, eta, beta, gamma, w_in, m_in))
    ln_a, ln_b = _f64(ln_a), _f64(ln_b)
    B, H, T, d = q.shape
    P = param_count(d, dh, fw)
    assert w_in.shape == (B, H, P), (w_in.shape, (B, H, P))
    out = np.zeros((B, H, T, d))
    w_out = np.zeros((B, H, P))
    m_out = np.zeros((B, H, P))
    rc = _load().e2ttt_oracle_forward(B, H, T, d, dh, C, fw, flags, eps, _p(q), _p(k), _p(v),
                                      _p(eta), _p(beta), _p(gamma), _p(w_in), _p(m_in), _p(ln_a),
                                      _p(ln_b), _p(out), _p(w_out), _p(m_out),
                                      nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle forward rejected its arguments")
    return out, w_out, m_out


def backward(q, k, v, eta, beta, gamma, w_in, m_in, d_out, d_w_out=None, d_m_out=None, *, C, fw,
             dh, flags=0, eps=1e-5, nthreads=None, ln_a=None, ln_b=None):
    """Gradients of sum<d_out,out> + <d_w_out,w_out> + <d_m_out,m_out>.

    Returns a dict with dq, dk, dv, d_eta, d_beta, d_gamma (None if gamma is
    None), d_w_in, d_m_in, and with the LayerNorm affine (ln_a and ln_b [H, d],
    both or neither) d_ln_a, d_ln_b [H, d] summed over the batch, all float64.
    """
    q, k, v, eta, beta, gamma, w_in, m_in, d_out, d_w_out, d_m_out = map(
        _f64, (q, k, v, eta, beta, gamma, w_in, m_in, d_out, d_w_out, d_m_out))
    ln_a, ln_b = _f64(ln_a), _f64(ln_b)
    B, H, T, d = q.shape
    P = param_count(d, dh, fw)
    res = {n: np.zeros((B, H, T, d)) for n in ("dq", "dk", "dv")}
    for n in ("d_eta", "d_beta"):
        res[n] = np.zeros((B, H, T))
    res["d_gamma"] = None if gamma is None else np.zeros((B, H, T))
    res["d_w_in"] = np.zeros((B, H, P))
    res["d_m_in"] = np.zeros((B, H, P))
    aff = ln_a is not None or ln_b is not None
    if aff:
        res["d_ln_a"] = np.zeros((H, d))
        res["d_ln_b"] = np.zeros((H, d))
    rc = _load().e2ttt_oracle_backward(
        B, H, T, d, dh, C, fw, flags, eps, _p(q), _p(k), _p(v), _p(eta), _p(beta), _p(gamma),
        _p(w_in), _p(m_in), _p(ln_a), _p(ln_b), _p(d_out), _p(d_w_out), _p(d_m_out), _p(res["dq"]),
        _p(res["dk"]), _p(res["dv"]), _p(res["d_eta"]), _p(res["d_beta"]), _p(res["d_gamma"]),
        _p(res["d_w_in"]), _p(res["d_m_in"]), _p(res.get("d_ln_a")), _p(res.get("d_ln_b")),
        nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle backward rejected its arguments")
    return res


def chunk_coeffs(eta, beta, gamma=None):
    """Scalar kernels of one chunk: (kw[C], km[C], (cw, cm, cb))."""
    eta, beta, gamma = map(_f64, (eta, beta, gamma))
    C = eta.shape[0]
    kw = np.zeros(C)
    km = np.zeros(C)
    carry = np.zeros(3)
    rc = _load().e2ttt_oracle_chunk_coeffs(C, _p(eta), _p(beta), _p(gamma), _p(kw), _p(km),
                                           _p(carry))
    if rc != 0:
        raise ValueError("bad chunk")
    return kw, km, tuple(carry)


def net(W, x, *, fw, dh, flags=0, eps=1e-5, ln_a=None, ln_b=None):
    """f_W(x) for rows x[n, d] of one unit (ln_a, ln_b: its head's affine [d], or None)."""
    W, x, ln_a, ln_b = _f64(W), _f64(x), _f64(ln_a), _f64(ln_b)
    n, d = x.shape
    f = np.zeros((n, d))
    rc = _load().e2ttt_oracle_net(d, dh, fw, flags, eps, _p(W), _p(ln_a), _p(ln_b), n, _p(x),
                                  _p(f))
    if rc != 0:
        raise ValueError("bad net arguments")
    return f


def neg_grad(W, k, v, *, fw, dh, flags=0, eps=1e-5, ln_a=None, ln_b=None):
    """G[n, P] = -grad_W 1/2||f_W(k_r) - v_r||^2 for each row r."""
    W, k, v, ln_a, ln_b = _f64(W), _f64(k), _f64(v), _f64(ln_a), _f64(ln_b)
    n, d = k.shape
    P = param_count(d, dh, fw)
    G = np.zeros((n, P))
    rc = _load().e2ttt_oracle_neg_grad(d, dh, fw, flags, eps, _p(W), _p(ln_a), _p(ln_b), n, _p(k),
                                       _p(v), _p(G))
    if rc != 0:
        raise ValueError("bad grad arguments")
    return G
