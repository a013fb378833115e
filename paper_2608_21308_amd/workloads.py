"""Seeded synthetic workloads for the E2-TTT chunk update.

This module holds input recipes only (shapes, seeds, distributions and the
bf16 rounding of inputs); it contains none of the method's arithmetic.  Both
the HIP path and the fp64 oracle consume exactly the arrays it returns.

Recipe (the paper trains on text corpora that are not available here; these
synthetic draws stand in for them with the shapes of the paper-scale layer):
  * Q, K, V ~ N(0, 1) per element, L2-normalised per token over d (the paper
    L2-normalises queries and keys before the fast-weight net, Sec. 4), then
    rounded once to bf16 (round-to-nearest-even) for bf16 workloads.
  * eta_t = 0.1 * sigmoid(N(0,1)); beta_t = sigmoid(N(1,1));
    gamma_t = 1 - eta_t * alpha_t with alpha_t = 0.1 * sigmoid(N(0,1))
    (the coupling of eq. (14) with alpha_base = 0.1 of Table 7).  Gates fp32.
  * W_init ~ N(0, 0.02^2) per head, broadcast over the batch; M_init = 0.
  * d_out ~ N(0, 1) in the io dtype (backward workloads only).
Draw order: Q, K, V, eta-logits, beta-logits, alpha-logits, W_init, d_out,
then (small tests only) d_w_out, d_m_out.  Generator: numpy PCG64.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

FW_MLP = 0
FW_SWIGLU = 1


@dataclass(frozen=True)
class Workload:
    name: str
    fw: int                  # FW_MLP or FW_SWIGLU
    B: int
    H: int
    T: int
    d: int
    dh: int
    C: int
    io: str                  # "f32" or "bf16"
    backward: bool           # whether the workload includes the backward pass
    seed: int
    note: str = field(default="", compare=False)

    @property
    def units(self) -> int:
        return self.B * self.H

    @property
    def n_chunks(self) -> int:
        return (self.T + self.C - 1) // self.C

    @property
    def P(self) -> int:
        return (2 if self.fw == FW_MLP else 3) * self.d * self.dh

    def with_(self, **kw) -> "Workload":
        vals = {k: getattr(self, k) for k in self.__dataclass_fields__}
        vals.update(kw)
        return Workload(**vals)


# The five workloads of the measurement plan.  Index 3 is the 1.3B-model
# layer shape (d_model 1024 = 16 heads x 64) used for the headline number.
WORKLOADS = [
    Workload("tiny_mlp_f32", FW_MLP, 1, 1, 256, 16, 64, 16, "f32", False, 20260,
             "tiny fp32 correctness case, forward"),
    Workload("mlp_fwd_bf16", FW_MLP, 2, 4, 2048, 64, 256, 64, "bf16", False, 20261,
             "MLP fast weight, forward"),
    Workload("swiglu_train_bf16", FW_SWIGLU, 2, 4, 2048, 64, 172, 64, "bf16", True, 20262,
             "SwiGLU fast weight, forward + backward"),
    Workload("mlp_1p3b_train_bf16", FW_MLP, 8, 16, 4096, 64, 256, 64, "bf16", True, 20263,
             "1.3B layer shape, training step (forward + backward)"),
    Workload("swiglu_prefill_32k_bf16", FW_SWIGLU, 1, 16, 32768, 64, 172, 64, "bf16", False, 20264,
             "long-context prefill, 512 chunks, forward"),
]


# The paper's own throughput shape for its 1.3B model (Sec. 5: hidden 2048 over
# 16 heads, so head dim 128; sequences of 2K tokens, batch 2, chunk 512), with
# an MLP fast weight of hidden 4 d = 512 per head; the same recipe as above.
PAPER_1P3B = Workload("paper_1p3b_d128_c512_bf16", FW_MLP, 2, 16, 2048, 128, 512, 512, "bf16",
                      True, 20270, "paper-scale 1.3B layer: head dim 128, chunk 512, fwd + bwd")


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))
    r = ((u + bias) >> np.uint64(16)) << np.uint64(16)
    out = r.astype(np.uint32).view(np.float32)
    return np.where(np.isnan(x), x, out).astype(np.float32)


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def make_inputs(w: Workload, *, with_grads: bool | None = None, state_grads: bool = False,
                units: list[int] | None = None) -> dict:
    """Draw the inputs of workload ``w``.

    Returns float32 numpy arrays (bf16-representable for bf16 workloads):
    q, k, v [B,H,T,d]; eta, beta, gamma [B,H,T]; w_in [B,H,P]; m_in None;
    d_out [B,H,T,d] when the backward is requested; d_w_out, d_m_out [B,H,P]
    when ``state_grads``.  ``units`` (flat b*H+h indices) restricts the
    returned arrays to those units, drawn from the same full-size stream.
    """
    rng = np.random.Generator(np.random.PCG64(w.seed))
    B, H, T, d, P = w.B, w.H, w.T, w.d, w.P
    bf = w.io == "bf16"

    def tok():
        x = rng.standard_normal((B, H, T, d), dtype=np.float32)
        x /= np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True)).astype(np.float32)
        return round_bf16(x) if bf else x

    q = tok()
    k = tok()
    v = tok()
    eta = (0.1 * _sigmoid(rng.standard_normal((B, H, T)))).astype(np.float32)
    beta = _sigmoid(rng.normal(1.0, 1.0, (B, H, T))).astype(np.float32)
    alpha = (0.1 * _sigmoid(rng.standard_normal((B, H, T)))).astype(np.float32)
    gamma = (np.float32(1.0) - eta * alpha).astype(np.float32)
    w_head = (0.02 * rng.standard_normal((H, P))).astype(np.float32)
    w_in = np.ascontiguousarray(np.broadcast_to(w_head[None], (B, H, P)))
    res = dict(q=q, k=k, v=v, eta=eta, beta=beta, gamma=gamma, w_in=w_in, m_in=None)
    if with_grads is None:
        with_grads = w.backward
    if with_grads:
        do = rng.standard_normal((B, H, T, d), dtype=np.float32)
        res["d_out"] = round_bf16(do) if bf else do
    if state_grads:
        res["d_w_out"] = rng.standard_normal((B, H, P), dtype=np.float32)
        res["d_m_out"] = rng.standard_normal((B, H, P), dtype=np.float32)
    if units is not None:
        idx = np.asarray(units)
        for key, val in list(res.items()):
            if val is None:
                continue
            flat = val.reshape((B * H,) + val.shape[2:])
            res[key] = np.ascontiguousarray(flat[idx][None])
    return res


def small(w: Workload, **kw) -> Workload:
    """A reduced copy of ``w`` for oracle-speed tests (same kinds and dims)."""
    return w.with_(**kw)
