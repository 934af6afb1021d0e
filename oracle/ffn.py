"""SwiGLU experts and the MoE combine (Background, "Mixture-of-Experts (MoE)
based LLMs": each expert is an FFN of three linear layers, the block output is
the gate-weighted sum of the activated experts' outputs; the chunked-prefetching
section relies on the same three-matrix structure).

Per routed pair (t, r) with expert e = ids[t, r]:
  a   = Wg_e x_t,  b = Wu_e x_t                      (float64)
  act = silu(a) * b,  silu(u) = u / (1 + exp(-u))
  act <- bf16(act) for bf16 models (the GPU feeds its down projection bf16
         activations); unchanged for fp32 models
  Y[t, r] = Wd_e act
Shared experts (always resident): Ysh[t] = sum_j SwiGLU_j(x_t), computed the
same way.  Output:
  y[t] = sum_{r=0..k-1} w[t, r] Y[t, r]  (+ s[t] Ysh[t])
rounded once at the end to the model dtype.
"""
import numpy as np

from . import bf16


def silu(u: np.ndarray) -> np.ndarray:
    return u / (1.0 + np.exp(-u))


def swiglu(x: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray, act_bf16: bool) -> np.ndarray:
    """x [M, H], Wg/Wu [I, H], Wd [H, I] (float64) -> [M, H]."""
    a = x @ wg.T
    b = x @ wu.T
    act = silu(a) * b
    if act_bf16:
        act = bf16.round_rne(act)
    return act @ wd.T


def routed_outputs(x: np.ndarray, ids: np.ndarray, expert_fn, act_bf16: bool) -> np.ndarray:
    """Y [T, k, H]: Y[t, r] = SwiGLU_{ids[t,r]}(x[t]).  expert_fn(e) -> (Wg, Wu, Wd) float64."""
    T, k = ids.shape
    H = x.shape[1]
    Y = np.zeros((T, k, H), np.float64)
    for e in np.unique(ids):
        tok, rr = np.nonzero(ids == e)
        wg, wu, wd = expert_fn(int(e))
        Y[tok, rr] = swiglu(x[tok], wg, wu, wd, act_bf16)
    return Y


def shared_output(x: np.ndarray, parts, act_bf16: bool) -> np.ndarray:
    """Sum over the shared experts; parts = list of (Wg, Wu, Wd) float64."""
    out = np.zeros_like(x, dtype=np.float64)
    for wg, wu, wd in parts:
        out = out + swiglu(x, wg, wu, wd, act_bf16)
    return out


def combine(Y: np.ndarray, w: np.ndarray, ysh=None, s=None) -> np.ndarray:
    """y[t] = sum_r w[t,r] Y[t,r] in r order, plus the (gated) shared output."""
    T, k, H = Y.shape
    y = np.zeros((T, H), np.float64)
    for r in range(k):
        y = y + w[:, r:r + 1] * Y[:, r]
    if ysh is not None:
        y = y + (ysh if s is None else s[:, None] * ysh)
    return y


def round_out(y: np.ndarray, dtype: str) -> np.ndarray:
    """The single final rounding: bf16 (RNE) or fp32, returned as float64 values."""
    if dtype == "bf16":
        return bf16.round_rne(y)
    return y.astype(np.float32).astype(np.float64)


def moe_forward(x, ids, w, expert_fn, act_bf16: bool, shared_parts=None, s=None):
    """Unrounded float64 MoE block output for given routing."""
    Y = routed_outputs(x, ids, expert_fn, act_bf16)
    ysh = shared_output(x, shared_parts, act_bf16) if shared_parts else None
    return combine(Y, w, ysh, s)
