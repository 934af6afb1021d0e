"""Harness ops around the MoE block (the paper's transformer layer: attention,
normalisation and residual adds around the MoE FFN, Background section).  The
attention block is replaced by a seeded linear mix of the hidden state.

  rms(v)  = v / sqrt(mean(v^2) + 1e-6)
  h      <- h + Wa . q(rms(h))          q = bf16 rounding for bf16 models
  x       = q(rms(h))                   (MoE block input)
  h      <- h + y                       (y = MoE block output)
"""
import numpy as np

from . import bf16

EPS = 1e-6


def rms(v: np.ndarray) -> np.ndarray:
    v = np.asarray(v, np.float64)
    return v / np.sqrt(np.mean(v * v, axis=-1, keepdims=True) + EPS)


def quant(v: np.ndarray, dtype: str) -> np.ndarray:
    return bf16.round_rne(v) if dtype == "bf16" else np.asarray(v, np.float32).astype(np.float64)


def attn_surrogate(h: np.ndarray, wa: np.ndarray, dtype: str) -> np.ndarray:
    return np.asarray(h, np.float64) + quant(rms(h), dtype) @ np.asarray(wa, np.float64).T


def moe_input(h: np.ndarray, dtype: str) -> np.ndarray:
    return quant(rms(h), dtype)
