"""Seeded weight and input recipes for the synthetic MoE stacks.

Every tensor is an independent Philox stream keyed by (config seed,
stream_id(kind, layer, index)), so any tensor can be regenerated alone, in any
order, on any thread count.  Weights are N(0, 0.02) draws; bf16 configs store
their round-to-nearest-even bf16 bits (uint16 arrays), the fp32 config stores
float32.

Look-ahead predictor weights (the paper trains a small two-layer MLP per layer
offline from traces; with random weights there is nothing to learn from):
the predictor owned by layer l targets layer l+d and is built from that
layer's gate so that it reproduces a skip-based predictor plus noise:
    W1 = [Wg(l+d); -Wg(l+d); 0] + N(0, 0.005)      (pred_hidden x H)
    W2 = [I, -I, 0]                                  (E x pred_hidden)
so that W2 relu(W1 x) = Wg(l+d) x exactly when the noise is zero.  The fp32
config uses a single GEMV predictor Wp = Wg + N(0, 0.005) on its own layer.
"""
from __future__ import annotations

import numpy as np

from . import normal
from .configs import INT4_GROUP, MoEConfig

K_GATE, K_BIAS, K_EG, K_EU, K_ED, K_SG, K_SU, K_SD, K_SGATE, K_PN1, K_PN2, K_ATTN, K_H0, K_X = range(1, 15)


def stream_id(kind: int, layer: int = 0, index: int = 0) -> int:
    return (kind << 48) | (layer << 32) | index


def _bf16_bits(f32: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest even); data preparation only."""
    u = np.ascontiguousarray(f32, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _w(cfg: MoEConfig, kind: int, layer: int, index: int, n: int, std=None, out=None):
    std = cfg.weight_std if std is None else std
    return normal(cfg.seed, stream_id(kind, layer, index), n, std, dtype=cfg.dtype, out=out)


# ---------------------------------------------------------------- routed experts
def expert(cfg: MoEConfig, layer: int, e: int):
    """(Wg [I,H], Wu [I,H], Wd [H,I]) of routed expert e of a layer."""
    I, H = cfg.inter, cfg.hidden
    return (_w(cfg, K_EG, layer, e, I * H).reshape(I, H),
            _w(cfg, K_EU, layer, e, I * H).reshape(I, H),
            _w(cfg, K_ED, layer, e, H * I).reshape(H, I))


def write_expert(cfg: MoEConfig, layer: int, e: int, addr: int) -> None:
    """Write [Wg | Wu | Wd] of one routed expert to raw memory at addr (each
    matrix as codes then scales for the int4 format)."""
    n = cfg.inter * cfg.hidden
    if cfg.weight_format == "int4":
        from . import quant_int4
        for i, m in enumerate(expert(cfg, layer, e)):
            rows, K = m.shape
            base = addr + i * cfg.chunk_bytes
            quant_int4(m, rows, K, INT4_GROUP, base, base + rows * K // 2)
        return
    eb = cfg.elem_bytes
    _w(cfg, K_EG, layer, e, n, out=addr)
    _w(cfg, K_EU, layer, e, n, out=addr + n * eb)
    _w(cfg, K_ED, layer, e, n, out=addr + 2 * n * eb)


def quantize_int4(w: np.ndarray, group: int = INT4_GROUP):
    """Round-to-nearest symmetric 4-bit quantisation of fp32 rows w [R, K] in
    groups of `group` along K (data preparation only; write_expert uses the
    same recipe in C, synth.quant_int4, checked equal to this one on the CPU):
    scale s = bf16(absmax / 7),
    code = clamp(rint(w / s), -8, 7) + 8, two codes per byte (even k in the low
    nibble).  Returns (codes uint8 [R, K/2], scales bf16 bits uint16 [R, K/group])."""
    R, K = w.shape
    g = w.reshape(R, K // group, group)
    s_bits = _bf16_bits((np.abs(g).max(axis=2) / 7.0).astype(np.float32))
    s = bf16_to_f32(s_bits)[:, :, None]
    q = np.where(s > 0, np.rint(g / np.where(s > 0, s, 1.0)), 0.0)
    codes = (np.clip(q, -8, 7) + 8).astype(np.uint8).reshape(R, K)
    packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    return packed, s_bits


def expert_from_bytes(cfg: MoEConfig, buf: np.ndarray):
    """Split a flat [Wg|Wu|Wd] element array into its three matrices (for int4,
    `buf` is the raw bytes and each matrix is returned as its stored byte block)."""
    I, H = cfg.inter, cfg.hidden
    n = I * H
    if cfg.weight_format == "int4":
        cb = cfg.chunk_bytes
        return buf[:cb], buf[cb:2 * cb], buf[2 * cb:3 * cb]
    return buf[:n].reshape(I, H), buf[n:2 * n].reshape(I, H), buf[2 * n:3 * n].reshape(H, I)


# ---------------------------------------------------------------- gate / shared
def gate(cfg: MoEConfig, layer: int) -> np.ndarray:
    return _w(cfg, K_GATE, layer, 0, cfg.n_experts * cfg.hidden).reshape(cfg.n_experts, cfg.hidden)


def bias(cfg: MoEConfig, layer: int):
    if not cfg.router_bias:
        return None
    return normal(cfg.seed, stream_id(K_BIAS, layer), cfg.n_experts, 1.0, dtype="f32")


def shared_parts(cfg: MoEConfig, layer: int):
    """List of (Wg, Wu, Wd) for each shared expert of a layer (empty if none)."""
    I, H = cfg.shared_inter, cfg.hidden
    out = []
    for j in range(cfg.n_shared):
        out.append((_w(cfg, K_SG, layer, j, I * H).reshape(I, H),
                    _w(cfg, K_SU, layer, j, I * H).reshape(I, H),
                    _w(cfg, K_SD, layer, j, H * I).reshape(H, I)))
    return out


def shared_concat(cfg: MoEConfig, layer: int):
    """The shared experts of a layer as one expert of intermediate n_shared*shared_inter:
    gate/up rows stacked, down columns stacked.  Flat [Wg|Wu|Wd] element array."""
    parts = shared_parts(cfg, layer)
    if not parts:
        return None
    wg = np.concatenate([p[0] for p in parts], axis=0)
    wu = np.concatenate([p[1] for p in parts], axis=0)
    wd = np.concatenate([p[2] for p in parts], axis=1)
    return np.concatenate([wg.ravel(), wu.ravel(), np.ascontiguousarray(wd).ravel()])


def shared_gate_vec(cfg: MoEConfig, layer: int):
    if not cfg.shared_gate or not cfg.n_shared:
        return None
    return _w(cfg, K_SGATE, layer, 0, cfg.hidden)


# ---------------------------------------------------------------- predictor
def predictor_target(cfg: MoEConfig, layer: int):
    t = layer + cfg.lookahead
    return t if t < cfg.n_layers else None


def predictor(cfg: MoEConfig, layer: int):
    """Predictor owned by `layer` (targets layer + lookahead).  Returns (W1, W2) with
    W2 None for the single-GEMV form, or None when the target is past the last layer."""
    t = predictor_target(cfg, layer)
    if t is None:
        return None
    E, H, P = cfg.n_experts, cfg.hidden, cfg.pred_hidden
    g = gate(cfg, t)
    g32 = g.astype(np.float32) if cfg.dtype == "f32" else bf16_to_f32(g)
    if P == 0:
        n = normal(cfg.seed, stream_id(K_PN1, layer), E * H, cfg.pred_noise_std, dtype="f32").reshape(E, H)
        wp = g32 + n
        return (wp.astype(np.float32) if cfg.dtype == "f32" else _bf16_bits(wp)), None
    assert P >= 2 * E
    n1 = normal(cfg.seed, stream_id(K_PN1, layer), P * H, cfg.pred_noise_std, dtype="f32").reshape(P, H)
    w1 = n1.copy()
    w1[:E] += g32
    w1[E:2 * E] -= g32
    w2 = np.zeros((E, P), dtype=np.float32)
    w2[np.arange(E), np.arange(E)] = 1.0
    w2[np.arange(E), E + np.arange(E)] = -1.0
    if cfg.dtype == "f32":
        return w1.astype(np.float32), w2
    return _bf16_bits(w1), _bf16_bits(w2)


# ---------------------------------------------------------------- harness / inputs
def attn(cfg: MoEConfig, layer: int):
    if not cfg.attn_surrogate:
        return None
    return _w(cfg, K_ATTN, layer, 0, cfg.hidden * cfg.hidden).reshape(cfg.hidden, cfg.hidden)


def stack_input(cfg: MoEConfig, step: int, T: int, tag: int = 0) -> np.ndarray:
    """Residual-stream input h0 [T, H] (fp32 N(0,1)) of a step; a fresh vector per
    step and sequence."""
    idx = (tag << 24) | step
    return normal(cfg.seed, stream_id(K_H0, 0, idx), T * cfg.hidden, 1.0, dtype="f32").reshape(T, cfg.hidden)


def layer_input(cfg: MoEConfig, layer: int, T: int, tag: int = 0) -> np.ndarray:
    """MoE-block input x [T, H] ~ N(0,1) for a single-layer case: fp32, or bf16 bits."""
    return normal(cfg.seed, stream_id(K_X, layer, tag), T * cfg.hidden, 1.0,
                  dtype=cfg.dtype).reshape(T, cfg.hidden)
