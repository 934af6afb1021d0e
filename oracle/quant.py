"""Decoder of the 4-bit expert storage (test infrastructure, like the rest of
this package).

The paper runs its larger models with 4-bit weights quantised by GPTQ
(Sec. "Evaluation", setup and the bits-per-weight study).  The library stores
such experts group-wise: every expert matrix of R rows and reduction length K
is R x K/2 bytes of codes, row-major, two per byte (even k in the low nibble,
odd k in the high nibble), followed by R x K/G bf16 scales (G = 128, row-major);
the weight at (r, k) is (code - 8) * scale[r][k // G].  This module reads that
layout back into float64 matrices.
"""
import numpy as np

from . import bf16 as obf16

GROUP = 128


def decode_matrix(block: np.ndarray, rows: int, K: int, group: int = GROUP) -> np.ndarray:
    """float64 [rows, K] from one stored matrix (uint8 bytes: codes then scales)."""
    block = np.asarray(block, dtype=np.uint8)
    n_codes = rows * K // 2
    n_scales = rows * (K // group)
    codes = block[:n_codes].reshape(rows, K // 2)
    scale_bits = block[n_codes:n_codes + 2 * n_scales].view(np.uint16).reshape(rows, K // group)
    q = np.empty((rows, K), dtype=np.float64)
    q[:, 0::2] = codes & 0x0F
    q[:, 1::2] = codes >> 4
    scale = obf16.decode(scale_bits)
    return (q - 8.0) * np.repeat(scale, group, axis=1)


def decode_expert(raw: np.ndarray, inter: int, hidden: int):
    """(Wg [I,H], Wu [I,H], Wd [H,I]) float64 from an expert's stored bytes."""
    raw = np.asarray(raw, dtype=np.uint8)
    cb = inter * hidden // 2 + (inter * hidden // GROUP) * 2
    return (decode_matrix(raw[:cb], inter, hidden),
            decode_matrix(raw[cb:2 * cb], inter, hidden),
            decode_matrix(raw[2 * cb:3 * cb], hidden, inter))
