"""bfloat16 helpers for the oracle.

bf16 is the upper 16 bits of an IEEE-754 binary32.  Decoding is exact
(shift into the high half).  Encoding rounds to nearest, ties to even, on the
binary32 value: add 0x7FFF plus the lowest kept bit, then truncate.  Values
already in float64 are first rounded to binary32 (one extra rounding that the
GPU, which holds fp32, does not see; tests compare within bf16 tolerances).
"""
import numpy as np


def decode(bits) -> np.ndarray:
    """raw bf16 bits (uint16) -> float64, exactly (a signalling-NaN pattern
    becomes a quiet NaN, as any widening conversion makes it)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def encode_rne(x) -> np.ndarray:
    """float -> raw bf16 bits (uint16), round to nearest even; NaN stays NaN."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        rounded = np.where(nan, (u >> 16).astype(np.uint16) | np.uint16(0x40), rounded)
    return rounded


def round_rne(x) -> np.ndarray:
    """float -> nearest bf16 value, returned as float64."""
    return decode(encode_rne(x))


def to_f64(a, dtype: str) -> np.ndarray:
    """Tensor stored as fp32 values ('f32') or bf16 bits ('bf16') -> float64."""
    if dtype == "bf16":
        return decode(a)
    return np.asarray(a, dtype=np.float32).astype(np.float64)
