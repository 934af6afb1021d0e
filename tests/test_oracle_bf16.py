"""Pins of the oracle's bf16 rounding against the binary32 bit layout."""
import numpy as np

from oracle import bf16


def test_roundtrip_every_pattern():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    vals = bf16.decode(bits)
    back = bf16.encode_rne(vals)
    finite_or_inf = ~np.isnan(vals)
    assert np.array_equal(back[finite_or_inf], bits[finite_or_inf])
    assert np.isnan(bf16.decode(bf16.encode_rne(vals[~finite_or_inf]))).all()


def test_ties_to_even_and_known_values():
    f = np.array([0x3F808000, 0x3F818000, 0x3F808001, 0x3F807FFF], dtype=np.uint32).view(np.float32)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> 1 + 2^-6
    assert list(bf16.encode_rne(f)) == [0x3F80, 0x3F82, 0x3F81, 0x3F80]
    assert bf16.encode_rne(np.array([1.0]))[0] == 0x3F80
    assert bf16.encode_rne(np.array([-2.0]))[0] == 0xC000
    assert bf16.encode_rne(np.array([np.inf]))[0] == 0x7F80
    # largest finite float32 rounds up to infinity in bf16
    assert bf16.encode_rne(np.array([np.finfo(np.float32).max]))[0] == 0x7F80


def test_rounding_error_bound():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(100000)
    r = bf16.round_rne(x)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0 ** -8 + 1e-45)
