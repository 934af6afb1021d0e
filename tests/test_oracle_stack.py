"""Pins of the harness ops."""
import numpy as np

from oracle import stack


def test_rms_closed_forms():
    v = np.full((1, 16), 3.0)
    assert np.allclose(stack.rms(v), 3.0 / np.sqrt(9.0 + 1e-6))
    # at |v| = 1e-3 the epsilon (1e-6) equals mean(v^2): rms = 1/sqrt(2) exactly
    v = np.full((1, 8), 1e-3)
    assert np.allclose(stack.rms(v), 1e-3 / np.sqrt(2e-6), rtol=1e-12)
    rng = np.random.default_rng(0)
    v = rng.standard_normal((4, 64))
    r = stack.rms(v)
    assert np.allclose(np.mean(r * r, axis=1), np.mean(v * v, 1) / (np.mean(v * v, 1) + 1e-6))
    assert np.allclose(stack.rms(5 * v), stack.rms(v), rtol=1e-6)


def test_attn_surrogate_loops():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((2, 6))
    wa = rng.standard_normal((6, 6))
    out = stack.attn_surrogate(h, wa, "f32")
    for t in range(2):
        u = (h[t] / np.sqrt((h[t] ** 2).mean() + 1e-6)).astype(np.float32).astype(np.float64)
        ref = [h[t, i] + sum(wa[i, j] * u[j] for j in range(6)) for i in range(6)]
        assert np.allclose(out[t], ref)
