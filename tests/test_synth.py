"""The seeded input generator: Philox known answers, distribution, determinism."""
import os

import numpy as np

import synth
from synth import configs, model

HERE = os.path.dirname(os.path.abspath(__file__))


def test_philox_known_answers():
    rows = []
    with open(os.path.join(HERE, "golden", "philox_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append([int(v, 16) for v in line.split()])
    assert len(rows) == 3
    for r in rows:
        out = synth.philox4x32_10(r[0:4], r[4:6])
        assert [int(v) for v in out] == r[6:10]


def test_normal_moments_and_offsets():
    z = synth.normal(7, 11, 2_000_000, 1.0)
    assert abs(z.mean()) < 3e-3 and abs(z.std() - 1) < 3e-3
    assert abs((z ** 4).mean() - 3.0) < 0.03          # Gaussian kurtosis
    part = synth.normal(7, 11, 1000, 1.0, offset=12345)
    assert np.array_equal(part, z[12345:13345])
    w = synth.normal(7, 11, 1000, 0.02, dtype="bf16")
    f = model.bf16_to_f32(w)
    assert np.allclose(f, 0.02 * z[:1000], rtol=2 ** -8, atol=0)
    assert not np.array_equal(synth.normal(7, 12, 100, 1.0), z[:100])


def test_model_tensors_shapes_and_predictor_identity():
    c = configs.C2.with_(n_layers=3, pred_noise_std=0.0)
    w1, w2 = model.predictor(c, 0)
    g = model.bf16_to_f32(model.gate(c, 1))
    assert np.array_equal(model.bf16_to_f32(w1)[:64], g)
    assert np.array_equal(model.bf16_to_f32(w1)[64:128], -g)
    assert model.predictor(c, 2) is None
    sh = model.shared_concat(configs.C2.with_(n_layers=1), 0)
    assert sh.size == 3 * 2816 * 2048
