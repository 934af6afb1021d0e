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


def test_int4_storage_in_c_equals_the_numpy_recipe():
    # write_expert stores 4-bit experts through synth.quant_int4 (C); it must
    # give the same bytes as model.quantize_int4 (numpy), rounding ties to even
    rng = np.random.default_rng(3)
    R, K = 24, 512
    w = model._bf16_bits((rng.standard_normal((R, K)) * 0.02).astype(np.float32))
    w[0, :128] = 0                                   # an all-zero group: scale 0, codes 8
    s = 0.5 * np.arange(-16, 16, dtype=np.float32)   # exact halves of a power-of-two scale: ties
    w[1, 128:256] = model._bf16_bits(np.resize(s, 128) * np.float32(2.0 ** -7))
    w[1, 128] = model._bf16_bits(np.array([7.0 * 2.0 ** -7], np.float32))[0]   # absmax 7 * 2^-7: scale 2^-7
    codes_np, scales_np = model.quantize_int4(model.bf16_to_f32(w))
    codes = np.zeros((R, K // 2), np.uint8)
    scales = np.zeros((R, K // 128), np.uint16)
    synth.quant_int4(w, R, K, 128, codes.ctypes.data, scales.ctypes.data)
    assert np.array_equal(scales, scales_np) and np.array_equal(codes, codes_np)
    assert scales[0, 0] == 0 and np.all(codes[0, :64] == 0x88)
