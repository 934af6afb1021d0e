"""Pins of the oracle's 4-bit expert decoder: a hand-worked example, the
round trip through the input generator's (separately written) quantiser, and
values already on the quantisation grid."""
import json
import os

import numpy as np

from oracle import quant
from synth import configs, model as sm

HERE = os.path.dirname(os.path.abspath(__file__))


def _block(codes, scales):
    return np.concatenate([codes.reshape(-1), scales.reshape(-1).view(np.uint8)])


def test_hand_worked_example():
    g = json.load(open(os.path.join(HERE, "golden", "int4_block_example.json")))
    rows, K = g["rows"], g["K"]
    codes = np.full(rows * K // 2, g["fill_byte"], dtype=np.uint8)
    for i, v in g["bytes"].items():
        codes[int(i)] = v
    scales = np.array(g["scales_bf16"], dtype=np.uint16)
    w = quant.decode_matrix(_block(codes, scales), rows, K)
    expect = np.zeros((rows, K))
    for i, v in g["expected_nonzero"].items():
        expect[0, int(i)] = v
    assert np.array_equal(w, expect)


def test_round_trip_through_the_quantiser():
    rng = np.random.default_rng(0)
    w = rng.normal(0, 0.02, (16, 512)).astype(np.float32)
    w[3, :128] = 0.0                        # an all-zero group: scale 0, codes 8
    codes, scales = sm.quantize_int4(w)
    d = quant.decode_matrix(_block(codes, scales), 16, 512)
    g = np.abs(w.reshape(16, 4, 128)).max(axis=2)
    s = sm.bf16_to_f32(scales).astype(np.float64)
    # error: half a step, plus the clamp at +7 when the bf16 scale rounded below absmax/7
    bound = np.repeat(s / 2 + g * 2.0 ** -8, 128, axis=1)
    assert np.all(np.abs(d - w) <= bound + 1e-12)
    assert np.all(d[3, :128] == 0.0)
    # the decoded values lie on the grid of their group
    q = d / np.repeat(np.where(s > 0, s, 1.0), 128, axis=1)
    assert np.allclose(q, np.rint(q)) and q.min() >= -8 and q.max() <= 7


def test_values_on_the_grid_are_exact():
    rng = np.random.default_rng(1)
    s = sm.bf16_to_f32(sm._bf16_bits(rng.uniform(1e-3, 1e-2, (8, 2)).astype(np.float32)))
    q = rng.integers(-7, 8, (8, 256)).astype(np.float64)
    q[:, 0], q[:, 128] = 7, -7              # each group reaches |q| = 7, so absmax / 7 = s
    w = (q * np.repeat(s, 128, axis=1)).astype(np.float32)
    codes, scales = sm.quantize_int4(w)
    assert np.array_equal(sm.bf16_to_f32(scales), s)
    assert np.array_equal(quant.decode_matrix(_block(codes, scales), 8, 256), w.astype(np.float64))


def test_expert_blocks_are_split_in_order():
    cfg = configs.C1.with_(dtype="bf16", hidden=256, inter=128, weight_format="int4")
    rng = np.random.default_rng(2)
    mats = [rng.normal(0, 0.02, (128, 256)).astype(np.float32), rng.normal(0, 0.02, (128, 256)).astype(np.float32),
            rng.normal(0, 0.02, (256, 128)).astype(np.float32)]
    raw = np.concatenate([_block(*sm.quantize_int4(m)) for m in mats])
    assert raw.nbytes == cfg.expert_bytes
    wg, wu, wd = quant.decode_expert(raw, 128, 256)
    for a, b in zip((wg, wu, wd), mats):
        assert a.shape == b.shape and np.abs(a - b).max() < 0.02 / 7 * 4
