"""Pins of the oracle expert FFN and combine."""
import numpy as np

from oracle import bf16, brute, ffn, router


def _experts(E, H, I, seed):
    rng = np.random.default_rng(seed)
    return [(rng.standard_normal((I, H)) * 0.3, rng.standard_normal((I, H)) * 0.3,
             rng.standard_normal((H, I)) * 0.3) for _ in range(E)]


def test_swiglu_matches_textbook_loops():
    H, I = 8, 16
    (wg, wu, wd), = _experts(1, H, I, 0)
    x = np.random.default_rng(1).standard_normal((3, H))
    y = ffn.swiglu(x, wg, wu, wd, act_bf16=False)
    for t in range(3):
        assert np.allclose(y[t], brute.loop_swiglu(x[t], wg, wu, wd), rtol=1e-12, atol=1e-12)


def test_sparse_equals_dense_masked():
    E, H, I, T, k = 6, 8, 12, 9, 2
    ex = _experts(E, H, I, 2)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((T, H))
    z = rng.standard_normal((T, E))
    ids, w, _ = router.route(z, k)
    for act_bf16 in (False, True):
        sparse = ffn.moe_forward(x, ids, w, lambda e: ex[e], act_bf16)
        dense = brute.dense_moe(x, ids, w, lambda e: ex[e], E, act_bf16, ffn.swiglu)
        assert np.allclose(sparse, dense, rtol=1e-12, atol=1e-12)


def test_k1_weight1_is_plain_mlp_and_shared_concat_identity():
    E, H, I, T = 3, 8, 16, 4
    ex = _experts(E, H, I, 4)
    x = np.random.default_rng(5).standard_normal((T, H))
    ids = np.array([[1]] * T)
    y = ffn.moe_forward(x, ids, np.ones((T, 1)), lambda e: ex[e], False)
    assert np.allclose(y, ffn.swiglu(x, *ex[1], False))
    # two shared experts == one expert with stacked gate/up rows and stacked down columns
    a, b = ex[0], ex[2]
    cat = (np.vstack([a[0], b[0]]), np.vstack([a[1], b[1]]), np.hstack([a[2], b[2]]))
    for q in (False, True):
        assert np.allclose(ffn.shared_output(x, [a, b], q), ffn.swiglu(x, *cat, q), rtol=1e-12, atol=1e-12)


def test_combine_order_and_gate():
    Y = np.arange(2 * 3 * 4, dtype=float).reshape(2, 3, 4)
    w = np.array([[0.5, 0.3, 0.2], [1.0, 0.0, 0.0]])
    ysh = np.ones((2, 4))
    s = np.array([0.25, 0.0])
    y = ffn.combine(Y, w, ysh, s)
    ref = np.einsum("tr,trh->th", w, Y) + s[:, None] * ysh
    assert np.allclose(y, ref)
    assert np.allclose(ffn.combine(Y, w, ysh), np.einsum("tr,trh->th", w, Y) + 1.0)


def test_activation_rounding_only_for_bf16():
    H, I = 4, 8
    (wg, wu, wd), = _experts(1, H, I, 6)
    x = np.random.default_rng(7).standard_normal((2, H))
    a = x @ wg.T
    act = a / (1 + np.exp(-a)) * (x @ wu.T)
    assert np.allclose(ffn.swiglu(x, wg, wu, wd, True), bf16.round_rne(act) @ wd.T, rtol=0, atol=0)
    assert not np.allclose(ffn.swiglu(x, wg, wu, wd, True), act @ wd.T, rtol=0, atol=0)
    assert np.allclose(ffn.round_out(np.array([1.0 + 2 ** -9]), "bf16"), [1.0])
