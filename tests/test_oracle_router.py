"""Pins of the oracle router: brute-force top-k, closed forms, invariants."""
import numpy as np
import scipy.special

from oracle import brute, router


def _rand(T, E, H, seed):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((T, H)), rng.standard_normal((E, H)) * 0.1


def test_logits_match_loops():
    x, wg = _rand(3, 5, 7, 0)
    z = router.gate_logits(x, wg)
    for t in range(3):
        assert np.allclose(z[t], brute.loop_matvec(wg, x[t]), rtol=1e-13, atol=1e-13)
    b = np.arange(5.0)
    assert np.allclose(router.gate_logits(x, wg, b) - z, b[None, :])


def test_topk_matches_full_sort_including_ties():
    rng = np.random.default_rng(1)
    z = np.round(rng.standard_normal((200, 8)), 1)      # many exact ties
    for k in (1, 2, 3, 8):
        ids = router.topk(z, k)
        for t in range(z.shape[0]):
            assert list(ids[t]) == brute.sort_topk(z[t], k)
    z = np.zeros((1, 6))
    assert list(router.topk(z, 3)[0]) == [0, 1, 2]


def test_renormalised_weights_closed_form_and_sum():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((50, 16)) * 3
    ids, w, p = router.route(z, 4, renorm=True)
    sel = np.take_along_axis(z, ids.astype(np.int64), axis=1)
    closed = np.exp(sel - sel[:, :1]) / np.exp(sel - sel[:, :1]).sum(1, keepdims=True)
    assert np.allclose(w, closed, rtol=1e-12, atol=1e-15)
    assert np.allclose(w.sum(1), 1.0, atol=1e-12)
    assert np.all(np.diff(w, axis=1) <= 0)              # rank order = descending weight
    _, w_nr, _ = router.route(z, 4, renorm=False)
    assert np.all(w_nr.sum(1) < 1.0)
    assert np.allclose(w_nr, np.take_along_axis(scipy.special.softmax(z, axis=1), ids.astype(np.int64), 1))


def test_k_equals_e_is_plain_softmax():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((10, 6))
    ids, w, p = router.route(z, 6, renorm=True)
    ref = scipy.special.softmax(z, axis=1)
    assert np.allclose(np.take_along_axis(ref, ids.astype(np.int64), 1), w, rtol=1e-12)
    assert np.allclose(p, ref, rtol=1e-12)


def test_bias_changes_selection_before_topk():
    z = np.array([[1.0, 0.9, 0.0, -1.0]])
    ids, _, _ = router.route(router.gate_logits(np.eye(4)[:1], np.diag([1.0, 0.9, 0.0, -1.0]),
                                                np.array([0.0, 0.0, 5.0, 0.0])), 2)
    assert list(ids[0]) == [2, 0]
    assert list(router.topk(z, 2)[0]) == [0, 1]


def test_margins():
    z = np.array([[3.0, 1.0, 2.0, 1.5]])
    b, inner = router.margins(z, 2)
    assert np.isclose(b[0], 0.5) and np.isclose(inner[0], 1.0)


def test_shared_scale_is_sigmoid():
    x = np.array([[1.0, -2.0], [0.0, 0.0]])
    s = router.shared_scale(x, np.array([0.5, 0.25]))
    assert np.allclose(s, scipy.special.expit([0.0, 0.0]))
    s = router.shared_scale(x, np.array([1.0, 0.0]))
    assert np.allclose(s, scipy.special.expit([1.0, 0.0]))


def test_weights_for_on_route_ids_equals_route_weights():
    # evaluated on the oracle's own selection, the helper reproduces route()
    rng = np.random.default_rng(4)
    z = rng.standard_normal((40, 12)) * 2
    for k in (1, 3, 12):
        for renorm in (True, False):
            ids, w, p = router.route(z, k, renorm)
            assert np.array_equal(router.weights_for(p, ids, renorm), w)


def test_weights_for_arbitrary_ids_closed_form():
    # on any distinct ids (not the top-k, any order) the renormalised weights are
    # the softmax over exactly those logits, in the given order; without
    # renormalisation they are the full softmax's values at those ids
    rng = np.random.default_rng(5)
    T, E, k = 30, 9, 3
    z = rng.standard_normal((T, E)) * 3
    p = scipy.special.softmax(z, axis=1)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    w = router.weights_for(p, ids, renorm=True)
    for t in range(T):
        sel = z[t, ids[t]]
        expect = np.exp(sel - sel.max()) / np.exp(sel - sel.max()).sum()
        assert np.allclose(w[t], expect, rtol=1e-12, atol=1e-15)
    w_nr = router.weights_for(p, ids, renorm=False)
    for t in range(T):
        for r in range(k):
            assert w_nr[t, r] == p[t, ids[t, r]]
    # a permutation of the ids permutes the weights the same way (no axis mix-up)
    perm = ids[:, ::-1]
    assert np.allclose(router.weights_for(p, perm, True), w[:, ::-1], rtol=1e-14, atol=0)
