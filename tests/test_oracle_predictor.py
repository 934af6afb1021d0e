"""Pins of the oracle predictor: the skip-predictor identity, vote brute force."""
import itertools

import numpy as np

from oracle import predictor, router
from synth import configs, model


def test_mlp_without_noise_reproduces_target_gate_exactly():
    c = configs.C2.with_(n_layers=2, pred_noise_std=0.0)
    w1, w2 = model.predictor(c, 0)
    from oracle import bf16
    x = bf16.decode(model.layer_input(c, 0, 4))
    q = predictor.logits(x, bf16.decode(w1), bf16.decode(w2))
    z = router.gate_logits(x, bf16.decode(model.gate(c, 1)))
    assert np.array_equal(q, z)


def test_single_gemv_form():
    rng = np.random.default_rng(0)
    x, w = rng.standard_normal((3, 5)), rng.standard_normal((4, 5))
    assert np.allclose(predictor.logits(x, w), x @ w.T)


def test_vote_single_token_is_topk_in_rank_order():
    q = np.array([[0.1, 0.9, 0.5, 0.7, -1.0]])
    ids = predictor.per_token(q, 3)
    Q, votes, best = predictor.vote(ids, 5, cap=10)
    assert Q == [1, 3, 2]
    Q, _, _ = predictor.vote(ids, 5, cap=2)
    assert Q == [1, 3]


def test_vote_brute_force_small():
    # compare with an independent formulation: score tuples built from counts
    rng = np.random.default_rng(5)
    E, k = 5, 2
    for trial in range(200):
        T = int(rng.integers(1, 5))
        ids = np.array([rng.permutation(E)[:k] for _ in range(T)])
        cap = int(rng.integers(1, E + 1))
        Q, _, _ = predictor.vote(ids, E, cap)
        score = {}
        for e in range(E):
            appearances = [r for t in range(T) for r in range(k) if ids[t, r] == e]
            if appearances:
                score[e] = (len(appearances), -min(appearances), -e)
        ref = sorted(score, key=lambda e: score[e], reverse=True)[:cap]
        assert Q == ref


def test_vote_never_exceeds_cap_and_counts_all_tokens():
    ids = np.array(list(itertools.permutations(range(4), 2)))   # 12 tokens
    Q, votes, best = predictor.vote(ids, 4, cap=3)
    assert len(Q) == 3 and votes.sum() == ids.size and (best == 0).all()
