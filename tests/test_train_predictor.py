"""CPU checks of the offline predictor trainer on planted routings."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2410_22134_amd import train_predictor as tp  # noqa: E402


def _planted(N=6000, H=32, E=8, k=2, seed=0):
    g = torch.Generator().manual_seed(seed)
    G = torch.randn(E, H, generator=g)
    X = torch.randn(N, H, generator=g)
    ids = (X @ G.t()).topk(k, dim=1).indices
    return X, ids, G


def test_skip_predictor_construction_is_exact():
    # W1 = [G; -G; 0], W2 = [I, -I, 0]: W2 relu(W1 x) = G x, so the top-k is the routing
    X, ids, G = _planted()
    E, H = G.shape
    P = 3 * E
    w1 = torch.zeros(P, H)
    w1[:E], w1[E:2 * E] = G, -G
    w2 = torch.zeros(E, P)
    w2[torch.arange(E), torch.arange(E)] = 1.0
    w2[torch.arange(E), E + torch.arange(E)] = -1.0
    logits = torch.relu(X @ w1.t()) @ w2.t()
    assert torch.allclose(logits, X @ G.t(), atol=1e-4)
    assert tp.topk_accuracy(logits, ids) == 1.0
    # a random ranking scores about k/E
    r = torch.randn(X.shape[0], E, generator=torch.Generator().manual_seed(3))
    assert abs(tp.topk_accuracy(r, ids) - 2 / 8) < 0.03


def test_training_learns_a_planted_routing():
    X, ids, G = _planted()
    E, H = G.shape
    g = torch.Generator().manual_seed(1)
    w1 = 0.1 * torch.randn(64, H, generator=g)
    w2 = 0.1 * torch.randn(E, 64, generator=g)
    _, _, m = tp.train_layer(X, ids, E, w1, w2, epochs=30, lr=3e-3, batch=256)
    assert m["acc_start"] < 0.5
    assert m["acc_trained"] > 0.85, m


def test_bf16_export_rounds_to_nearest_even():
    w = torch.tensor([1.0, 1.00390625, 1.01171875, -2.5, 3.0e-3])
    b = tp.to_model_dtype(w, "bf16").numpy().view(np.uint16)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa -> 1.0 (0x3F80)
    assert b[0] == 0x3F80 and b[1] == 0x3F80
    # 1 + 3*2^-8 ties between 1 + 2^-7 and 1 + 2^-6: even -> 1 + 2^-6 (0x3F82)
    assert b[2] == 0x3F82
    assert b[3] == 0xC020
