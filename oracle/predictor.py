"""Look-ahead expert predictor (Sec. "Learning-based Predictor" and
"Stride Prefetching").

The predictor owned by layer l reads that layer's MoE input and scores the
experts of layer l+d.  Its output is a priority over experts like a gate's; for
every token the k highest-priority experts are taken (k = the model's top-k),
by the same total order as the router (value descending, id ascending).

With T > 1 tokens the per-token picks are merged into one list by an integer
vote (a reading: the paper states only the per-token rule):
  votes[e] = number of tokens whose top-k contains e
  best[e]  = smallest rank at which e appears in any token's top-k
  Q        = experts with votes > 0, sorted by (votes desc, best asc, e asc),
             truncated to the cache capacity C.
"""
import numpy as np

from .router import topk


def logits(x: np.ndarray, w1: np.ndarray, w2=None) -> np.ndarray:
    """Single GEMV form (w2 None): q = W1 x.  MLP form: q = W2 relu(W1 x)."""
    h = np.asarray(x, np.float64) @ np.asarray(w1, np.float64).T
    if w2 is None:
        return h
    return np.maximum(h, 0.0) @ np.asarray(w2, np.float64).T


def per_token(q: np.ndarray, k: int) -> np.ndarray:
    return topk(q, k)


def vote(pred_ids: np.ndarray, n_experts: int, cap: int):
    """-> (Q list, votes[E], best[E]); best = k for experts never picked."""
    pred_ids = np.asarray(pred_ids)
    T, k = pred_ids.shape
    votes = np.zeros(n_experts, np.int64)
    best = np.full(n_experts, k, np.int64)
    for t in range(T):
        for r in range(k):
            e = int(pred_ids[t, r])
            votes[e] += 1
            best[e] = min(best[e], r)
    cand = [e for e in range(n_experts) if votes[e] > 0]
    cand.sort(key=lambda e: (-votes[e], best[e], e))
    return cand[:cap], votes, best
