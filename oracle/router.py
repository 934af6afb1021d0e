"""Gate and top-k routing (Background, "Mixture-of-Experts (MoE) based LLMs";
early-preemption section: the experts a layer needs are all known once the
gate finishes).

For every token t:
  z[t, e] = sum_h Wg[e, h] x[t, h] (+ b[e])         float64
  p[t, :] = softmax(z[t, :])
  top-k ids by the total order (z descending, expert id ascending)
  w[t, r] = p[t, id_r] / sum_r' p[t, id_r']           (renormalised), or p[t, id_r]
  s[t]    = sigmoid(w_sg . x[t])                      (gated shared expert)
"""
import numpy as np


def gate_logits(x: np.ndarray, wg: np.ndarray, bias=None) -> np.ndarray:
    z = np.asarray(x, np.float64) @ np.asarray(wg, np.float64).T
    if bias is not None:
        z = z + np.asarray(bias, np.float64)[None, :]
    return z


def softmax(z: np.ndarray) -> np.ndarray:
    m = z.max(axis=1, keepdims=True)
    ez = np.exp(z - m)
    return ez / ez.sum(axis=1, keepdims=True)


def rank_order(z: np.ndarray) -> np.ndarray:
    """Per row, expert ids sorted by (value descending, id ascending)."""
    # a stable sort of -z keeps equal values in ascending id order
    return np.argsort(-z, axis=1, kind="stable")


def topk(z: np.ndarray, k: int) -> np.ndarray:
    return rank_order(z)[:, :k].astype(np.int32)


def margins(z: np.ndarray, k: int):
    """Per token: the gap between the k-th and (k+1)-th largest logits (inf if k == E),
    and the smallest gap between adjacent selected logits (inf if k == 1)."""
    zs = -np.sort(-z, axis=1)
    E = z.shape[1]
    boundary = zs[:, k - 1] - zs[:, k] if k < E else np.full(z.shape[0], np.inf)
    inner = (zs[:, :k - 1] - zs[:, 1:k]).min(axis=1) if k > 1 else np.full(z.shape[0], np.inf)
    return boundary, inner


def route(z: np.ndarray, k: int, renorm: bool = True):
    """-> ids [T, k] int32, w [T, k] float64, p [T, E] float64."""
    p = softmax(z)
    ids = topk(z, k)
    w = np.take_along_axis(p, ids.astype(np.int64), axis=1)
    if renorm:
        w = w / w.sum(axis=1, keepdims=True)
    return ids, w, p


def weights_for(p: np.ndarray, ids: np.ndarray, renorm: bool = True) -> np.ndarray:
    """Gate weights of a given id selection (used to evaluate the GPU's own ids)."""
    w = np.take_along_axis(p, np.asarray(ids, np.int64), axis=1)
    if renorm:
        w = w / w.sum(axis=1, keepdims=True)
    return w


def shared_scale(x: np.ndarray, wsg: np.ndarray) -> np.ndarray:
    u = np.asarray(x, np.float64) @ np.asarray(wsg, np.float64)
    return 1.0 / (1.0 + np.exp(-u))
