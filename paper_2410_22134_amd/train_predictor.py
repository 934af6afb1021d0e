"""Offline training of the look-ahead predictors (Sec. "Learning-based Predictor",
"Stride Prefetching"; predictor training in Sec. "Implementation").

The predictor owned by layer l reads layer l's MoE input x_l and ranks the
experts of layer l + d.  Traces pair x_l with the experts the gate of layer
l + d actually routed, for every token; they come from the library's own
forward pass on synthetic inputs, with every expert resident (the hidden states
and routing do not depend on the cache policy).  Each layer's predictor is the
paper's two-layer MLP, W2 relu(W1 x) (no biases), trained with a softmax
cross-entropy against the routed set (1/k on each routed expert) on 90% of the
tokens and scored on the other 10%: the share of a token's k predicted experts
that its gate routes.  Training starts from the given predictor weights, so a
trained predictor is never worse on the training split than where it started.

Training runs in plain PyTorch: it is offline, not part of the serving path.
"""
from __future__ import annotations

import math

import numpy as np


def collect_traces(model, steps: int, T: int, seed0: int = 5000):
    """Run `steps` forward steps of T tokens through the stack and return
    (x, ids): x[l] = bf16 bits [steps*T, H] of layer l's MoE input (int16 torch
    tensor on the device), ids[l] = routed experts [steps*T, k] (int64)."""
    import torch
    from synth import model as sm
    from .stack import Stack
    cfg = model.cfg
    L, H, k, n = cfg.n_layers, cfg.hidden, cfg.top_k, steps * T
    st = Stack(model, T)
    xs = [torch.empty(n, H, dtype=st.x.dtype, device=model.device) for _ in range(L)]
    ids = [torch.empty(n, k, dtype=torch.int64, device=model.device) for _ in range(L)]
    for i in range(steps):
        sl = slice(i * T, (i + 1) * T)

        def rec(stage, l, s, order=None, q=None):
            if stage == "x":
                xs[l][sl].copy_(s.x)
            elif stage == "moe":
                ids[l][sl].copy_(s.ids)
        h0 = torch.from_numpy(sm.stack_input(cfg, seed0 + i, T)).to(model.device)
        st.step(h0, predict=False, record=rec)
    model.ctx.sync()
    return xs, ids


def _to_f32(x, dtype: str):
    import torch
    if dtype == "bf16":
        return (x.to(torch.int32) << 16).view(torch.float32) if x.dtype == torch.int16 else x.float()
    return x.float()


def topk_accuracy(logits, ids) -> float:
    """Mean share of each token's top-k predicted experts found among its routed ones."""
    import torch
    k = ids.shape[1]
    pred = logits.topk(k, dim=1).indices
    hit = (pred.unsqueeze(2) == ids.unsqueeze(1)).any(dim=2).float().sum(dim=1)
    return float((hit / k).mean())


def train_layer(X, ids, n_experts: int, w1, w2, epochs: int = 8, lr: float = 1e-3, batch: int = 512,
                weight_decay: float = 0.0, seed: int = 0):
    """Fit W2 relu(W1 x) to the routed experts of the target layer.

    X [N, H] fp32 and ids [N, k] int64 (same device); w1 [P, H], w2 [E, P] fp32
    starting weights.  The first 90% of the rows train, the last 10% evaluate.
    Returns (w1, w2, {"acc_start": ..., "acc_trained": ..., "acc_train": ...})."""
    import torch
    torch.manual_seed(seed)
    N = X.shape[0]
    n_tr = int(math.floor(0.9 * N))
    Xtr, Xev, Ytr, Yev = X[:n_tr], X[n_tr:], ids[:n_tr], ids[n_tr:]
    W1 = torch.nn.Parameter(w1.clone().float())
    W2 = torch.nn.Parameter(w2.clone().float())

    def fwd(x):
        return torch.relu(x @ W1.t()) @ W2.t()

    with torch.no_grad():
        acc0 = topk_accuracy(fwd(Xev), Yev)
    target = torch.zeros(n_tr, n_experts, device=X.device)
    target.scatter_(1, Ytr, 1.0 / ids.shape[1])
    opt = torch.optim.Adam([W1, W2], lr=lr, weight_decay=weight_decay)
    for _ in range(epochs):
        perm = torch.randperm(n_tr, device=X.device)
        for b0 in range(0, n_tr, batch):
            sel = perm[b0:b0 + batch]
            logp = torch.log_softmax(fwd(Xtr[sel]), dim=1)
            loss = -(target[sel] * logp).sum(dim=1).mean()
            opt.zero_grad()
            loss.backward()
            opt.step()
    with torch.no_grad():
        acc1 = topk_accuracy(fwd(Xev), Yev)
        acc_tr = topk_accuracy(fwd(Xtr[: min(n_tr, 8192)]), Ytr[: min(n_tr, 8192)])
    return W1.detach(), W2.detach(), {"acc_start": acc0, "acc_trained": acc1, "acc_train": acc_tr}


def train_all(model, xs, ids, lookahead: int, epochs: int = 8, lr: float = 1e-3):
    """Train the predictor of every layer l with l + lookahead < L, starting from
    the model's predictor when its target matches, else from the skip predictor
    built from the target gate.  Returns {l: (w1, w2, metrics)} with fp32 weights."""
    import torch
    from synth import model as sm
    cfg = model.cfg.with_(lookahead=lookahead)
    out = {}
    for l in range(cfg.n_layers):
        t = sm.predictor_target(cfg, l)
        if t is None:
            continue
        p = sm.predictor(cfg, l)
        w1 = torch.from_numpy(_np_f32(p[0], cfg.dtype)).to(model.device)
        w2 = torch.from_numpy(_np_f32(p[1], cfg.dtype)).to(model.device)
        X = _to_f32(xs[l], cfg.dtype)
        out[l] = train_layer(X, ids[t], cfg.n_experts, w1, w2, epochs=epochs, lr=lr, seed=l)
    return out


def _np_f32(a, dtype):
    if dtype == "bf16":
        return (a.astype(np.uint32) << 16).view(np.float32)
    return a.astype(np.float32)


def to_model_dtype(w, dtype: str):
    """fp32 torch weights -> the library's storage (bf16 bits as int16, or fp32)."""
    import torch
    if dtype == "bf16":
        return w.to(torch.bfloat16).view(torch.int16).contiguous()
    return w.float().contiguous()


def install(model, trained):
    """Use trained predictors in the model: the device weights the next
    model.open() hands to the library, and the host copy of the same stored
    values (bf16 bits or fp32) that model.np_pred exposes as data."""
    cfg = model.cfg
    for l, (w1, w2, _) in trained.items():
        d1, d2 = to_model_dtype(w1, cfg.dtype), to_model_dtype(w2, cfg.dtype)
        model.d_pred[l] = (d1, d2)
        host = [t.cpu().numpy() for t in (d1, d2)]
        if cfg.dtype == "bf16":
            host = [h.view(np.uint16) for h in host]
        model.np_pred[l] = (host[0], host[1])
