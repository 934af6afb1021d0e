"""Stack driver: the transformer-layer loop around the MoE block for the
synthetic configs (prefill or decode steps), calling the library per layer:
attention surrogate -> route -> predict -> expert_ffn -> residual add (predict
before route when the look-ahead is 0)."""
from __future__ import annotations

from ._abi import FLAG_NO_PREFETCH
from .model import SyntheticModel


class Stack:
    def __init__(self, model: SyntheticModel, T: int):
        import torch
        cfg = model.cfg
        self.m, self.T = model, T
        dev = model.device
        xdt = torch.int16 if cfg.dtype == "bf16" else torch.float32
        H, k = cfg.hidden, cfg.top_k
        self.h = torch.zeros(T, H, dtype=torch.float32, device=dev)
        self.x = torch.zeros(T, H, dtype=xdt, device=dev)
        self.y = torch.zeros(T, H, dtype=xdt, device=dev)
        self.ids = torch.zeros(T, k, dtype=torch.int32, device=dev)
        self.w = torch.zeros(T, k, dtype=torch.float32, device=dev)
        self.s = torch.zeros(T, dtype=torch.float32, device=dev)
        self.pred_ids = torch.zeros(T, k, dtype=torch.int32, device=dev)
        # device addresses of the buffers above, passed to every per-layer call
        self._h, self._x, self._y = self.h.data_ptr(), self.x.data_ptr(), self.y.data_ptr()
        self._ids, self._w, self._s = self.ids.data_ptr(), self.w.data_ptr(), self.s.data_ptr()
        self._pred = self.pred_ids.data_ptr()
        self._cuda = str(dev).startswith("cuda")

    def moe_layer(self, l: int, predict: bool = True, want_q: bool = False, stream=None):
        """route -> predict -> ffn on self.x (predict first at look-ahead 0); returns (order, q).

        With a look-ahead the prediction is made after the route, so the
        speculative copies it queues for layer l + d go behind the precise copies
        of layer l and fill the link while layer l computes (measured 35.8 ->
        37.1 tok/s on the DeepSeek-16B decode)."""
        ctx, T = self.m.ctx, self.T
        s = _handle(stream) if self._cuda else stream
        first = self.m.cfg.lookahead == 0
        q = None
        if predict and not first and not want_q:
            # one call: the predictor's launches fill the route's wait for its plan
            order = ctx.route_predict(l, self._x, T, self._ids, self._w, self._s, self._pred, stream=s)
            ctx.expert_ffn(l, self._x, T, self._ids, self._w, self._s, self._y, stream=s)
            return order, None
        if predict and first:
            q = ctx.predict(l, self._x, T, self._pred, want_q=want_q, stream=s)
        order = ctx.route(l, self._x, T, self._ids, self._w, self._s, stream=s)
        if predict and not first:
            q = ctx.predict(l, self._x, T, self._pred, want_q=want_q, stream=s)
        ctx.expert_ffn(l, self._x, T, self._ids, self._w, self._s, self._y, stream=s)
        return order, q

    def step(self, h0, predict: bool | None = None, record=None, stream=None, native: bool = True):
        """One step over all layers from residual input h0 [T, H] (fp32, device),
        on `stream` (default: the current stream, looked up once per step).
        predict=None: the predictor runs unless the context was opened without
        prefetching (then nothing would read its output).  Without a record
        callback the whole loop is one library call (promoe_stack_step) unless
        native=False."""
        ctx, T = self.m.ctx, self.T
        s = _handle(stream) if self._cuda else stream
        if predict is None:
            predict = not getattr(self.m, "flags", 0) & FLAG_NO_PREFETCH
        self.h.copy_(h0)
        if native and record is None and hasattr(ctx, "stack_step"):
            ctx.stack_step(self._h, T, self._x, self._y, self._ids, self._w, self._s, self._pred, predict, stream=s)
            return self.h
        for l in range(self.m.cfg.n_layers):
            if record is not None:
                record("h", l, self)
            ctx.attn_surrogate(l, self._h, T, self._x, stream=s)
            if record is not None:
                record("x", l, self)
            order, q = self.moe_layer(l, predict, want_q=record is not None, stream=s)
            if record is not None:
                record("moe", l, self, order=order, q=q)
            ctx.residual_add(self._h, self._y, T, stream=s)
        return self.h


def _handle(stream) -> int:
    """A hipStream_t as an int: the given stream's, or the current stream's."""
    if isinstance(stream, int):
        return stream
    import torch
    return (stream if stream is not None else torch.cuda.current_stream()).cuda_stream
