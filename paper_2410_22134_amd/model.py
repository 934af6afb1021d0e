"""Synthetic MoE model on the GPU: seeded weights (from ``synth``) placed where the
library expects them -- routed experts in pinned host memory, gates, predictors,
shared experts and the attention surrogate in device memory, an HBM cache region
of n_layers x slots expert slots -- and a context bound to them."""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor

import numpy as np

from synth import model as sm
from synth.configs import MoEConfig

from ._abi import PROMOE_BF16, PROMOE_F32, WEIGHTS_DENSE, WEIGHTS_INT4, Config, Context, HostBuffer


def lib_config(cfg: MoEConfig, max_tokens: int, flags: int = 0, window: int = 0, subchunk: int = 0,
               spec_fill_limit: int = 0) -> Config:
    c = Config()
    c.n_layers, c.hidden, c.n_experts, c.top_k, c.inter = cfg.n_layers, cfg.hidden, cfg.n_experts, cfg.top_k, cfg.inter
    c.shared_inter, c.shared_gate = cfg.shared_total, cfg.shared_gate if cfg.n_shared else 0
    c.renorm, c.router_bias = cfg.renorm, cfg.router_bias
    c.slots_per_layer, c.lookahead, c.pred_hidden = cfg.slots, cfg.lookahead, cfg.pred_hidden
    c.max_tokens = max_tokens
    c.dtype = PROMOE_BF16 if cfg.dtype == "bf16" else PROMOE_F32
    c.copy_subchunk_bytes, c.copy_window, c.flags = subchunk, window, flags
    c.spec_fill_limit = spec_fill_limit
    c.weight_format = WEIGHTS_INT4 if cfg.weight_format == "int4" else WEIGHTS_DENSE
    return c


def _dev(arr: np.ndarray, device):
    import torch
    a = np.ascontiguousarray(arr)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


class SyntheticModel:
    def __init__(self, cfg: MoEConfig, device="cuda", max_tokens=None, flags=0, window=0, subchunk=0, spec_fill_limit=0,
                 warm=True, gen_threads=4):
        import torch
        self.cfg = cfg
        self.device = device
        self.max_tokens = max_tokens or cfg.max_tokens
        L, E = cfg.n_layers, cfg.n_experts
        eb = cfg.expert_bytes
        # routed experts: pinned host memory, one buffer per layer
        self.host = [HostBuffer(E * eb) for _ in range(L)]

        def fill(le):
            l, e = le
            sm.write_expert(cfg, l, e, self.host[l].addr + e * eb)
        with ThreadPoolExecutor(max_workers=gen_threads) as ex:
            list(ex.map(fill, [(l, e) for l in range(L) for e in range(E)]))
        # resident weights
        self.np_gate = [sm.gate(cfg, l) for l in range(L)]
        self.np_bias = [sm.bias(cfg, l) for l in range(L)]
        self.np_pred = [sm.predictor(cfg, l) for l in range(L)]
        self.np_sgate = [sm.shared_gate_vec(cfg, l) for l in range(L)]
        self.d_gate = [_dev(g, device) for g in self.np_gate]
        self.d_bias = [None if b is None else _dev(b, device) for b in self.np_bias]
        self.d_pred = [(None, None) if p is None else (_dev(p[0], device), None if p[1] is None else _dev(p[1], device))
                       for p in self.np_pred]
        self.d_shared = [None if not cfg.n_shared else _dev(sm.shared_concat(cfg, l), device) for l in range(L)]
        self.d_sgate = [None if v is None else _dev(v, device) for v in self.np_sgate]
        self.d_attn = [None if not cfg.attn_surrogate else _dev(sm.attn(cfg, l), device) for l in range(L)]
        self.cache = torch.empty(L * cfg.slots * eb, dtype=torch.uint8, device=device)
        self.ctx = None
        self.open(flags, window, subchunk, spec_fill_limit, warm)

    def open(self, flags=0, window=0, subchunk=0, spec_fill_limit=0, warm=True, slots=None):
        """(Re)create the context over the same weights, e.g. to run another cache
        policy or (slots=...) another cache size; the cache starts over from the
        warm set."""
        import torch
        if self.ctx is not None:
            self.ctx.close()
            self.ctx = None
        self.flags = flags
        if slots is not None and slots != self.cfg.slots:
            self.cfg = self.cfg.with_(slots=slots)
            self.cache = None
            self.cache = torch.empty(self.cfg.n_layers * slots * self.cfg.expert_bytes, dtype=torch.uint8,
                                     device=self.device)
        cfg, L, E, eb = self.cfg, self.cfg.n_layers, self.cfg.n_experts, self.cfg.expert_bytes
        self.ctx = Context(lib_config(cfg, self.max_tokens, flags, window, subchunk, spec_fill_limit),
                           self.cache.data_ptr(), self.cache.numel())
        for l in range(L):
            p1, p2 = self.d_pred[l]
            self.ctx.set_layer(l, self.d_gate[l], self.d_bias[l], p1, p2, self.d_shared[l], self.d_sgate[l])
            if self.d_attn[l] is not None:
                self.ctx.set_attn(l, self.d_attn[l])
            for e in range(E):
                self.ctx.set_expert_host(l, e, self.host[l].addr + e * eb)
            if warm:
                self.ctx.set_initial_cache(l, list(range(min(cfg.slots, E))))

    # host views for the oracle (data, not code)
    def expert_host(self, layer: int, e: int) -> np.ndarray:
        cfg = self.cfg
        if cfg.weight_format == "int4":
            return self.host[layer].numpy(np.uint8, count=cfg.expert_bytes, offset=e * cfg.expert_bytes)
        n = 3 * cfg.inter * cfg.hidden
        dt = np.uint16 if cfg.dtype == "bf16" else np.float32
        return self.host[layer].numpy(dt, count=n, offset=e * cfg.expert_bytes)

    def close(self):
        self.ctx.close()
        for h in self.host:
            h.free()
