"""The five synthetic workload shapes (shapes only; no arithmetic of the method).

Sizes follow the model families the paper evaluates (its MoE model table:
DeepSeek-MoE, Qwen1.5-MoE, Mixtral-8x7B, Qwen2-MoE) at random init.

Readings taken where the workload statement is silent:
* every config renormalises the top-k gate weights;
* the two DeepSeek shared experts are stored as one resident SwiGLU expert of
  intermediate 2 x 1408 (equal by concatenation), weight 1;
* Qwen shared experts are gated by sigmoid(w_sg . x);
* Mixtral gets an N(0,1) per-expert router bias, and a look-ahead of 2 (the
  paper's stride prefetching distance);
* the Qwen2-57B cache budget is 32 GiB of routed slots -> 22 slots per layer;
* the tiny config predicts its own (single) layer: look-ahead 0.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    kind: str          # "decode" or "prefill"
    tokens: int        # tokens per step (batch for decode, prompt length for prefill)
    steps: int         # number of steps


INT4_GROUP = 128


@dataclass(frozen=True)
class MoEConfig:
    name: str
    seed: int
    n_layers: int
    hidden: int
    n_experts: int
    top_k: int
    inter: int
    slots: int                 # expert-cache slots per layer (C)
    lookahead: int             # predictor distance d
    pred_hidden: int           # 0: single GEMV predictor [E x H]; else 2-layer MLP hidden width
    dtype: str                 # "f32" or "bf16"
    n_shared: int = 0
    shared_inter: int = 0      # per shared expert
    shared_gate: int = 0       # 0: weight 1; 1: sigmoid gate
    renorm: int = 1
    router_bias: int = 0
    weight_std: float = 0.02
    pred_noise_std: float = 0.005
    attn_surrogate: int = 1    # stack has a hidden x hidden linear mix per layer
    workloads: tuple = field(default_factory=tuple)
    # routed-expert storage: "dense" (dtype) or "int4" (4-bit codes in groups of
    # INT4_GROUP along the reduction dimension, one bf16 scale per group)
    weight_format: str = "dense"

    @property
    def shared_total(self) -> int:
        return self.n_shared * self.shared_inter

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def matrix_elems(self) -> int:
        return self.inter * self.hidden

    @property
    def chunk_bytes(self) -> int:
        """Bytes of one expert matrix as stored (codes then scales for int4)."""
        if self.weight_format == "int4":
            return self.matrix_elems // 2 + (self.matrix_elems // INT4_GROUP) * 2
        return self.matrix_elems * self.elem_bytes

    @property
    def expert_bytes(self) -> int:
        return 3 * self.chunk_bytes

    @property
    def max_tokens(self) -> int:
        return max(w.tokens for w in self.workloads)

    def with_(self, **kw) -> "MoEConfig":
        d = dict(self.__dict__)
        d.update(kw)
        return MoEConfig(**d)


C1 = MoEConfig(name="c1_tiny_fp32", seed=1, n_layers=1, hidden=256, n_experts=8, top_k=2, inter=512,
               slots=4, lookahead=0, pred_hidden=0, dtype="f32", attn_surrogate=0,
               workloads=(Workload("prefill", 16, 1), Workload("decode", 1, 16)))
C2 = MoEConfig(name="c2_deepseek_moe_16b", seed=2, n_layers=27, hidden=2048, n_experts=64, top_k=6,
               inter=1408, slots=32, lookahead=1, pred_hidden=512, dtype="bf16",
               n_shared=2, shared_inter=1408, shared_gate=0,
               workloads=(Workload("decode", 1, 256),))
C3 = MoEConfig(name="c3_qwen15_moe_a27b", seed=3, n_layers=24, hidden=2048, n_experts=60, top_k=4,
               inter=1408, slots=30, lookahead=2, pred_hidden=512, dtype="bf16",
               n_shared=1, shared_inter=5632, shared_gate=1,
               workloads=(Workload("prefill", 512, 1), Workload("decode", 1, 128)))
C4 = MoEConfig(name="c4_mixtral_8x7b", seed=4, n_layers=32, hidden=4096, n_experts=8, top_k=2,
               inter=14336, slots=2, lookahead=2, pred_hidden=512, dtype="bf16", router_bias=1,
               workloads=(Workload("prefill", 256, 1), Workload("decode", 1, 128)))
C5 = MoEConfig(name="c5_qwen2_57b_a14b", seed=5, n_layers=28, hidden=3584, n_experts=64, top_k=8,
               inter=2560, slots=22, lookahead=1, pred_hidden=512, dtype="bf16",
               n_shared=1, shared_inter=20480, shared_gate=1,
               workloads=(Workload("prefill", 1024, 1), Workload("decode", 1, 128), Workload("decode", 8, 128)))

ALL = (C1, C2, C3, C4, C5)
BY_NAME = {c.name: c for c in ALL}
