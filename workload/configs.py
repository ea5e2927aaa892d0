"""Workload configurations for the offloaded-MoE decode hot path.

Each configuration fixes the shapes of a synthetic MoE decode stack and the
recipe of its seeded inputs.  The shapes follow the two models the paper
evaluates (Section "Experimental Setup": Qwen3-VL-30B-A3B with 128 routed
experts and top-8, DeepSeek-VL2-Tiny with 64 routed experts, top-6 and shared
experts); the values are synthetic (no checkpoint or dataset is used).

This module holds no arithmetic of the method: it only names sizes, seeds and
distributions.  Both the CPU oracle and the device path read it.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Tuple


Q4_BLOCK = 32  # elements per scale in the "q4" expert codec


@dataclass(frozen=True)
class MoEConfig:
    """Shapes, storage precision and input recipe of one synthetic decode stack.

    Notation follows the paper's problem formulation: ``L`` MoE layers, ``n``
    routed experts per layer, top-``K`` routing, hidden size ``D``; the adapter
    rank ``r`` (Section "Expert Prediction Adapter").  ``I`` is the SwiGLU
    intermediate size of one routed expert, ``S`` the number of accelerator
    expert slots per layer (the capacity of the available set), ``windows``
    the prefetch window capacities (in whole expert transfers) the budget is
    evaluated at.
    """

    name: str
    L: int
    D: int
    n: int
    K: int
    I: int
    r: int
    S: int
    windows: Tuple[int, ...]
    tokens: int
    batch: int = 1
    n_shared: int = 0
    has_proj: bool = False
    dtype: str = "bf16"          # storage dtype of weights and hidden states: "bf16" | "f32"
    seed: int = 0
    rho: float = 0.8             # AR(1) coefficient of the layer-0 hidden states
    sigma: float = 0.6           # AR(1) innovation scale
    w_std: float = 0.02          # std of router, expert, shared-expert and projection weights
    adapter_noise: float = 0.005  # std of the noise added to the SVD-built adapters
    rms_eps: float = 1e-6
    # 0: every layer has its own experts.  E > 0: layer l's expert weights are
    # those of layer l mod E (a tied offload tier that bounds pinned host
    # memory; routers, adapters and slot pools stay per layer).
    expert_layers: int = 0
    # expert weight codec: "plain" (the storage dtype) or "q4": 4-bit codes q in
    # 0..15 in blocks of 32 with one fp16 scale per block, w = scale * (q - 8);
    # blocks run along D for gate rows, up rows and down columns alike
    codec: str = "plain"
    # routing predictability.  router_rank > 0: each router is an exact
    # rank-router_rank matrix (entries still of std w_std), in place of a
    # full-rank i.i.d. one; update_scale scales every expert's down projection
    # (routed and shared; for "q4" its block scales), i.e. the size of a
    # layer's update of the residual stream relative to the stream itself.
    router_rank: int = 0
    update_scale: float = 1.0

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    @property
    def blob_elems(self) -> int:
        """Elements of one expert: gate [I,D] + up [I,D] + down [D,I]."""
        return 3 * self.I * self.D

    @property
    def blob_bytes(self) -> int:
        """Bytes of one expert: 3 I D elements, or for "q4" 3 I D half-bytes plus
        one 2-byte scale per 32 elements."""
        if self.codec == "q4":
            return self.I * (3 * self.D // 2 + 3 * (self.D // Q4_BLOCK) * 2)
        return self.blob_elems * self.elem_bytes

    def expert_layer(self, layer: int) -> int:
        """The layer whose seeded expert weights layer `layer` uses."""
        return layer % self.expert_layers if self.expert_layers > 0 else layer

    @property
    def host_layers(self) -> int:
        """Distinct expert-weight layers in the offload tier."""
        return min(self.expert_layers, self.L) if self.expert_layers > 0 else self.L

    @property
    def window(self) -> int:
        """Default window capacity (first entry of ``windows``)."""
        return self.windows[0]

    def with_(self, **kw) -> "MoEConfig":
        return dataclasses.replace(self, **kw)


# Tiny fp32 parity case: 2 layers, 8 experts, top-2.
C0 = MoEConfig(name="tiny_f32_L2_D256_n8_k2", L=2, D=256, n=8, K=2, I=512, r=16,
               S=4, windows=(1,), tokens=64, dtype="f32", seed=0)

# Qwen3-VL-30B-A3B-shaped MoE layer pair in bf16 (layer 0 is the predictor's
# source, layer 1 the prefetch target): 128 experts, top-8, 9.44 MB per expert.
C1 = MoEConfig(name="qwen3vl30b_a3b_layer_bf16", L=2, D=2048, n=128, K=8, I=768, r=64,
               S=32, windows=(2,), tokens=256, seed=0)

# Full 48-layer Qwen3-VL-30B-A3B-shaped stack with a dense 2048x2048 stand-in
# projection per layer in place of attention; 25% of experts resident.
C2 = MoEConfig(name="qwen3vl30b_a3b_stack48_bf16", L=48, D=2048, n=128, K=8, I=768, r=64,
               S=32, windows=(1, 2, 4), tokens=512, has_proj=True, seed=0)

# DeepSeek-VL2-Tiny-shaped stack: 12 layers, 64 routed experts, top-6, two
# always-resident shared experts; 30% of routed experts resident (floor).
C3 = MoEConfig(name="deepseekvl2_tiny_stack12_bf16", L=12, D=1280, n=64, K=6, I=896, r=32,
               S=19, windows=(2,), tokens=512, n_shared=2, seed=0)

# Batched Qwen3-VL-30B-A3B-shaped stack at 64 concurrent decode sequences.
C4 = MoEConfig(name="qwen3vl30b_a3b_stack48_b64_bf16", L=48, D=2048, n=128, K=8, I=768, r=64,
               S=32, windows=(4,), tokens=256, batch=64, has_proj=True, seed=0)

# The same shapes with 4-bit experts (the paper's on-device setting runs a 4-bit
# DeepSeek-VL2-Tiny, 1.94 MB per expert; the "q4" codec gives exactly that size).
C1Q4 = C1.with_(name="qwen3vl30b_a3b_layer_q4", codec="q4")
C3Q4 = C3.with_(name="deepseekvl2_tiny_stack12_q4", codec="q4")

# Recall-calibrated variants: rank-32 routers and expert updates scaled by 0.25
# make the next layer's routing as predictable from the current layer as the
# paper measures for its trained adapters (ExpertRecall@{K/2, K, K+2} of about
# 0.49 / 0.87 / 0.95 with the SVD adapters here, against 49.5 / 89.4 / 95.5%
# printed for Qwen3-VL-30B-A3B); the i.i.d. routers above give 0.35 / 0.50 /
# 0.58.  Same shapes, sizes and seeds otherwise.
_PREDICTABLE = dict(router_rank=32, update_scale=0.25)
C1P = C1.with_(name="qwen3vl30b_a3b_layer_bf16_calibrated", **_PREDICTABLE)
C1PQ4 = C1Q4.with_(name="qwen3vl30b_a3b_layer_q4_calibrated", **_PREDICTABLE)
C3P = C3.with_(name="deepseekvl2_tiny_stack12_bf16_calibrated", **_PREDICTABLE)
C3PQ4 = C3Q4.with_(name="deepseekvl2_tiny_stack12_q4_calibrated", **_PREDICTABLE)

CONFIGS = {"c0": C0, "c1": C1, "c2": C2, "c3": C3, "c4": C4, "c1q4": C1Q4, "c3q4": C3Q4,
           "c1p": C1P, "c1pq4": C1PQ4, "c3p": C3P, "c3pq4": C3PQ4}


def get(name: str, **overrides) -> MoEConfig:
    cfg = CONFIGS[name]
    return cfg.with_(**overrides) if overrides else cfg
