"""Shapes of the five synthetic MoE-layer workloads.

Mixtral-shaped layers: hidden 4096, 8 experts, top-2, expert ffn 14336.
Fine-grained layer: hidden 2048, 64 routed experts top-6 plus 2 shared
experts, expert ffn 1408.  The paper's models (Mixtral-8x7B, DeepSeek-V2-Lite)
and ShareGPT traffic are not available; these layers take the models' shapes
and a Zipf-skewed router that imitates the skewed expert activation the paper
shows (section III-B).
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class MoEConfig:
    name: str
    cid: int            # workload id, part of every tensor seed
    T: int              # tokens per layer call
    C: int              # model hidden size
    E: int              # routed experts
    k: int              # experts per token
    R: int              # expert ffn size
    S: int = 0          # shared experts (always on, weight 1)
    act: str = "bf16"   # activation dtype: "f32" or "bf16"
    zipf_s: float = 0.0  # router bias b_e = -zipf_s * ln(rank(e) + 1); 0 = no bias
    layers: int = 1     # MoE layers in the stack
    resident: int = 0   # experts per layer resident on the GPU (0 = all)
    pred_hidden: int = 0  # predictor MLP hidden width (0 = no predictor)
    pred_group: int = 0   # token rows pooled per predictor evaluation
    w_std: float = 0.02   # expert weight standard deviation

    @property
    def G(self) -> int:
        return self.E + self.S


CONFIGS = {
    "tiny": MoEConfig("tiny", 1, T=16, C=256, E=4, k=2, R=512, act="f32"),
    "mixtral_decode": MoEConfig("mixtral_decode", 2, T=1, C=4096, E=8, k=2, R=14336,
                                zipf_s=1.2),
    "mixtral_prefill": MoEConfig("mixtral_prefill", 3, T=512, C=4096, E=8, k=2, R=14336,
                                 zipf_s=1.2),
    "beam_stack": MoEConfig("beam_stack", 4, T=8, C=4096, E=8, k=2, R=14336, zipf_s=1.2,
                            layers=32, resident=4, pred_hidden=512, pred_group=8),
    "fine_grained": MoEConfig("fine_grained", 5, T=2048, C=2048, E=64, k=6, R=1408, S=2,
                              zipf_s=1.0),
}


def get_config(name: str) -> MoEConfig:
    return CONFIGS[name]
