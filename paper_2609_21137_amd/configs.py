"""Workload shapes of the compressed-MoE decode layer.

Each workload is one MoE layer (or a stack of them) with the expert matrices
stored as blockwise VQ codes plus a shared-basis low-rank term. Shapes follow
the Qwen3-30B-A3B MoE layer of the paper's model table (Table 2: H=2048,
I=768, E=128, top-8) with the rank and code-book sizes fixed per workload.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    H: int          # hidden size
    I: int          # expert intermediate size
    E: int          # experts per layer
    top_k: int      # experts selected per token
    d: int          # VQ block length (along the input dimension)
    K: int          # code words per code book
    r: int          # rank of the shared low-rank basis
    B: int          # decode batch (tokens per step)
    seed: int
    layers: int = 1
    hot_experts: tuple = ()      # experts whose router logit gets +hot_bias
    hot_bias: float = 0.0
    rotate_layers: int = 0       # layers a benchmark rotates over (0: its default)
    act: str = "silu_glu"        # expert activation: "silu_glu" (gate+up) or "relu2_up" (up only)
    description: str = field(default="", compare=False)

    @property
    def shape(self):
        return (self.H, self.I, self.E, self.top_k, self.d, self.K, self.r)


TINY = Workload("tiny_h256_i128_e8_top2_b1", H=256, I=128, E=8, top_k=2, d=4, K=16, r=8,
                B=1, seed=0, description="tiny layer, d=4, K=16, r=8, batch 1")
QWEN3_B1 = Workload("qwen3_30b_a3b_moe_layer_b1", H=2048, I=768, E=128, top_k=8, d=8, K=256,
                    r=128, B=1, seed=1,
                    description="Qwen3-30B-A3B-shaped MoE layer, d=8, K=256, r=128, batch 1")
QWEN3_B16 = Workload("qwen3_30b_a3b_moe_layer_b16", H=2048, I=768, E=128, top_k=8, d=8, K=256,
                     r=128, B=16, seed=1,
                     description="Qwen3-30B-A3B-shaped MoE layer, batch 16")
WIDE_SKEW_B4 = Workload("wide_h4096_i1536_e64_top6_b4_skewed", H=4096, I=1536, E=64, top_k=6,
                        d=8, K=256, r=256, B=4, seed=2, hot_experts=tuple(range(8)),
                        hot_bias=2.0,
                        description="wider layer, r=256, batch 4, 8 hot experts (+2.0 logit)")
QWEN3_48L_B16 = Workload("qwen3_48_layer_decode_step_b16", H=2048, I=768, E=128, top_k=8, d=8,
                         K=256, r=128, B=16, seed=1, layers=48,
                         description="48 stacked Qwen3-shaped layers, RMS-normalised between")

# the other gate+up models of the paper's model table (Table 2), at their
# (d, K, r); two rotated layers already exceed the last-level cache
DSV2_LITE_B1 = Workload("deepseek_v2_lite_moe_layer_b1", H=2048, I=1408, E=64, top_k=6, d=8, K=256,
                        r=384, B=1, seed=3, rotate_layers=2,
                        description="DeepSeek-V2-Lite-shaped MoE layer, d=8, K=256, r=384, batch 1")
OLMOE_B1 = Workload("olmoe_1b_7b_moe_layer_b1", H=2048, I=1024, E=64, top_k=8, d=4, K=256, r=256,
                    B=1, seed=4, rotate_layers=2,
                    description="OLMoE-1B-7B-shaped MoE layer, d=4, K=256, r=256, batch 1")
GEMMA4_B1 = Workload("gemma4_26b_a4b_moe_layer_b1", H=2816, I=704, E=128, top_k=8, d=8, K=256,
                     r=384, B=1, seed=5, rotate_layers=2,
                     description="Gemma-4-26B-A4B-shaped MoE layer, d=8, K=256, r=384, batch 1")
OTHER_MODELS_B1 = (DSV2_LITE_B1, OLMOE_B1, GEMMA4_B1)

# the up-only model of the table: experts p = max(u, 0)^2 without a gate
# projection; H = 2688 and I = 1856 are already multiples of the kernels'
# 64 and 32 (no padding of either dimension)
NEMOTRON3_B1 = Workload("nemotron3_nano_moe_layer_b1", H=2688, I=1856, E=128, top_k=6, d=8, K=256,
                        r=512, B=1, seed=6, rotate_layers=2, act="relu2_up",
                        description="Nemotron-3-Nano-shaped up-only squared-ReLU MoE layer, d=8, K=256, "
                                    "r=512, batch 1")
NEMOTRON3_B16 = dataclasses.replace(NEMOTRON3_B1, name="nemotron3_nano_moe_layer_b16", B=16,
                                    description="Nemotron-3-Nano-shaped up-only layer, batch 16")

WORKLOADS = {w.name: w for w in (TINY, QWEN3_B1, QWEN3_B16, WIDE_SKEW_B4, QWEN3_48L_B16,
                                 *OTHER_MODELS_B1, NEMOTRON3_B1, NEMOTRON3_B16)}
