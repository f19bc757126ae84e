"""The five synthetic workloads of the BOM hot path.

Shapes follow the paper's fine-tuning and language-model workloads (classification heads
with C = 10 and C = 1000 outputs; next-token heads with V = 32,000 / 50,304 / 128,256).
Everything is seeded and synthetic: features H ~ N(0, 1), head W ~ N(0, 0.02) (the paper's
initialisation standard deviation for its language models), flat parameters theta ~ N(0, 0.02),
backbone gradients u ~ N(0, 1e-3), logits Z ~ N(0, sqrt(0.0004 * d)), labels uniform (heads with
C <= 1000) or truncated Zipf(1.1) (vocabularies). "N(0, x)" means standard deviation x.

Hyperparameters are the paper's fixed coefficients: lambda = 0.5, beta1 = 0.9, beta2 = 0.999,
eps = 1e-8; decoupled decay 0.01 for fine-tuning heads (bias exempt) and 0.1 for language models.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    N: int                 # rows of Z: examples or valid next-token positions
    d: int                 # head input width
    V: int                 # output width (classes or vocabulary)
    P: int                 # flat parameter count (head W first, then bias if any, then backbone)
    dtype: str             # "f32" or "bf16" for H, W, Z, R
    labels: str            # "uniform" or "zipf"
    lr: float
    weight_decay: float
    has_bias: bool = False
    factored: bool = False  # second moment factored per block_rows x block_cols block
    block_rows: int = 4096
    block_cols: int = 4096
    steps: int = 3          # parity steps (bias corrections and history become non-trivial)
    lam: float = 0.5
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    ignore_index: int = -100
    notes: str = field(default="", compare=False)

    @property
    def logit_std(self) -> float:
        return math.sqrt(0.0004 * self.d)

    @property
    def head_params(self) -> int:
        return self.d * self.V + (self.V if self.has_bias else 0)

    def segments(self):
        """(offset, length, weight_decay) triples: weight decay exempts the bias only."""
        if self.has_bias:
            dv = self.d * self.V
            return [(0, dv, self.weight_decay), (dv, self.V, 0.0), (dv + self.V, self.P - dv - self.V,
                                                                   self.weight_decay)]
        return [(0, self.P, self.weight_decay)]


WORKLOADS = [
    Workload("tiny_linear_c10", N=256, d=128, V=10, P=1290, dtype="f32", labels="uniform", lr=1e-2,
             weight_decay=0.01, has_bias=True, steps=20,
             notes="10-class linear softmax classifier, 20 BOM steps, flat buffer = W (1280) + b (10)"),
    Workload("vision_head_c1000", N=1024, d=768, V=1000, P=86_000_000, dtype="bf16", labels="uniform",
             lr=3e-5, weight_decay=0.01,
             notes="ImageNet-1k-shaped 1000-class head on 768-d pooled features, 86M flat parameters"),
    Workload("lm_small_v32000", N=4096, d=768, V=32000, P=124_000_000, dtype="bf16", labels="zipf",
             lr=1e-3, weight_decay=0.1, notes="B=8 x T=512 tokens, V=32,000, 124M flat parameters"),
    Workload("lm_1b_v50304", N=8192, d=2048, V=50304, P=1_100_000_000, dtype="bf16", labels="zipf",
             lr=1e-3, weight_decay=0.1, notes="B=8 x T=1024 tokens, V=50,304, 1.1B flat parameters"),
    Workload("lm_8b_v128256", N=16384, d=4096, V=128256, P=8_000_000_000, dtype="bf16", labels="zipf",
             lr=1e-3, weight_decay=0.1, factored=True,
             notes="B=16 x T=1024 tokens, V=128,256, 8.0B flat parameters, factored second moment"),
]

BY_NAME = {w.name: w for w in WORKLOADS}
