"""The five synthetic workloads: shapes, trit distribution, salient fraction.

Matrix shapes (N out x K in, PyTorch nn.Linear orientation) follow the fused
linears of one decoder layer of each model family.  The stacks repeat the
same four shapes per layer with independent seeds per (layer, matrix).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from fractions import Fraction


@dataclass(frozen=True)
class Workload:
    name: str
    shapes: tuple  # ((role, N, K), ...) per layer
    layers: int
    batches: tuple
    p0: Fraction = Fraction(2, 5)
    frac: Fraction = Fraction(2, 100)
    note: str = ""
    resid: str = "fp16"  # residual value storage: "fp16" or "e4m3"
    groups: int = 0  # columns per quantization group (0: one group per row)

    def matrices(self):
        """Yield (layer, mat, role, N, K) in per-token execution order."""
        for layer in range(self.layers):
            for mat, (role, N, K) in enumerate(self.shapes):
                yield layer, mat, role, N, K


LLAMA3_8B = (("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096), ("down", 4096, 14336))
QWEN3_14B = (("qkv", 7168, 5120), ("o", 5120, 5120), ("gate_up", 34816, 5120), ("down", 5120, 17408))
LLAMA3_70B = (("qkv", 10240, 8192), ("o", 8192, 8192), ("gate_up", 57344, 8192), ("down", 8192, 28672))

WORKLOADS = {
    "gemv_4096x4096": Workload("gemv_4096x4096", (("single", 4096, 4096),), 1, (1,),
                               note="single 4096x4096 GEMV"),
    "llama3_8b_layer": Workload("llama3_8b_layer", LLAMA3_8B, 1, (1,),
                                note="one Llama-3-8B-shaped decoder layer's linears"),
    "llama3_8b_stack": Workload("llama3_8b_stack", LLAMA3_8B, 32, (1, 4),
                                note="32-layer Llama-3-8B-shaped linear stack"),
    "qwen3_14b_stack": Workload("qwen3_14b_stack", QWEN3_14B, 40, (1, 8, 16),
                                frac=Fraction(3, 100),
                                note="40-layer Qwen3-14B-shaped linear stack, 3% salient"),
    "llama3_70b_stack": Workload("llama3_70b_stack", LLAMA3_70B, 80, (1, 16),
                                 p0=Fraction(1, 2),
                                 note="80-layer Llama-3-70B-shaped linear stack, P(0)=0.5"),
    # the paper's evaluation storage: 5% salient columns, FP8 E4M3 residual
    # values, a column bitmap (1.7 bits per weight in its accounting)
    "llama3_8b_stack_e4m3": Workload("llama3_8b_stack_e4m3", LLAMA3_8B, 32, (1, 4),
                                     frac=Fraction(5, 100), resid="e4m3",
                                     note="32-layer Llama-3-8B-shaped stack, 5% salient, E4M3 residual"),
    # the paper's full format: 128-column groups with scale and bias, 26-byte
    # packs, 5% salient columns with E4M3 residual values and a bitmap
    "llama3_8b_stack_g128": Workload("llama3_8b_stack_g128", LLAMA3_8B, 32, (1,),
                                     frac=Fraction(5, 100), resid="e4m3", groups=128,
                                     note="32-layer Llama-3-8B-shaped stack in the paper's grouped format"),
}

ORDER = ["gemv_4096x4096", "llama3_8b_layer", "llama3_8b_stack", "qwen3_14b_stack", "llama3_70b_stack"]
