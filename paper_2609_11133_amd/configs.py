"""Shapes of the MoE decode-layer workloads.

Each entry describes one decode layer of a Mixture-of-Experts model in the form the
library consumes: hidden size H, expert count E, top-k, SwiGLU intermediate size I,
activation / router dtypes, the expert weight format, the router bias recipe and the
per-step token counts (decode batch sizes) it is exercised at.  The 235B- and
480B-shaped layers follow the two MoE models the paper deploys (Experimental Setup,
models table row): Qwen3-235B-A22B and Qwen3-Coder-480B-A35B.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

SEED = 1234  # the paper's workload generator seed (Experimental Setup, workloads)


@dataclass(frozen=True)
class LayerConfig:
    name: str
    hidden: int
    n_experts: int
    topk: int
    inter: int
    act: str  # "bf16" or "f32"
    router: str  # "bf16" or "f32"
    wfmt: str  # "fp8" (E4M3, 128x128 fp32 block scales), "mxfp4" (E2M1, E8M0 per 32) or
    #            "nvfp4" (E2M1, E4M3 per 16, fp32 per matrix)
    bias: Optional[str]  # None, "normal:0.5" (sd) or "zipf:1.1"
    tokens: List[int] = field(default_factory=list)
    layers: int = 1

    @property
    def wfmt_id(self) -> int:
        return {"fp8": 0, "mxfp4": 1, "nvfp4": 2}[self.wfmt]

    def expert_weight_bytes(self) -> int:
        H, I = self.hidden, self.inter
        return 3 * H * I if self.wfmt == "fp8" else 3 * H * I // 2

    def expert_scale_bytes(self) -> int:
        H, I = self.hidden, self.inter
        if self.wfmt == "fp8":
            return 4 * 3 * (H // 128) * (I // 128)
        if self.wfmt == "mxfp4":
            return 3 * H * I // 32
        return 16 + 3 * H * I // 16

    def matrix_bytes(self, mat: int) -> int:
        """Weight + scale bytes of one matrix of one expert (0 gate, 1 up, 2 down);
        the NVFP4 matrix scales (16 bytes per expert) are counted with the gate."""
        H, I = self.hidden, self.inter
        if self.wfmt == "fp8":
            return H * I + 4 * (H // 128) * (I // 128)
        if self.wfmt == "mxfp4":
            return H * I // 2 + H * I // 32
        return H * I // 2 + H * I // 16 + (16 if mat == 0 else 0)

    def expert_bytes(self) -> int:
        """Algorithmic bytes streamed per activated expert (weights + scales)."""
        return self.expert_weight_bytes() + self.expert_scale_bytes()

    def w13_bytes(self) -> int:
        """Gate+up bytes (weights + scales) of one expert."""
        return self.matrix_bytes(0) + self.matrix_bytes(1)

    def w2_bytes(self) -> int:
        return self.matrix_bytes(2)


TINY = LayerConfig("tiny", 256, 8, 2, 128, "f32", "f32", "fp8", None, [4])
QWEN3_235B = LayerConfig("qwen3-235b-a22b", 4096, 128, 8, 1536, "bf16", "bf16", "fp8", None, [1, 8, 32, 64])
QWEN3_480B = LayerConfig(
    "qwen3-coder-480b-a35b", 6144, 160, 8, 2560, "bf16", "bf16", "fp8", "normal:0.5", [1, 16, 64, 128]
)
# One GPU's share of the 480B layer in the paper's TP4 decode lane (Experimental Setup):
# every expert's intermediate dimension split four ways, I = 2560 / 4 = 640 (5 blocks of
# 128); T up to the lane's decode concurrency of 48 and beyond.
QWEN3_480B_TP4 = LayerConfig(
    "qwen3-coder-480b-a35b-tp4", 6144, 160, 8, 640, "bf16", "bf16", "fp8", "normal:0.5", [1, 16, 48, 64, 128]
)
QWEN3_480B_X12 = LayerConfig(
    "qwen3-coder-480b-a35b-x12",
    6144,
    160,
    8,
    2560,
    "bf16",
    "bf16",
    "fp8",
    "normal:0.5",
    [1, 2, 4, 8, 16, 32, 64, 128, 256],
    layers=12,
)
QWEN3_235B_MXFP4 = LayerConfig(
    "qwen3-235b-a22b-mxfp4-zipf", 4096, 128, 8, 1536, "bf16", "bf16", "mxfp4", "zipf:1.1", [256]
)

# The paper deploys Qwen3-235B-A22B in NVFP4 (Experimental Setup, models row).
QWEN3_235B_NVFP4 = LayerConfig("qwen3-235b-a22b-nvfp4", 4096, 128, 8, 1536, "bf16", "bf16", "nvfp4", None, [1, 8, 32, 64])
QWEN3_235B_NVFP4_ZIPF = LayerConfig(
    "qwen3-235b-a22b-nvfp4-zipf", 4096, 128, 8, 1536, "bf16", "bf16", "nvfp4", "zipf:1.1", [256]
)

ALL = [TINY, QWEN3_235B, QWEN3_480B, QWEN3_480B_TP4, QWEN3_480B_X12, QWEN3_235B_MXFP4, QWEN3_235B_NVFP4, QWEN3_235B_NVFP4_ZIPF]
BY_NAME = {c.name: c for c in ALL}
