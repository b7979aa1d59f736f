"""Synthetic decode-layer workloads: seeded host tensors for a layer configuration
and their device copies.

Recipe (same for every configuration):
  x        [T,H]  N(0,1) rounded to bf16 (fp32 for fp32-activation layers)
  router_w [E,H]  N(0, 1/sqrt(H)), same dtype rule
  bias     [E]    none, N(0, sd) in fp32 ("normal:sd"), or -s*ln(rank) ("zipf:s")
  experts         gate/up N(0, 1/sqrt(H)), down N(0, 1/sqrt(I)), quantised to
                  FP8-E4M3 with 128x128 fp32 block scales or to MXFP4
Gaussian draws are Irwin-Hall(12) from a counter-based SplitMix64 stream keyed by
(seed, tensor, layer / batch, expert).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

from . import synth
from .configs import SEED, LayerConfig


@dataclass
class HostLayer:
    cfg: LayerConfig
    router_w: np.ndarray  # uint16 (bf16 bits) or float32
    bias: Optional[np.ndarray]
    expert_w: np.ndarray  # uint8 [E, expert bytes]
    scales: np.ndarray  # float32 [E, n] (FP8) or uint8 [E, n] (MXFP4)


def host_x(cfg: LayerConfig, T: int, batch: int = 0, seed: int = SEED) -> np.ndarray:
    if cfg.act == "bf16":
        return synth.x_bf16(seed, batch, T, cfg.hidden)
    return synth.x_f32(seed, batch, T, cfg.hidden)


def host_layer(cfg: LayerConfig, layer: int = 0, seed: int = SEED) -> HostLayer:
    E, H, I = cfg.n_experts, cfg.hidden, cfg.inter
    rw = synth.router_bf16(seed, layer, E, H) if cfg.router == "bf16" else synth.router_f32(seed, layer, E, H)
    bias = None
    if cfg.bias:
        kind, val = cfg.bias.split(":")
        if kind == "normal":
            bias = synth.bias_normal(seed, layer, E, float(val))
        elif kind == "zipf":
            bias = synth.bias_zipf(seed, layer, E, float(val))
        else:
            raise ValueError(cfg.bias)
    w, s = synth.experts(seed, layer, cfg.wfmt_id, E, H, I)
    return HostLayer(cfg, rw, bias, w, s)


def to_device(a: Optional[np.ndarray], device="cuda"):
    """Copy a host array to the device as raw bytes of the same shape (bf16 bits
    travel as int16)."""
    import torch

    if a is None:
        return None
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def empty_y(cfg: LayerConfig, T: int, device="cuda"):
    import torch

    return torch.empty((T, cfg.hidden), dtype=torch.bfloat16 if cfg.act == "bf16" else torch.float32, device=device)


def y_to_f64(y) -> np.ndarray:
    import torch

    return y.detach().to("cpu", torch.float64).numpy()


def binding_config(cfg: LayerConfig, max_tokens: int, mfma_min_tokens: int = 0, screen_min_tokens: int = 0,
                   weight_layout: int = 0):
    from . import binding as B

    return B.make_config(
        cfg.hidden, cfg.n_experts, cfg.inter, cfg.topk, max_tokens,
        act_dtype=B.MOE_DTYPE_BF16 if cfg.act == "bf16" else B.MOE_DTYPE_F32,
        router_dtype=B.MOE_DTYPE_BF16 if cfg.router == "bf16" else B.MOE_DTYPE_F32,
        wfmt=cfg.wfmt_id, mfma_min_tokens=mfma_min_tokens, screen_min_tokens=screen_min_tokens,
        weight_layout=weight_layout,
    )
