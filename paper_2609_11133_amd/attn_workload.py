"""Synthetic decode-attention workloads: seeded host tensors for one decode step of
grouped-query attention over a paged KV cache, and their device copies.

Shapes.  Query/key-value head counts of the paper's two MoE models (their public model
configurations): Qwen3-235B-A22B 64 query / 4 key-value heads, Qwen3-Coder-480B-A35B 96
/ 8, head dimension 128; the 480B decode lane runs TP4 (Experimental Setup table), so one
GPU holds 24 query / 2 key-value heads of it.  Batch = the decode concurrency of the
Experimental Setup (24 for 235B, 48 for 480B).  Pages of 16 tokens.

Context lengths (the paper's two workloads, Experimental Setup, workloads paragraph):
  standard  input length from {64, 128, 256, 512, 1024, 2048} with weights
            {0.18, 0.24, 0.26, 0.18, 0.10, 0.04}, output length from {32, 64, 128, 256,
            512, 1024} with weights {0.16, 0.22, 0.26, 0.20, 0.12, 0.04}; a decode step
            at a uniform point of the generation: L = input + u, u uniform in 1..output
  agentic   4 tool-calling turns, base input 512, 128 generated tokens per turn, a
            256-token tool result appended after each turn: turn i uniform in 0..3,
            L = 512 + i * (128 + 256) + u, u uniform in 1..128
  long:N    every sequence at N tokens (a long-context point)
Values: q, K and V ~ N(0, 1) rounded to bf16 (counter-based streams of ``synth``);
physical pages are a seeded permutation of the pool, so a sequence's pages are
scattered; the page pool holds every sequence's pages plus 10 % unused ones filled with
NaN bit patterns, which no result may depend on.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

from . import synth
from .configs import SEED

STANDARD_IN = ([64, 128, 256, 512, 1024, 2048], [0.18, 0.24, 0.26, 0.18, 0.10, 0.04])
STANDARD_OUT = ([32, 64, 128, 256, 512, 1024], [0.16, 0.22, 0.26, 0.20, 0.12, 0.04])
NAN_BF16 = 0x7FC1


@dataclass(frozen=True)
class AttnConfig:
    name: str
    n_q_heads: int
    n_kv_heads: int
    batch: int
    mix: str  # "standard", "agentic" or "long:N"
    head_dim: int = 128
    page: int = 16
    capacity: Optional[int] = None  # tokens a block-table row holds (None: the longest context)


ATTN_CONFIGS = [
    AttnConfig("qwen3-235b-a22b-attn-agentic", 64, 4, 24, "agentic"),
    AttnConfig("qwen3-235b-a22b-attn-standard", 64, 4, 24, "standard"),
    AttnConfig("qwen3-coder-480b-a35b-tp4-attn-agentic", 24, 2, 48, "agentic"),
    AttnConfig("qwen3-235b-a22b-attn-long32k", 64, 4, 24, "long:32768"),
    # the agentic step on a configuration sized for 32K-token contexts (block-table rows
    # of 2048 pages), as a server that also admits long contexts would size it
    AttnConfig("qwen3-235b-a22b-attn-agentic-cap32k", 64, 4, 24, "agentic", capacity=32768),
]
ATTN_BY_NAME = {c.name: c for c in ATTN_CONFIGS}


def context_lengths(mix: str, batch: int, seed: int = SEED, draw: int = 0) -> np.ndarray:
    """Seeded context lengths of `batch` sequences in decode under the given mix."""
    rng = np.random.default_rng([seed, 9001, draw])
    if mix == "standard":
        inp = rng.choice(STANDARD_IN[0], size=batch, p=STANDARD_IN[1])
        out = rng.choice(STANDARD_OUT[0], size=batch, p=STANDARD_OUT[1])
        L = inp + 1 + (rng.random(batch) * out).astype(np.int64)
    elif mix == "agentic":
        turn = rng.integers(0, 4, size=batch)
        L = 512 + turn * (128 + 256) + 1 + (rng.random(batch) * 128).astype(np.int64)
    elif mix.startswith("long:"):
        L = np.full(batch, int(mix.split(":")[1]), np.int64)
    else:
        raise ValueError(f"unknown length mix {mix!r}")
    return L.astype(np.int32)


@dataclass
class HostAttn:
    q: np.ndarray            # uint16 [B, Hq, D]
    k_cache: np.ndarray      # uint16 [n_pages, Hkv, P, D]
    v_cache: np.ndarray      # uint16 [n_pages, Hkv, D, P]
    block_table: np.ndarray  # int32 [B, max_pages]
    ctx: np.ndarray          # int32 [B]

    @property
    def n_pages(self) -> int:
        return self.k_cache.shape[0]

    def kv_bytes(self, n_kv_heads: int, head_dim: int = 128) -> int:
        """Bytes of K and V the step must read: every context token's key and value."""
        return int(self.ctx.astype(np.int64).sum()) * n_kv_heads * head_dim * 2 * 2


def host_attn(cfg: AttnConfig, seed: int = SEED, draw: int = 0, ctx: Optional[np.ndarray] = None,
              max_pages: Optional[int] = None, garbage: bool = True) -> HostAttn:
    """Host tensors of one decode step; `ctx` overrides the mix's lengths."""
    B, Hq, Hkv, D, P = cfg.batch, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.page
    L = context_lengths(cfg.mix, B, seed, draw) if ctx is None else np.asarray(ctx, np.int32)
    pages = (L.astype(np.int64) + P - 1) // P
    if max_pages is None and cfg.capacity:
        max_pages = (cfg.capacity + P - 1) // P
    mp = int(max(1, pages.max())) if max_pages is None else max_pages
    used = int(pages.sum())
    n_pages = max(1, used + used // 10)
    rng = np.random.default_rng([seed, 9002, draw])
    perm = rng.permutation(n_pages).astype(np.int32)
    bt = np.zeros((B, mp), np.int32)
    o = 0
    for b in range(B):
        bt[b, : pages[b]] = perm[o: o + pages[b]]
        o += pages[b]
    q = synth.normal_bf16(seed, "q", draw, 0, B * Hq * D).reshape(B, Hq, D)
    kc = synth.normal_bf16(seed, "k", draw, 0, n_pages * Hkv * P * D).reshape(n_pages, Hkv, P, D)
    vc = synth.normal_bf16(seed, "v", draw, 0, n_pages * Hkv * D * P).reshape(n_pages, Hkv, D, P)
    if garbage:
        # unused pages, and the slots past each context in its last page, hold NaN bits
        unused = perm[used:]
        kc[unused] = NAN_BF16
        vc[unused] = NAN_BF16
        for b in range(B):
            if pages[b] and L[b] % P:
                last = bt[b, pages[b] - 1]
                kc[last, :, L[b] % P:, :] = NAN_BF16
                vc[last, :, :, L[b] % P:] = NAN_BF16
    return HostAttn(q, kc, vc, bt, L)


def to_device(h: HostAttn, device="cuda"):
    import torch

    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)  # noqa: E731
    return dict(q=t(h.q.view(np.int16)), k_cache=t(h.k_cache.view(np.int16)), v_cache=t(h.v_cache.view(np.int16)),
                block_table=t(h.block_table), ctx=t(h.ctx))
