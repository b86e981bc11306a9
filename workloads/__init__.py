"""Seeded synthetic inputs for the sparsity-aware fused attention forward.

This module is shared by the CPU oracle side (tests, the CPU baseline) and by
the GPU side (tests, bench, smoke).  It only draws numbers and builds block
masks; it holds none of the attention arithmetic, so neither side can borrow
a step of the method from here.

Workloads.  The paper evaluates attention shapes only: BERT attention with 12
heads and head dimension 64 (Section V-B, V-C) and Llama3.1-1B attention with
32 heads, head dimension 64, sequence lengths 2048 to 32768 (Section V-D).  No
dataset or trained weight enters the method, so every input here is drawn
from a seeded generator.  The five named configurations below are the ones the
throughput metric is quoted on; their masks exercise the three tile cases of
Section IV-A (skipped, unmasked, partially masked) including the windowed
variant the same paragraph names.

Generation recipe (all on the CPU, bit-reproducible):

* one ``torch.Generator`` seeded with ``seed`` draws Q, then K, then V as
  float32 N(0,1) tensors of shape [B, H, S, D] (H = Hq for Q, Hkv for K, V);
* for the low-rank workload it then draws, per head, U [S, r] and W [D, r]
  i.i.d. N(0,1) from the same generator, forms L = scale_lr * U W^T / sqrt(r)
  and adds the same L to that head's Q and K (a shared component);
* every tensor is then rounded to bfloat16 with round-to-nearest-even;
* block masks are uint8 [B, Hq, nQB, nKB], nonzero = live; ``None`` means
  "every block live" (the causal structure is applied by the consumer).
"""
from __future__ import annotations

import dataclasses
import math
from fractions import Fraction
from typing import Optional

import numpy as np
import torch

BLK = 64


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    B: int
    Hq: int
    Hkv: int
    S_q: int
    S_k: int
    D: int
    causal: bool
    mask: str            # "none" | "bernoulli" | "window_sink" | "topk_meanpool"
    seed: int = 0
    p_keep: float = 0.25           # bernoulli
    window_blocks: int = 16        # window_sink: 1024 tokens / 64
    sink_blocks: int = 1           # window_sink: first 64 tokens
    topk_frac: float = 0.10        # topk_meanpool
    lowrank_rank: int = 0          # shared low-rank component on Q and K
    lowrank_scale: float = 0.0
    blk: int = BLK

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)

    @property
    def nQB(self) -> int:
        return (self.S_q + self.blk - 1) // self.blk

    @property
    def nKB(self) -> int:
        return (self.S_k + self.blk - 1) // self.blk

    def describe(self) -> dict:
        return {
            "workload": self.name, "B": self.B, "Hq": self.Hq, "Hkv": self.Hkv,
            "S_q": self.S_q, "S_k": self.S_k, "D": self.D, "causal": self.causal,
            "mask": self.mask, "blk": self.blk, "seed": self.seed,
        }


# The five throughput/parity workloads.  Names state what they are.
CONFIGS = {
    "mha1_s512_d64_causal": Config(
        "mha1_s512_d64_causal", 1, 1, 1, 512, 512, 64, True, "none"),
    "gqa32x8_s4096_d128_causal": Config(
        "gqa32x8_s4096_d128_causal", 1, 32, 8, 4096, 4096, 128, True, "none"),
    "gqa32x8_s8192_d128_causal_bernoulli25": Config(
        "gqa32x8_s8192_d128_causal_bernoulli25", 1, 32, 8, 8192, 8192, 128, True,
        "bernoulli"),
    "gqa32x8_s16384_d128_window1024_sink64": Config(
        "gqa32x8_s16384_d128_window1024_sink64", 1, 32, 8, 16384, 16384, 128, True,
        "window_sink"),
    "mha24_s32768_d64_causal_top10_lowrank4": Config(
        "mha24_s32768_d64_causal_top10_lowrank4", 1, 24, 24, 32768, 32768, 64, True,
        "topk_meanpool", lowrank_rank=4, lowrank_scale=2.0),
}
CONFIG_ORDER = list(CONFIGS)


def make_qkv(cfg: Config):
    """Draw bf16 Q [B,Hq,S_q,D], K and V [B,Hkv,S_k,D] on the CPU."""
    g = torch.Generator().manual_seed(cfg.seed)
    q = torch.randn((cfg.B, cfg.Hq, cfg.S_q, cfg.D), generator=g, dtype=torch.float32)
    k = torch.randn((cfg.B, cfg.Hkv, cfg.S_k, cfg.D), generator=g, dtype=torch.float32)
    v = torch.randn((cfg.B, cfg.Hkv, cfg.S_k, cfg.D), generator=g, dtype=torch.float32)
    if cfg.lowrank_rank > 0:
        if cfg.Hq != cfg.Hkv or cfg.S_q != cfg.S_k:
            raise ValueError("the shared low-rank component needs Hq == Hkv and S_q == S_k")
        r = cfg.lowrank_rank
        for b in range(cfg.B):
            for h in range(cfg.Hq):
                u = torch.randn((cfg.S_q, r), generator=g, dtype=torch.float32)
                w = torch.randn((cfg.D, r), generator=g, dtype=torch.float32)
                low = (cfg.lowrank_scale / math.sqrt(r)) * (u @ w.T)
                q[b, h] += low
                k[b, h] += low
    return (q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16))


def bernoulli_mask(cfg: Config) -> np.ndarray:
    """Each block kept with probability p, seeded per query head; diagonal kept."""
    m = np.zeros((cfg.B, cfg.Hq, cfg.nQB, cfg.nKB), dtype=np.uint8)
    for b in range(cfg.B):
        for h in range(cfg.Hq):
            g = torch.Generator().manual_seed(1000 * cfg.seed + h + 100003 * b)
            keep = (torch.rand((cfg.nQB, cfg.nKB), generator=g) < cfg.p_keep).numpy()
            keep = keep.astype(np.uint8)
            d = np.arange(min(cfg.nQB, cfg.nKB))
            keep[d, d] = 1
            m[b, h] = keep
    return m


def window_sink_mask(cfg: Config) -> np.ndarray:
    """Block-level sliding window of ``window_blocks`` blocks ending at the
    diagonal block, plus the first ``sink_blocks`` key blocks."""
    qb = np.arange(cfg.nQB)[:, None]
    kb = np.arange(cfg.nKB)[None, :]
    keep = ((kb <= qb) & (kb > qb - cfg.window_blocks)) | (kb < cfg.sink_blocks)
    m = np.broadcast_to(keep.astype(np.uint8), (cfg.B, cfg.Hq, cfg.nQB, cfg.nKB))
    return np.ascontiguousarray(m)


def topk_meanpool_mask(cfg: Config, q_bf16: torch.Tensor, k_bf16: torch.Tensor) -> np.ndarray:
    """Per (b, h, qb): rank the causal candidate blocks kb <= qb by the product of
    the mean-pooled query block and the mean-pooled key block (fp64, from the
    bf16 values), keep the top ceil(frac*(qb+1)) (ties to the smaller kb), then
    add the diagonal block."""
    blk = cfg.blk
    nQB, nKB = cfg.nQB, cfg.nKB
    G = cfg.Hq // cfg.Hkv
    m = np.zeros((cfg.B, cfg.Hq, nQB, nKB), dtype=np.uint8)
    for b in range(cfg.B):
        for h in range(cfg.Hq):
            qf = q_bf16[b, h].to(torch.float64).numpy()
            kf = k_bf16[b, h // G].to(torch.float64).numpy()
            qpad = np.zeros((nQB * blk, cfg.D)); qpad[: cfg.S_q] = qf
            kpad = np.zeros((nKB * blk, cfg.D)); kpad[: cfg.S_k] = kf
            qcnt = np.minimum(blk, cfg.S_q - np.arange(nQB) * blk)[:, None]
            kcnt = np.minimum(blk, cfg.S_k - np.arange(nKB) * blk)[:, None]
            qm = qpad.reshape(nQB, blk, cfg.D).sum(1) / qcnt
            km = kpad.reshape(nKB, blk, cfg.D).sum(1) / kcnt
            sc = qm @ km.T
            for qb in range(nQB):
                ncand = min(qb + 1, nKB)
                keep_n = math.ceil(Fraction(str(cfg.topk_frac)) * ncand)
                cand = sc[qb, :ncand]
                # stable sort on -score: ties keep the smaller kb first
                idx = np.argsort(-cand, kind="stable")[:keep_n]
                m[b, h, qb, idx] = 1
                if qb < nKB:
                    m[b, h, qb, qb] = 1
    return m


def make_block_mask(cfg: Config, q=None, k=None) -> Optional[np.ndarray]:
    if cfg.mask == "none":
        return None
    if cfg.mask == "bernoulli":
        return bernoulli_mask(cfg)
    if cfg.mask == "window_sink":
        return window_sink_mask(cfg)
    if cfg.mask == "topk_meanpool":
        if q is None or k is None:
            raise ValueError("topk_meanpool needs the bf16 Q and K")
        return topk_meanpool_mask(cfg, q, k)
    raise ValueError(f"unknown mask kind {cfg.mask!r}")


def make_workload(cfg: Config):
    """(q, k, v, block_mask) on the CPU: bf16 torch tensors and a uint8 numpy
    mask (or None)."""
    q, k, v = make_qkv(cfg)
    return q, k, v, make_block_mask(cfg, q, k)


def random_block_mask(rng: np.random.Generator, B, Hq, nQB, nKB, p=0.5, kill_rows=0):
    """Small random masks for parity cases; ``kill_rows`` rows are zeroed
    entirely (dead query blocks)."""
    m = (rng.random((B, Hq, nQB, nKB)) < p).astype(np.uint8)
    for _ in range(kill_rows):
        m[rng.integers(B), rng.integers(Hq), rng.integers(nQB), :] = 0
    return m


def small_qkv(seed, B, Hq, Hkv, S_q, S_k, D, std=1.0):
    g = torch.Generator().manual_seed(seed)
    q = (std * torch.randn((B, Hq, S_q, D), generator=g)).to(torch.bfloat16)
    k = (std * torch.randn((B, Hkv, S_k, D), generator=g)).to(torch.bfloat16)
    v = torch.randn((B, Hkv, S_k, D), generator=g).to(torch.bfloat16)
    return q, k, v
