"""GPU parity of the structured-mask forms (window + sink blocks generated from
block coordinates, no mask tensor) through the C ABI.

The structured mask is by definition the block mask
    M[qb, kb] = (qb - W < kb <= qb) or (kb < sink),
so each case checks the window form (1) against the float64 oracle given that
mask as a tensor, to the same bar as every attention output (max-abs <= 1e-2,
mean-abs <= 1e-3), and (2) bit for bit against the mask-tensor form of the
library: both build the same live lists, so they run the same arithmetic.
"""
import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads
from workloads import CONFIGS, small_qkv

pytestmark = pytest.mark.gpu

MAX_ABS = 1e-2
MEAN_ABS = 1e-3


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


def window_mask(B, Hq, S_q, S_k, W, sink):
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    qb = np.arange(nQB)[:, None]
    kb = np.arange(nKB)[None, :]
    keep = ((kb <= qb) & (kb > qb - W)) | (kb < sink)
    return np.ascontiguousarray(np.broadcast_to(keep.astype(np.uint8), (B, Hq, nQB, nKB)))


CASES = [
    # name, B, Hq, Hkv, S_q, S_k, D, causal, window_blocks, sink_blocks
    ("gqa4_ragged_d128", 1, 8, 2, 600, 600, 128, True, 3, 1),
    ("mha_sq_lt_sk_d64", 2, 4, 4, 300, 500, 64, True, 2, 0),
    ("noncausal_sink2", 1, 4, 2, 448, 448, 128, False, 4, 2),
    ("window_wider_than_grid", 1, 2, 1, 200, 200, 64, True, 50, 0),
    ("packs_multi_item", 4, 32, 8, 1024, 1024, 128, True, 4, 1),
    ("sink_only_diag", 1, 4, 1, 512, 512, 128, True, 1, 3),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_window_form_matches_oracle_and_mask_form(case):
    name, B, Hq, Hkv, S_q, S_k, D, causal, W, sink = case
    say(f"[window] {name}: B={B} Hq={Hq} Hkv={Hkv} S_q={S_q} S_k={S_k} D={D} causal={causal} "
        f"window={W} sink={sink}")
    s = steel()
    dev = torch.device("cuda:0")
    q, k, v = small_qkv(zlib.crc32(name.encode()) % 1000, B, Hq, Hkv, S_q, S_k, D)
    m = window_mask(B, Hq, S_q, S_k, W, sink)
    scale = 1.0 / math.sqrt(D)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    got = s.attn_fwd_window(qd, kd, vd, W, sink, scale=scale, causal=causal)
    ref = s.attn_fwd(qd, kd, vd, torch.from_numpy(m).to(dev), scale=scale, causal=causal)
    plan = s.Plan(None, B, Hq, Hkv, S_q, S_k, causal=causal, device=dev, window=(W, sink))
    via_plan = plan.run(qd, kd, vd, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(got, ref), "window form differs from the mask-tensor form"
    assert torch.equal(got, via_plan), "window plan + run differs from the fused window call"
    want = oracle.attention(q, k, v, m, scale, causal, 64)
    err = np.abs(got.cpu().numpy().astype(np.float64) - want)
    say(f"  {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


def test_window_plan_full_size_window_sink_workload():
    """At the full window/sink workload (S = 16384, 32/8 heads, D = 128) the
    window plan equals the mask-tensor plan bit for bit; the mask-tensor path
    is checked against the oracle at this size in test_gpu_parity."""
    s = steel()
    cfg = CONFIGS["gqa32x8_s16384_d128_window1024_sink64"]
    say("[window] full-size window/sink workload: window plan vs mask plan")
    dev = torch.device("cuda:0")
    q, k, v, m = workloads.make_workload(cfg)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    p_mask = s.Plan(torch.from_numpy(m).to(dev), cfg.B, cfg.Hq, cfg.Hkv, cfg.S_q, cfg.S_k,
                    causal=cfg.causal, device=dev)
    p_win = s.Plan(None, cfg.B, cfg.Hq, cfg.Hkv, cfg.S_q, cfg.S_k, causal=cfg.causal, device=dev,
                   window=(cfg.window_blocks, cfg.sink_blocks))
    a = p_mask.run(qd, kd, vd, scale=cfg.scale)
    b = p_win.run(qd, kd, vd, scale=cfg.scale)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
