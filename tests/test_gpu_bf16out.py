"""GPU checks of the bf16-output form (steel_attn_fwd_ex with out_bf16 = 1).

Every bf16 output value is the round-to-nearest-even of the fp32 result the
default form writes, so the two are compared bit for bit after rounding the
fp32 output with torch (RNE); the bf16 form is also held to the attention
bar against the float64 oracle (max-abs <= 1e-2, mean-abs <= 1e-3), on small
cases and on sampled rows of the full low-rank top-10% workload, the case
with the largest outputs (the measured error budget of this form).
"""
import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads
from workloads import CONFIGS, small_qkv, random_block_mask

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


CASES = [
    ("packs4_d128_ragged", 1, 8, 2, 600, 600, 128, True, 0.6),
    ("single_d64", 2, 3, 3, 300, 450, 64, True, None),
    ("packs2_d128_noncausal", 1, 4, 2, 256, 320, 128, False, 0.5),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_bf16_output_is_rounded_fp32_output(case):
    name, B, Hq, Hkv, S_q, S_k, D, causal, p = case
    say(f"[bf16out] {name}")
    s = steel()
    dev = torch.device("cuda:0")
    q, k, v = small_qkv(zlib.crc32(name.encode()) % 1000, B, Hq, Hkv, S_q, S_k, D)
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    m = None if p is None else random_block_mask(np.random.default_rng(2), B, Hq, nQB, nKB, p=p)
    md = None if m is None else torch.from_numpy(m).to(dev)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    o32, l32 = s.attn_fwd_lse(qd, kd, vd, md, causal=causal)
    o16, l16 = s.attn_fwd_lse(qd, kd, vd, md, causal=causal, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert o16.dtype == torch.bfloat16
    assert torch.equal(o16, o32.to(torch.bfloat16)), "bf16 output is not the RNE of the fp32 output"
    assert torch.equal(l16, l32)
    want = oracle.attention(q, k, v, m, 1 / math.sqrt(D), causal, 64)
    err = np.abs(o16.float().cpu().numpy() - want)
    say(f"  {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= 1e-2 and err.mean() <= 1e-3


def test_bf16_output_error_budget_full_size_topk_workload():
    s = steel()
    cfg = CONFIGS["mha24_s32768_d64_causal_top10_lowrank4"]
    say("[bf16out] full-size low-rank top-10% workload")
    q, k, v, m = workloads.make_workload(cfg)
    dev = torch.device("cuda:0")
    o16, _ = s.attn_fwd_lse(q.to(dev), k.to(dev), v.to(dev), torch.from_numpy(m).to(dev),
                            scale=cfg.scale, causal=True, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    idx = np.array([(0, int(h), int(i)) for h in rng.integers(0, cfg.Hq, 8)
                    for i in rng.integers(0, cfg.S_q, 16)], dtype=np.int64)
    want = oracle.attention_rows(q, k, v, idx, m, cfg.scale, True, 64)
    got = o16.float().cpu().numpy()[idx[:, 0], idx[:, 1], idx[:, 2]]
    err = np.abs(got - want)
    say(f"  sampled rows: max_abs={err.max():.3e} mean_abs={err.mean():.3e} (|O| max {np.abs(want).max():.3f})")
    assert err.max() <= 1e-2 and err.mean() <= 1e-3
