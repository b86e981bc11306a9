"""The layer-by-layer comparison baseline in bench.py (scores and P written to
HBM in bf16 between hipBLASLt GEMMs and torch softmax/mask passes) computes
attention: checked against the float64 oracle on small cases.  Its bar is
looser than the library's (max-abs <= 5e-2, mean-abs <= 5e-3): it rounds the
scores to bf16 before the softmax, which the fused pass never does.
"""
import math
import sys

import numpy as np
import pytest
import torch

import bench
import oracle
from workloads import small_qkv, random_block_mask

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("case", [
    ("mha_causal", 1, 2, 2, 512, 512, 64, True, None),
    ("gqa_masked", 1, 8, 2, 384, 384, 128, True, 0.6),
])
def test_unfused_baseline_against_oracle(case):
    name, B, Hq, Hkv, S_q, S_k, D, causal, p = case
    print(f"[unfused] {name}", file=sys.stderr, flush=True)
    q, k, v = small_qkv(3, B, Hq, Hkv, S_q, S_k, D)
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    m = None
    if p is not None:
        m = random_block_mask(np.random.default_rng(4), B, Hq, nQB, nKB, p=p)
        m[:, :, np.arange(nQB), np.arange(nQB)] = 1  # every row keeps its diagonal block
    dev = torch.device("cuda:0")
    md = None if m is None else torch.from_numpy(m).to(dev)
    hidden = bench.hidden_scores(md, B, Hq, S_q, S_k, causal, dev)
    got = bench.unfused_attention(q.to(dev), k.to(dev), v.to(dev), hidden, 1 / math.sqrt(D))
    got = got.float().cpu().numpy().astype(np.float64)
    want = oracle.attention(q, k, v, m, 1 / math.sqrt(D), causal, 64)
    err = np.abs(got - want)
    print(f"  {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", file=sys.stderr, flush=True)
    assert err.max() <= 5e-2 and err.mean() <= 5e-3
