"""GPU parity of the top-k mean-pooled block selection (steel_topk_block_mask)
through the C ABI: the mask is an integer output decided by float64
arithmetic that the library and the oracle carry out in the same order, so
the bar is bit-exact equality with the oracle's mask.
"""
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads
from workloads import CONFIGS, small_qkv

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


CASES = [
    # name, B, Hq, Hkv, S_q, S_k, D, causal, keep_num, keep_den
    ("mha_causal_10pct_d64", 1, 2, 2, 2048, 2048, 64, True, 1, 10),
    ("gqa4_ragged_d128", 2, 8, 2, 1000, 1000, 128, True, 1, 4),
    ("noncausal_sq_lt_sk", 1, 4, 2, 700, 1500, 64, False, 3, 10),
    ("keep_all", 1, 1, 1, 640, 640, 128, True, 1, 1),
    ("many_key_blocks", 1, 2, 1, 300, 64 * 300 + 17, 64, False, 1, 20),
    ("one_block", 1, 1, 1, 10, 10, 64, True, 1, 10),
    # 2000 key blocks: two rows per select workgroup instead of four
    ("wide_rows", 1, 2, 1, 200, 64 * 2000 - 5, 64, False, 1, 10),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_topk_mask_matches_oracle(case):
    name, B, Hq, Hkv, S_q, S_k, D, causal, kn, kd = case
    say(f"[topk] {name}: B={B} Hq={Hq} Hkv={Hkv} S_q={S_q} S_k={S_k} D={D} causal={causal} keep={kn}/{kd}")
    s = steel()
    dev = torch.device("cuda:0")
    q, k, _ = small_qkv(zlib.crc32(name.encode()) % 1000, B, Hq, Hkv, S_q, S_k, D)
    got = s.topk_block_mask(q.to(dev), k.to(dev), kn, kd, causal=causal)
    torch.cuda.synchronize()
    want = oracle.topk_meanpool_mask(q, k, kn, kd, causal)
    got = got.cpu().numpy()
    assert got.shape == want.shape
    assert np.array_equal(got, want), f"{int((got != want).sum())} mask bytes differ"


def test_topk_mask_full_size_sparse_workload():
    """The 24-head S = 32768 D = 64 workload whose mask is defined by this
    rule: the device mask equals the oracle's and the workload generator's
    (which the benchmark feeds to the attention pass)."""
    s = steel()
    cfg = CONFIGS["mha24_s32768_d64_causal_top10_lowrank4"]
    say("[topk] full-size top-10% workload: generating inputs")
    q, k, v, m = workloads.make_workload(cfg)
    dev = torch.device("cuda:0")
    say("[topk] full-size top-10% workload: GPU selection")
    got = s.topk_block_mask(q.to(dev), k.to(dev), 1, 10, causal=True)
    torch.cuda.synchronize()
    got = got.cpu().numpy()
    say("[topk] full-size top-10% workload: oracle selection")
    want = oracle.topk_meanpool_mask(q, k, 1, 10, causal=True)
    assert np.array_equal(got, want), f"{int((got != want).sum())} mask bytes differ from the oracle"
    assert np.array_equal(got, m), "device mask differs from the workload's mask"


def test_topk_mask_feeds_the_pass():
    """Selection and attention chained on the device equal the attention
    with the oracle's mask, bit for bit (same mask, same pass)."""
    s = steel()
    dev = torch.device("cuda:0")
    q, k, v = small_qkv(21, 1, 4, 4, 1536, 1536, 64)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = s.topk_block_mask(qd, kd, 1, 10, causal=True)
    a = s.attn_fwd(qd, kd, vd, md, causal=True)
    want_m = torch.from_numpy(oracle.topk_meanpool_mask(q, k, 1, 10, causal=True)).to(dev)
    b = s.attn_fwd(qd, kd, vd, want_m, causal=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def _tie_inputs(kind, B, Hq, Hkv, S_q, S_k, D):
    q, k, _ = small_qkv(77, B, Hq, Hkv, S_q, S_k, D)
    if kind == "equal":
        # every row of Q and of K the same vector: every block mean, hence every
        # score of a row, is the same number
        q = q[:, :, :1].expand(-1, -1, S_q, -1).contiguous()
        k = k[:, :, :1].expand(-1, -1, S_k, -1).contiguous()
    else:
        # Q = 0: every score is exactly zero (the products are signed zeros,
        # and a sum that starts at +0 stays +0)
        q = torch.zeros_like(q)
    return q, k


@pytest.mark.parametrize("kind", ["equal", "zero"])
@pytest.mark.parametrize("causal", [True, False])
def test_topk_mask_ties(kind, causal):
    """All candidates of a row tie: the kept blocks are the smallest kb (the
    oracle's order), on the radix path (rows of <= 512 key blocks) and on the
    sorting path (longer rows)."""
    s = steel()
    dev = torch.device("cuda:0")
    for S_k in (64 * 300 + 5, 64 * 700):
        say(f"[topk] ties {kind}: causal={causal} S_k={S_k}")
        q, k = _tie_inputs(kind, 1, 4, 2, 640, S_k, 64)
        got = s.topk_block_mask(q.to(dev), k.to(dev), 1, 10, causal=causal)
        torch.cuda.synchronize()
        want = oracle.topk_meanpool_mask(q, k, 1, 10, causal)
        got = got.cpu().numpy()
        assert np.array_equal(got, want), f"{int((got != want).sum())} mask bytes differ"
