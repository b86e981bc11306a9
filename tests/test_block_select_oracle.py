"""Pins of the top-k mean-pooled block selection oracle (CPU).

* exact rational brute force: the means and scores computed with Fraction
  from the bf16 values, the selection by sorting (-score, kb), on small
  random inputs (causal and not, GQA, ragged blocks);
* the tie rule: equal scores keep the smaller kb;
* a constructed ranking whose order is known in closed form;
* row invariants: the diagonal is set, no causal row keeps a block past it,
  each row keeps keep_n candidates plus the diagonal;
* agreement with the workload generator's own construction of the sparse
  workload's mask (an independent implementation of the same rule, with a
  different summation order) on a reduced size.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import workloads
from workloads import small_qkv


def brute_mask(q, k, keep_num, keep_den, causal, blk=64):
    qn = q.float().numpy()
    kn = k.float().numpy()
    B, Hq, S_q, D = qn.shape
    _, Hkv, S_k, _ = kn.shape
    G = Hq // Hkv
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)

    def means(x, S, nb):
        out = []
        for i in range(nb):
            rows = range(i * blk, min((i + 1) * blk, S))
            out.append([sum(Fraction(float(x[r, d])) for r in rows) / len(rows) for d in range(D)])
        return out

    m = np.zeros((B, Hq, nQB, nKB), dtype=np.uint8)
    for b in range(B):
        for h in range(Hq):
            qm = means(qn[b, h], S_q, nQB)
            km = means(kn[b, h // G], S_k, nKB)
            for qb in range(nQB):
                ncand = min(qb + 1, nKB) if causal else nKB
                keep = -(-keep_num * ncand // keep_den)
                scored = sorted(range(ncand), key=lambda kb: (-sum(a * c for a, c in zip(qm[qb], km[kb])), kb))
                for kb in scored[:keep]:
                    m[b, h, qb, kb] = 1
                if qb < nKB:
                    m[b, h, qb, qb] = 1
    return m


@pytest.mark.parametrize("case", [
    # seed, B, Hq, Hkv, S_q, S_k, D, causal, keep_num, keep_den
    (1, 1, 2, 1, 640, 640, 8, True, 1, 10),
    (2, 1, 4, 2, 700, 500, 8, True, 1, 4),
    (3, 2, 2, 2, 300, 1000, 16, False, 3, 10),
    (4, 1, 1, 1, 1100, 1100, 4, True, 1, 1),
])
def test_oracle_matches_exact_rational_brute_force(case):
    seed, B, Hq, Hkv, S_q, S_k, D, causal, kn, kd = case
    q, k, _ = small_qkv(seed, B, Hq, Hkv, S_q, S_k, D)
    got = oracle.topk_meanpool_mask(q, k, kn, kd, causal)
    want = brute_mask(q, k, kn, kd, causal)
    assert np.array_equal(got, want)


def test_block_means_of_ragged_blocks_against_fractions():
    q, _, _ = small_qkv(7, 1, 1, 1, 150, 150, 8)
    x = q[0, 0].float().numpy()
    got = oracle.block_means(x, 64)
    assert got.shape == (3, 8)
    for i, (lo, hi) in enumerate([(0, 64), (64, 128), (128, 150)]):
        for d in range(8):
            exact = sum(Fraction(float(x[r, d])) for r in range(lo, hi)) / (hi - lo)
            # one rounding at most: the row sum of bf16 values here is exact
            assert got[i, d] == float(exact)


def test_equal_scores_keep_the_smaller_blocks():
    # every key block has the same rows, so all candidate scores are equal
    D, S = 8, 64 * 12
    q = torch.randn(1, 1, S, D).to(torch.bfloat16)
    row = torch.randn(64, D)
    k = row.repeat(12, 1).reshape(1, 1, S, D).to(torch.bfloat16)
    m = oracle.topk_meanpool_mask(q, k, 1, 4, causal=True)
    for qb in range(12):
        keep = -(-(qb + 1) // 4)
        want = set(range(keep)) | {qb}
        assert set(np.nonzero(m[0, 0, qb])[0].tolist()) == want


def test_constructed_ranking():
    # Q rows all ones; key block kb has every entry equal to c[kb], so
    # score(qb, kb) = D * c[kb]: the top blocks are the largest c among the
    # candidates
    D, nb = 4, 10
    c = np.array([0.5, -1.0, 3.0, 2.0, 0.25, 4.0, -2.0, 1.0, 1.5, 0.75])
    q = torch.ones(1, 1, 64 * nb, D, dtype=torch.bfloat16)
    k = torch.from_numpy(np.repeat(c, 64)[:, None] * np.ones((1, D))).reshape(1, 1, 64 * nb, D)
    k = k.to(torch.bfloat16)
    m = oracle.topk_meanpool_mask(q, k, 3, 10, causal=True)
    for qb in range(nb):
        cand = list(range(qb + 1))
        keep = -(-3 * (qb + 1) // 10)
        top = sorted(cand, key=lambda j: (-c[j], j))[:keep]
        assert set(np.nonzero(m[0, 0, qb])[0].tolist()) == set(top) | {qb}


def test_row_invariants():
    q, k, _ = small_qkv(11, 2, 4, 2, 1000, 1000, 16)
    m = oracle.topk_meanpool_mask(q, k, 1, 10, causal=True)
    nQB = m.shape[2]
    for b in range(2):
        for h in range(4):
            for qb in range(nQB):
                row = m[b, h, qb]
                assert row[qb] == 1
                assert not row[qb + 1:].any()
                keep = -(-(qb + 1) // 10)
                assert row.sum() in (keep, keep + 1)


def test_agrees_with_workload_generator_reduced():
    cfg = workloads.Config("topk_reduced", 1, 3, 3, 4096, 4096, 64, True, "topk_meanpool",
                           lowrank_rank=4, lowrank_scale=2.0)
    q, k, v = workloads.make_qkv(cfg)
    want = workloads.topk_meanpool_mask(cfg, q, k)
    got = oracle.topk_meanpool_mask(q, k, 1, 10, causal=True)
    assert np.array_equal(got, want)
