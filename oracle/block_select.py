"""Top-k mean-pooled key-block selection (test infrastructure only).

The step before the attention pass for learned-free sparse prefill: the block
mask is produced from the inputs themselves.  The paper generates its masks
from tile coordinates on the compute core instead of fetching them (Section
III-B), and treats any block mask through the same three tile classes
(Section IV-A); the selection rule here is the one the sparse workload of
this library is defined with:

* for every (b, query head h, query block qb): the mean of the query block's
  rows of Q, and for every key block kb the mean of its rows of K (key/value
  head g = h // (Hq/Hkv)), both in float64 from the bf16 values; a ragged
  last block averages over the rows it has;
* score(qb, kb) = dot(mean_q(qb), mean_k(kb));
* candidates are kb < ncand with ncand = min(qb + 1, nKB) when causal (the
  blocks at or before the block diagonal), else nKB;
* keep_n = ceil(keep_num / keep_den * ncand) candidates with the largest
  scores are kept, equal scores going to the smaller kb; the diagonal block
  kb = qb (when qb < nKB) is kept as well; every other block is 0.

Floating point decides the selection, so the arithmetic order is fixed here
and the library follows the same order in the same precision: each block sum
adds the rows in increasing order, the mean is that sum divided by the row
count, and each score adds the D products in increasing d, every product and
sum rounded on its own (no fused multiply-add).  With that order fixed the
mask is unique and compared bit for bit.

Pinned by ``tests/test_block_select_oracle.py``: exact rational brute force
on small inputs, the tie rule on equal scores, a constructed ranking, and the
row invariants.
"""
from __future__ import annotations

import numpy as np


def block_means(x, blk: int = 64) -> np.ndarray:
    """x: [S, D] (any float type holding bf16 values) -> [ceil(S/blk), D]
    float64 means, rows summed in increasing order."""
    x = np.asarray(x, dtype=np.float64)
    S, D = x.shape
    nb = -(-S // blk)
    pad = np.zeros((nb * blk, D))
    pad[:S] = x
    pad = pad.reshape(nb, blk, D)
    acc = np.zeros((nb, D))
    for r in range(blk):  # row r of every block; padding rows add exact zeros
        acc = acc + pad[:, r, :]
    cnt = np.minimum(blk, S - np.arange(nb) * blk).astype(np.float64)
    return acc / cnt[:, None]


def block_scores(qm: np.ndarray, km: np.ndarray) -> np.ndarray:
    """[nQB, D] x [nKB, D] -> [nQB, nKB]: dot products accumulated over d in
    increasing order, products and sums rounded separately."""
    s = np.zeros((qm.shape[0], km.shape[0]))
    for d in range(qm.shape[1]):
        s = s + np.multiply.outer(qm[:, d], km[:, d])
    return s


def keep_count(ncand: int, keep_num: int, keep_den: int) -> int:
    return (keep_num * ncand + keep_den - 1) // keep_den


def select_row(scores_row: np.ndarray, ncand: int, keep_n: int) -> np.ndarray:
    """Indices of the keep_n largest of scores_row[:ncand], ties to the
    smaller index."""
    cand = scores_row[:ncand]
    order = np.lexsort((np.arange(ncand), -cand))  # by -score, then by kb
    return np.sort(order[:keep_n])


def topk_meanpool_mask(q, k, keep_num: int, keep_den: int, causal: bool, blk: int = 64) -> np.ndarray:
    """q: [B, Hq, S_q, D], k: [B, Hkv, S_k, D] (bf16 values as torch or numpy)
    -> uint8 block mask [B, Hq, nQB, nKB]."""
    q = np.asarray(q.float().numpy() if hasattr(q, "float") else q, dtype=np.float64)
    k = np.asarray(k.float().numpy() if hasattr(k, "float") else k, dtype=np.float64)
    B, Hq, S_q, _ = q.shape
    _, Hkv, S_k, _ = k.shape
    G = Hq // Hkv
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    mask = np.zeros((B, Hq, nQB, nKB), dtype=np.uint8)
    for b in range(B):
        kms = [block_means(k[b, g], blk) for g in range(Hkv)]
        for h in range(Hq):
            qm = block_means(q[b, h], blk)
            sc = block_scores(qm, kms[h // G])
            for qb in range(nQB):
                ncand = min(qb + 1, nKB) if causal else nKB
                kn = keep_count(ncand, keep_num, keep_den)
                mask[b, h, qb, select_row(sc[qb], ncand, kn)] = 1
                if qb < nKB:
                    mask[b, h, qb, qb] = 1
    return mask
