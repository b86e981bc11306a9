"""Tile classification, compressed live-block lists and work order (test
infrastructure only).

Section IV-A: every core knows the coordinates (i, j) of the score tile it
handles and treats it in one of three ways -- a fully masked tile is skipped,
an unmasked tile is processed normally, a partially masked tile gets the mask
applied locally.  Here the tiles are 64x64 blocks of the score matrix of one
(batch, query head); the block mask and the causal structure decide the class:

* rows of block qb are ``[qb*blk, min((qb+1)*blk, S_q))``, keys of block kb are
  ``[kb*blk, min((kb+1)*blk, S_k))``; causal visibility is ``j <= i + delta``
  with ``delta = S_k - S_q``;
* **dead** (skipped): the block-mask byte is 0, or the attention is causal and
  the first key of the block lies beyond what the last real row can see,
  ``kb*blk > last_row + delta``;
* **partial** (masked locally): live, and either causal with the last key of
  the block beyond what the first row can see, ``(kb+1)*blk - 1 > qb*blk +
  delta``, or the block runs past the last key, ``(kb+1)*blk > S_k``;
* **full**: live and not partial.

Compressed list (one row per (b, h, qb), rows numbered
``r = (b*Hq + h)*nQB + qb``): ``row_ptr`` is the exclusive prefix sum of the
live counts, ``col[row_ptr[r]:row_ptr[r+1]]`` lists the live kb in increasing
order, with bit 31 set when the tile is partial.

Work order (Section IV-C balances the masked work over the pipelines that
share a broadcast; on a GPU the same concern is load balance across compute
units): the rows sorted by live count, heaviest first, ties by row number.
The paper fixes no resolution for "heaviest"; counts are compared through a
monotone bin code that is exact below 128 and keeps 16 steps per octave
above (relative resolution 1/16), so that every order uses at most 512 bins.
"""
from __future__ import annotations

import numpy as np

PARTIAL_BIT = np.uint32(1 << 31)


def tile_classes(block_mask, B, Hq, S_q, S_k, blk, causal):
    """(live, partial) boolean arrays [B, Hq, nQB, nKB] from coordinates."""
    nQB = -(-S_q // blk)
    nKB = -(-S_k // blk)
    delta = S_k - S_q
    qb = np.arange(nQB)[:, None]
    kb = np.arange(nKB)[None, :]
    first_row = qb * blk
    last_row = np.minimum((qb + 1) * blk, S_q) - 1
    if block_mask is None:
        bits = np.ones((B, Hq, nQB, nKB), dtype=bool)
    else:
        bits = np.asarray(block_mask).reshape(B, Hq, nQB, nKB) != 0
    if causal:
        dead_c = kb * blk > last_row + delta
        part_c = (kb + 1) * blk - 1 > first_row + delta
    else:
        dead_c = np.zeros((nQB, nKB), dtype=bool)
        part_c = np.zeros((nQB, nKB), dtype=bool)
    tail = np.broadcast_to((kb + 1) * blk > S_k, (nQB, nKB))
    live = bits & ~dead_c[None, None]
    partial = live & (part_c | tail)[None, None]
    return live, partial


N_BINS = 512


def count_bin(counts) -> np.ndarray:
    """Bin of a live count: the count itself below 128; above, with
    e = floor(log2 c), 128 + 16*(e - 7) + (the four bits of c below its
    leading one).  Monotone in c; bins < 512 for every c < 2**31."""
    c = np.asarray(counts, dtype=np.int64)
    if np.any(c < 0) or np.any(c >= 2 ** 31):
        raise ValueError("live counts lie in [0, 2**31)")
    e = np.zeros_like(c)
    for k in range(1, 31):                      # e = position of the leading one
        e += (c >> k) > 0
    shift = np.maximum(e - 4, 0)
    big = 128 + 16 * (e - 7) + ((c >> shift) & 15)
    return np.where(c < 128, c, big)


def work_order(counts: np.ndarray) -> np.ndarray:
    """Rows by live count bin, heaviest first; equal bins keep row order."""
    return np.argsort(-count_bin(counts), kind="stable").astype(np.int32)


def build_index(block_mask, B, Hq, S_q, S_k, blk=64, causal=True):
    """Returns (row_ptr int32 [R+1], col uint32 [N_live], order int32 [R])."""
    live, partial = tile_classes(block_mask, B, Hq, S_q, S_k, blk, causal)
    nKB = live.shape[-1]
    live2 = live.reshape(-1, nKB)
    part2 = partial.reshape(-1, nKB)
    counts = live2.sum(axis=1)
    row_ptr = np.zeros(live2.shape[0] + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(counts)
    r_idx, kb_idx = np.nonzero(live2)          # row-major: rows in order, kb ascending
    col = kb_idx.astype(np.uint32)
    col[part2[r_idx, kb_idx]] |= PARTIAL_BIT
    return row_ptr.astype(np.int32), col, work_order(counts)
