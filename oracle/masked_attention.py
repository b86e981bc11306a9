"""Plain float64 attention with a block mask (test infrastructure only).

Definition followed (Section II-A, Eq. 1): for one head,
``A = Q K^T * scale`` and ``O = softmax(A) V`` with the softmax taken over each
row of A independently.  The paper's fused method (Algorithm 1: running row
maximum, exponentials, running row sum, rescaled accumulation, final division
by the row sum) reaches exactly this value in exact arithmetic, so the oracle
is the definition itself, not the algorithm.

Masking (Section IV-A: tiles that are fully masked are skipped, partially
masked tiles are masked element by element).  An element (i, j) of a head is
*visible* iff its 64x64 block is marked live in the block mask and, when the
attention is causal, ``j <= i + (S_k - S_q)`` (bottom-right alignment, which is
plain lower-triangular attention when S_q == S_k).  Invisible elements take the
value -inf before the row maximum, so they get probability exactly 0.  A row
with no visible element has no defined softmax; its output is 0.

Grouped-query heads: query head h reads key/value head ``h // (Hq // Hkv)``.

Inputs are the exact bf16 values converted to float64 (a lossless widening);
the scale is used as given.  Score rows are materialised in full, a chunk of
query rows at a time; each row is complete, so chunking changes nothing.
"""
from __future__ import annotations

import numpy as np

try:  # torch is only needed to unpack bf16 tensors
    import torch
except Exception:  # pragma: no cover
    torch = None


def _f64(x) -> np.ndarray:
    if torch is not None and isinstance(x, torch.Tensor):
        return x.detach().to("cpu").to(torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def kv_head(h: int, Hq: int, Hkv: int) -> int:
    """Key/value head read by query head h (contiguous groups)."""
    return h // (Hq // Hkv)


def element_visibility(block_row_bits: np.ndarray, rows: np.ndarray, S_q: int,
                       S_k: int, blk: int, causal: bool, offset=None) -> np.ndarray:
    """Boolean [len(rows), S_k]: which keys each listed query row may see.

    ``block_row_bits`` is the [nQB, nKB] block mask of one (b, h), or None.
    ``offset``: causal key limit ``j <= i + offset`` (default S_k - S_q).
    """
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.arange(S_k, dtype=np.int64)
    if block_row_bits is None:
        vis = np.ones((rows.size, S_k), dtype=bool)
    else:
        bits = np.asarray(block_row_bits) != 0
        vis = bits[rows // blk][:, cols // blk]
    if causal:
        vis &= cols[None, :] <= rows[:, None] + ((S_k - S_q) if offset is None else offset)
    return vis


def _head_rows(qh, kh, vh, vis, scale):
    """Output rows for one head: qh [R, D], kh/vh [S_k, D], vis [R, S_k]."""
    s = (qh @ kh.T) * scale
    s = np.where(vis, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    dead = ~np.isfinite(m[:, 0])
    m = np.where(np.isfinite(m), m, 0.0)
    p = np.exp(s - m)                      # exp(-inf) = 0 on invisible entries
    denom = p.sum(axis=1, keepdims=True)
    o = (p @ vh) / np.where(denom > 0, denom, 1.0)
    o[dead] = 0.0
    return o


def attention(q, k, v, block_mask=None, scale=None, causal=True, blk=64, chunk=1024):
    """Full output, float64 [B, Hq, S_q, D]."""
    qf, kf, vf = _f64(q), _f64(k), _f64(v)
    B, Hq, S_q, D = qf.shape
    Hkv, S_k = kf.shape[1], kf.shape[2]
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    bm = None if block_mask is None else np.asarray(block_mask)
    out = np.zeros((B, Hq, S_q, D), dtype=np.float64)
    for b in range(B):
        for h in range(Hq):
            g = kv_head(h, Hq, Hkv)
            bits = None if bm is None else bm[b, h]
            for r0 in range(0, S_q, chunk):
                rows = np.arange(r0, min(S_q, r0 + chunk))
                vis = element_visibility(bits, rows, S_q, S_k, blk, causal)
                out[b, h, rows] = _head_rows(qf[b, h, rows], kf[b, g], vf[b, g], vis, scale)
    return out


def attention_rows(q, k, v, index, block_mask=None, scale=None, causal=True, blk=64):
    """Output rows for a sample: ``index`` is an int array [n, 3] of (b, h, i).

    Returns float64 [n, D] in the order of ``index``.
    """
    qt, kt, vt = q, k, v
    index = np.asarray(index, dtype=np.int64).reshape(-1, 3)
    B, Hq, S_q, D = tuple(qt.shape)
    Hkv, S_k = int(kt.shape[1]), int(kt.shape[2])
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    bm = None if block_mask is None else np.asarray(block_mask)
    out = np.zeros((index.shape[0], D), dtype=np.float64)
    keys = index[:, 0] * Hq + index[:, 1]
    for key in np.unique(keys):
        sel = np.nonzero(keys == key)[0]
        b, h = int(key // Hq), int(key % Hq)
        g = kv_head(h, Hq, Hkv)
        rows = index[sel, 2]
        qh = _f64(qt[b, h])[rows]
        kh, vh = _f64(kt[b, g]), _f64(vt[b, g])
        bits = None if bm is None else bm[b, h]
        vis = element_visibility(bits, rows, S_q, S_k, blk, causal)
        out[sel] = _head_rows(qh, kh, vh, vis, scale)
    return out
