"""Row log-sum-exp and the merge of partial results (test infrastructure only).

Section II-A (Eq. 1) together with the running statistics the fused method
carries per row -- the row maximum m and the row sum l of Algorithm 1 -- gives
every query row the value

    lse_i = log sum_{j visible to i} exp(scale * q_i . k_j)

(-inf when no key is visible).  Attention over the union of disjoint key sets
is the weighted average of the attentions over each set, with weights
exp(lse_c - lse) and lse = log sum_c exp(lse_c): the step that combines
partial results computed over separate key chunks (chunked prefill, keys
split over devices).

``attention_lse`` is the plain definition in float64 with an explicit causal
limit ``j <= i + causal_offset``: a chunk of keys [k0, k1) of a longer
sequence is causal with ``causal_offset = (S_k_total - S_q) - k0``.
``merge_partials`` is the combination rule written out.

Pinned by ``tests/test_lse_merge_oracle.py``: chunked keys merged back equal
the unchunked result, lse against brute-force log(sum(exp)), the closed form
for equal scores, and rows with no visible key.
"""
from __future__ import annotations

import numpy as np

from .masked_attention import _f64, element_visibility, kv_head


def attention_lse(q, k, v, block_mask=None, scale=None, causal=True, blk=64,
                  causal_offset=None, chunk=1024):
    """(O float64 [B, Hq, S_q, D], lse float64 [B, Hq, S_q])."""
    qf, kf, vf = _f64(q), _f64(k), _f64(v)
    B, Hq, S_q, D = qf.shape
    Hkv, S_k = kf.shape[1], kf.shape[2]
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    bm = None if block_mask is None else np.asarray(block_mask)
    out = np.zeros((B, Hq, S_q, D))
    lse = np.full((B, Hq, S_q), -np.inf)
    for b in range(B):
        for h in range(Hq):
            g = kv_head(h, Hq, Hkv)
            bits = None if bm is None else bm[b, h]
            for r0 in range(0, S_q, chunk):
                rows = np.arange(r0, min(S_q, r0 + chunk))
                vis = element_visibility(bits, rows, S_q, S_k, blk, causal, causal_offset)
                s = (qf[b, h, rows] @ kf[b, g].T) * scale
                s = np.where(vis, s, -np.inf)
                m = s.max(axis=1)
                live = np.isfinite(m)
                msafe = np.where(live, m, 0.0)
                p = np.exp(s - msafe[:, None])
                den = p.sum(axis=1)
                o = (p @ vf[b, g]) / np.where(den > 0, den, 1.0)[:, None]
                o[~live] = 0.0
                out[b, h, rows] = o
                lse[b, h, rows] = np.where(live, msafe + np.log(np.where(den > 0, den, 1.0)), -np.inf)
    return out, lse


def merge_partials(o_parts, lse_parts):
    """o_parts [n, ..., D], lse_parts [n, ...] -> (O [..., D], lse [...])."""
    o = np.asarray(o_parts, dtype=np.float64)
    l = np.asarray(lse_parts, dtype=np.float64)
    top = l.max(axis=0)
    live = np.isfinite(top)
    tsafe = np.where(live, top, 0.0)
    w = np.exp(l - tsafe[None])                # 0 for parts with lse = -inf
    den = w.sum(axis=0)
    out = (w[..., None] * o).sum(axis=0) / np.where(den > 0, den, 1.0)[..., None]
    out[~live] = 0.0
    lse = np.where(live, tsafe + np.log(np.where(den > 0, den, 1.0)), -np.inf)
    return out, lse
