"""Float64 model of the fp8 (E4M3) form of the fused pass (test infrastructure).

The paper computes both products of Algorithm 1 with bf16 operands and fp32
accumulation (Section II-C, the AIE datapath).  The library's fp8 form keeps
Algorithm 1's order of operations (query block by query block, live key
blocks in increasing order, running row maximum, rescaled accumulation, final
division by the row sum) and changes only the operands of its two products:

* E4M3, the OCP 8-bit floating-point format: 1 sign bit, 4 exponent bits
  with bias 7, 3 mantissa bits, subnormals (quantum 2^-9 below 2^-6), largest
  finite magnitude 448, no infinities.  Rounding is to nearest, ties to even.
* Power-of-two scales.  A tensor X whose largest magnitude is a is quantized
  as E4M3(X * s) with s = 2^floor(log2(448 / a)) (s = 1 when a = 0); the
  product is divided by s afterwards.  Q has one scale per query row; K and V
  one scale each per (batch, key/value head).
* P.  The running row maximum m (log2 units) follows every increase (no
  deferred rescale), so the weights 2^(S - m + 8) lie in (0, 256]; they are
  rounded to E4M3 for the P V product.  The +8 keeps weights down to
  2^-14 of the row maximum in E4M3's normal range.  The row sum l adds the
  weights before that rounding.

Everything else is float64:
  S      = (Q8 K8^T) / (s_q s_k) * scale * log2(e)     (visible keys; -inf else)
  m'     = max(m, rowmax S);  alpha = 2^(m - m')        (1 when m' = -inf)
  P      = 2^(S - m' + 8);    l = alpha l + rowsum P
  O      = alpha O + E4M3(P) V8 / s_v
  out    = O / l (0 for a row with no visible key);  lse = (m - 8 + log2 l) ln 2.

With ``qk_fp8=False`` (the library's P V-only fp8 form) Q and K are not
quantized: S = (Q K^T) * scale * log2(e) from the bf16 values, and only V and
P take E4M3 operands.

Visibility is that of ``masked_attention`` (block mask and causal limit).  A
live tile in which a row sees no key leaves that row's state unchanged, so
iterating over the key blocks in which the row block sees any key is the
same as iterating over the library's live list.
"""
from __future__ import annotations

import math

import numpy as np

from .masked_attention import _f64, element_visibility, kv_head

E4M3_MAX = 448.0
E4M3_MIN_NORMAL = 2.0 ** -6
E4M3_QUANTUM_SUB = 2.0 ** -9
P_OFFSET = 8.0  # log2 offset of the P weights


def e4m3_round(x) -> np.ndarray:
    """Round float64 values to the E4M3 grid (nearest, ties to even).

    Magnitudes above 448 are not representable and raise: every value the
    model rounds is at most 448 by construction (scaled tensors) or 256 (P).
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    if np.any(a > E4M3_MAX) or np.any(~np.isfinite(a)):
        raise ValueError("value outside the finite E4M3 range")
    # quantum: 2^(e - 3) for a in [2^e, 2^(e+1)), e >= -6; 2^-9 below 2^-6
    _, E = np.frexp(np.where(a > 0, a, 1.0))           # a = f 2^E, f in [0.5, 1)
    quantum = np.where(a >= E4M3_MIN_NORMAL, np.ldexp(1.0, E - 1 - 3), E4M3_QUANTUM_SUB)
    r = np.rint(a / quantum) * quantum                  # a / quantum is exact
    return np.copysign(r, x)


def round_p(p) -> np.ndarray:
    """The P operand: the weights rounded to E4M3."""
    return e4m3_round(p)


def pow2_scale(amax) -> np.ndarray:
    """2^floor(log2(448 / amax)), 1 where amax == 0 (float64)."""
    amax = np.asarray(amax, dtype=np.float64)
    safe = np.where(amax > 0, amax, E4M3_MAX)
    _, E = np.frexp(E4M3_MAX / safe)
    return np.where(amax > 0, np.ldexp(1.0, E - 1), 1.0)


def quantize_rows(x: np.ndarray):
    """E4M3 values and scales of x [..., n], one scale per row."""
    s = pow2_scale(np.abs(x).max(axis=-1))
    return e4m3_round(x * s[..., None]), s


def quantize_tensor(x: np.ndarray):
    """E4M3 values and the one scale of the whole array x."""
    s = float(pow2_scale(np.abs(x).max() if x.size else 0.0))
    return e4m3_round(x * s), s


def _block_rows(q8, sq, k8, sk, v8, sv, vis, c):
    """One query block of one head: q8 [R, D] with scales sq [R], k8/v8
    [S_k, D] with scales sk, sv, vis [R, S_k], c = scale * log2(e).  Returns
    (O / l, lse).  Unquantized operands come with scale 1."""
    R, S_k = vis.shape
    D = q8.shape[1]
    m = np.full(R, -np.inf)
    l = np.zeros(R)
    o = np.zeros((R, D))
    nkb = -(-S_k // 64)
    for kb in range(nkb):
        cols = slice(64 * kb, min(64 * (kb + 1), S_k))
        tv = vis[:, cols]
        if not tv.any():
            continue
        s = (q8 @ k8[cols].T) / (sq[:, None] * sk) * c
        s = np.where(tv, s, -np.inf)
        m_new = np.maximum(m, s.max(axis=1))
        alpha = np.where(m_new == -np.inf, 1.0, np.exp2(m - np.where(m_new == -np.inf, 0.0, m_new)))
        ms = np.where(m_new == -np.inf, 0.0, m_new)
        p = np.exp2(s - ms[:, None] + P_OFFSET)          # exp2(-inf) = 0
        l = alpha * l + p.sum(axis=1)
        o = alpha[:, None] * o + (round_p(p) @ v8[cols]) / sv
        m = m_new
    live = l > 0
    out = np.where(live[:, None], o / np.where(live, l, 1.0)[:, None], 0.0)
    lse = np.where(live, (m - P_OFFSET + np.log2(np.where(live, l, 1.0))) * math.log(2.0), -np.inf)
    return out, lse


def attention_fp8(q, k, v, block_mask=None, scale=None, causal=True, blk=64, causal_offset=None,
                  heads=None, qblocks=None, qk_fp8=True):
    """fp8 model of the fused pass.  Returns (out, lse): float64
    [B, Hq, S_q, D] and [B, Hq, S_q]; rows outside the selected ``heads``
    ((b, h) pairs) or ``qblocks`` (query-block indices) are NaN.
    ``qk_fp8``: Q and K in E4M3 too (else only P and V)."""
    if blk != 64:
        raise ValueError("the model follows the library's 64 x 64 tiles")
    qf, kf, vf = _f64(q), _f64(k), _f64(v)
    B, Hq, S_q, D = qf.shape
    Hkv, S_k = kf.shape[1], kf.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    c = float(scale) * math.log2(math.e)
    offset = (S_k - S_q) if causal_offset is None else causal_offset
    mask = None if block_mask is None else np.asarray(_f64(block_mask)) != 0
    out = np.full((B, Hq, S_q, D), np.nan)
    lse = np.full((B, Hq, S_q), np.nan)
    kv = {}
    nqb = -(-S_q // blk)
    pairs = [(b, h) for b in range(B) for h in range(Hq)] if heads is None else list(heads)
    for b, h in pairs:
        g = kv_head(h, Hq, Hkv)
        if (b, g) not in kv:
            k8, sk = quantize_tensor(kf[b, g]) if qk_fp8 else (kf[b, g], 1.0)
            v8, sv = quantize_tensor(vf[b, g])
            kv[(b, g)] = (k8, sk, v8, sv)
        k8, sk, v8, sv = kv[(b, g)]
        for qb in (range(nqb) if qblocks is None else qblocks):
            rows = np.arange(qb * blk, min((qb + 1) * blk, S_q))
            vis = element_visibility(None if mask is None else mask[b, h], rows, S_q, S_k, blk,
                                     causal, offset)
            if qk_fp8:
                q8, sq = quantize_rows(qf[b, h, rows])
            else:
                q8, sq = qf[b, h, rows], np.ones(len(rows))
            o, ls = _block_rows(q8, sq, k8, sk, v8, sv, vis, c)
            out[b, h, rows] = o
            lse[b, h, rows] = ls
    return out, lse
