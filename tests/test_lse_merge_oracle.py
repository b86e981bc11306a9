"""Pins of the log-sum-exp / partial-merge oracle (CPU).

* keys split into chunks (each chunk with its own causal limit) and merged
  back equal the unchunked attention and lse: an identity of the softmax
  that the oracle's two functions must satisfy together;
* lse against brute-force log(sum(exp(.))) written out per element;
* equal scores: lse = s + log(number of visible keys) in closed form;
* rows with no visible key: O = 0, lse = -inf, also through the merge;
* the causal limit: offset S_k - S_q reproduces the attention oracle, a
  large offset is the non-causal attention.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from workloads import small_qkv, random_block_mask


@pytest.mark.parametrize("case", [
    # seed, B, Hq, Hkv, S_q, S_k, D, causal, mask p, chunk bounds
    (1, 1, 2, 1, 96, 300, 16, True, None, [0, 70, 128, 300]),
    (2, 2, 4, 2, 200, 200, 8, True, 0.6, [0, 64, 190, 200]),
    (3, 1, 2, 2, 50, 257, 8, False, 0.5, [0, 1, 256, 257]),
])
def test_chunked_keys_merge_to_the_whole(case):
    seed, B, Hq, Hkv, S_q, S_k, D, causal, p, bounds = case
    q, k, v = small_qkv(seed, B, Hq, Hkv, S_q, S_k, D)
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    m = None if p is None else random_block_mask(np.random.default_rng(seed), B, Hq, nQB, nKB, p=p)
    scale = 1 / math.sqrt(D)
    o_full, l_full = oracle.attention_lse(q, k, v, m, scale, causal, 64)
    parts_o, parts_l = [], []
    for k0, k1 in zip(bounds[:-1], bounds[1:]):
        # a key chunk keeps the global visibility: element mask of the full
        # problem restricted to its columns (block mask columns of the chunk
        # are not whole blocks here, so the mask is applied per element)
        vis = np.zeros((B, Hq, S_q, k1 - k0), dtype=bool)
        for b in range(B):
            for h in range(Hq):
                bits = None if m is None else m[b, h]
                vis[b, h] = oracle.element_visibility(bits, np.arange(S_q), S_q, S_k, 64, causal)[:, k0:k1]
        o_c, l_c = _masked_chunk(q, k[:, :, k0:k1], v[:, :, k0:k1], vis, scale)
        parts_o.append(o_c)
        parts_l.append(l_c)
    o, l = oracle.merge_partials(parts_o, parts_l)
    assert np.allclose(o, o_full, atol=1e-12, rtol=0)
    assert np.array_equal(np.isinf(l), np.isinf(l_full))
    fin = np.isfinite(l_full)
    assert np.allclose(l[fin], l_full[fin], atol=1e-12, rtol=0)


def _masked_chunk(q, k, v, vis, scale):
    """Direct softmax over an element mask (independent of the oracle's
    block-mask path), for building chunk partials."""
    qf = q.double().numpy()
    kf = k.double().numpy()
    vf = v.double().numpy()
    B, Hq, S_q, D = qf.shape
    G = Hq // kf.shape[1]
    o = np.zeros((B, Hq, S_q, D))
    lse = np.full((B, Hq, S_q), -np.inf)
    for b in range(B):
        for h in range(Hq):
            s = qf[b, h] @ kf[b, h // G].T * scale
            for i in range(S_q):
                sel = vis[b, h, i]
                if not sel.any():
                    continue
                e = np.exp(s[i, sel] - s[i, sel].max())
                o[b, h, i] = e @ vf[b, h // G][sel] / e.sum()
                lse[b, h, i] = s[i, sel].max() + math.log(e.sum())
    return o, lse


def test_lse_against_brute_force():
    q, k, v = small_qkv(5, 1, 2, 1, 70, 90, 8)
    m = random_block_mask(np.random.default_rng(1), 1, 2, 2, 2, p=0.7)
    m[0, :, 1, 0] = 1
    _, lse = oracle.attention_lse(q, k, v, m, 0.3, True, 64)
    qf, kf = q.double().numpy(), k.double().numpy()
    for h in range(2):
        for i in range(70):
            tot = 0.0
            for j in range(90):
                visible = m[0, h, i // 64, j // 64] and j <= i + 20
                if visible:
                    tot += math.exp(0.3 * float(qf[0, h, i] @ kf[0, 0, j]))
            want = math.log(tot) if tot > 0 else -math.inf
            assert lse[0, h, i] == pytest.approx(want, rel=0, abs=1e-12) if tot > 0 else lse[0, h, i] == -math.inf


def test_equal_scores_closed_form():
    # all keys equal: every visible score is s = scale * q_i . k
    D, S = 8, 130
    q = torch.randn(1, 1, S, D).to(torch.bfloat16)
    krow = torch.randn(D)
    k = krow.repeat(S, 1).reshape(1, 1, S, D).to(torch.bfloat16)
    v = torch.randn(1, 1, S, D).to(torch.bfloat16)
    _, lse = oracle.attention_lse(q, k, v, None, 0.5, True, 64)
    qf, kf = q.double().numpy()[0, 0], k.double().numpy()[0, 0, 0]
    for i in range(S):
        assert lse[0, 0, i] == pytest.approx(0.5 * float(qf[i] @ kf) + math.log(i + 1), abs=1e-12)


def test_dead_rows_and_merge_of_dead_parts():
    q, k, v = small_qkv(8, 1, 1, 1, 128, 64, 8)
    # causal with S_q > S_k: rows i < S_q - S_k see no key
    o, lse = oracle.attention_lse(q, k, v, None, 0.35, True, 64)
    assert np.all(o[0, 0, :64] == 0) and np.all(np.isneginf(lse[0, 0, :64]))
    assert np.all(np.isfinite(lse[0, 0, 64:]))
    mo, ml = oracle.merge_partials([o, np.zeros_like(o)], [lse, np.full_like(lse, -np.inf)])
    assert np.array_equal(mo, o) and np.array_equal(np.isinf(ml), np.isinf(lse))
    fin = np.isfinite(lse)
    assert np.array_equal(ml[fin], lse[fin])


def test_causal_offset_limits():
    q, k, v = small_qkv(9, 1, 2, 1, 100, 160, 8)
    o_def, _ = oracle.attention_lse(q, k, v, None, 0.3, True, 64)
    assert np.allclose(o_def, oracle.attention(q, k, v, None, 0.3, True, 64), atol=1e-13, rtol=0)
    o_big, l_big = oracle.attention_lse(q, k, v, None, 0.3, True, 64, causal_offset=10 ** 6)
    o_nc, l_nc = oracle.attention_lse(q, k, v, None, 0.3, False, 64)
    assert np.array_equal(o_big, o_nc) and np.array_equal(l_big, l_nc)
