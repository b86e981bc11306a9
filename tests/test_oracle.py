"""Pins for the float64 oracle (CPU only).

The oracle is checked against things other than itself:

* brute force on tiny inputs -- pure-Python loops over the definition of
  Section II-A, Eq. 1, with the visibility of every element decided from its
  own coordinates (no helper of the oracle is used), and a softmax written
  without the max-subtraction the oracle uses;
* a library routine -- ``torch.nn.functional.scaled_dot_product_attention`` in
  float64 on the CPU with a boolean mask (the unmasked/dense case and the
  "block-skipped equals dense with -inf entries" case both reduce to it);
* closed forms -- causal row 0 equals the first value row; Q = 0 gives the mean
  of the visible value rows; two keys give a logistic mixture;
* invariants -- probabilities of a live row sum to 1 (V = 1 gives O = 1), every
  output lies in the range of the visible value rows, joint permutation of the
  keys and values leaves a non-causal result unchanged, adding to all keys a
  vector shifts each score row by a constant and changes nothing;
* planted mistakes -- plausible slips planted into a copy of the oracle on the
  CPU (wrong head mapping, softmax over the wrong axis, off-by-one causal
  diagonal, dropped block mask, transposed operand, dropped scale) each fail at
  least one of the pins above.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import masked_attention as oatt
from workloads import small_qkv, random_block_mask


# ---------------------------------------------------------------- brute force
def brute_force(q, k, v, block_mask, scale, causal, blk):
    """Pure-Python loops; returns nested lists [B][Hq][S_q][D]."""
    qf = q.to(torch.float64).tolist()
    kf = k.to(torch.float64).tolist()
    vf = v.to(torch.float64).tolist()
    B, Hq, S_q, D = q.shape
    Hkv, S_k = k.shape[1], k.shape[2]
    group = Hq // Hkv
    out = []
    for b in range(B):
        ob = []
        for h in range(Hq):
            g = h // group
            oh = []
            for i in range(S_q):
                weights = []
                for j in range(S_k):
                    visible = True
                    if block_mask is not None and block_mask[b][h][i // blk][j // blk] == 0:
                        visible = False
                    if causal and j > i + (S_k - S_q):
                        visible = False
                    if visible:
                        s = 0.0
                        for d in range(D):
                            s += qf[b][h][i][d] * kf[b][g][j][d]
                        weights.append((j, math.exp(s * scale)))
                total = math.fsum(w for _, w in weights)
                row = []
                for d in range(D):
                    if not weights:
                        row.append(0.0)
                    else:
                        row.append(math.fsum(w * vf[b][g][j][d] for j, w in weights) / total)
                oh.append(row)
            ob.append(oh)
        out.append(ob)
    return np.array(out, dtype=np.float64)


TINY = [
    # (B, Hq, Hkv, S_q, S_k, D, blk, causal, mask kind)
    (1, 1, 1, 1, 1, 1, 64, True, "none"),
    (1, 1, 1, 2, 2, 8, 64, True, "none"),
    (1, 1, 1, 3, 3, 8, 64, False, "none"),
    (1, 2, 1, 17, 17, 8, 4, True, "random"),
    (1, 1, 1, 63, 63, 4, 64, True, "none"),
    (1, 1, 1, 64, 64, 4, 64, False, "none"),
    (1, 1, 1, 65, 65, 4, 64, True, "none"),
    (2, 4, 2, 20, 20, 4, 4, True, "random"),
    (1, 2, 2, 24, 24, 4, 8, True, "diag"),
    (1, 2, 1, 16, 16, 4, 4, False, "deadrow"),
    (1, 2, 2, 12, 20, 4, 4, True, "random"),    # S_q < S_k: bottom-right diagonal
    (1, 1, 1, 20, 12, 4, 4, True, "none"),      # S_q > S_k: first rows see nothing
]


def _mask(kind, B, Hq, S_q, S_k, blk, seed):
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    rng = np.random.default_rng(seed)
    if kind == "none":
        return None
    if kind == "random":
        return random_block_mask(rng, B, Hq, nQB, nKB, p=0.6)
    if kind == "diag":
        m = np.zeros((B, Hq, nQB, nKB), dtype=np.uint8)
        for t in range(min(nQB, nKB)):
            m[:, :, t, t] = 1
        return m
    if kind == "deadrow":
        m = random_block_mask(rng, B, Hq, nQB, nKB, p=0.7)
        m[0, 1, 1, :] = 0
        return m
    raise ValueError(kind)


@pytest.mark.parametrize("case", TINY, ids=[f"c{i}" for i in range(len(TINY))])
def test_oracle_matches_brute_force(case):
    B, Hq, Hkv, S_q, S_k, D, blk, causal, kind = case
    q, k, v = small_qkv(7 + S_q, B, Hq, Hkv, S_q, S_k, D)
    m = _mask(kind, B, Hq, S_q, S_k, blk, seed=S_q)
    scale = 1.0 / math.sqrt(D)
    got = oracle.attention(q, k, v, m, scale, causal, blk)
    want = brute_force(q, k, v, m, scale, causal, blk)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


# ---------------------------------------------------------------- library routine
def sdpa_reference(q, k, v, block_mask, scale, causal, blk):
    """torch SDPA in float64 on the CPU with an explicit boolean mask."""
    B, Hq, S_q, D = q.shape
    Hkv, S_k = k.shape[1], k.shape[2]
    qd, kd, vd = (t.to(torch.float64) for t in (q, k, v))
    kd = kd.repeat_interleave(Hq // Hkv, dim=1)
    vd = vd.repeat_interleave(Hq // Hkv, dim=1)
    allow = torch.ones((B, Hq, S_q, S_k), dtype=torch.bool)
    if block_mask is not None:
        bm = torch.from_numpy(np.asarray(block_mask) != 0)
        allow &= bm.repeat_interleave(blk, 2)[:, :, :S_q].repeat_interleave(blk, 3)[..., :S_k]
    if causal:
        i = torch.arange(S_q)[:, None]
        j = torch.arange(S_k)[None, :]
        allow &= (j <= i + (S_k - S_q))
    o = torch.nn.functional.scaled_dot_product_attention(qd, kd, vd, attn_mask=allow, scale=scale)
    live = allow.any(-1)
    return o.numpy(), live.numpy()


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("masked", [False, True])
def test_oracle_matches_sdpa(seed, causal, masked):
    B, Hq, Hkv, S, D, blk = 2, 4, 2, 200, 32, 64
    q, k, v = small_qkv(seed, B, Hq, Hkv, S, S, D)
    m = random_block_mask(np.random.default_rng(seed), B, Hq, 4, 4, p=0.5, kill_rows=1) if masked else None
    got = oracle.attention(q, k, v, m, 1 / math.sqrt(D), causal, blk)
    want, live = sdpa_reference(q, k, v, m, 1 / math.sqrt(D), causal, blk)
    np.testing.assert_allclose(got[live], want[live], rtol=0, atol=1e-12)
    assert np.all(got[~live] == 0.0)


def test_all_ones_mask_equals_no_mask():
    q, k, v = small_qkv(3, 1, 2, 2, 130, 130, 16)
    ones = np.ones((1, 2, 3, 3), dtype=np.uint8)
    for causal in (False, True):
        a = oracle.attention(q, k, v, None, 0.25, causal, 64)
        b = oracle.attention(q, k, v, ones, 0.25, causal, 64)
        assert np.array_equal(a, b)


def test_attention_rows_equals_full():
    q, k, v = small_qkv(5, 1, 4, 2, 150, 150, 16)
    m = random_block_mask(np.random.default_rng(5), 1, 4, 3, 3, p=0.6)
    full = oracle.attention(q, k, v, m, 0.25, True, 64)
    idx = np.array([(0, h, i) for h in range(4) for i in (0, 1, 63, 64, 127, 128, 149)])
    rows = oracle.attention_rows(q, k, v, idx, m, 0.25, True, 64)
    np.testing.assert_array_equal(rows, full[idx[:, 0], idx[:, 1], idx[:, 2]])


# ---------------------------------------------------------------- closed forms
def test_causal_row0_is_first_value_row():
    q, k, v = small_qkv(11, 1, 4, 2, 96, 96, 16)
    o = oracle.attention(q, k, v, None, 0.25, True, 64)
    for h in range(4):
        np.testing.assert_array_equal(o[0, h, 0], v[0, h // 2, 0].to(torch.float64).numpy())


def test_zero_query_gives_mean_of_visible_values():
    _, k, v = small_qkv(12, 1, 2, 1, 80, 80, 8)
    q = torch.zeros((1, 2, 80, 8), dtype=torch.bfloat16)
    m = np.ones((1, 2, 2, 2), dtype=np.uint8)
    m[0, 1, 1, 0] = 0                                  # head 1, rows 64..79 cannot see keys 0..63
    o = oracle.attention(q, k, v, m, 0.5, True, 64)
    vv = v[0, 0].to(torch.float64).numpy()
    for i in range(80):
        np.testing.assert_allclose(o[0, 0, i], vv[: i + 1].mean(0), rtol=0, atol=1e-13)
    for i in range(64, 80):
        np.testing.assert_allclose(o[0, 1, i], vv[64: i + 1].mean(0), rtol=0, atol=1e-13)


def test_two_keys_logistic():
    q, k, v = small_qkv(13, 1, 1, 1, 5, 2, 8)
    o = oracle.attention(q, k, v, None, 0.3, False, 64)
    qf, kf, vf = (t[0, 0].to(torch.float64).numpy() for t in (q, k, v))
    for i in range(5):
        a = 0.3 * (qf[i] @ kf[0] - qf[i] @ kf[1])
        w0 = 1.0 / (1.0 + math.exp(-a))
        np.testing.assert_allclose(o[0, 0, i], w0 * vf[0] + (1 - w0) * vf[1], rtol=0, atol=1e-13)


# ---------------------------------------------------------------- invariants
def test_live_rows_sum_to_one_dead_rows_zero():
    q, k, _ = small_qkv(14, 1, 2, 2, 140, 140, 16)
    v = torch.ones((1, 2, 140, 16), dtype=torch.bfloat16)
    m = random_block_mask(np.random.default_rng(14), 1, 2, 3, 3, p=0.5, kill_rows=2)
    o = oracle.attention(q, k, v, m, 0.25, True, 64)
    _, live = sdpa_reference(q, k, v, m, 0.25, True, 64)
    np.testing.assert_allclose(o[live], 1.0, rtol=0, atol=1e-12)
    assert np.all(o[~live] == 0.0)


def test_output_in_range_of_visible_values():
    q, k, v = small_qkv(15, 1, 1, 1, 100, 100, 8)
    o = oracle.attention(q, k, v, None, 1.0, True, 64)[0, 0]
    vv = v[0, 0].to(torch.float64).numpy()
    for i in range(100):
        lo, hi = vv[: i + 1].min(0), vv[: i + 1].max(0)
        assert np.all(o[i] >= lo - 1e-12) and np.all(o[i] <= hi + 1e-12)


def test_joint_key_permutation_invariance():
    q, k, v = small_qkv(16, 1, 2, 1, 50, 70, 8)
    perm = torch.from_numpy(np.random.default_rng(0).permutation(70))
    a = oracle.attention(q, k, v, None, 0.35, False, 64)
    b = oracle.attention(q, k[:, :, perm], v[:, :, perm], None, 0.35, False, 64)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_key_translation_invariance():
    # adding u to every key adds q_i.u to the whole score row i
    q, k, v = small_qkv(17, 1, 1, 1, 60, 60, 8)
    u = torch.tensor([0.5, -0.25, 0, 0, 1.0, 0, 0, -0.5], dtype=torch.float64)
    k2 = k.to(torch.float64) + u
    a = oracle.attention(q, k, v, None, 0.25, True, 64)
    b = oracle.attention(q.to(torch.float64), k2, v.to(torch.float64), None, 0.25, True, 64)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-11)


def test_gqa_equals_repeated_mha():
    q, k, v = small_qkv(18, 1, 8, 2, 90, 90, 8)
    m = random_block_mask(np.random.default_rng(18), 1, 8, 2, 2, p=0.7)
    a = oracle.attention(q, k, v, m, 0.25, True, 64)
    b = oracle.attention(q, k.repeat_interleave(4, 1), v.repeat_interleave(4, 1), m, 0.25, True, 64)
    np.testing.assert_array_equal(a, b)


def test_scale_folds_into_query():
    q, k, v = small_qkv(19, 1, 1, 1, 40, 40, 8)
    a = oracle.attention(q, k, v, None, 0.125, True, 64)
    b = oracle.attention(q.to(torch.float64) * 0.125, k, v, None, 1.0, True, 64)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


# ---------------------------------------------------------------- planted mistakes
def _pins_pass():
    """Run a compact set of the pins above; True iff all pass."""
    try:
        for case in (TINY[3], TINY[7], TINY[10], TINY[11]):
            test_oracle_matches_brute_force(case)
        test_oracle_matches_sdpa(0, True, True)
        test_oracle_matches_sdpa(1, False, False)
        test_causal_row0_is_first_value_row()
        test_zero_query_gives_mean_of_visible_values()
        test_two_keys_logistic()
        test_live_rows_sum_to_one_dead_rows_zero()
        test_gqa_equals_repeated_mha()
    except AssertionError:
        return False
    return True


def _mut_head_rows_axis0(qh, kh, vh, vis, scale):
    s = np.where(vis, (qh @ kh.T) * scale, -np.inf)
    m = np.where(np.isfinite(s.max(0, keepdims=True)), s.max(0, keepdims=True), 0.0)
    p = np.exp(s - m)
    return (p / np.maximum(p.sum(0, keepdims=True), 1e-300)) @ vh


def _mut_head_rows_no_scale(qh, kh, vh, vis, scale):
    return _ORIG_HEAD_ROWS(qh, kh, vh, vis, 1.0)


def _mut_head_rows_transposed(qh, kh, vh, vis, scale):
    # uses V where K belongs
    return _ORIG_HEAD_ROWS(qh, vh, vh, vis, scale)


def _mut_visibility_strict(bits, rows, S_q, S_k, blk, causal):
    vis = _ORIG_VIS(bits, rows, S_q, S_k, blk, False)
    if causal:
        cols = np.arange(S_k)
        vis &= cols[None, :] < np.asarray(rows)[:, None] + (S_k - S_q)
    return vis


def _mut_visibility_top_left(bits, rows, S_q, S_k, blk, causal):
    vis = _ORIG_VIS(bits, rows, S_q, S_k, blk, False)
    if causal:
        vis &= np.arange(S_k)[None, :] <= np.asarray(rows)[:, None]
    return vis


def _mut_visibility_no_mask(bits, rows, S_q, S_k, blk, causal):
    return _ORIG_VIS(None, rows, S_q, S_k, blk, causal)


_ORIG_HEAD_ROWS = oatt._head_rows
_ORIG_VIS = oatt.element_visibility

MUTATIONS = {
    "kv_head_modulo": ("kv_head", lambda h, Hq, Hkv: h % Hkv),
    "softmax_axis0": ("_head_rows", _mut_head_rows_axis0),
    "scale_dropped": ("_head_rows", _mut_head_rows_no_scale),
    "k_replaced_by_v": ("_head_rows", _mut_head_rows_transposed),
    "causal_strict": ("element_visibility", _mut_visibility_strict),
    "causal_top_left": ("element_visibility", _mut_visibility_top_left),
    "block_mask_dropped": ("element_visibility", _mut_visibility_no_mask),
}


def test_pins_pass_on_the_oracle():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(oatt, attr, fn)
    assert not _pins_pass(), f"planted mistake {name} went unnoticed"
