"""Pins of the fp8 model (oracle/fp8_attention.py) against things other than
itself: torch's own E4M3 conversion, the code table of the format, closed
forms of special inputs, exact power-of-two invariances, pure-Python brute
force on one tile, and the distance to exact attention."""
import math

import numpy as np
import pytest
import torch

from oracle import attention
from oracle.fp8_attention import (attention_fp8, e4m3_round, pow2_scale, quantize_rows,
                                  quantize_tensor)


def _codes():
    """All finite non-negative E4M3 values from the format definition."""
    vals = []
    for e in range(16):
        for m in range(8):
            if e == 15 and m == 7:
                continue  # NaN
            vals.append(m / 8 * 2.0 ** -6 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))
    return np.array(sorted(vals))


def test_code_table_fixed_points_and_ties_to_even():
    grid = _codes()
    assert grid[-1] == 448.0 and grid[1] == 2.0 ** -9
    assert np.array_equal(e4m3_round(grid), grid)
    assert np.array_equal(e4m3_round(-grid), -grid)
    mids = (grid[:-1] + grid[1:]) / 2
    got = e4m3_round(mids)
    # the even neighbour: the code with an even mantissa field (step index)
    idx = np.arange(len(grid))
    even = np.where(idx[:-1] % 2 == 0, grid[:-1], grid[1:])
    assert np.array_equal(got, even)


def test_hand_values():
    cases = {1.0625: 1.0, 1.1875: 1.25, 1.07: 1.125, 2.0 ** -10: 0.0, 3 * 2.0 ** -10: 2.0 ** -8,
             0.3: 0.3125, 440.0: 448.0, 100.0: 96.0, 104.0: 104.0, 232.0: 224.0}
    for x, want in cases.items():
        assert e4m3_round(x) == want, x
    with pytest.raises(ValueError):
        e4m3_round(449.0)


def test_matches_torch_float8_e4m3fn():
    bits = (np.uint32(0x3A000000) + np.arange(0, 20200, dtype=np.uint32) * np.uint32(0x2000))
    x = bits.view(np.float32).astype(np.float64)
    x = x[x <= 448.0]
    x = np.concatenate([x, -x, np.random.default_rng(0).uniform(-448, 448, 100000)])
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(e4m3_round(x), ref)


def test_pow2_scale():
    assert pow2_scale(448.0) == 1.0
    assert pow2_scale(224.0) == 2.0
    assert pow2_scale(224.5) == 1.0
    assert pow2_scale(1.0) == 256.0
    assert pow2_scale(449.0) == 0.5
    assert pow2_scale(0.0) == 1.0
    a = np.random.default_rng(1).lognormal(0, 6, 10000)
    s = pow2_scale(a)
    assert np.all(a * s <= 448.0) and np.all(a * s > 224.0)
    assert np.all(np.log2(s) == np.round(np.log2(s)))


def _inputs(B, Hq, Hkv, S_q, S_k, D, seed, spread=1.0):
    g = torch.Generator().manual_seed(seed)
    q = (torch.randn(B, Hq, S_q, D, generator=g) * spread).to(torch.bfloat16)
    k = torch.randn(B, Hkv, S_k, D, generator=g).to(torch.bfloat16)
    v = torch.randn(B, Hkv, S_k, D, generator=g).to(torch.bfloat16)
    return q, k, v


def test_zero_query_is_mean_of_quantized_values():
    # all scores 0: every visible key gets weight 2^8 exactly, so the output
    # is the plain mean of E4M3(V s_v) / s_v over the visible keys
    _, k, v = _inputs(1, 2, 1, 130, 130, 16, 3)
    q = torch.zeros(1, 2, 130, 16, dtype=torch.bfloat16)
    out, lse = attention_fp8(q, k, v, causal=True)
    v8, sv = quantize_tensor(v[0, 0].double().numpy())
    vq = v8 / sv
    for i in (0, 1, 63, 64, 100, 129):
        want = vq[: i + 1].mean(axis=0)
        np.testing.assert_allclose(out[0, 0, i], want, rtol=0, atol=1e-15)
        assert lse[0, 1, i] == pytest.approx(math.log(i + 1), abs=1e-12)


def test_offset_keeps_small_weights():
    # one key 12 log2 units above 1000 others: without the +8 offset the small
    # weights (2^-12 of the maximum) would fall below E4M3's range and vanish;
    # with it they are 2^-4, exactly representable, and carry half the mass
    D, n = 8, 4097
    c = math.log2(math.e) / math.sqrt(D)
    q = torch.zeros(1, 1, 1, D, dtype=torch.bfloat16)
    q[0, 0, 0, 0] = 1.0
    k = torch.zeros(1, 1, n, D, dtype=torch.bfloat16)
    k[0, 0, 0, 0] = 12.0 / c   # not exact in bf16: take the actual score below
    v = torch.zeros(1, 1, n, D, dtype=torch.bfloat16)
    v[0, 0, 0, 1] = 1.0
    v[0, 0, 1:, 2] = 1.0
    out, _ = attention_fp8(q, k, v, causal=False)
    k0 = float(k[0, 0, 0, 0]) * pow2_scale(abs(float(k[0, 0, 0, 0])))
    s_top = float(e4m3_round(k0)) / pow2_scale(abs(float(k[0, 0, 0, 0]))) * 1.0 * c
    # q scale: row amax 1 -> s_q 256, q8 = 256, divided back out exactly
    w_small = float(e4m3_round(2.0 ** (0 - s_top + 8)))
    w_top = 256.0
    l = w_top + (n - 1) * 2.0 ** (0 - s_top + 8)
    np.testing.assert_allclose(out[0, 0, 0, 1], w_top / l, rtol=1e-14)
    np.testing.assert_allclose(out[0, 0, 0, 2], (n - 1) * w_small / l, rtol=1e-14)
    assert 0.4 < out[0, 0, 0, 2] < 0.6


def test_power_of_two_invariances():
    q, k, v = _inputs(1, 2, 2, 200, 200, 32, 5)
    out, lse = attention_fp8(q, k, v, scale=0.125)
    # V * 2^3: the same E4M3 codes under the scale, output * 2^3 exactly
    out_v, lse_v = attention_fp8(q, k, v * 8, scale=0.125)
    assert np.array_equal(out_v, out * 8) and np.array_equal(lse_v, lse)
    # Q * 2^-2 with scale * 2^2: row scales absorb the factor, scores equal
    out_q, lse_q = attention_fp8(q * 0.25, k, v, scale=0.5)
    assert np.array_equal(out_q, out) and np.array_equal(lse_q, lse)


def _brute_one_tile(q, k, v, scale):
    """Pure-Python loops, S_q = S_k <= 64, causal, one head."""
    S, D = len(q), len(q[0])
    c = scale * math.log2(math.e)
    ka = max(abs(x) for row in k for x in row)
    va = max(abs(x) for row in v for x in row)
    sk, sv = float(pow2_scale(ka)), float(pow2_scale(va))
    k8 = [[float(e4m3_round(x * sk)) for x in row] for row in k]
    v8 = [[float(e4m3_round(x * sv)) for x in row] for row in v]
    out = []
    for i in range(S):
        sq = float(pow2_scale(max(abs(x) for x in q[i])))
        q8 = [float(e4m3_round(x * sq)) for x in q[i]]
        s = [sum(q8[d] * k8[j][d] for d in range(D)) / (sq * sk) * c for j in range(i + 1)]
        mx = max(s)
        p = [2.0 ** (sj - mx + 8) for sj in s]
        l = sum(p)
        out.append([sum(float(e4m3_round(p[j])) * v8[j][d] for j in range(i + 1)) / sv / l
                    for d in range(D)])
    return out


def test_single_tile_brute_force():
    q, k, v = _inputs(1, 1, 1, 40, 40, 8, 7, spread=3.0)
    out, _ = attention_fp8(q, k, v, scale=0.3)
    want = _brute_one_tile(q[0, 0].double().tolist(), k[0, 0].double().tolist(),
                           v[0, 0].double().tolist(), 0.3)
    np.testing.assert_allclose(out[0, 0], np.array(want), rtol=1e-12, atol=1e-14)


def test_close_to_exact_attention_but_not_equal():
    # several tiles, GQA, a block mask with dead rows, ragged sizes
    B, Hq, Hkv, S_q, S_k, D = 1, 4, 2, 200, 260, 64
    q, k, v = _inputs(B, Hq, Hkv, S_q, S_k, D, 9)
    rng = np.random.default_rng(2)
    mask = (rng.random((B, Hq, 4, 5)) < 0.6).astype(np.uint8)
    mask[0, 0, 1, :] = 0
    out, lse = attention_fp8(q, k, v, mask, causal=True)
    exact = attention(q, k, v, torch.from_numpy(mask), causal=True)
    err = np.abs(out - exact)
    assert np.isfinite(out).all()
    # loose bound: each term's operands carry at most 2^-4 relative rounding
    # and the score error moves each weight by a few percent, so every output
    # stays within 1/32 of the largest |V| (about 4 here) of the exact one
    vmax = float(v.abs().max())
    assert err.max() < vmax / 32 and err.mean() < 0.01
    assert err.mean() > 1e-4        # the operands really are rounded
    assert np.all(out[0, 0, 64:128] == 0) and np.all(lse[0, 0, 64:128] == -np.inf)


def test_pv_only_form():
    # scores from the unrounded bf16 values: a single tile against loops
    q, k, v = _inputs(1, 1, 1, 30, 30, 8, 13, spread=3.0)
    out, lse = attention_fp8(q, k, v, scale=0.3, qk_fp8=False)
    qd, kd, vd = (t[0, 0].double().numpy() for t in (q, k, v))
    v8, sv = quantize_tensor(vd)
    c = 0.3 * math.log2(math.e)
    for i in (0, 7, 29):
        s_ = [float(np.dot(qd[i], kd[j])) * c for j in range(i + 1)]
        mx = max(s_)
        p = [2.0 ** (x - mx + 8) for x in s_]
        want = sum(float(e4m3_round(p[j])) * v8[j] for j in range(i + 1)) / sv / sum(p)
        np.testing.assert_allclose(out[0, 0, i], want, rtol=1e-12, atol=1e-14)
        assert lse[0, 0, i] == pytest.approx(math.log(sum(2.0 ** x for x in s_)), rel=1e-12)
    # peaked scores (large |s|): the P V-only form stays near exact attention,
    # the form with E4M3 scores does not
    q, k, v = _inputs(1, 2, 2, 128, 128, 64, 15, spread=4.0)
    exact = attention(q, k, v, None, causal=True)
    err_pv = np.abs(attention_fp8(q, k, v, qk_fp8=False)[0] - exact)
    err_all = np.abs(attention_fp8(q, k, v)[0] - exact)
    assert err_pv.mean() < 0.5 * err_all.mean()


def test_subset_rows_equal_full_run():
    q, k, v = _inputs(2, 2, 1, 150, 150, 16, 11)
    full, lse = attention_fp8(q, k, v)
    part, lsep = attention_fp8(q, k, v, heads=[(1, 0)], qblocks=[2])
    assert np.array_equal(part[1, 0, 128:150], full[1, 0, 128:150])
    assert np.isnan(part[0, 0]).all()


@pytest.mark.parametrize("mistake", ["no_p_round", "no_offset", "no_v_descale"])
def test_planted_mistakes_are_caught(mistake, monkeypatch):
    """Each plausible slip in the model fails one of the pins above."""
    import oracle.fp8_attention as F

    if mistake == "no_p_round":
        monkeypatch.setattr(F, "round_p", lambda p: np.asarray(p, dtype=np.float64))
        with pytest.raises(AssertionError):
            test_single_tile_brute_force()
    elif mistake == "no_offset":
        monkeypatch.setattr(F, "P_OFFSET", 0.0)
        with pytest.raises(AssertionError):
            test_offset_keeps_small_weights()
    else:
        real = F.quantize_tensor
        monkeypatch.setattr(F, "quantize_tensor", lambda x: (real(x)[0], 1.0))
        with pytest.raises(AssertionError):
            test_zero_query_is_mean_of_quantized_values()
