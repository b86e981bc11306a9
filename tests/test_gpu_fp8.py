"""GPU checks of the fp8 forms of steel_attn_fwd_ex: STEEL_FP8 (E4M3 operands
for both products, mode "all") and STEEL_FP8_PV (for P V only, mode "pv").

Two references, both from the oracle package:
* the float64 model of the fp8 form (oracle/fp8_attention.py): the same
  E4M3 operands and scales, the same recurrence in float64.  The kernels
  reach the same quantized Q, K and V codes; what remains is fp32 arithmetic
  (scores accumulated in fp32, exp2 in fp32) and, for about one weight in
  10^4, a weight within a few fp32 ulps of an E4M3 rounding boundary that
  rounds the other way: that moves one weight by one E4M3 step (at most 1/8
  of it) and the row's outputs by up to 1/8 of that weight's share of the
  row times |v - O|.  Bar (FP8_MODEL_*): mean, 99th percentile and max of
  the elementwise difference.
* exact attention (oracle.attention): the error budget of each form, stated
  below (BUDGET) and measured on small cases and on sampled rows of the
  full-size window/sink and low-rank top-10% workloads.  E4M3 scores lose
  the most where scores are large: the low-rank workload (sharply peaked
  rows) has its own, much wider budget in mode "all".
"""
import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads
from oracle.fp8_attention import attention_fp8
from workloads import CONFIGS, small_qkv, random_block_mask

pytestmark = pytest.mark.gpu

FP8_MODEL_MAX = 5e-2     # against the fp8 model, any element
FP8_MODEL_P99 = 1e-3     # 99% of the elements
FP8_MODEL_MEAN = 1e-4
# against exact attention: (max-abs, mean-abs) per mode and input kind
BUDGET = {
    ("all", "small"): (0.25, 1.5e-2),     # N(0,1) Q, K, V
    ("pv", "small"): (0.25, 1.5e-2),
    ("all", "gqa32x8_s16384_d128_window1024_sink64"): (0.25, 1.5e-2),
    ("pv", "gqa32x8_s16384_d128_window1024_sink64"): (0.25, 1.5e-2),
    ("all", "mha24_s32768_d64_causal_top10_lowrank4"): (3.0, 6e-2),
    ("pv", "mha24_s32768_d64_causal_top10_lowrank4"): (0.25, 2.5e-2),
}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


def run_fp8(q, k, v, m, scale, causal, mode, causal_offset=None):
    s = steel()
    dev = torch.device("cuda:0")
    md = None if m is None else torch.from_numpy(np.ascontiguousarray(m)).to(dev)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    B, Hq, S_q, D = q.shape
    out = torch.full((B, Hq, S_q, D), float("nan"), dtype=torch.float32, device=dev)
    lse = torch.full((B, Hq, S_q), float("nan"), dtype=torch.float32, device=dev)
    s.attn_fwd_lse(qd, kd, vd, md, scale=scale, causal=causal, causal_offset=causal_offset,
                   out=out, lse=lse, fp8=mode)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def compare(got, want, label, mx_bar, mean_bar, p99_bar=None):
    err = np.abs(got - want)
    mx, mean, p99 = float(err.max()), float(err.mean()), float(np.quantile(err, 0.99))
    say(f"  {label}: max_abs={mx:.3e} p99={p99:.3e} mean_abs={mean:.3e} "
        f"(>1e-3: {int((err > 1e-3).sum())} of {err.size})")
    assert np.all(np.isfinite(got)), f"{label}: non-finite output"
    assert mx <= mx_bar, f"{label}: max abs error {mx}"
    assert mean <= mean_bar, f"{label}: mean abs error {mean}"
    if p99_bar is not None:
        assert p99 <= p99_bar, f"{label}: 99th percentile error {p99}"
    return mx, mean


def compare_model(got, want, label):
    return compare(got, want, label, FP8_MODEL_MAX, FP8_MODEL_MEAN, FP8_MODEL_P99)


# name, B, Hq, Hkv, S_q, S_k, D, causal, mask keep probability (None: no mask)
CASES = [
    ("packs4_d128_ragged_masked", 1, 8, 2, 600, 600, 128, True, 0.6),
    ("uniform_packs4_d128", 2, 8, 2, 320, 320, 128, True, None),
    ("single_d64_sq_lt_sk", 2, 3, 3, 300, 450, 64, True, None),
    ("packs2_d128_noncausal_masked", 1, 4, 2, 256, 320, 128, False, 0.5),
    ("uniform_packs4_d64_noncausal", 1, 8, 2, 640, 640, 64, False, None),
    ("mha_d128_ragged", 2, 2, 2, 130, 130, 128, True, None),
    ("one_tile_d64", 1, 1, 1, 64, 64, 64, True, None),
]


@pytest.mark.parametrize("mode", ["all", "pv"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fp8_small_cases(case, mode):
    name, B, Hq, Hkv, S_q, S_k, D, causal, p = case
    say(f"[fp8 {mode}] {name}")
    q, k, v = small_qkv(zlib.crc32(name.encode()) % 1000, B, Hq, Hkv, S_q, S_k, D)
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    m = None if p is None else random_block_mask(np.random.default_rng(3), B, Hq, nQB, nKB, p=p,
                                                 kill_rows=1)
    scale = 1 / math.sqrt(D)
    got, lse = run_fp8(q, k, v, m, scale, causal, mode)
    want, wlse = attention_fp8(q, k, v, m, scale, causal, qk_fp8=mode == "all")
    compare_model(got, want, f"{name} vs fp8 model")
    live = np.isfinite(wlse)
    assert np.array_equal(np.isfinite(lse), live)
    compare_model(lse[live], wlse[live], f"{name} lse vs fp8 model")
    assert np.all(got[~live] == 0)
    exact = oracle.attention(q, k, v, m, scale, causal, 64)
    compare(got, exact, f"{name} vs exact", *BUDGET[(mode, "small")])


@pytest.mark.parametrize("mode", ["all", "pv"])
def test_fp8_causal_offset_chunk(mode):
    # a key chunk of a longer sequence (causal_offset), rows that see nothing
    name = "offset_chunk"
    say(f"[fp8 {mode}] {name}")
    q, k, v = small_qkv(17, 1, 4, 2, 200, 190, 128)
    got, lse = run_fp8(q, k, v, None, 0.09, True, mode, causal_offset=-70)
    want, wlse = attention_fp8(q, k, v, None, 0.09, True, causal_offset=-70,
                               qk_fp8=mode == "all")
    compare_model(got, want, f"{name} vs fp8 model")
    assert np.all(got[:, :, :70] == 0) and np.all(lse[:, :, :70] == -np.inf)


@pytest.mark.parametrize("mode", ["all", "pv"])
@pytest.mark.parametrize("wl", ["gqa32x8_s16384_d128_window1024_sink64",
                                "mha24_s32768_d64_causal_top10_lowrank4"])
def test_fp8_error_budget_full_size(wl, mode):
    """Full-size workload through an fp8 form: every output finite; sampled
    query blocks against the fp8 model and against exact attention."""
    cfg = CONFIGS[wl]
    say(f"[fp8 {mode}] full size {wl}")
    q, k, v, m = workloads.make_workload(cfg)
    got, lse = run_fp8(q, k, v, m, cfg.scale, cfg.causal, mode)
    assert np.all(np.isfinite(got)) and np.all(np.isfinite(lse))
    rng = np.random.default_rng(5)
    heads = [(0, int(h)) for h in rng.choice(cfg.Hq, 4, replace=False)]
    qbs = sorted({0, cfg.nQB - 1, *[int(x) for x in rng.integers(0, cfg.nQB, 3)]})
    want, wlse = attention_fp8(q, k, v, m, cfg.scale, cfg.causal, heads=heads, qblocks=qbs,
                               qk_fp8=mode == "all")
    rows = np.concatenate([np.arange(64 * qb, min(64 * qb + 64, cfg.S_q)) for qb in qbs])
    sel_got = np.stack([got[b, h][rows] for b, h in heads])
    sel_want = np.stack([want[b, h][rows] for b, h in heads])
    compare_model(sel_got, sel_want, f"{wl} sampled blocks vs fp8 model")
    idx = np.array([(b, h, r) for b, h in heads for r in rows], dtype=np.int64)
    exact = oracle.attention_rows(q, k, v, idx, m, cfg.scale, cfg.causal, 64)
    bmax, bmean = BUDGET[(mode, wl)]
    mx, mean = compare(sel_got.reshape(-1, cfg.D), exact, f"{wl} sampled blocks vs exact",
                       bmax, bmean)
    say(f"  {wl} ({mode}): |O| max {np.abs(exact).max():.3f}, budget used {mx / bmax:.2f} (max) "
        f"{mean / bmean:.2f} (mean)")
