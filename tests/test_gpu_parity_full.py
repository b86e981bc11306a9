"""GPU parity where the kernels branch only at scale (Section IV-A tile
classes; Section IV-C placement), against the float64 oracle.

* The window/sink workload at full size (S = 16384, 32/8 heads): the output
  buffer starts as NaN and every element must come back finite (a skipped or
  duplicated work item would leave NaN behind); every row of one query head
  per key/value group (8 x 16384 rows, each head at a different wave position
  of its pack) is compared with the oracle element by element.
* More than 1024 head-pack items, so the packed kernel deals its work order
  to the XCDs in groups of 16 (the dealing the full-size window/sink workload
  uses), against the full oracle, with S_k a multiple of 64 and ragged.
* The index build above 12288 rows (per-chunk histograms in global memory)
  with live counts of 128 and more (where count bins merge counts), bit for
  bit against the index oracle.
* Uniform head packs of 4 at D = 64 (the packed 32-row kernel), against the
  full oracle.

Bar: max-abs <= 1e-2 and mean-abs <= 1e-3 over all compared elements; index
outputs bit for bit.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import workloads
from workloads import CONFIGS, small_qkv

pytestmark = pytest.mark.gpu

MAX_ABS = 1e-2
MEAN_ABS = 1e-3


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


def fused(q, k, v, m, scale, causal):
    s = steel()
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = None if m is None else torch.from_numpy(np.ascontiguousarray(m)).to(dev)
    out = torch.full(tuple(q.shape), float("nan"), dtype=torch.float32, device=dev)
    s.attn_fwd(qd, kd, vd, md, scale=scale, causal=causal, out=out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def window_mask(B, Hq, nQB, nKB, win, sink):
    qb = np.arange(nQB)[:, None]
    kb = np.arange(nKB)[None, :]
    keep = ((kb <= qb) & (kb > qb - win)) | (kb < sink)
    return np.ascontiguousarray(np.broadcast_to(keep.astype(np.uint8), (B, Hq, nQB, nKB)))


@pytest.mark.timeout(900)
def test_window_sink_full_size_every_row_of_one_head_per_group():
    cfg = CONFIGS["gqa32x8_s16384_d128_window1024_sink64"]
    say(f"[parity-full] {cfg.name}: generating inputs")
    q, k, v, m = workloads.make_workload(cfg)
    say(f"[parity-full] {cfg.name}: GPU run (NaN-prefilled output)")
    got = fused(q, k, v, m, cfg.scale, cfg.causal)
    assert np.all(np.isfinite(got)), "an output element was never written"
    G = cfg.Hq // cfg.Hkv
    heads = [g * G + (g % G) for g in range(cfg.Hkv)]  # one per group, every wave position
    abs_sum, n_el, mx = 0.0, 0, 0.0
    chunk = 2048
    for h in heads:
        say(f"[parity-full] {cfg.name}: oracle, all {cfg.S_q} rows of head {h}")
        for r0 in range(0, cfg.S_q, chunk):
            rows = np.arange(r0, min(cfg.S_q, r0 + chunk))
            idx = np.stack([np.zeros_like(rows), np.full_like(rows, h), rows], 1)
            want = oracle.attention_rows(q, k, v, idx, m, cfg.scale, cfg.causal, 64)
            err = np.abs(got[0, h, rows].astype(np.float64) - want)
            mx = max(mx, float(err.max()))
            abs_sum += float(err.sum())
            n_el += err.size
    mean = abs_sum / n_el
    say(f"  {cfg.name}: {len(heads)} heads x {cfg.S_q} rows: max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert mx <= MAX_ABS
    assert mean <= MEAN_ABS


# B, Hq, Hkv, S, D: 8 * (32/4) * nQB >= 2048 head-pack items (> 1024: groups of 16)
GROUP16 = [("aligned_s2048", 8, 32, 8, 2048, 128), ("ragged_s2100", 8, 32, 8, 2100, 128)]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", GROUP16, ids=[c[0] for c in GROUP16])
def test_pack_dealing_in_groups_of_16_full_oracle(case):
    name, B, Hq, Hkv, S, D = case
    nQB = -(-S // 64)
    n_items = B * (Hq // 4) * nQB
    assert n_items > 1024
    say(f"[parity-full] groups of 16: {name}, {n_items} pack items")
    q, k, v = small_qkv(17 + S, B, Hq, Hkv, S, S, D)
    m = window_mask(B, Hq, nQB, nQB, 16, 1)
    scale = 1.0 / math.sqrt(D)
    got = fused(q, k, v, m, scale, True)
    assert np.all(np.isfinite(got))
    want = oracle.attention(q, k, v, m, scale, True, 64)
    err = np.abs(got.astype(np.float64) - want)
    say(f"  {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


INDEX_LARGE = [
    # name, B, Hq, S, causal, mask p (None: no mask)
    ("causal_32heads_s32768", 1, 32, 32768, True, None),
    ("random_2x13heads_s32768", 2, 13, 32768, True, 0.6),
    ("noncausal_random_1x25heads_s32768", 1, 25, 32768, False, 0.3),
]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", INDEX_LARGE, ids=[c[0] for c in INDEX_LARGE])
def test_index_above_12288_rows_bit_exact(case):
    name, B, Hq, S, causal, p = case
    s = steel()
    nQB = nKB = -(-S // 64)
    R = B * Hq * nQB
    assert R > 12288
    m = None if p is None else workloads.random_block_mask(np.random.default_rng(R), B, Hq, nQB, nKB, p=p)
    want_rp, want_col, want_order = oracle.build_index(m, B, Hq, S, S, 64, causal)
    counts = np.diff(want_rp)
    assert counts.max() >= 128, "the case must reach the merged count bins"
    say(f"[parity-full] index {name}: R={R}, live counts up to {counts.max()}")
    md = None if m is None else torch.from_numpy(m).cuda()
    rp, col, order = s.block_index(md, B, Hq, S, S, causal=causal, device=torch.device("cuda:0"))
    torch.cuda.synchronize()
    assert np.array_equal(rp.cpu().numpy(), want_rp)
    n = int(want_rp[-1])
    assert np.array_equal(col.cpu().numpy()[:n].view(np.uint32), want_col)
    assert np.array_equal(order.cpu().numpy(), want_order)


def test_fused_call_above_12288_rows():
    """The fused call over an index built by the large-problem path: 13 heads
    (single-head items), S = 65536 keys per head with only the diagonal and
    two random blocks per row live, sampled rows against the oracle and the
    whole output finite."""
    B, Hq, Hkv, S, D = 1, 13, 13, 61440, 64
    nQB = S // 64
    assert B * Hq * nQB > 12288
    rng = np.random.default_rng(5)
    m = np.zeros((B, Hq, nQB, nQB), dtype=np.uint8)
    i = np.arange(nQB)
    m[:, :, i, i] = 1
    for h in range(Hq):
        m[0, h, i, rng.integers(0, nQB, nQB)] = 1
        m[0, h, i, rng.integers(0, nQB, nQB)] = 1
    q, k, v = small_qkv(23, B, Hq, Hkv, S, S, D)
    scale = 1.0 / math.sqrt(D)
    say("[parity-full] fused call above 12288 rows")
    got = fused(q, k, v, m, scale, True)
    assert np.all(np.isfinite(got))
    rows = np.r_[0, 1, 63, 64, 4095, 30000, S - 1, rng.integers(0, S, 40)]
    idx = np.array([(0, h, r) for h in (0, 6, 12) for r in rows], dtype=np.int64)
    want = oracle.attention_rows(q, k, v, idx, m, scale, True, 64)
    err = np.abs(got[idx[:, 0], idx[:, 1], idx[:, 2]].astype(np.float64) - want)
    say(f"  sampled rows: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


UNIFORM_D64 = [("gqa8x2_s640_d64_causal", 1, 8, 2, 640, True),
               ("gqa8x2_s640_d64_noncausal", 2, 8, 2, 640, False)]


@pytest.mark.parametrize("case", UNIFORM_D64, ids=[c[0] for c in UNIFORM_D64])
def test_uniform_packs_of_4_at_d64_full_oracle(case):
    name, B, Hq, Hkv, S, causal = case
    D = 64
    say(f"[parity-full] uniform packs of 4 at D=64: {name}")
    q, k, v = small_qkv(31, B, Hq, Hkv, S, S, D)
    scale = 1.0 / math.sqrt(D)
    got = fused(q, k, v, None, scale, causal)
    want = oracle.attention(q, k, v, None, scale, causal, 64)
    err = np.abs(got.astype(np.float64) - want)
    say(f"  {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert np.all(np.isfinite(got))
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


# name, B, heads (Hq = Hkv), S: more than 16,384 single-head items (the XCD
# bucket pass takes the work order in two slices), with 5 heads per bucket
# (one head range each) and with 18 heads per bucket (8 ranges of up to 3)
BUCKET_RANGES = [("5_heads_per_bucket_s32768", 1, 40, 32768),
                 ("18_heads_per_bucket_s8192", 2, 72, 8192)]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", BUCKET_RANGES, ids=[c[0] for c in BUCKET_RANGES])
def test_single_head_buckets_in_head_ranges(case):
    """Single-head items dealt to the XCD buckets head range by head range:
    every output element written (NaN-prefilled output), sampled rows of the
    first and last heads of several buckets against the oracle."""
    name, B, H, S = case
    D = 64
    nQB = S // 64
    assert B * H * nQB > 16384
    rng = np.random.default_rng(B * H + S)
    m = workloads.random_block_mask(rng, B, H, nQB, nQB, p=0.05)
    m[:, :, np.arange(nQB), np.arange(nQB)] = 1  # every row has its diagonal block
    q, k, v = small_qkv(41, B, H, H, S, S, D)
    scale = 1.0 / math.sqrt(D)
    say(f"[parity-full] bucket head ranges: {name}, {B * H * nQB} single-head items")
    got = fused(q, k, v, m, scale, True)
    assert np.all(np.isfinite(got)), "an output element was never written"
    rows = np.r_[0, 63, 64, S - 1, rng.integers(0, S, 24)]
    heads = [(b, h) for b in range(B) for h in (0, 7, 8, H - 1)]
    idx = np.array([(b, h, r) for b, h in heads for r in rows], dtype=np.int64)
    want = oracle.attention_rows(q, k, v, idx, m, scale, True, 64)
    err = np.abs(got[idx[:, 0], idx[:, 1], idx[:, 2]].astype(np.float64) - want)
    say(f"  {name}: sampled rows: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


@pytest.mark.timeout(600)
def test_short_pack_list_among_many_single_head_rows():
    """A few uniform head packs (fewer than 64) among at least 1,024
    single-head items: the packs' rows are dealt with the single-head items.
    NaN-prefilled output all finite; every row of every uniform pack and
    sampled other rows against the oracle."""
    B, Hq, Hkv, S, D = 2, 16, 4, 4096, 128
    G = Hq // Hkv
    nQB = S // 64
    rng = np.random.default_rng(77)
    m = workloads.random_block_mask(rng, B, Hq, nQB, nQB, p=0.3)
    i = np.arange(nQB)
    m[:, :, i, i] = 1
    for _ in range(12):  # a dozen more uniform packs: one head's row copied to its group
        b, g, qb = int(rng.integers(B)), int(rng.integers(Hkv)), int(rng.integers(nQB))
        m[b, G * g + 1:G * g + G, qb, :] = m[b, G * g, qb, :]
    alive = np.tril(np.ones((nQB, nQB), dtype=bool))
    live = (m != 0) & alive
    uniform = [(b, g, qb) for b in range(B) for g in range(Hkv) for qb in range(nQB)
               if all(np.array_equal(live[b, G * g, qb], live[b, G * g + h, qb]) for h in range(1, G))]
    n_single = B * Hq * nQB - G * len(uniform)
    assert 0 < len(uniform) < 64 and n_single >= 1024, (len(uniform), n_single)
    q, k, v = small_qkv(43, B, Hq, Hkv, S, S, D)
    scale = 1.0 / math.sqrt(D)
    say(f"[parity-full] short pack list: {len(uniform)} uniform packs, {n_single} single-head rows")
    got = fused(q, k, v, m, scale, True)
    assert np.all(np.isfinite(got)), "an output element was never written"
    idx = [(b, G * g + h, 64 * qb + r) for b, g, qb in uniform for h in range(G) for r in range(64)]
    idx += [(int(rng.integers(B)), int(rng.integers(Hq)), int(rng.integers(S))) for _ in range(256)]
    idx = np.array(idx, dtype=np.int64)
    want = oracle.attention_rows(q, k, v, idx, m, scale, True, 64)
    err = np.abs(got[idx[:, 0], idx[:, 1], idx[:, 2]].astype(np.float64) - want)
    say(f"  {len(idx)} rows: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS
