"""GPU parity: libsteel (through the C ABI) against the float64 oracle.

Bar (bf16 inputs, fp32 accumulation): max-abs error <= 1e-2 and mean-abs
error <= 1e-3 against the float64 oracle on the same seeded inputs.  Integer
outputs of the index build must match the index oracle bit for bit.

Small cases run the full oracle and span several tiles with ragged tails; the
five named workloads run at full size and are compared on sampled rows that
the oracle computes one by one (first/last rows of blocks, the causal
diagonal, random rows), plus properties that hold at any size.
"""
import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads
from workloads import CONFIGS, small_qkv, random_block_mask

pytestmark = pytest.mark.gpu

MAX_ABS = 1e-2
MEAN_ABS = 1e-3


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


def run(q, k, v, m, scale, causal, stream=None):
    """One fused call; the output buffer starts as NaN, so an element the
    kernels skip (a work item lost or a row never stored) cannot pass."""
    s = steel()
    dev = torch.device("cuda:0")
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    md = None if m is None else torch.from_numpy(np.ascontiguousarray(m)).to(dev)
    out = torch.full(tuple(q.shape), float("nan"), dtype=torch.float32, device=dev)
    s.attn_fwd(qd, kd, vd, md, scale=scale, causal=causal, stream=stream, out=out)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def check_close(got, want, label):
    err = np.abs(got - want)
    mx, mean = float(err.max()), float(err.mean())
    say(f"  {label}: max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert np.all(np.isfinite(got)), f"{label}: non-finite output"
    assert mx <= MAX_ABS, f"{label}: max abs error {mx}"
    assert mean <= MEAN_ABS, f"{label}: mean abs error {mean}"


SMALL = [
    # name, B, Hq, Hkv, S_q, S_k, D, causal, mask kind
    ("one_tile", 1, 1, 1, 64, 64, 64, True, "none"),
    ("ragged_causal", 1, 2, 2, 200, 200, 64, True, "none"),
    ("ragged_noncausal", 2, 2, 1, 130, 190, 128, False, "none"),
    ("sq_lt_sk", 1, 4, 2, 100, 300, 128, True, "random"),
    ("sq_gt_sk_dead_rows", 1, 2, 1, 300, 100, 64, True, "none"),
    ("gqa8_uniform_mask", 1, 8, 1, 256, 256, 128, True, "uniform"),
    ("gqa4_packs_ragged_d128", 2, 8, 2, 200, 200, 128, True, "none"),
    # more head-pack items than the packed kernel's 256 persistent
    # workgroups: each takes two or three, so item transitions (next item's
    # first tiles and Q rows, output staging) are checked against the full
    # oracle; the uniform mask mixes items with 0, 1, 2 and more live tiles
    ("packs_multi_item_causal", 8, 32, 8, 512, 512, 128, True, "none"),
    ("packs_multi_item_masked_ragged", 8, 32, 8, 600, 600, 128, True, "uniform"),
    ("gqa4_random_mask", 2, 8, 2, 320, 320, 64, True, "random"),
    ("gqa2_mixed_packs", 1, 4, 2, 384, 384, 128, True, "mixed"),
    ("dead_query_blocks", 1, 4, 4, 256, 256, 64, False, "deadrows"),
    ("tiny_S1", 1, 1, 1, 1, 1, 64, True, "none"),
    ("S65_D128", 3, 3, 1, 65, 65, 128, True, "none"),
    ("noncausal_masked", 1, 2, 2, 448, 448, 128, False, "random"),
    # mixed head packs, 126 of them uniform
    ("gqa4_mixed_packs_126", 2, 16, 4, 1024, 1024, 128, True, "mixed"),
    # single heads at D = 64 with S_k a multiple of 64 (the key-split kernel)
    ("sq_gt_sk_aligned_d64", 1, 2, 2, 256, 128, 64, True, "random"),
    ("sq_lt_sk_aligned_d64_noncausal", 2, 3, 3, 128, 320, 64, False, "random"),
]


def small_mask(kind, B, Hq, S_q, S_k, seed):
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    rng = np.random.default_rng(seed)
    if kind == "none":
        return None
    if kind == "random":
        return random_block_mask(rng, B, Hq, nQB, nKB, p=0.5)
    if kind == "uniform":
        m = random_block_mask(rng, B, 1, nQB, nKB, p=0.6)
        return np.ascontiguousarray(np.broadcast_to(m, (B, Hq, nQB, nKB)))
    if kind == "mixed":
        # some head packs share their lists, others differ in one block
        m = np.ascontiguousarray(np.broadcast_to(random_block_mask(rng, B, 1, nQB, nKB, p=0.6),
                                                 (B, Hq, nQB, nKB)))
        m[0, 1, 2, 1] ^= 1
        m[0, 3, 5, 0] ^= 1
        return m
    if kind == "deadrows":
        m = random_block_mask(rng, B, Hq, nQB, nKB, p=0.7)
        m[0, 0, 1, :] = 0
        m[0, 3, :, :] = 0
        return m
    raise ValueError(kind)


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_cases_full_oracle(case):
    name, B, Hq, Hkv, S_q, S_k, D, causal, kind = case
    say(f"[parity] small {name}: B={B} Hq={Hq} Hkv={Hkv} S_q={S_q} S_k={S_k} D={D} causal={causal} mask={kind}")
    q, k, v = small_qkv(zlib.crc32(name.encode()) % 1000, B, Hq, Hkv, S_q, S_k, D)
    m = small_mask(kind, B, Hq, S_q, S_k, seed=len(name))
    scale = 1.0 / math.sqrt(D)
    got = run(q, k, v, m, scale, causal)
    want = oracle.attention(q, k, v, m, scale, causal, 64)
    check_close(got, want, name)
    live, _ = oracle.tile_classes(m, B, Hq, S_q, S_k, 64, causal)
    # rows with no visible key are exactly zero
    vis_rows = np.zeros((B, Hq, S_q), dtype=bool)
    for b in range(B):
        for h in range(Hq):
            rows = np.arange(S_q)
            vis = oracle.element_visibility(None if m is None else m[b, h], rows, S_q, S_k, 64, causal)
            vis_rows[b, h] = vis.any(1)
    assert np.all(got[~vis_rows] == 0.0)


def sample_rows(cfg, rng, n_random=64):
    idx = []
    heads = sorted(set([0, cfg.Hq - 1] + rng.integers(0, cfg.Hq, 6).tolist()))
    for h in heads:
        rows = {0, 1, 63, 64, cfg.S_q - 1, cfg.S_q // 2, cfg.S_q // 2 + 63}
        rows |= set(rng.integers(0, cfg.S_q, n_random // len(heads) + 1).tolist())
        for i in sorted(rows):
            idx.append((0, h, i))
    return np.array(idx, dtype=np.int64)


@pytest.mark.parametrize("name", workloads.CONFIG_ORDER)
def test_named_workloads(name):
    cfg = CONFIGS[name]
    say(f"[parity] workload {name}: generating inputs")
    q, k, v, m = workloads.make_workload(cfg)
    say(f"[parity] workload {name}: GPU run")
    got = run(q, k, v, m, cfg.scale, cfg.causal)
    if cfg.S_q * cfg.Hq <= 4096:
        want = oracle.attention(q, k, v, m, cfg.scale, cfg.causal, 64)
        check_close(got, want, name + " (full)")
        return
    idx = sample_rows(cfg, np.random.default_rng(0))
    say(f"[parity] workload {name}: oracle on {len(idx)} sampled rows")
    want = oracle.attention_rows(q, k, v, idx, m, cfg.scale, cfg.causal, 64)
    check_close(got[idx[:, 0], idx[:, 1], idx[:, 2]], want, name + " (sampled rows)")
    assert np.all(np.isfinite(got))


def test_block_index_matches_oracle():
    s = steel()
    cases = [
        ("causal_none", 1, 3, 300, 300, True, None),
        ("random", 2, 4, 200, 330, True, 0.5),
        ("noncausal_tail", 1, 2, 130, 250, False, 0.6),
        ("sq_gt_sk", 1, 2, 400, 150, True, 0.7),
    ]
    for name, B, Hq, S_q, S_k, causal, p in cases:
        say(f"[parity] block_index {name}")
        nQB, nKB = -(-S_q // 64), -(-S_k // 64)
        m = None if p is None else random_block_mask(np.random.default_rng(B + Hq), B, Hq, nQB, nKB, p=p)
        md = None if m is None else torch.from_numpy(m).cuda()
        rp, col, order = s.block_index(md, B, Hq, S_q, S_k, causal=causal, device=torch.device("cuda:0"))
        torch.cuda.synchronize()
        want_rp, want_col, want_order = oracle.build_index(m, B, Hq, S_q, S_k, 64, causal)
        assert np.array_equal(rp.cpu().numpy(), want_rp)
        n = int(want_rp[-1])
        assert np.array_equal(col.cpu().numpy()[:n].view(np.uint32), want_col)
        assert np.array_equal(order.cpu().numpy(), want_order)


@pytest.mark.parametrize("name", ["gqa32x8_s8192_d128_causal_bernoulli25",
                                  "mha24_s32768_d64_causal_top10_lowrank4"])
def test_block_index_named_workloads(name):
    s = steel()
    cfg = CONFIGS[name]
    say(f"[parity] block_index {name}")
    q, k, v, m = workloads.make_workload(cfg)
    md = torch.from_numpy(m).cuda()
    rp, col, order = s.block_index(md, cfg.B, cfg.Hq, cfg.S_q, cfg.S_k, causal=cfg.causal,
                                   device=torch.device("cuda:0"))
    torch.cuda.synchronize()
    want_rp, want_col, want_order = oracle.build_index(m, cfg.B, cfg.Hq, cfg.S_q, cfg.S_k, 64, cfg.causal)
    assert np.array_equal(rp.cpu().numpy(), want_rp)
    assert np.array_equal(col.cpu().numpy()[: int(want_rp[-1])].view(np.uint32), want_col)
    assert np.array_equal(order.cpu().numpy(), want_order)


def test_bitwise_deterministic_and_stream():
    say("[parity] determinism and non-default stream")
    q, k, v = small_qkv(5, 1, 8, 2, 1000, 1000, 128)
    m = random_block_mask(np.random.default_rng(3), 1, 8, 16, 16, p=0.6)
    a = run(q, k, v, m, 0.0884, True)
    b = run(q, k, v, m, 0.0884, True)
    assert np.array_equal(a, b)
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        c = run(q, k, v, m, 0.0884, True, stream=st)
    assert np.array_equal(a, c)


def test_overwrites_output_buffer():
    say("[parity] out buffer fully overwritten")
    s = steel()
    q, k, v = small_qkv(6, 1, 2, 2, 200, 200, 64)
    dev = torch.device("cuda:0")
    m = np.zeros((1, 2, 4, 4), dtype=np.uint8)  # everything dead -> all zeros
    out = torch.full((1, 2, 200, 64), float("nan"), device=dev)
    s.attn_fwd(q.to(dev), k.to(dev), v.to(dev), torch.from_numpy(m).to(dev), causal=True, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 0).item()


def test_plan_run_equals_fused_call_and_rejects_mismatch():
    say("[parity] plan + run == attn_fwd; mismatched plan leaves out untouched")
    s = steel()
    dev = torch.device("cuda:0")
    q, k, v = small_qkv(9, 1, 8, 2, 640, 640, 128)
    m = random_block_mask(np.random.default_rng(9), 1, 8, 10, 10, p=0.5)
    qd, kd, vd, md = q.to(dev), k.to(dev), v.to(dev), torch.from_numpy(m).to(dev)
    a = s.attn_fwd(qd, kd, vd, md, causal=True)
    plan = s.Plan(md, 1, 8, 2, 640, 640, causal=True, device=dev)
    b1 = plan.run(qd, kd, vd)
    b2 = plan.run(qd, kd, vd)
    torch.cuda.synchronize()
    assert torch.equal(a, b1) and torch.equal(a, b2)
    # a plan for the non-causal problem run as causal: header mismatch, out untouched
    plan_nc = s.Plan(md, 1, 8, 2, 640, 640, causal=False, device=dev)
    plan_nc.causal = True
    out = torch.full((1, 8, 640, 128), 7.0, device=dev)
    plan_nc.run(qd, kd, vd, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0).item()
