"""Pins for the block-index oracle and the seeded workloads (CPU only).

* Tile classes are checked against element-level brute force: a tile is live
  iff at least one of its real elements is visible, partial iff it is live and
  needs element masking (some real element invisible, or the tile runs past
  the last key) -- the three cases of Section IV-A.
* Live counts of the named workloads have closed forms: a causal 512x512 head
  has 1+2+...+8 = 36 live tiles, a causal 4096 head 64*65/2 = 2080, the window
  of 16 blocks plus a sink block over 256 query blocks 136 + 240*17 = 4216.
* The work order is checked against Python's stable ``sorted``.
* A planted mistake in the oracle's classification is caught.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import block_index as obi
import workloads
from workloads import CONFIGS, random_block_mask


def brute_classes(block_mask, B, Hq, S_q, S_k, blk, causal):
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    live = np.zeros((B, Hq, nQB, nKB), dtype=bool)
    part = np.zeros_like(live)
    for b in range(B):
        for h in range(Hq):
            for qb in range(nQB):
                for kb in range(nKB):
                    vis_any, invis_any = False, False
                    for i in range(qb * blk, min((qb + 1) * blk, S_q)):
                        for j in range(kb * blk, min((kb + 1) * blk, S_k)):
                            ok = block_mask is None or block_mask[b, h, qb, kb] != 0
                            ok = ok and (not causal or j <= i + S_k - S_q)
                            vis_any |= ok
                            invis_any |= not ok
                    live[b, h, qb, kb] = vis_any
                    part[b, h, qb, kb] = vis_any and (invis_any or (kb + 1) * blk > S_k)
    return live, part


CLASS_CASES = [
    # B, Hq, S_q, S_k, blk, causal, mask p
    (1, 1, 40, 40, 8, True, None),
    (1, 2, 40, 40, 8, True, 0.5),
    (2, 2, 37, 45, 8, True, 0.6),     # ragged, S_q < S_k
    (1, 2, 45, 30, 8, True, 0.7),     # S_q > S_k
    (1, 2, 33, 33, 8, False, 0.5),    # key tail only
    (1, 1, 64, 64, 16, True, None),
]


@pytest.mark.parametrize("case", CLASS_CASES, ids=[f"c{i}" for i in range(len(CLASS_CASES))])
def test_tile_classes_match_element_brute_force(case):
    B, Hq, S_q, S_k, blk, causal, p = case
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    m = None if p is None else random_block_mask(np.random.default_rng(S_q), B, Hq, nQB, nKB, p=p)
    live, part = oracle.tile_classes(m, B, Hq, S_q, S_k, blk, causal)
    blive, bpart = brute_classes(m, B, Hq, S_q, S_k, blk, causal)
    assert np.array_equal(live, blive)
    assert np.array_equal(part, bpart)


@pytest.mark.parametrize("case", CLASS_CASES, ids=[f"c{i}" for i in range(len(CLASS_CASES))])
def test_csr_structure(case):
    B, Hq, S_q, S_k, blk, causal, p = case
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    m = None if p is None else random_block_mask(np.random.default_rng(S_q), B, Hq, nQB, nKB, p=p)
    row_ptr, col, order = oracle.build_index(m, B, Hq, S_q, S_k, blk, causal)
    live, part = brute_classes(m, B, Hq, S_q, S_k, blk, causal)
    live2, part2 = live.reshape(-1, nKB), part.reshape(-1, nKB)
    assert row_ptr[0] == 0 and row_ptr[-1] == col.size
    for r in range(live2.shape[0]):
        seg = col[row_ptr[r]: row_ptr[r + 1]]
        kbs = (seg & 0x7FFFFFFF).astype(int).tolist()
        assert kbs == [kb for kb in range(nKB) if live2[r, kb]]
        assert [(int(c) >> 31) == 1 for c in seg] == [bool(part2[r, kb]) for kb in kbs]
    counts = np.diff(row_ptr)
    assert counts.max() < 128          # the bin code is the identity here
    want = sorted(range(len(counts)), key=lambda r: (-counts[r], r))
    assert order.tolist() == want


def brute_bin(c):
    """The bin code from its definition, on Python ints."""
    if c < 128:
        return c
    e = c.bit_length() - 1
    return 128 + 16 * (e - 7) + ((c >> (e - 4)) & 15)


def test_count_bin_closed_forms():
    cs = list(range(0, 5000)) + [2 ** k + d for k in range(12, 31) for d in (-1, 0, 1)] + [2 ** 31 - 1]
    got = oracle.count_bin(np.array(cs)).tolist()
    assert got == [brute_bin(c) for c in cs]
    assert got[:128] == list(range(128))
    # octave starts: 128 -> 128, 256 -> 144, 512 -> 160; last bin of 2**31 - 1
    assert [brute_bin(c) for c in (128, 255, 256, 511, 512)] == [128, 143, 144, 159, 160]
    assert brute_bin(2 ** 31 - 1) == oracle.N_BINS - 1
    # monotone, and one bin never spans more than 1/16 of its smallest count
    assert all(a <= b for a, b in zip(got[:5000], got[1:5000]))
    lo = {}
    for c in range(128, 5000):
        lo.setdefault(brute_bin(c), c)
    for c in range(128, 5000):
        assert c - lo[brute_bin(c)] < lo[brute_bin(c)] / 16
    with pytest.raises(ValueError):
        oracle.count_bin([2 ** 31])


def test_work_order_bins_large_counts():
    # 130, 135 and 129 share bin 128; 200 is bin 137; 127 is bin 127
    counts = np.array([130, 200, 135, 127, 129, 300])
    assert oracle.work_order(counts).tolist() == [5, 1, 0, 2, 4, 3]
    # the plain count sort would put 135 before 130: the bins keep row order
    assert np.argsort(-counts, kind="stable").tolist() == [5, 1, 2, 0, 4, 3]


def test_live_count_closed_forms():
    c1 = CONFIGS["mha1_s512_d64_causal"]
    rp, _, _ = oracle.build_index(None, c1.B, c1.Hq, c1.S_q, c1.S_k, 64, True)
    assert rp[-1] == 36
    c2 = CONFIGS["gqa32x8_s4096_d128_causal"]
    rp, _, _ = oracle.build_index(None, 1, 1, c2.S_q, c2.S_k, 64, True)
    assert rp[-1] == 64 * 65 // 2 == 2080
    c4 = CONFIGS["gqa32x8_s16384_d128_window1024_sink64"]
    m = workloads.window_sink_mask(c4)
    rp, _, _ = oracle.build_index(m[:, :1], 1, 1, c4.S_q, c4.S_k, 64, True)
    assert rp[-1] == sum(range(1, 17)) + 240 * 17 == 4216
    # every query block's diagonal tile is the only partial one in a causal config
    _, col, _ = oracle.build_index(m[:, :1], 1, 1, c4.S_q, c4.S_k, 64, True)
    assert int(np.count_nonzero(col >> 31)) == c4.nQB


def test_planted_classification_mistake_is_caught(monkeypatch):
    # non-causal, ragged: only the key-tail rule makes tiles partial
    B, Hq, S_q, S_k, blk, causal, p = CLASS_CASES[4]
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    m = random_block_mask(np.random.default_rng(S_q), B, Hq, nQB, nKB, p=p)
    orig = obi.tile_classes

    def no_tail(block_mask, B, Hq, S_q, S_k, blk, causal):
        # forgets that a tile running past the last key needs element masking
        live, _ = orig(block_mask, B, Hq, S_q, S_k, blk, causal)
        qb = np.arange(live.shape[2])[:, None]
        kb = np.arange(live.shape[3])[None, :]
        part_c = causal & ((kb + 1) * blk - 1 > qb * blk + S_k - S_q)
        return live, live & part_c

    monkeypatch.setattr(obi, "tile_classes", no_tail)
    live, part = obi.tile_classes(m, B, Hq, S_q, S_k, blk, causal)
    blive, bpart = brute_classes(m, B, Hq, S_q, S_k, blk, causal)
    assert np.array_equal(live, blive)
    assert not np.array_equal(part, bpart)


# ---------------------------------------------------------------- workloads
def test_generators_are_deterministic():
    cfg = workloads.Config("t", 1, 4, 2, 256, 256, 64, True, "bernoulli", seed=3)
    a = workloads.make_workload(cfg)
    b = workloads.make_workload(cfg)
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
    assert np.array_equal(a[3], b[3])


def test_bernoulli_mask_properties():
    cfg = CONFIGS["gqa32x8_s8192_d128_causal_bernoulli25"]
    m = workloads.bernoulli_mask(cfg)
    assert m.shape == (1, 32, 128, 128)
    d = np.arange(128)
    assert np.all(m[:, :, d, d] == 1)
    off = m.astype(bool).copy()
    off[:, :, d, d] = False
    dens = off.sum() / (32 * 128 * 127)
    assert abs(dens - 0.25) < 0.01
    assert not np.array_equal(m[0, 0], m[0, 1])       # seeded per head


def test_topk_meanpool_mask_properties():
    cfg = workloads.Config("t5", 1, 2, 2, 1024, 1024, 16, True, "topk_meanpool",
                           lowrank_rank=4, lowrank_scale=2.0)
    q, k, v = workloads.make_qkv(cfg)
    m = workloads.topk_meanpool_mask(cfg, q, k)
    for h in range(2):
        qm = q[0, h].to(torch.float64).reshape(16, 64, 16).mean(1)
        km = k[0, h].to(torch.float64).reshape(16, 64, 16).mean(1)
        for qb in range(16):
            keep = math.ceil((qb + 1) / 10)
            scores = [(float(qm[qb] @ km[kb]), kb) for kb in range(qb + 1)]
            top = sorted(scores, key=lambda t: (-t[0], t[1]))[:keep]
            want = {kb for _, kb in top} | {qb}
            assert set(np.nonzero(m[0, h, qb])[0].tolist()) == want


def test_lowrank_component_shared_on_q_and_k():
    cfg = workloads.Config("t5", 1, 1, 1, 512, 512, 64, True, "none", lowrank_rank=4,
                           lowrank_scale=2.0)
    q, k, v = workloads.make_qkv(cfg)
    plain = workloads.Config("p", 1, 1, 1, 512, 512, 64, True, "none")
    q0, k0, v0 = workloads.make_qkv(plain)
    assert torch.equal(v, v0)
    dq = q.float() - q0.float()
    dk = k.float() - k0.float()
    # the same rank-4 matrix of entry std 2 was added to both (up to bf16 rounding)
    assert abs(dq.std().item() - 2.0) < 0.1
    assert torch.allclose(dq, dk, atol=0.2)
    s = torch.linalg.svdvals(dq[0, 0].double())
    assert s[4] < 0.05 * s[3]
