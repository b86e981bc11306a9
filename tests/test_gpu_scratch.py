"""Fused calls from several streams and several host threads.  Each stream
keeps its own scratch buffer for the live-block index (the float64 workspace
of the mask producer lives there too); calls on one stream reuse it in
stream order, and two threads enqueueing on one stream take turns.

Each call's result must equal, bit for bit, the result of the same call made
alone on one stream (the library's results are reproducible run to run), and
one case is anchored to the float64 oracle.  A call whose index needs more
scratch than any earlier call on its stream makes that stream's buffer grow
while calls are queued on both streams.
"""
import math
import sys
import threading

import numpy as np
import pytest
import torch

import oracle
from workloads import small_qkv, random_block_mask

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


# name, B, Hq, Hkv, S_q, S_k, D, causal, mask p (None: no mask, "diag": only
# the diagonal blocks)
CASES = {
    "packs_masked": (1, 8, 2, 700, 700, 128, True, 0.5),
    "mha_d64": (2, 3, 3, 333, 400, 64, True, None),
    "noncausal_gqa": (1, 4, 2, 256, 640, 128, False, 0.7),
    # 6144 x 6144 blocks: a 144 MiB live-list capacity, more scratch than any
    # other GPU test asks for, so the buffer grows when this call arrives
    "wide_diag": (1, 1, 1, 64 * 6144, 64 * 6144, 64, True, "diag"),
}


def make(name, dev):
    B, Hq, Hkv, S_q, S_k, D, causal, p = CASES[name]
    q, k, v = small_qkv(sum(map(ord, name)) % 997, B, Hq, Hkv, S_q, S_k, D)
    nQB, nKB = -(-S_q // 64), -(-S_k // 64)
    if p is None:
        m = None
    elif p == "diag":
        m = np.zeros((B, Hq, nQB, nKB), dtype=np.uint8)
        i = np.arange(min(nQB, nKB))
        m[:, :, i, i] = 1
    else:
        m = random_block_mask(np.random.default_rng(len(name)), B, Hq, nQB, nKB, p=p)
    dv = [t.to(dev) for t in (q, k, v)]
    md = None if m is None else torch.from_numpy(m).to(dev)
    return (q, k, v, m), (*dv, md), dict(scale=1 / math.sqrt(D), causal=causal)


def call(s, name, inputs, kw, stream):
    qd, kd, vd, md = inputs
    with torch.cuda.stream(stream):
        out = torch.empty(qd.shape, dtype=torch.float32, device=qd.device)
    s.attn_fwd(qd, kd, vd, md, out=out, stream=stream, **kw)
    return out


def test_fused_calls_on_two_streams():
    s = steel()
    dev = torch.device("cuda:0")
    data = {n: make(n, dev) for n in CASES}
    say("[scratch] references, one stream")
    ref = {}
    for n in ("packs_masked", "mha_d64", "noncausal_gqa"):
        ref[n] = call(s, n, data[n][1], data[n][2], torch.cuda.current_stream())
    torch.cuda.synchronize()

    # anchor: one reference against the oracle
    (q, k, v, m), _, kw = data["packs_masked"]
    want = oracle.attention(q, k, v, m, kw["scale"], kw["causal"], 64)
    err = np.abs(ref["packs_masked"].cpu().numpy().astype(np.float64) - want)
    say(f"[scratch] anchor: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= 1e-2 and err.mean() <= 1e-3

    say("[scratch] interleaved calls on two streams, the wide index in the middle")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    seq = [(s1, "packs_masked"), (s2, "mha_d64"), (s1, "noncausal_gqa"), (s2, "packs_masked"),
           (s1, "wide_diag"), (s2, "noncausal_gqa"), (s1, "mha_d64"), (s2, "packs_masked")]
    got = [(n, call(s, n, data[n][1], data[n][2], st)) for st, n in seq]
    torch.cuda.synchronize()
    for i, (n, o) in enumerate(got):
        if n in ref:
            assert torch.equal(o, ref[n]), f"call {i} ({n}) differs from the one-stream result"
    # the wide case: each row sees only its diagonal block (keys up to the row)
    (q, k, v, _), _, kw = data["wide_diag"]
    o = got[4][1][0, 0].cpu().numpy().astype(np.float64)
    rows = np.r_[0:3, 64 * 1000 + 5, 64 * 6144 - 1]
    qf, kf, vf = (t[0, 0].double().numpy() for t in (q, k, v))
    for r in rows:
        lo = (r // 64) * 64
        sc = kw["scale"] * (kf[lo:r + 1] @ qf[r])
        p = np.exp(sc - sc.max())
        want_r = p @ vf[lo:r + 1] / p.sum()
        assert np.abs(o[r] - want_r).max() <= 1e-2, f"wide_diag row {r}"


def test_fused_calls_from_two_threads():
    s = steel()
    dev = torch.device("cuda:0")
    names = ["packs_masked", "mha_d64", "noncausal_gqa"]
    data = {n: make(n, dev) for n in names}
    ref = {n: call(s, n, data[n][1], data[n][2], torch.cuda.current_stream()) for n in names}
    torch.cuda.synchronize()
    results = {0: [], 1: []}
    errors = []

    def worker(t):
        try:
            st = torch.cuda.Stream()
            for r in range(6):
                n = names[(r + t) % 3]
                results[t].append((n, call(s, n, data[n][1], data[n][2], st)))
            st.synchronize()
        except Exception as e:  # reported in the main thread
            errors.append(repr(e))

    say("[scratch] two host threads, one stream each")
    th = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for t in range(2):
        assert len(results[t]) == 6
        for n, o in results[t]:
            assert torch.equal(o, ref[n]), f"thread {t}: {n} differs from the one-stream result"


def test_two_threads_on_one_stream():
    """Both threads enqueue on the same stream and so reuse one scratch
    buffer: the per-stream lock keeps each call's index build and attention
    pass together."""
    s = steel()
    dev = torch.device("cuda:0")
    names = ["packs_masked", "mha_d64", "noncausal_gqa"]
    data = {n: make(n, dev) for n in names}
    ref = {n: call(s, n, data[n][1], data[n][2], torch.cuda.current_stream()) for n in names}
    torch.cuda.synchronize()
    shared = torch.cuda.Stream()
    results = {0: [], 1: []}
    errors = []

    def worker(t):
        try:
            for r in range(8):
                n = names[(r + t) % 3]
                results[t].append((n, call(s, n, data[n][1], data[n][2], shared)))
        except Exception as e:  # reported in the main thread
            errors.append(repr(e))

    say("[scratch] two host threads, one shared stream")
    th = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    shared.synchronize()
    assert not errors, errors
    for t in range(2):
        assert len(results[t]) == 8
        for n, o in results[t]:
            assert torch.equal(o, ref[n]), f"thread {t}: {n} differs from the one-stream result"
