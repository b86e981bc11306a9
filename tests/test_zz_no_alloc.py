"""steel_attn_fwd_noalloc through the C ABI: the entry point for callers that
cannot allocate builds the index in the library's fixed per-device array and
must give exactly what steel_attn_fwd gives (same kernels), call after call,
also when a smaller problem follows a larger one (the array keeps the last
call's index; nothing in it may leak into the next call)."""
import ctypes
import math
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def lib():
    from paper_2607_09385_amd import _lib
    return _lib


def inputs(seed, B, Hq, Hkv, S_q, S_k, D, p, dev):
    g = torch.Generator(device=dev).manual_seed(seed)
    q = torch.randn((B, Hq, S_q, D), generator=g, device=dev).to(torch.bfloat16)
    k = torch.randn((B, Hkv, S_k, D), generator=g, device=dev).to(torch.bfloat16)
    v = torch.randn((B, Hkv, S_k, D), generator=g, device=dev).to(torch.bfloat16)
    m = None
    if p is not None:
        nQB, nKB = -(-S_q // 64), -(-S_k // 64)
        m = (torch.rand((B, Hq, nQB, nKB), generator=g, device=dev) < p).to(torch.uint8)
    return q, k, v, m


def call(fn, q, k, v, m, out, causal):
    B, Hq, S_q, D = q.shape
    Hkv, S_k = k.shape[1], k.shape[2]
    st = fn(q.data_ptr(), k.data_ptr(), v.data_ptr(), None if m is None else m.data_ptr(),
            out.data_ptr(), B, Hq, Hkv, S_q, S_k, D, 64, 1.0 / math.sqrt(D), causal,
            torch.cuda.current_stream().cuda_stream)
    lib().check(st)


# the largest named index (24 heads, S = 32768: 25.5 MiB of the 32 MiB array)
# first, then smaller problems of other shapes and masks
SEQ = [
    ("mha24_s32768_d64_sparse", 1, 24, 24, 32768, 32768, 64, 0.02, 1),
    ("gqa8x2_s700_d128_masked", 1, 8, 2, 700, 700, 128, 0.5, 1),
    ("gqa4x1_s300x450_d64_noncausal", 2, 4, 1, 300, 450, 64, None, 0),
]


def test_noalloc_equals_fused_call_twice_in_a_row_then_smaller():
    L = lib()
    cl = L.load()
    dev = torch.device("cuda:0")
    data = []
    for name, B, Hq, Hkv, S_q, S_k, D, p, causal in SEQ:
        q, k, v, m = inputs(len(name), B, Hq, Hkv, S_q, S_k, D, p, dev)
        data.append((name, q, k, v, m, causal))
    outs = []
    say("[noalloc] calls back to back: large, large again, then smaller ones")
    order = [0, 0, 1, 2, 1]
    for i in order:
        name, q, k, v, m, causal = data[i]
        o = torch.full(tuple(q.shape), float("nan"), device=dev)
        call(cl.steel_attn_fwd_noalloc, q, k, v, m, o, causal)
        outs.append(o)
    torch.cuda.synchronize()
    for j, i in enumerate(order):
        name, q, k, v, m, causal = data[i]
        ref = torch.full(tuple(q.shape), float("nan"), device=dev)
        call(cl.steel_attn_fwd, q, k, v, m, ref, causal)
        torch.cuda.synchronize()
        assert torch.all(torch.isfinite(outs[j])).item(), f"call {j} ({name}): unwritten output"
        assert torch.equal(outs[j], ref), f"call {j} ({name}) differs from steel_attn_fwd"
        say(f"  call {j} ({name}): bitwise equal to steel_attn_fwd")


def test_noalloc_rejects_problems_beyond_the_array():
    L = lib()
    cl = L.load()
    dev = torch.device("cuda:0")
    q = torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16, device=dev)
    out = torch.full((1, 1, 64, 64), 7.0, device=dev)
    # 32 heads at S = 65536: 16384 rows x 1024 key blocks, a 64 MiB list
    st = cl.steel_attn_fwd_noalloc(q.data_ptr(), q.data_ptr(), q.data_ptr(), None, out.data_ptr(),
                                   1, 32, 8, 65536, 65536, 64, 64, 0.125, 1,
                                   torch.cuda.current_stream().cuda_stream)
    assert st == L.STEEL_ERR_UNSUPPORTED and "noalloc" in L.last_error()
    torch.cuda.synchronize()
    assert torch.all(out == 7.0).item()
