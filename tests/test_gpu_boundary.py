"""The two-phase boundary on the GPU: a plan run with other sizes than it was
made for leaves the output untouched (the kernels compare the plan's header
with their arguments: Section II-A's problem sizes, the causal structure and
the head packing), and the binding refuses output buffers the kernels could
overrun."""
import math
import sys

import numpy as np
import pytest
import torch

from workloads import small_qkv

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def steel():
    import paper_2607_09385_amd as s
    s.load()
    return s


def raw_run(plan, q, k, v, out, B, Hq, Hkv, S_q, S_k, causal):
    """steel_attn_run through the C ABI with explicit sizes (the binding would
    refuse the mismatch before the call)."""
    from paper_2607_09385_amd import _lib
    D = q.shape[-1]
    st = _lib.load().steel_attn_run(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, Hq, Hkv, S_q, S_k, D, 64,
        1.0 / math.sqrt(D), causal, plan.workspace.data_ptr(), plan.workspace.numel(),
        torch.cuda.current_stream().cuda_stream)
    _lib.check(st)


@pytest.mark.parametrize("plan_shape,run_shape,plan_causal,run_causal", [
    # same key-block count (64 blocks) but a ragged S_k: the last block would
    # not be treated as partial
    ((1, 8, 2, 4096, 4096), (1, 8, 2, 4033, 4033), 0, 0),
    # B and Hq swapped at the same row count R = B * Hq * nQB
    ((2, 4, 2, 256, 256), (1, 8, 2, 256, 256), 1, 1),
    # another Hkv with the same pack of 2 heads (G = 6 and G = 2)
    ((1, 12, 2, 512, 512), (1, 12, 6, 512, 512), 1, 1),
    # S_q and S_k both differ with the same block counts and the same S_k - S_q
    ((1, 4, 1, 500, 600), (1, 4, 1, 510, 610), 0, 0),
    # the causal flag
    ((1, 8, 2, 640, 640), (1, 8, 2, 640, 640), 0, 1),
], ids=["ragged_sk_same_nkb", "b_hq_swapped", "other_hkv_same_pack", "other_sizes_same_blocks", "causal_flag"])
def test_mismatched_run_leaves_out_untouched(plan_shape, run_shape, plan_causal, run_causal):
    s = steel()
    dev = torch.device("cuda:0")
    say(f"[boundary] plan {plan_shape} causal={plan_causal} run {run_shape} causal={run_causal}")
    plan = s.Plan(None, *plan_shape, causal=bool(plan_causal), device=dev)
    B, Hq, Hkv, S_q, S_k = run_shape
    q, k, v = small_qkv(3, B, Hq, Hkv, S_q, S_k, 128)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    out = torch.full((B, Hq, S_q, 128), 7.0, device=dev)
    raw_run(plan, qd, kd, vd, out, B, Hq, Hkv, S_q, S_k, run_causal)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0).item()
    # the matching run does write it
    plan_ok = s.Plan(None, *run_shape, causal=bool(run_causal), device=dev)
    raw_run(plan_ok, qd, kd, vd, out, B, Hq, Hkv, S_q, S_k, run_causal)
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(out)).item() and not torch.all(out == 7.0).item()


def test_plan_run_rejects_bad_out_buffers():
    s = steel()
    dev = torch.device("cuda:0")
    plan = s.Plan(None, 1, 4, 2, 256, 256, causal=True, device=dev)
    q, k, v = (t.to(dev) for t in small_qkv(4, 1, 4, 2, 256, 256, 64))
    bad = [torch.empty((1, 4, 255, 64), device=dev),                       # too short
           torch.empty((1, 4, 256, 64), dtype=torch.bfloat16, device=dev),  # wrong dtype
           torch.empty((1, 4, 64, 256), device=dev).transpose(2, 3),        # not contiguous
           torch.empty((1, 4, 256, 64))]                                     # host memory
    for out in bad:
        with pytest.raises(ValueError):
            plan.run(q, k, v, out=out)
    with pytest.raises(ValueError):
        plan.run(q, k, v[:, :, :128].contiguous())
    good = plan.run(q, k, v, out=torch.empty((1, 4, 256, 64), device=dev))
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(good)).item()
