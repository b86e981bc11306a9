"""The C ABI on the CPU: the library builds, loads, exports every symbol the
header declares, and rejects invalid arguments before any HIP call (no GPU
needed: nothing is dereferenced or enqueued on those paths)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_09385_amd as steel
from paper_2607_09385_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "steel.h")

FAKE = 0x100000  # 16-byte aligned, never dereferenced on the checked paths


BENCH_HEADER = os.path.join(ROOT, "include", "steel_bench.h")


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(steel_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    names = declared_functions()
    assert {"steel_attn_fwd", "steel_block_index", "steel_last_error", "steel_version"} <= set(names)
    for name in names + declared_functions(BENCH_HEADER):
        assert hasattr(lib, name), f"{name} declared in include/ but not exported"


def test_mfma_peak_rejects_invalid_before_launch():
    lib = _lib.load()
    assert lib.steel_mfma_peak(None, 10, 256, 4, FAKE, FAKE, None) == 1
    assert lib.steel_mfma_peak(FAKE, 0, 256, 4, FAKE, FAKE, None) == 1
    assert lib.steel_mfma_peak(FAKE, 10, 256, 17, FAKE, FAKE, None) == 1


def test_lds_and_copy_rate_reject_invalid_before_launch():
    lib = _lib.load()
    assert lib.steel_mix_rate(0, 0, FAKE, 10, FAKE, 10, 256, FAKE, FAKE, None) == 1   # no role
    assert lib.steel_mix_rate(3, 2, FAKE, 10, FAKE, 10, 256, FAKE, FAKE, None) == 1   # bad vop
    assert lib.steel_mix_rate(1, 0, None, 10, None, 0, 256, FAKE, FAKE, None) == 1    # no operands
    assert lib.steel_mix_rate(2, 0, None, 0, None, 10, 256, FAKE, FAKE, None) == 1    # no seed
    assert lib.steel_mix_rate(3, 1, FAKE, 10, FAKE, 10, 0, FAKE, FAKE, None) == 1     # empty grid
    assert lib.steel_lds_rate(3, 10, 256, 4, FAKE, FAKE, None) == 1
    assert lib.steel_lds_rate(0, 0, 256, 4, FAKE, FAKE, None) == 1
    assert lib.steel_lds_rate(0, 10, 256, 17, FAKE, FAKE, None) == 1
    assert lib.steel_lds_rate(0, 10, 256, 4, None, FAKE, None) == 1
    assert lib.steel_copy_rate(FAKE, 1 << 20, 10, 256, 3, FAKE, FAKE, None) == 1   # not a power of 2
    assert lib.steel_copy_rate(FAKE, 1 << 18, 10, 256, 4, FAKE, FAKE, None) == 1   # source too small
    assert lib.steel_copy_rate(FAKE + 8, 1 << 20, 10, 256, 4, FAKE, FAKE, None) == 1  # misaligned
    assert lib.steel_copy_rate(None, 1 << 20, 10, 256, 4, FAKE, FAKE, None) == 1


def test_version_and_empty_error():
    assert "gfx950" in steel.version()


def attn(**kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, mask=None, out=FAKE, B=1, Hq=4, Hkv=2, S_q=128, S_k=128,
                D=64, blk=64, scale=0.125, causal=1, stream=None)
    args.update(kw)
    lib = _lib.load()
    st = lib.steel_attn_fwd(args["q"], args["k"], args["v"], args["mask"], args["out"],
                            args["B"], args["Hq"], args["Hkv"], args["S_q"], args["S_k"],
                            args["D"], args["blk"], args["scale"], args["causal"], args["stream"])
    return st, _lib.last_error()


@pytest.mark.parametrize("kw,code,text", [
    (dict(q=None), 1, "non-NULL"),
    (dict(out=None), 1, "non-NULL"),
    (dict(k=FAKE + 8), 1, "aligned"),
    (dict(out=FAKE + 4), 1, "aligned"),
    (dict(Hq=3, Hkv=2), 1, "multiple"),
    (dict(B=0), 1, ">= 1"),
    (dict(S_q=0), 1, ">= 1"),
    (dict(S_k=-5), 1, ">= 1"),
    (dict(scale=float("nan")), 1, "scale"),
    (dict(scale=float("inf")), 1, "scale"),
    (dict(scale=0.0), 1, "scale"),
    (dict(scale=-0.1), 1, "scale"),
    (dict(causal=2), 1, "causal"),
    (dict(D=96), 2, "D=96"),
    (dict(D=256), 2, "D=256"),
    (dict(blk=128), 2, "blk=128"),
    (dict(B=1 << 20, Hq=1 << 10, Hkv=1, S_q=1 << 20), 2, "too large"),
])
def test_invalid_arguments_rejected(kw, code, text):
    st, msg = attn(**kw)
    assert st == code
    assert text in msg


def test_error_text_is_thread_local_and_cleared():
    import threading
    st, msg = attn(D=96)
    assert st == 2 and "D=96" in msg
    seen = []
    t = threading.Thread(target=lambda: seen.append(_lib.last_error()))
    t.start(); t.join()
    assert seen == [""]
    attn(Hq=3, Hkv=2)
    assert "multiple" in _lib.last_error()


def test_block_index_rejects_invalid():
    lib = _lib.load()
    st = lib.steel_block_index(None, 1, 1, 64, 64, 64, 1, None, FAKE, FAKE, None)
    assert st == 1 and "non-NULL" in _lib.last_error()
    st = lib.steel_block_index(None, 1, 1, 64, 64, 32, 1, FAKE, FAKE, FAKE, None)
    assert st == 2 and "blk" in _lib.last_error()
    st = lib.steel_block_index(None, 1, 1, 64, 0, 64, 1, FAKE, FAKE, FAKE, None)
    assert st == 1


def test_python_binding_checks(monkeypatch):
    torch = pytest.importorskip("torch")
    q = torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        steel.attn_fwd(q, q, q)
    with pytest.raises(TypeError):
        steel.attn_fwd(None, q, q)


def test_valid_call_without_gpu_reports_hip_error():
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a GPU is present; covered by the GPU tests")
    st, msg = attn()
    assert st == 3 and "HIP" in msg


def test_workspace_bytes_and_plan_run_checks():
    lib = _lib.load()
    n = lib.steel_attn_workspace_bytes(1, 32, 8, 16384, 16384, 64)
    assert n > 256 * 256 * 8 * 4            # holds at least the live list capacity
    assert lib.steel_attn_workspace_bytes(1, 3, 2, 64, 64, 64) == 0
    assert "multiple" in _lib.last_error()
    # plan: NULL / misaligned / short workspace, all before any HIP call
    st = lib.steel_attn_plan(None, 1, 4, 2, 128, 128, 64, 1, None, n, None)
    assert st == 1 and "workspace" in _lib.last_error()
    st = lib.steel_attn_plan(None, 1, 4, 2, 128, 128, 64, 1, FAKE + 16, n, None)
    assert st == 1 and "256-byte" in _lib.last_error()
    need = lib.steel_attn_workspace_bytes(1, 4, 2, 128, 128, 64)
    st = lib.steel_attn_plan(None, 1, 4, 2, 128, 128, 64, 1, FAKE, need - 1, None)
    assert st == 1 and "smaller" in _lib.last_error()
    st = lib.steel_attn_run(FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 128, 128, 96, 64, 0.1, 1, FAKE, need,
                            None)
    assert st == 2 and "D=96" in _lib.last_error()
    st = lib.steel_attn_run(FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 0.1, 1, FAKE, 16,
                            None)
    assert st == 1 and "smaller" in _lib.last_error()


def test_window_forms_reject_invalid_window():
    lib = _lib.load()
    need = lib.steel_attn_workspace_bytes(1, 4, 2, 128, 128, 64)
    st = lib.steel_attn_plan_window(1, 4, 2, 128, 128, 64, 1, 0, 1, FAKE, need, None)
    assert st == 1 and "window_blocks" in _lib.last_error()
    st = lib.steel_attn_plan_window(1, 4, 2, 128, 128, 64, 1, 2, -1, FAKE, need, None)
    assert st == 1 and "sink_blocks" in _lib.last_error()
    st = lib.steel_attn_plan_window(1, 4, 2, 128, 128, 64, 1, 2, 1, FAKE, need - 1, None)
    assert st == 1 and "smaller" in _lib.last_error()
    st = lib.steel_attn_fwd_window(FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 0.125, 1,
                                   0, 0, None)
    assert st == 1 and "window_blocks" in _lib.last_error()
    st = lib.steel_attn_fwd_window(FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 128, 128, 96, 64, 0.125, 1,
                                   2, 0, None)
    assert st == 2 and "D=96" in _lib.last_error()


def test_topk_block_mask_rejects_invalid():
    lib = _lib.load()
    st = lib.steel_topk_block_mask(FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 1, 1, 10, None, None)
    assert st == 1 and "non-NULL" in _lib.last_error()
    st = lib.steel_topk_block_mask(FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 1, 0, 10, FAKE, None)
    assert st == 1 and "keep fraction" in _lib.last_error()
    st = lib.steel_topk_block_mask(FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 1, 11, 10, FAKE, None)
    assert st == 1 and "keep fraction" in _lib.last_error()
    st = lib.steel_topk_block_mask(FAKE, FAKE, 1, 4, 2, 128, 128, 80, 64, 1, 1, 10, FAKE, None)
    assert st == 2 and "D=80" in _lib.last_error()
    st = lib.steel_topk_block_mask(FAKE, FAKE, 1, 4, 2, 128, 64 * 4097, 64, 64, 1, 1, 10, FAKE,
                                   None)
    assert st == 2 and "4096" in _lib.last_error()
    st = lib.steel_topk_block_mask(FAKE, FAKE, 1, 3, 2, 128, 128, 64, 64, 1, 1, 10, FAKE, None)
    assert st == 1 and "multiple" in _lib.last_error()


def test_lse_and_merge_entry_points_reject_invalid():
    lib = _lib.load()
    st = lib.steel_attn_fwd_ex(FAKE, FAKE, FAKE, None, FAKE, FAKE, 1, 4, 2, 128, 128, 96, 64, 0.1, 1,
                               0, 0, None)
    assert st == 2 and "D=96" in _lib.last_error()
    st = lib.steel_attn_fwd_ex(FAKE, FAKE, FAKE, None, None, FAKE, 1, 4, 2, 128, 128, 64, 64, 0.1, 1,
                               0, 0, None)
    assert st == 1 and "non-NULL" in _lib.last_error()
    st = lib.steel_attn_fwd_ex(FAKE, FAKE, FAKE, None, FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 0.1, 1,
                               0, 8, None)
    assert st == 1 and "flags" in _lib.last_error()
    st = lib.steel_attn_fwd_ex(FAKE, FAKE, FAKE, None, FAKE, FAKE, 1, 4, 2, 128, 128, 64, 64, 0.1, 1,
                               0, -1, None)
    assert st == 1 and "flags" in _lib.last_error()
    st = lib.steel_attn_merge(FAKE, FAKE, 0, 10, 64, FAKE, None, None)
    assert st == 1 and "n_parts" in _lib.last_error()
    st = lib.steel_attn_merge(FAKE, FAKE, 2, 10, 66, FAKE, None, None)
    assert st == 1 and "multiple of 4" in _lib.last_error()
    st = lib.steel_attn_merge(None, FAKE, 2, 10, 64, FAKE, None, None)
    assert st == 1 and "non-NULL" in _lib.last_error()
    st = lib.steel_attn_merge(FAKE + 4, FAKE, 2, 10, 64, FAKE, None, None)
    assert st == 1 and "aligned" in _lib.last_error()


def test_output_buffer_validation():
    """The binding's check of caller-supplied fp32 outputs (used by attn_fwd,
    attn_fwd_window and Plan.run) runs on the host."""
    torch = pytest.importorskip("torch")
    from paper_2607_09385_amd import _check_out
    dev = torch.device("cpu")
    _check_out(torch.empty((1, 2, 64, 64)), (1, 2, 64, 64), dev)
    with pytest.raises(ValueError, match="contiguous float32"):
        _check_out(torch.empty((1, 2, 63, 64)), (1, 2, 64, 64), dev)
    with pytest.raises(ValueError, match="contiguous float32"):
        _check_out(torch.empty((1, 2, 64, 64), dtype=torch.bfloat16), (1, 2, 64, 64), dev)
    with pytest.raises(ValueError, match="contiguous float32"):
        _check_out(torch.empty((1, 2, 64, 64)).transpose(2, 3), (1, 2, 64, 64), dev)
    with pytest.raises(ValueError, match="device"):
        _check_out(torch.empty((1, 2, 64, 64)), (1, 2, 64, 64), torch.device("cuda", 0))
    with pytest.raises(TypeError):
        _check_out(np.zeros((1, 2, 64, 64), dtype=np.float32), (1, 2, 64, 64), dev)


def test_noalloc_rejects_oversized_index_before_any_hip_call():
    lib = _lib.load()
    # 32 heads at S = 65536: the index needs 64 MiB, the fixed array holds 32
    st = lib.steel_attn_fwd_noalloc(FAKE, FAKE, FAKE, None, FAKE, 1, 32, 8, 65536, 65536, 64, 64,
                                    0.125, 1, None)
    assert st == 2 and "noalloc" in _lib.last_error()
    need = lib.steel_attn_workspace_bytes(1, 32, 8, 65536, 65536, 64)
    assert need > 32 << 20
    # the largest named index fits
    assert lib.steel_attn_workspace_bytes(1, 24, 24, 32768, 32768, 64) <= 32 << 20
    st = lib.steel_attn_fwd_noalloc(FAKE, FAKE, FAKE, None, FAKE, 1, 4, 2, 128, 128, 96, 64,
                                    0.125, 1, None)
    assert st == 2 and "D=96" in _lib.last_error()
