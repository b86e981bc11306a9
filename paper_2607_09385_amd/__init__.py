"""libsteel: sparsity-aware fused attention forward on MI355X (gfx950).

``attn_fwd`` computes softmax(Q K^T * scale + mask) V in one fused pass over
64x64 tiles, visiting only the key blocks that the block mask and the causal
structure leave live (the STEEL paper: Section II-A Eq. 1, Algorithm 1,
Section IV-A).  ``block_index`` exposes the compressed live-block list and the
heaviest-first work order the pass walks.

PyTorch provides device memory and the current stream; all arithmetic runs in
the library's HIP kernels.
"""
from __future__ import annotations

import math
from typing import Optional

from . import _lib
from ._lib import SteelError, load, last_error, version  # noqa: F401

BLK = 64
STEEL_OUT_BF16 = 1  # steel_attn_fwd_ex flags (include/steel.h)
STEEL_FP8 = 2
STEEL_FP8_PV = 4


def _torch():
    import torch
    return torch


def _stream_handle(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _check_bf16(name, t, ndim=4):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU device (got {t.device})")
    if t.dtype != torch.bfloat16:
        raise ValueError(f"{name} must be bfloat16 (got {t.dtype})")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims [B, H, S, D] (got {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_out(out, shape, device):
    """A caller-supplied fp32 output: the kernels write every element of a
    contiguous [B, Hq, S_q, D] float32 buffer on q's device, nothing less."""
    torch = _torch()
    if not isinstance(out, torch.Tensor):
        raise TypeError("out must be a torch.Tensor")
    if out.dtype != torch.float32 or tuple(out.shape) != tuple(shape) or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous float32 tensor {list(shape)} "
                         f"(got {out.dtype} {tuple(out.shape)})")
    if out.device != device:
        raise ValueError(f"out must be on q's device {device} (got {out.device})")


def attn_fwd(q, k, v, block_mask=None, *, scale: Optional[float] = None, causal: bool = True,
             blk: int = BLK, out=None, stream=None):
    """Fused masked attention forward.

    q: bf16 [B, Hq, S_q, D]; k, v: bf16 [B, Hkv, S_k, D]; block_mask: uint8
    [B, Hq, ceil(S_q/blk), ceil(S_k/blk)] or None (all live).  Returns fp32
    [B, Hq, S_q, D] (or fills ``out``).  Asynchronous on the current stream.
    """
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_bf16(name, t)
    B, Hq, S_q, D = q.shape
    Bk, Hkv, S_k, Dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or Bk != B or Dk != D:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    if q.device != k.device or q.device != v.device:
        raise ValueError("q, k and v must be on the same device")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    mask_ptr = None
    if block_mask is not None:
        nQB, nKB = -(-S_q // blk), -(-S_k // blk)
        if not isinstance(block_mask, torch.Tensor) or block_mask.dtype != torch.uint8:
            raise ValueError("block_mask must be a uint8 torch.Tensor")
        if tuple(block_mask.shape) != (B, Hq, nQB, nKB):
            raise ValueError(f"block_mask must be [{B}, {Hq}, {nQB}, {nKB}] (got {tuple(block_mask.shape)})")
        if block_mask.device != q.device or not block_mask.is_contiguous():
            raise ValueError("block_mask must be contiguous and on q's device")
        mask_ptr = block_mask.data_ptr()
    if out is None:
        out = torch.empty((B, Hq, S_q, D), dtype=torch.float32, device=q.device)
    else:
        _check_out(out, (B, Hq, S_q, D), q.device)
    with torch.cuda.device(q.device):
        st = _lib.load().steel_attn_fwd(
            q.data_ptr(), k.data_ptr(), v.data_ptr(), mask_ptr, out.data_ptr(),
            B, Hq, Hkv, S_q, S_k, D, blk, float(scale), 1 if causal else 0, _stream_handle(stream))
    _lib.check(st)
    return out


def attn_fwd_lse(q, k, v, block_mask=None, *, scale: Optional[float] = None, causal: bool = True,
                 causal_offset: Optional[int] = None, blk: int = BLK, out=None, lse=None,
                 out_dtype=None, fp8=False, stream=None):
    """``attn_fwd`` that also returns the row log-sum-exp (fp32 [B, Hq, S_q],
    natural log, -inf for rows with no visible key) and takes an explicit
    causal limit ``j <= i + causal_offset`` (default S_k - S_q).  ``out_dtype``
    torch.float32 (default) or torch.bfloat16 (the fp32 result rounded to
    nearest even).  ``fp8``: False (bf16 operands), "pv" (E4M3 operands for
    P V: STEEL_FP8_PV) or True / "all" (both products: STEEL_FP8)."""
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_bf16(name, t)
    B, Hq, S_q, D = q.shape
    Bk, Hkv, S_k, Dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or Bk != B or Dk != D:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    if q.device != k.device or q.device != v.device:
        raise ValueError("q, k and v must be on the same device")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if causal_offset is None:
        causal_offset = S_k - S_q
    mask_ptr = None
    if block_mask is not None:
        nQB, nKB = -(-S_q // blk), -(-S_k // blk)
        if block_mask.dtype != torch.uint8 or tuple(block_mask.shape) != (B, Hq, nQB, nKB) \
                or not block_mask.is_contiguous() or block_mask.device != q.device:
            raise ValueError(f"block_mask must be a contiguous uint8 [{B}, {Hq}, {nQB}, {nKB}] on q's device")
        mask_ptr = block_mask.data_ptr()
    if fp8 is False or fp8 is None:
        fp8_flag = 0
    elif fp8 is True or fp8 == "all":
        fp8_flag = STEEL_FP8
    elif fp8 == "pv":
        fp8_flag = STEEL_FP8_PV
    else:
        raise ValueError('fp8 must be False, "pv", True or "all"')
    odt = torch.float32 if out_dtype is None else out_dtype
    if odt not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
    if out is None:
        out = torch.empty((B, Hq, S_q, D), dtype=odt, device=q.device)
    if lse is None:
        lse = torch.empty((B, Hq, S_q), dtype=torch.float32, device=q.device)
    if out.dtype != odt or tuple(out.shape) != (B, Hq, S_q, D) or not out.is_contiguous() \
            or out.device != q.device:
        raise ValueError(f"out must be a contiguous {odt} tensor [B, Hq, S_q, D] on q's device")
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, Hq, S_q) or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 tensor [B, Hq, S_q] on q's device")
    with torch.cuda.device(q.device):
        st = _lib.load().steel_attn_fwd_ex(
            q.data_ptr(), k.data_ptr(), v.data_ptr(), mask_ptr, out.data_ptr(), lse.data_ptr(),
            B, Hq, Hkv, S_q, S_k, D, blk, float(scale), 1 if causal else 0, int(causal_offset),
            (STEEL_OUT_BF16 if odt == torch.bfloat16 else 0) | fp8_flag,
            _stream_handle(stream))
    _lib.check(st)
    return out, lse


def attn_merge(o_parts, lse_parts, *, out=None, lse_out=None, stream=None):
    """Combine partial results over disjoint key sets: o_parts fp32
    [n, ..., D] and lse_parts fp32 [n, ...] (stacked outputs of attn_fwd_lse)
    -> (out [..., D], lse [...])."""
    torch = _torch()
    if o_parts.dtype != torch.float32 or lse_parts.dtype != torch.float32:
        raise ValueError("o_parts and lse_parts must be float32")
    if not o_parts.is_contiguous() or not lse_parts.is_contiguous():
        raise ValueError("o_parts and lse_parts must be contiguous")
    if tuple(o_parts.shape[:-1]) != tuple(lse_parts.shape):
        raise ValueError("o_parts must be lse_parts' shape plus a last dimension D")
    n, D = o_parts.shape[0], o_parts.shape[-1]
    rows = lse_parts[0].numel()
    if out is None:
        out = torch.empty(o_parts.shape[1:], dtype=torch.float32, device=o_parts.device)
    if lse_out is None:
        lse_out = torch.empty(lse_parts.shape[1:], dtype=torch.float32, device=o_parts.device)
    with torch.cuda.device(o_parts.device):
        st = _lib.load().steel_attn_merge(o_parts.data_ptr(), lse_parts.data_ptr(), n, rows, D,
                                          out.data_ptr(), lse_out.data_ptr(), _stream_handle(stream))
    _lib.check(st)
    return out, lse_out


def attn_fwd_window(q, k, v, window_blocks: int, sink_blocks: int = 0, *,
                    scale: Optional[float] = None, causal: bool = True, blk: int = BLK, out=None,
                    stream=None):
    """``attn_fwd`` with the block mask generated from coordinates: block
    (qb, kb) is live iff qb - window_blocks < kb <= qb or kb < sink_blocks
    (then causal as usual); no mask tensor is read."""
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_bf16(name, t)
    B, Hq, S_q, D = q.shape
    Bk, Hkv, S_k, Dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or Bk != B or Dk != D:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    if q.device != k.device or q.device != v.device:
        raise ValueError("q, k and v must be on the same device")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty((B, Hq, S_q, D), dtype=torch.float32, device=q.device)
    else:
        _check_out(out, (B, Hq, S_q, D), q.device)
    with torch.cuda.device(q.device):
        st = _lib.load().steel_attn_fwd_window(
            q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, Hq, Hkv, S_q, S_k, D, blk,
            float(scale), 1 if causal else 0, int(window_blocks), int(sink_blocks),
            _stream_handle(stream))
    _lib.check(st)
    return out


def topk_block_mask(q, k, keep_num: int = 1, keep_den: int = 10, *, causal: bool = True,
                    blk: int = BLK, out=None, stream=None):
    """Block mask uint8 [B, Hq, nQB, nKB]: per query block the top
    ceil(keep_num/keep_den * candidates) key blocks by mean-pooled q.k score
    (ties to the smaller block), plus the diagonal block; computed on the GPU."""
    torch = _torch()
    _check_bf16("q", q)
    _check_bf16("k", k)
    B, Hq, S_q, D = q.shape
    Bk, Hkv, S_k, Dk = k.shape
    if Bk != B or Dk != D:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)}")
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    if out is None:
        out = torch.empty((B, Hq, nQB, nKB), dtype=torch.uint8, device=q.device)
    elif out.dtype != torch.uint8 or tuple(out.shape) != (B, Hq, nQB, nKB) or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous uint8 tensor [{B}, {Hq}, {nQB}, {nKB}]")
    with torch.cuda.device(q.device):
        st = _lib.load().steel_topk_block_mask(
            q.data_ptr(), k.data_ptr(), B, Hq, Hkv, S_q, S_k, D, blk, 1 if causal else 0,
            int(keep_num), int(keep_den), out.data_ptr(), _stream_handle(stream))
    _lib.check(st)
    return out


def block_index(block_mask, B: int, Hq: int, S_q: int, S_k: int, *, causal: bool = True,
                blk: int = BLK, device=None, stream=None):
    """Live-block list: returns (row_ptr int32 [R+1], col int32 [R*nKB]
    (valid up to row_ptr[-1]; bit 31 = partial), order int32 [R])."""
    torch = _torch()
    nQB, nKB = -(-S_q // blk), -(-S_k // blk)
    R = B * Hq * nQB
    if block_mask is not None:
        if block_mask.dtype != torch.uint8 or tuple(block_mask.shape) != (B, Hq, nQB, nKB):
            raise ValueError("block_mask must be uint8 [B, Hq, nQB, nKB]")
        if not block_mask.is_contiguous() or block_mask.device.type != "cuda":
            raise ValueError("block_mask must be a contiguous GPU tensor")
        device = block_mask.device
    device = device or torch.device("cuda")
    row_ptr = torch.empty(R + 1, dtype=torch.int32, device=device)
    col = torch.empty(max(R * nKB, 1), dtype=torch.int32, device=device)
    order = torch.empty(R, dtype=torch.int32, device=device)
    with torch.cuda.device(device):
        st = _lib.load().steel_block_index(
            None if block_mask is None else block_mask.data_ptr(), B, Hq, S_q, S_k, blk,
            1 if causal else 0, row_ptr.data_ptr(), col.data_ptr(), order.data_ptr(),
            _stream_handle(stream))
    _lib.check(st)
    return row_ptr, col, order


class Plan:
    """Live-block index built once for a mask and reused by ``run`` (the
    two-phase form of ``attn_fwd``).  ``window=(window_blocks, sink_blocks)``
    plans the structured mask of ``attn_fwd_window`` instead (block_mask must
    then be None)."""

    def __init__(self, block_mask, B: int, Hq: int, Hkv: int, S_q: int, S_k: int, *,
                 causal: bool = True, blk: int = BLK, device=None, stream=None, window=None):
        torch = _torch()
        lib = _lib.load()
        nbytes = lib.steel_attn_workspace_bytes(B, Hq, Hkv, S_q, S_k, blk)
        if nbytes == 0:
            raise SteelError(_lib.STEEL_ERR_INVALID_ARGUMENT, last_error())
        if block_mask is not None:
            nQB, nKB = -(-S_q // blk), -(-S_k // blk)
            if block_mask.dtype != torch.uint8 or tuple(block_mask.shape) != (B, Hq, nQB, nKB):
                raise ValueError("block_mask must be uint8 [B, Hq, nQB, nKB]")
            if not block_mask.is_contiguous() or block_mask.device.type != "cuda":
                raise ValueError("block_mask must be a contiguous GPU tensor")
            device = block_mask.device
        device = device or torch.device("cuda")
        self.shape = (B, Hq, Hkv, S_q, S_k)
        self.causal, self.blk, self.device = bool(causal), blk, device
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        with torch.cuda.device(device):
            if window is not None:
                if block_mask is not None:
                    raise ValueError("pass either block_mask or window, not both")
                wb, sb = window
                st = lib.steel_attn_plan_window(B, Hq, Hkv, S_q, S_k, blk, 1 if causal else 0,
                                                int(wb), int(sb), self.workspace.data_ptr(), nbytes,
                                                _stream_handle(stream))
            else:
                st = lib.steel_attn_plan(None if block_mask is None else block_mask.data_ptr(),
                                         B, Hq, Hkv, S_q, S_k, blk, 1 if causal else 0,
                                         self.workspace.data_ptr(), nbytes, _stream_handle(stream))
        _lib.check(st)

    def run(self, q, k, v, *, scale: Optional[float] = None, out=None, stream=None):
        torch = _torch()
        for name, t in (("q", q), ("k", k), ("v", v)):
            _check_bf16(name, t)
        B, Hq, Hkv, S_q, S_k = self.shape
        D = q.shape[-1]
        if tuple(q.shape) != (B, Hq, S_q, D) or tuple(k.shape) != (B, Hkv, S_k, D) \
                or tuple(v.shape) != tuple(k.shape):
            raise ValueError("q, k, v do not match the planned shape")
        if q.device != k.device or q.device != v.device or q.device != self.workspace.device:
            raise ValueError("q, k, v and the plan's workspace must be on the same device")
        if scale is None:
            scale = 1.0 / math.sqrt(D)
        if out is None:
            out = torch.empty((B, Hq, S_q, D), dtype=torch.float32, device=q.device)
        else:
            _check_out(out, (B, Hq, S_q, D), q.device)
        with torch.cuda.device(q.device):
            st = _lib.load().steel_attn_run(
                q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, Hq, Hkv, S_q, S_k,
                D, self.blk, float(scale), 1 if self.causal else 0, self.workspace.data_ptr(),
                self.workspace.numel(), _stream_handle(stream))
        _lib.check(st)
        return out
