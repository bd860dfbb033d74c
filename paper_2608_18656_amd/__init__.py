"""MI355X (gfx950) FlashAttention forward: MHA / GQA / MQA, prefill and decode.

Thin Python layer over the C ABI in include/fa.h (see ``_lib``); PyTorch is
used only for device memory and the current HIP stream.  Import is cheap: the
HIP library is loaded on first use and its absence raises (no CPU fallback).
"""
from __future__ import annotations

import math

__all__ = ["fwd", "fwd_splitkv", "fwd_splitkv_noalloc", "fwd_kvcache", "fwd_kvcache_paged", "fwd_unfused",
           "unfused_workspace_bytes", "q8_0_gemv", "FaError", "validate", "workspace_bytes", "release_workspace",
           "set_workspace", "version", "DTYPE_CODES"]


class FaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


def _torch():
    import torch

    return torch


def _codes():
    torch = _torch()
    return {torch.float16: 0, torch.bfloat16: 1, torch.float32: 2}


DTYPE_CODES = {"f16": 0, "bf16": 1, "f32": 2}


def _check(lib, st: int):
    if st != 0:
        raise FaError(st, lib.fa_status_string(st).decode())


def _prepare(q, k, v, out, lse, out_dtype, return_lse):
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous ([B, N, H, D] row-major)")
        if t.dim() != 4:
            raise ValueError(f"{name} must be 4-D [B, N, H, D]")
    if not (q.device == k.device == v.device):
        raise ValueError("q, k, v must be on the same device")
    if not (q.dtype == k.dtype == v.dtype) or q.dtype not in _codes():
        raise ValueError("q, k, v must share one dtype among float16, bfloat16, float32")
    B, Nq, Hq, D = q.shape
    Bk, Nk, Hkv, Dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or Bk != B or Dk != D:
        raise ValueError("k and v must be [B, Nk, Hkv, D] with q's B and D")
    odt = q.dtype if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((B, Nq, Hq, D), dtype=odt, device=q.device)
    elif (tuple(out.shape) != (B, Nq, Hq, D) or out.dtype != odt or not out.is_contiguous()
          or out.device != q.device):
        raise ValueError("out must be a contiguous [B, Nq, Hq, D] tensor of the output dtype")
    if lse is None and return_lse:
        lse = torch.empty((B, Hq, Nq), dtype=torch.float32, device=q.device)
    elif lse is not None and (tuple(lse.shape) != (B, Hq, Nq) or lse.dtype != torch.float32
                              or not lse.is_contiguous() or lse.device != q.device):
        raise ValueError("lse must be a contiguous float32 [B, Hq, Nq] tensor")
    return (B, Hq, Hkv, Nq, Nk, D), out, lse, odt


def _workspace_arg(workspace, device):
    """(pointer, bytes) of a caller-owned decode workspace tensor."""
    torch = _torch()
    if (workspace.dtype != torch.uint8 or not workspace.is_contiguous()
            or workspace.device != device):
        raise ValueError("workspace must be a contiguous uint8 tensor on q's device")
    return workspace.data_ptr(), workspace.numel()


def fwd(q, k, v, causal: bool = False, scale: float | None = None, out=None, lse=None,
        out_dtype=None, return_lse: bool = True, num_splits: int | None = None,
        heads_per_workgroup: int | None = None, workspace=None, slots_per_workgroup: int | None = None):
    """Attention forward o = softmax(scale * q k^T) v on the GPU.

    q [B, Nq, Hq, D], k and v [B, Nk, Hkv, D] (contiguous, same dtype and
    device); Hq must be a multiple of Hkv (query head h uses key/value head
    h // (Hq // Hkv)); ``causal`` uses the bottom-right mask (key j visible to
    query i iff j <= i + Nk - Nq).  ``scale`` defaults to 1/sqrt(D).
    ``out_dtype=torch.float32`` returns the kernel's fp32 result before the
    final rounding.  ``num_splits`` forces the decode split count (decode
    shapes only); ``heads_per_workgroup`` (1, 2 or 4) forces the prefill
    query-head packing (see fa_fwd_packed) and ``slots_per_workgroup`` (1, 2, 4
    or 8) the prefill workgroup layout (fa_fwd_slots).  ``workspace`` (a contiguous uint8
    GPU tensor of at least workspace_bytes(...) bytes) is this call's own
    decode workspace (fa_fwd_ws); otherwise the library-owned one of the
    current stream is used.  Returns (out, lse) with lse
    [B, Hq, Nq] float32 natural-log
    log-sum-exp (None if return_lse is False and no lse tensor was given).
    """
    from . import _lib

    lib = _lib.load()
    torch = _torch()
    (B, Hq, Hkv, Nq, Nk, D), out, lse, odt = _prepare(q, k, v, out, lse, out_dtype, return_lse)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    codes = _codes()
    stream = torch.cuda.current_stream(q.device).cuda_stream
    args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
            lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Nq, Nk, D,
            int(bool(causal)), float(scale), stream, codes[q.dtype], codes.get(odt, -1))
    with torch.cuda.device(q.device):
        if (heads_per_workgroup is not None and slots_per_workgroup is None
                and (num_splits is not None or workspace is not None)):
            raise ValueError("heads_per_workgroup excludes num_splits and workspace")
        if slots_per_workgroup is not None:
            if num_splits is not None or workspace is not None:
                raise ValueError("slots_per_workgroup excludes num_splits and workspace")
            st = lib.fa_fwd_slots(*args, int(slots_per_workgroup), int(heads_per_workgroup or 0))
        elif workspace is not None:
            st = lib.fa_fwd_ws(*args, int(num_splits or 0), *_workspace_arg(workspace, q.device))
        elif num_splits is not None:
            st = lib.fa_fwd_splitkv(*args, int(num_splits))
        elif heads_per_workgroup is not None:
            st = lib.fa_fwd_packed(*args, int(heads_per_workgroup))
        else:
            st = lib.fa_fwd(*args)
    _check(lib, st)
    return out, lse


def unfused_workspace_bytes(B: int, Hq: int, Nq: int, Nk: int) -> int:
    """Workspace bytes of fwd_unfused (fa_unfused_workspace_bytes)."""
    from . import _lib

    return int(_lib.load().fa_unfused_workspace_bytes(B, Hq, Nq, Nk))


def fwd_unfused(q, k, v, causal: bool = False, scale: float | None = None, out=None, lse=None,
                out_dtype=None, return_lse: bool = True, workspace=None):
    """Unfused self-attention (fa_fwd_unfused): the result of ``fwd`` with the
    score matrix materialised -- S = scale q k^T in fp32, P = softmax(S) in
    fp16, then O = P v, three kernels through HBM.  fp16 / bf16, D in {64,
    128}.  ``workspace``: a contiguous uint8 GPU tensor of at least
    unfused_workspace_bytes(B, Hq, Nq, Nk) bytes (allocated per call when
    None); afterwards it holds S [B, Hq, Nq, NkP] fp32 followed by P
    [B, Hq, Nq, NkP] fp16 (NkP = Nk rounded up to 64) on each row's visible
    keys.  Returns (out, lse) as ``fwd``.
    """
    from . import _lib

    lib = _lib.load()
    torch = _torch()
    (B, Hq, Hkv, Nq, Nk, D), out, lse, odt = _prepare(q, k, v, out, lse, out_dtype, return_lse)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    need = int(lib.fa_unfused_workspace_bytes(B, Hq, Nq, Nk))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    elif (workspace.dtype != torch.uint8 or not workspace.is_contiguous()
          or workspace.device != q.device):
        raise ValueError("workspace must be a contiguous uint8 tensor on q's device")
    codes = _codes()
    stream = torch.cuda.current_stream(q.device).cuda_stream
    with torch.cuda.device(q.device):
        st = lib.fa_fwd_unfused(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Nq, Nk,
                                D, int(bool(causal)), float(scale), stream, codes[q.dtype],
                                codes.get(odt, -1), workspace.data_ptr(), workspace.numel())
    _check(lib, st)
    return out, lse


def fwd_kvcache(q, k_cache, v_cache, seqlens_k, causal: bool = False, scale: float | None = None,
                out=None, lse=None, out_dtype=None, return_lse: bool = True, workspace=None):
    """Attention against K/V caches [B, Nk, Hkv, D] of which the first
    ``seqlens_k[b]`` rows are valid (``seqlens_k``: int32 [B] on the same
    device); q [B, Nq, Hq, D] holds each sequence's last Nq positions (decode
    for Nq = 1, chunked prefill otherwise).  Rows that see no key give 0 and
    lse -inf.  ``workspace``: this call's own decode workspace (uint8 GPU
    tensor; fa_fwd_kvcache_ws).  See fa_fwd_kvcache in include/fa.h."""
    from . import _lib

    lib = _lib.load()
    torch = _torch()
    (B, Hq, Hkv, Nq, Nk, D), out, lse, odt = _prepare(q, k_cache, v_cache, out, lse, out_dtype,
                                                      return_lse)
    if (not seqlens_k.is_cuda or seqlens_k.dtype != torch.int32 or tuple(seqlens_k.shape) != (B,)
            or not seqlens_k.is_contiguous() or seqlens_k.device != q.device):
        raise ValueError("seqlens_k must be a contiguous int32 [B] tensor on q's device")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    codes = _codes()
    stream = torch.cuda.current_stream(q.device).cuda_stream
    args = (q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), out.data_ptr(),
            lse.data_ptr() if lse is not None else None, seqlens_k.data_ptr(),
            B, Hq, Hkv, Nq, Nk, D, int(bool(causal)), float(scale), stream,
            codes[q.dtype], codes.get(odt, -1))
    with torch.cuda.device(q.device):
        if workspace is not None:
            st = lib.fa_fwd_kvcache_ws(*args, *_workspace_arg(workspace, q.device))
        else:
            st = lib.fa_fwd_kvcache(*args)
    _check(lib, st)
    return out, lse


def fwd_kvcache_paged(q, k_pages, v_pages, block_table, seqlens_k, causal: bool = False,
                      scale: float | None = None, out=None, lse=None, out_dtype=None,
                      return_lse: bool = True, workspace=None):
    """Attention against a paged K/V cache: ``k_pages``, ``v_pages``
    [num_pages, page_size, Hkv, D] (page_size a multiple of 64), ``block_table``
    int32 [B, max_pages] (page of each block of page_size keys of each
    sequence), ``seqlens_k`` int32 [B]; q [B, Nq, Hq, D] holds each sequence's
    last Nq positions.  ``workspace``: this call's own decode workspace
    (uint8 GPU tensor; fa_fwd_kvcache_paged_ws).  See fa_fwd_kvcache_paged in
    include/fa.h."""
    from . import _lib

    lib = _lib.load()
    torch = _torch()
    for name, t in (("q", q), ("k_pages", k_pages), ("v_pages", v_pages)):
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
            raise ValueError(f"{name} must be a contiguous 4-D GPU tensor")
    if not (q.device == k_pages.device == v_pages.device):
        raise ValueError("q and the page pools must be on the same device")
    if not (q.dtype == k_pages.dtype == v_pages.dtype) or q.dtype not in _codes():
        raise ValueError("q and the page pools must share one dtype")
    if tuple(k_pages.shape) != tuple(v_pages.shape):
        raise ValueError("k_pages and v_pages must have the same shape")
    B, Nq, Hq, D = q.shape
    num_pages, page_size, Hkv, Dk = k_pages.shape
    if Dk != D:
        raise ValueError("the page pools' head size differs from q's")
    for name, t, shp in (("block_table", block_table, None), ("seqlens_k", seqlens_k, (B,))):
        if (not t.is_cuda or t.dtype != torch.int32 or not t.is_contiguous() or t.device != q.device
                or (shp is not None and tuple(t.shape) != shp)):
            raise ValueError(f"{name} must be a contiguous int32 tensor on q's device")
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B, max_pages]")
    max_pages = block_table.shape[1]
    odt = q.dtype if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((B, Nq, Hq, D), dtype=odt, device=q.device)
    elif (tuple(out.shape) != (B, Nq, Hq, D) or out.dtype != odt or not out.is_contiguous()
          or out.device != q.device):
        raise ValueError("out must be a contiguous [B, Nq, Hq, D] tensor of the output dtype")
    if lse is None and return_lse:
        lse = torch.empty((B, Hq, Nq), dtype=torch.float32, device=q.device)
    elif lse is not None and (tuple(lse.shape) != (B, Hq, Nq) or lse.dtype != torch.float32
                              or not lse.is_contiguous() or lse.device != q.device):
        raise ValueError("lse must be a contiguous float32 [B, Hq, Nq] tensor")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    codes = _codes()
    stream = torch.cuda.current_stream(q.device).cuda_stream
    args = (q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(), out.data_ptr(),
            lse.data_ptr() if lse is not None else None, seqlens_k.data_ptr(), block_table.data_ptr(),
            B, Hq, Hkv, Nq, D, page_size, max_pages, num_pages, int(bool(causal)), float(scale),
            stream, codes[q.dtype], codes.get(odt, -1))
    with torch.cuda.device(q.device):
        if workspace is not None:
            st = lib.fa_fwd_kvcache_paged_ws(*args, *_workspace_arg(workspace, q.device))
        else:
            st = lib.fa_fwd_kvcache_paged(*args)
    _check(lib, st)
    return out, lse


def q8_0_gemv(w, x, out=None, out_dtype=None):
    """Q8_0 matrix-vector product y = W x (the decode-time linear layers).

    ``w``: uint8 GPU tensor holding M rows of K / 32 Q8_0 blocks of 34 bytes
    (binary16 scale, little-endian, then 32 int8 values), shaped [M, K/32, 34]
    or [M, K/32 * 34], contiguous.  ``x``: [K] float16, bfloat16 or float32 on
    the same device.  Returns y [M] in ``out_dtype`` (x's dtype, or float32).
    See fa_q8_0_gemv in include/fa.h."""
    from . import _lib

    lib = _lib.load()
    torch = _torch()
    if not (w.is_cuda and x.is_cuda) or w.device != x.device:
        raise ValueError("w and x must be GPU tensors on one device")
    if w.dtype != torch.uint8 or not w.is_contiguous() or w.dim() not in (2, 3):
        raise ValueError("w must be a contiguous uint8 [M, K/32, 34] or [M, K/32*34] tensor")
    if x.dim() != 1 or not x.is_contiguous() or x.dtype not in _codes():
        raise ValueError("x must be a contiguous 1-D float16, bfloat16 or float32 tensor")
    M, K = w.shape[0], x.shape[0]
    row_bytes = w[0].numel() if M > 0 else 0
    if (w.dim() == 3 and w.shape[2] != 34) or K % 32 != 0 or row_bytes != K // 32 * 34:
        raise ValueError("w must hold K/32 blocks of 34 bytes per row, K = len(x) a multiple of 32")
    odt = x.dtype if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((M,), dtype=odt, device=x.device)
    elif tuple(out.shape) != (M,) or out.dtype != odt or not out.is_contiguous() or out.device != x.device:
        raise ValueError("out must be a contiguous [M] tensor of the output dtype")
    codes = _codes()
    stream = torch.cuda.current_stream(x.device).cuda_stream
    with torch.cuda.device(x.device):
        st = lib.fa_q8_0_gemv(w.data_ptr(), x.data_ptr(), out.data_ptr(), M, K, codes[x.dtype],
                              codes.get(odt, -1), stream)
    _check(lib, st)
    return out


def fwd_splitkv_noalloc(q, k, v, num_splits: int = 0, causal: bool = False, scale: float | None = None,
                        out=None, lse=None, out_dtype=None, return_lse: bool = True):
    """fa_fwd_splitkv_noalloc: the decode forward with its split-KV partial
    results in the library's fixed device scratch (32 MiB per GPU) -- the C
    call allocates nothing (pass ``out``/``lse`` to keep this function from
    allocating them).  Calls that overlap on one GPU share the scratch and
    must be ordered."""
    from . import _lib

    lib = _lib.load()
    torch = _torch()
    (B, Hq, Hkv, Nq, Nk, D), out, lse, odt = _prepare(q, k, v, out, lse, out_dtype, return_lse)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    codes = _codes()
    stream = torch.cuda.current_stream(q.device).cuda_stream
    with torch.cuda.device(q.device):
        st = lib.fa_fwd_splitkv_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                        lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Nq, Nk,
                                        D, int(bool(causal)), float(scale), stream, codes[q.dtype],
                                        codes.get(odt, -1), int(num_splits))
    _check(lib, st)
    return out, lse


def fwd_splitkv(q, k, v, num_splits: int, **kw):
    """``fwd`` with an explicit decode split count (0 = default choice)."""
    return fwd(q, k, v, num_splits=num_splits, **kw)


def validate(q_ptr, k_ptr, v_ptr, o_ptr, lse_ptr, B, Hq, Hkv, Nq, Nk, D, causal, scale,
             in_dtype: str, out_dtype: str | None = None) -> int:
    """Status code of the library's host-side argument checks (no GPU use)."""
    from . import _lib

    lib = _lib.load()
    def code(x):
        return DTYPE_CODES[x] if x in DTYPE_CODES else int(x)

    in_code = code(in_dtype)
    out_code = in_code if out_dtype is None else code(out_dtype)
    return int(lib.fa_validate(q_ptr, k_ptr, v_ptr, o_ptr, lse_ptr, B, Hq, Hkv, Nq, Nk, D,
                               int(causal), float(scale), in_code, out_code))


def workspace_bytes(B, Hq, Hkv, Nq, Nk, D, in_dtype: str, num_splits: int = 0) -> int:
    from . import _lib

    return int(_lib.load().fa_workspace_bytes(B, Hq, Hkv, Nq, Nk, D, DTYPE_CODES[in_dtype],
                                              num_splits))


def release_workspace():
    from . import _lib

    lib = _lib.load()
    _check(lib, lib.fa_release_workspace())


_USER_WORKSPACE = {}   # device index -> caller tensor kept alive while set


def set_workspace(buf=None):
    """Use the device tensor ``buf`` (contiguous, on the current device) as
    the decode workspace of its device, or return to the library-owned one
    with ``None``; see fa_set_workspace in include/fa.h."""
    from . import _lib

    torch = _torch()
    lib = _lib.load()
    if buf is None:
        dev = torch.cuda.current_device()
        _check(lib, lib.fa_set_workspace(None, 0))
        _USER_WORKSPACE.pop(dev, None)
        return
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor")
    if buf.device.index != torch.cuda.current_device():
        raise ValueError("workspace must be on the current device")
    nbytes = buf.numel() * buf.element_size()
    _check(lib, lib.fa_set_workspace(buf.data_ptr() if nbytes else None, nbytes))
    _USER_WORKSPACE[buf.device.index] = buf


def version() -> tuple:
    from . import _lib

    v = _lib.load().fa_version()
    return (v >> 16, (v >> 8) & 0xFF, v & 0xFF)
