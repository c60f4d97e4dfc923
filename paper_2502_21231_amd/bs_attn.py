"""Python binding of libbs_attn.so (argument marshalling only).

Each function has the name of the C entry point it calls and takes torch
tensors on the GPU.  Every step of the computation runs in the library's HIP
kernels; torch only allocates device memory (outputs, workspace) and supplies
the current stream.  If the library has not been built this module raises
instead of computing anything another way.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbs_attn.so")

BS_OK, BS_ERR_INVALID_ARG, BS_ERR_UNSUPPORTED, BS_ERR_WORKSPACE, BS_ERR_HIP, BS_ERR_DEVICE_STATUS = range(6)
BS_F32, BS_BF16 = 0, 1
(BS_OP_VARLEN_FWD, BS_OP_VARLEN_BWD, BS_OP_CHUNK_FWD, BS_OP_CHUNK_BWD, BS_OP_PACKED_CHUNK_FWD,
 BS_OP_PACKED_CHUNK_BWD) = range(6)

EXPORTS = (
    "bs_attn_workspace_size", "bs_attn_varlen_fwd", "bs_attn_varlen_bwd", "bs_attn_chunk_fwd",
    "bs_attn_chunk_bwd", "bs_attn_packed_chunk_fwd", "bs_attn_packed_chunk_bwd",
    "bs_attn_chunk_fwd_merge", "bs_attn_packed_chunk_fwd_merge", "bs_copy_async",
    "bs_softmax_xent",
    "bs_dq_finalize", "bs_lse_merge", "bs_read_device_status",
    "bs_attn_plan_export", "bs_set_profiling", "bs_profile_read", "bs_last_error",
    "bs_attn_varlen_fwd_noalloc",
)
BS_NOALLOC_SCRATCH_BYTES = 4 << 20  # the per-device plan scratch of bs_attn_varlen_fwd_noalloc
(BS_KERNEL_PLAN, BS_KERNEL_FWD, BS_KERNEL_PREPROCESS, BS_KERNEL_BWD_DQ, BS_KERNEL_BWD_DKDV,
 BS_KERNEL_FINALIZE, BS_KERNEL_MERGE, BS_KERNEL_XENT) = range(8)


class BsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"bs_attn status {status}: {message}")
        self.status = status


class bs_dims(ctypes.Structure):
    _fields_ = [("total_q", ctypes.c_int64), ("total_k", ctypes.c_int64), ("hq", ctypes.c_int32),
                ("hkv", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


_LIB = None
_P = ctypes.c_void_p
_I32, _I64, _F, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
_DIMS = ctypes.POINTER(bs_dims)


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libbs_attn.so and declares the signatures of every export."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2502_21231_amd.build`")
    lib = ctypes.CDLL(path)
    sig = {
        "bs_attn_workspace_size": (_SZ, [ctypes.c_int, _DIMS, _I32, _I32]),
        "bs_attn_varlen_fwd": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _I32, _I32, ctypes.c_int, _F,
                                              _P, _P, _P, _SZ, _P]),
        "bs_attn_varlen_fwd_noalloc": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _I32, _I32,
                                                      ctypes.c_int, _F, _P, _P, _P]),
        "bs_attn_varlen_bwd": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _I32,
                                              ctypes.c_int, _F, _P, _P, _P, _P, _SZ, _P]),
        "bs_attn_chunk_fwd": (ctypes.c_int, [_DIMS, _P, _P, _P, _I64, _I64, ctypes.c_int, _F, _P, _P,
                                             _P, _SZ, _P]),
        "bs_attn_chunk_bwd": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _P, _I64, _I64, ctypes.c_int,
                                             _F, _P, _P, _P, ctypes.c_int, _P, _SZ, _P]),
        "bs_attn_packed_chunk_fwd": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _P, _P, _I32, _I32,
                                                    ctypes.c_int, _F, _P, _P, _P, _SZ, _P]),
        "bs_attn_packed_chunk_bwd": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                                    _I32, _I32, ctypes.c_int, _F, _P, _P, _P,
                                                    ctypes.c_int, _P, _SZ, _P]),
        "bs_attn_chunk_fwd_merge": (ctypes.c_int, [_DIMS, _P, _P, _P, _I64, _I64, ctypes.c_int, _F,
                                                   _P, _P, ctypes.c_int, _P, _P, _SZ, _P]),
        "bs_attn_packed_chunk_fwd_merge": (ctypes.c_int, [_DIMS, _P, _P, _P, _P, _P, _P, _P, _I32,
                                                          _I32, ctypes.c_int, _F, _P, _P,
                                                          ctypes.c_int, _P, _P, _SZ, _P]),
        "bs_dq_finalize": (ctypes.c_int, [_DIMS, _P, _P, _P]),
        "bs_lse_merge": (ctypes.c_int, [_DIMS, _P, _P, _I32, _P, _P, _P]),
        "bs_copy_async": (ctypes.c_int, [_P, _P, _SZ, _P]),
        "bs_softmax_xent": (ctypes.c_int, [_I64, _I64, ctypes.c_int, _P, _P, _I64, _F, _P, _P, _P, _P]),
        "bs_read_device_status": (ctypes.c_int, [_P, _P]),
        "bs_attn_plan_export": (ctypes.c_int, [ctypes.c_int, _DIMS, _P, _P, _I32, _I32, _I64, _I64,
                                               _P, _P, ctypes.c_int, _P, _SZ, _P, _SZ,
                                               ctypes.POINTER(_SZ), ctypes.POINTER(_I32),
                                               ctypes.POINTER(_I32), _P]),
        "bs_set_profiling": (ctypes.c_int, [ctypes.c_int]),
        "bs_profile_read": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(_I64)]),
        "bs_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def bs_last_error() -> str:
    return load_library().bs_last_error().decode()


def _check(status: int) -> None:
    if status != BS_OK:
        raise BsError(status, bs_last_error())


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr() if t.numel() > 0 else None


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BS_BF16
    if t.dtype == torch.float32:
        return BS_F32
    raise TypeError(f"unsupported dtype {t.dtype}: bfloat16 or float32")


def _need(t: torch.Tensor, name: str, dtype=None, ndim=None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions (got {t.dim()})")


def make_dims(q: torch.Tensor, k: torch.Tensor | None) -> bs_dims:
    return bs_dims(q.shape[0], k.shape[0] if k is not None else 0, q.shape[1],
                   k.shape[1] if k is not None else 1, q.shape[2], _dtype_code(q))


def bs_attn_workspace_size(op: int, dims: bs_dims, num_seqs: int = 1, max_seqlen: int = 0) -> int:
    n = load_library().bs_attn_workspace_size(op, ctypes.byref(dims), num_seqs, max_seqlen)
    if n == 0:
        raise BsError(BS_ERR_INVALID_ARG, bs_last_error())
    return int(n)


def alloc_workspace(op: int, dims: bs_dims, device, num_seqs: int = 1, max_seqlen: int = 0):
    return torch.empty(bs_attn_workspace_size(op, dims, num_seqs, max_seqlen), dtype=torch.uint8,
                       device=device)


def _qkv(q, k, v):
    _need(q, "q", ndim=3)
    _need(k, "k", q.dtype, 3)
    _need(v, "v", q.dtype, 3)
    if k.shape != v.shape or k.shape[2] != q.shape[2]:
        raise ValueError(f"shape mismatch q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")


def _scale(scale, d):
    return float(scale) if scale is not None else 1.0 / math.sqrt(d)


def bs_attn_varlen_fwd(q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen: int, causal: bool = True,
                       scale: float | None = None, out=None, lse=None, workspace=None):
    """Packed varlen forward. q [T,Hq,d], k/v [Tk,Hkv,d], cu_seqlens int32 [B+1] on the GPU.
    Returns (out [T,Hq,d], lse float32 [Hq,T])."""
    _qkv(q, k, v)
    _need(cu_seqlens_q, "cu_seqlens_q", torch.int32, 1)
    _need(cu_seqlens_k, "cu_seqlens_k", torch.int32, 1)
    if cu_seqlens_q.numel() != cu_seqlens_k.numel():
        raise ValueError("cu_seqlens_q and cu_seqlens_k must have the same length")
    dims = make_dims(q, k)
    nseq = cu_seqlens_q.numel() - 1
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(q.shape[1], q.shape[0], dtype=torch.float32, device=q.device) if lse is None else lse
    _need(out, "out", q.dtype)
    _need(lse, "lse", torch.float32)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_VARLEN_FWD, dims, q.device, nseq, max_seqlen)
    _check(load_library().bs_attn_varlen_fwd(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), nseq,
        int(max_seqlen), int(bool(causal)), _scale(scale, q.shape[2]), _ptr(out), _ptr(lse),
        _ptr(workspace), workspace.numel(), _stream(q.device)))
    return out, lse


def bs_attn_varlen_fwd_noalloc(q, k, v, cu_seqlens_q, cu_seqlens_k, max_seqlen: int,
                               causal: bool = True, scale: float | None = None, out=None, lse=None):
    """bs_attn_varlen_fwd with no workspace: the library plans into its own per-device scratch
    array.  Pass preallocated out / lse to make the call allocate nothing at all."""
    _qkv(q, k, v)
    _need(cu_seqlens_q, "cu_seqlens_q", torch.int32, 1)
    _need(cu_seqlens_k, "cu_seqlens_k", torch.int32, 1)
    if cu_seqlens_q.numel() != cu_seqlens_k.numel():
        raise ValueError("cu_seqlens_q and cu_seqlens_k must have the same length")
    dims = make_dims(q, k)
    nseq = cu_seqlens_q.numel() - 1
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(q.shape[1], q.shape[0], dtype=torch.float32, device=q.device) if lse is None else lse
    _need(out, "out", q.dtype)
    _need(lse, "lse", torch.float32)
    _check(load_library().bs_attn_varlen_fwd_noalloc(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), nseq,
        int(max_seqlen), int(bool(causal)), _scale(scale, q.shape[2]), _ptr(out), _ptr(lse),
        _stream(q.device)))
    return out, lse


def bs_attn_varlen_bwd(q, k, v, out, lse, dout, cu_seqlens_q, cu_seqlens_k, max_seqlen: int,
                       causal: bool = True, scale: float | None = None, dq=None, dk=None, dv=None,
                       workspace=None):
    """Packed varlen backward; returns (dq, dk, dv)."""
    _qkv(q, k, v)
    _need(out, "out", q.dtype)
    _need(dout, "dout", q.dtype)
    _need(lse, "lse", torch.float32)
    _need(cu_seqlens_q, "cu_seqlens_q", torch.int32, 1)
    _need(cu_seqlens_k, "cu_seqlens_k", torch.int32, 1)
    dims = make_dims(q, k)
    nseq = cu_seqlens_q.numel() - 1
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    if workspace is None:
        workspace = alloc_workspace(BS_OP_VARLEN_BWD, dims, q.device, nseq, max_seqlen)
    _check(load_library().bs_attn_varlen_bwd(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(dout),
        _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), nseq, int(max_seqlen), int(bool(causal)),
        _scale(scale, q.shape[2]), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), workspace.numel(),
        _stream(q.device)))
    return dq, dk, dv


def bs_attn_chunk_fwd(q, k, v, q_pos_offset: int, k_pos_offset: int, causal: bool = True,
                      scale: float | None = None, out=None, lse=None, workspace=None):
    """One context-parallel step; returns the partial (out, lse)."""
    _qkv(q, k, v)
    dims = make_dims(q, k)
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(q.shape[1], q.shape[0], dtype=torch.float32, device=q.device) if lse is None else lse
    _need(out, "out", q.dtype)
    _need(lse, "lse", torch.float32)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_CHUNK_FWD, dims, q.device)
    _check(load_library().bs_attn_chunk_fwd(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), int(q_pos_offset), int(k_pos_offset),
        int(bool(causal)), _scale(scale, q.shape[2]), _ptr(out), _ptr(lse), _ptr(workspace),
        workspace.numel(), _stream(q.device)))
    return out, lse


def bs_attn_chunk_bwd(q, k, v, out_merged, lse_merged, dout, q_pos_offset: int, k_pos_offset: int,
                      causal: bool = True, scale: float | None = None, dq_accum=None, dk=None,
                      dv=None, kv_accumulate: bool = False, workspace=None):
    """Backward of one context-parallel step: adds into dq_accum (float32, caller-zeroed) and
    returns (dq_accum, dk, dv) of this KV shard.  With kv_accumulate, dk and dv are float32
    accumulators (caller-zeroed) that this step's contribution is added to."""
    _qkv(q, k, v)
    _need(out_merged, "out_merged", q.dtype)
    _need(dout, "dout", q.dtype)
    _need(lse_merged, "lse_merged", torch.float32)
    dims = make_dims(q, k)
    if dq_accum is None:
        dq_accum = torch.zeros(q.shape, dtype=torch.float32, device=q.device)
    _need(dq_accum, "dq_accum", torch.float32)
    kv_dtype = torch.float32 if kv_accumulate else k.dtype
    if dk is None:
        dk = torch.zeros(k.shape, dtype=kv_dtype, device=k.device)
    if dv is None:
        dv = torch.zeros(v.shape, dtype=kv_dtype, device=v.device)
    _need(dk, "dk", kv_dtype)
    _need(dv, "dv", kv_dtype)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_CHUNK_BWD, dims, q.device)
    _check(load_library().bs_attn_chunk_bwd(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(out_merged), _ptr(lse_merged),
        _ptr(dout), int(q_pos_offset), int(k_pos_offset), int(bool(causal)),
        _scale(scale, q.shape[2]), _ptr(dq_accum), _ptr(dk), _ptr(dv), int(bool(kv_accumulate)),
        _ptr(workspace), workspace.numel(), _stream(q.device)))
    return dq_accum, dk, dv


def _segments(cu_seqlens_q, cu_seqlens_k, q_pos, k_pos):
    _need(cu_seqlens_q, "cu_seqlens_q", torch.int32, 1)
    _need(cu_seqlens_k, "cu_seqlens_k", torch.int32, 1)
    _need(q_pos, "q_pos", torch.int64, 1)
    _need(k_pos, "k_pos", torch.int64, 1)
    nseq = cu_seqlens_q.numel() - 1
    if cu_seqlens_k.numel() != nseq + 1 or q_pos.numel() != nseq or k_pos.numel() != nseq:
        raise ValueError("cu_seqlens_q/k need num_seqs+1 entries and q_pos/k_pos num_seqs")
    return nseq


def bs_attn_packed_chunk_fwd(q, k, v, cu_seqlens_q, cu_seqlens_k, q_pos, k_pos, max_seqlen: int,
                             causal: bool = True, scale: float | None = None, out=None, lse=None,
                             workspace=None):
    """One packed context-parallel step over many segments: segment b pairs query rows
    cu_seqlens_q[b]..cu_seqlens_q[b+1]-1 at global positions q_pos[b]+i with key rows
    cu_seqlens_k[b].. at k_pos[b]+j (int32 / int64 device tensors).  Returns the partial
    (out, lse)."""
    _qkv(q, k, v)
    nseq = _segments(cu_seqlens_q, cu_seqlens_k, q_pos, k_pos)
    dims = make_dims(q, k)
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(q.shape[1], q.shape[0], dtype=torch.float32, device=q.device) if lse is None else lse
    _need(out, "out", q.dtype)
    _need(lse, "lse", torch.float32)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_PACKED_CHUNK_FWD, dims, q.device, nseq, max_seqlen)
    _check(load_library().bs_attn_packed_chunk_fwd(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k),
        _ptr(q_pos), _ptr(k_pos), nseq, int(max_seqlen), int(bool(causal)), _scale(scale, q.shape[2]),
        _ptr(out), _ptr(lse), _ptr(workspace), workspace.numel(), _stream(q.device)))
    return out, lse


def _running(q, o_run, lse_run, out):
    _need(o_run, "o_run", torch.float32)
    _need(lse_run, "lse_run", torch.float32)
    if o_run.shape != q.shape or lse_run.shape != (q.shape[1], q.shape[0]):
        raise ValueError("o_run must be [T, hq, d] and lse_run [hq, T] of the queries")
    if out is not None:
        _need(out, "out", q.dtype)
        if out.shape != q.shape:
            raise ValueError("out must be [T, hq, d]")


def bs_attn_chunk_fwd_merge(q, k, v, q_pos_offset: int, k_pos_offset: int, o_run, lse_run,
                            accumulate: bool, causal: bool = True, scale: float | None = None,
                            out=None, workspace=None):
    """One context-parallel step folded into the running (o_run float32 [T,Hq,d],
    lse_run float32 [Hq,T]): replaced (accumulate False) or combined by log-sum-exp
    weights.  With `out` the combined output is written there in q's dtype instead of
    into o_run.  Returns (o_run, lse_run, out)."""
    _qkv(q, k, v)
    _running(q, o_run, lse_run, out)
    dims = make_dims(q, k)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_CHUNK_FWD, dims, q.device)
    _check(load_library().bs_attn_chunk_fwd_merge(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), int(q_pos_offset), int(k_pos_offset),
        int(bool(causal)), _scale(scale, q.shape[2]), _ptr(o_run), _ptr(lse_run),
        int(bool(accumulate)), _ptr(out), _ptr(workspace), workspace.numel(), _stream(q.device)))
    return o_run, lse_run, out


def bs_attn_packed_chunk_fwd_merge(q, k, v, cu_seqlens_q, cu_seqlens_k, q_pos, k_pos,
                                   max_seqlen: int, o_run, lse_run, accumulate: bool,
                                   causal: bool = True, scale: float | None = None, out=None,
                                   workspace=None):
    """Packed context-parallel step (segments as in bs_attn_packed_chunk_fwd) folded into
    the running (o_run, lse_run) as in bs_attn_chunk_fwd_merge.  Returns (o_run, lse_run, out)."""
    _qkv(q, k, v)
    nseq = _segments(cu_seqlens_q, cu_seqlens_k, q_pos, k_pos)
    _running(q, o_run, lse_run, out)
    dims = make_dims(q, k)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_PACKED_CHUNK_FWD, dims, q.device, nseq, max_seqlen)
    _check(load_library().bs_attn_packed_chunk_fwd_merge(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k),
        _ptr(q_pos), _ptr(k_pos), nseq, int(max_seqlen), int(bool(causal)),
        _scale(scale, q.shape[2]), _ptr(o_run), _ptr(lse_run), int(bool(accumulate)), _ptr(out),
        _ptr(workspace), workspace.numel(), _stream(q.device)))
    return o_run, lse_run, out


def bs_attn_packed_chunk_bwd(q, k, v, out_merged, lse_merged, dout, cu_seqlens_q, cu_seqlens_k,
                             q_pos, k_pos, max_seqlen: int, causal: bool = True,
                             scale: float | None = None, dq_accum=None, dk=None, dv=None,
                             kv_accumulate: bool = False, workspace=None):
    """Backward of one packed context-parallel step, with the conventions of
    bs_attn_chunk_bwd; returns (dq_accum, dk, dv)."""
    _qkv(q, k, v)
    _need(out_merged, "out_merged", q.dtype)
    _need(dout, "dout", q.dtype)
    _need(lse_merged, "lse_merged", torch.float32)
    nseq = _segments(cu_seqlens_q, cu_seqlens_k, q_pos, k_pos)
    dims = make_dims(q, k)
    if dq_accum is None:
        dq_accum = torch.zeros(q.shape, dtype=torch.float32, device=q.device)
    _need(dq_accum, "dq_accum", torch.float32)
    kv_dtype = torch.float32 if kv_accumulate else k.dtype
    if dk is None:
        dk = torch.zeros(k.shape, dtype=kv_dtype, device=k.device)
    if dv is None:
        dv = torch.zeros(v.shape, dtype=kv_dtype, device=v.device)
    _need(dk, "dk", kv_dtype)
    _need(dv, "dv", kv_dtype)
    if workspace is None:
        workspace = alloc_workspace(BS_OP_PACKED_CHUNK_BWD, dims, q.device, nseq, max_seqlen)
    _check(load_library().bs_attn_packed_chunk_bwd(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(out_merged), _ptr(lse_merged),
        _ptr(dout), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), _ptr(q_pos), _ptr(k_pos), nseq,
        int(max_seqlen), int(bool(causal)), _scale(scale, q.shape[2]), _ptr(dq_accum), _ptr(dk),
        _ptr(dv), int(bool(kv_accumulate)), _ptr(workspace), workspace.numel(), _stream(q.device)))
    return dq_accum, dk, dv


def bs_dq_finalize(dq_accum, dq):
    """Rounds the float32 accumulator into dq (bf16 RNE or float32 copy)."""
    _need(dq_accum, "dq_accum", torch.float32, 3)
    _need(dq, "dq", None, 3)
    dims = bs_dims(dq.shape[0], 0, dq.shape[1], 1, dq.shape[2], _dtype_code(dq))
    _check(load_library().bs_dq_finalize(ctypes.byref(dims), _ptr(dq_accum), _ptr(dq),
                                         _stream(dq.device)))
    return dq


def bs_lse_merge(out_partials, lse_partials, out=None, lse=None):
    """Merges n partials: out_partials [n,T,Hq,d], lse_partials float32 [n,Hq,T]."""
    _need(out_partials, "out_partials", None, 4)
    _need(lse_partials, "lse_partials", torch.float32, 3)
    n, T, hq, d = out_partials.shape
    if tuple(lse_partials.shape) != (n, hq, T):
        raise ValueError(f"lse_partials must be [{n},{hq},{T}]")
    dims = bs_dims(T, 0, hq, 1, d, _dtype_code(out_partials))
    out = torch.empty(T, hq, d, dtype=out_partials.dtype, device=out_partials.device) if out is None else out
    lse = torch.empty(hq, T, dtype=torch.float32, device=out_partials.device) if lse is None else lse
    _check(load_library().bs_lse_merge(ctypes.byref(dims), _ptr(out_partials), _ptr(lse_partials), n,
                                       _ptr(out), _ptr(lse), _stream(out_partials.device)))
    return out, lse


def bs_copy_async(dst, src):
    """dst.copy_(src) on the current stream by the GPU's DMA engines (same dtype and size,
    both contiguous on the GPU); returns dst."""
    _need(dst, "dst")
    _need(src, "src")
    if dst.dtype != src.dtype or dst.numel() != src.numel():
        raise ValueError("dst and src must have the same dtype and number of elements")
    _check(load_library().bs_copy_async(_ptr(dst), _ptr(src), src.numel() * src.element_size(),
                                        _stream(src.device)))
    return dst


def bs_softmax_xent(logits, labels, ignore_index: int = -100, grad_scale: float = 1.0,
                    loss=None, lse=None, dlogits=None, with_grad: bool = True):
    """Per-token cross-entropy of logits [T, V] (bf16 or float32) against int64 labels [T], with
    the fused gradient grad_scale * (softmax - onehot).  dlogits: a new tensor (default), a
    given one, or `logits` itself for an in-place gradient; with_grad=False computes the loss
    only.  Returns (loss float32 [T], lse float32 [T], dlogits or None)."""
    _need(logits, "logits", ndim=2)
    _need(labels, "labels", torch.int64, 1)
    T, V = logits.shape
    if labels.shape[0] != T:
        raise ValueError("one label per row of logits")
    dev = logits.device
    loss = torch.empty(T, dtype=torch.float32, device=dev) if loss is None else loss
    lse = torch.empty(T, dtype=torch.float32, device=dev) if lse is None else lse
    _need(loss, "loss", torch.float32, 1)
    _need(lse, "lse", torch.float32, 1)
    if with_grad:
        dlogits = torch.empty_like(logits) if dlogits is None else dlogits
        _need(dlogits, "dlogits", logits.dtype, 2)
        if dlogits.shape != logits.shape:
            raise ValueError("dlogits must have the shape of logits")
    else:
        dlogits = None
    _check(load_library().bs_softmax_xent(T, V, _dtype_code(logits), _ptr(logits), _ptr(labels),
                                          int(ignore_index), float(grad_scale), _ptr(loss), _ptr(lse),
                                          _ptr(dlogits), _stream(dev)))
    return loss, lse, dlogits


def bs_read_device_status(workspace) -> int:
    """Synchronises and returns BS_OK or raises BsError with the device planner's status."""
    _check(load_library().bs_read_device_status(_ptr(workspace), _stream(workspace.device)))
    return BS_OK


def bs_attn_plan_export(op: int, dims: bs_dims, cu_seqlens_q=None, cu_seqlens_k=None, max_seqlen=0,
                        q_pos_offset=0, k_pos_offset=0, causal=True, device="cuda", q_pos=None,
                        k_pos=None):
    """Runs the device planner of `op` and returns (items [n,12] int32 numpy, tile_m, tile_n)."""
    import numpy as np
    nseq = cu_seqlens_q.numel() - 1 if cu_seqlens_q is not None else 1
    ws = alloc_workspace(op, dims, device, nseq, max_seqlen)
    cap = bs_attn_workspace_size(op, dims, nseq, max_seqlen) // 48 + 1
    host = np.zeros((cap, 12), dtype=np.int32)
    count, tm, tn = _SZ(0), _I32(0), _I32(0)
    _check(load_library().bs_attn_plan_export(
        op, ctypes.byref(dims), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), nseq, int(max_seqlen),
        int(q_pos_offset), int(k_pos_offset), _ptr(q_pos), _ptr(k_pos), int(bool(causal)),
        _ptr(ws), ws.numel(),
        host.ctypes.data, cap, ctypes.byref(count), ctypes.byref(tm), ctypes.byref(tn),
        _stream(ws.device)))
    return host[:count.value].copy(), tm.value, tn.value


def bs_set_profiling(enable: bool) -> None:
    """Turns the per-kernel event timing on or off (and clears what was recorded)."""
    _check(load_library().bs_set_profiling(int(bool(enable))))


def bs_profile_read(kind: int) -> tuple[float, int]:
    """(total milliseconds, launches) of kernel class `kind` since profiling was enabled."""
    ms, n = ctypes.c_double(0), _I64(0)
    _check(load_library().bs_profile_read(kind, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
