"""Python binding of the pdyattn C-ABI (include/pdyattn.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of libpdyattn.so.  torch is used for device memory (outputs and the
workspace are torch allocations) and for the current stream.  There is no
fallback: if the library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("PDYATTN_LIB", os.path.join(_HERE, "libpdyattn.so"))

PDY_OK = 0
PDY_ERR_INVALID_ARG = -1
PDY_ERR_UNSUPPORTED = -2
PDY_ERR_WORKSPACE = -3
PDY_ERR_HIP = -4

# exported symbols, in the order include/pdyattn.h declares them
SYMBOLS = ("attn_fwd_workspace_size", "attn_bwd_workspace_size", "attn_fwd", "attn_bwd",
           "attn_fwd_chunk_workspace_size", "attn_bwd_chunk_workspace_size", "attn_fwd_chunk",
           "attn_bwd_chunk", "attn_merge",
           "attn_validate_cu_seqlens", "attn_bwd_noalloc", "pdy_status_string", "pdy_last_error",
           "pdy_kernel_count", "pdy_kernel_name", "pdy_profile_start", "pdy_profile_stop")


class PdyError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: status {status}: {detail}")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libpdyattn.so (built in-tree by paper_2511_13198_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2511_13198_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    i32, f32, vp, sz = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
    L.attn_fwd_workspace_size.argtypes = [i32] * 6
    L.attn_fwd_workspace_size.restype = sz
    L.attn_bwd_workspace_size.argtypes = [i32] * 6
    L.attn_bwd_workspace_size.restype = sz
    L.attn_fwd.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, f32, vp, vp, vp, sz, vp]
    L.attn_fwd.restype = i32
    L.attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, f32,
                           vp, vp, vp, vp, sz, vp]
    L.attn_bwd.restype = i32
    L.attn_fwd_chunk_workspace_size.argtypes = [i32] * 5
    L.attn_fwd_chunk_workspace_size.restype = sz
    L.attn_bwd_chunk_workspace_size.argtypes = [i32] * 5
    L.attn_bwd_chunk_workspace_size.restype = sz
    L.attn_fwd_chunk.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32, f32, vp, vp,
                                 vp, sz, vp]
    L.attn_fwd_chunk.restype = i32
    L.attn_bwd_chunk.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32,
                                 f32, vp, vp, vp, i32, vp, sz, vp]
    L.attn_bwd_chunk.restype = i32
    L.attn_merge.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, vp]
    L.attn_merge.restype = i32
    L.attn_validate_cu_seqlens.argtypes = [vp, i32, i32, ctypes.POINTER(i32), vp]
    L.attn_validate_cu_seqlens.restype = i32
    L.attn_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32,
                                   f32, vp, vp, vp, vp]
    L.attn_bwd_noalloc.restype = i32
    L.pdy_status_string.argtypes = [i32]
    L.pdy_status_string.restype = ctypes.c_char_p
    L.pdy_last_error.argtypes = []
    L.pdy_last_error.restype = ctypes.c_char_p
    L.pdy_kernel_count.argtypes = []
    L.pdy_kernel_count.restype = i32
    L.pdy_kernel_name.argtypes = [i32]
    L.pdy_kernel_name.restype = ctypes.c_char_p
    L.pdy_profile_start.argtypes = []
    L.pdy_profile_start.restype = i32
    L.pdy_profile_stop.argtypes = [ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double), i32]
    L.pdy_profile_stop.restype = i32
    _lib = L
    return L


def _check(status: int, where: str):
    if status != PDY_OK:
        L = lib()
        raise PdyError(status, where,
                       f"{L.pdy_status_string(status).decode()} ({L.pdy_last_error().decode()})")


def profile_start():
    """Start bracketing every kernel this thread launches with HIP events."""
    _check(lib().pdy_profile_start(), "pdy_profile_start")


def profile_stop() -> dict:
    """Stop timing; returns {kernel name: (launches, total ms)} for kernels
    launched since profile_start (waits for their events)."""
    L = lib()
    n = L.pdy_kernel_count()
    launches = (ctypes.c_int32 * n)()
    total = (ctypes.c_double * n)()
    _check(L.pdy_profile_stop(launches, total, n), "pdy_profile_stop")
    return {L.pdy_kernel_name(i).decode(): (int(launches[i]), float(total[i]))
            for i in range(n) if launches[i] > 0}


def last_error() -> str:
    return lib().pdy_last_error().decode()


def _stream_handle(device) -> int:
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def fwd_workspace_size(total_tokens, num_seqs, max_seqlen, hq, hkv, d) -> int:
    return int(lib().attn_fwd_workspace_size(total_tokens, num_seqs, max_seqlen, hq, hkv, d))


def bwd_workspace_size(total_tokens, num_seqs, max_seqlen, hq, hkv, d) -> int:
    return int(lib().attn_bwd_workspace_size(total_tokens, num_seqs, max_seqlen, hq, hkv, d))


def validate_cu_seqlens(cu_seqlens, total_tokens: int) -> int:
    """Checks cu_seqlens on the host (synchronising) and returns the longest
    segment length."""
    out = ctypes.c_int32(0)
    st = lib().attn_validate_cu_seqlens(cu_seqlens.data_ptr(), cu_seqlens.numel() - 1,
                                        total_tokens, ctypes.byref(out),
                                        _stream_handle(cu_seqlens.device))
    _check(st, "attn_validate_cu_seqlens")
    return int(out.value)


def _check_tensor(t, name, dtype, ndim):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _ws(nbytes: int, device):
    import torch
    return torch.empty(max(256, nbytes), dtype=torch.uint8, device=device)


def attn_fwd(q, k, v, cu_seqlens, max_seqlen: Optional[int] = None, causal: bool = True,
             scale: Optional[float] = None, out=None, lse=None, workspace=None):
    """O [T, Hq, d] bf16 and LSE [Hq, T] fp32 (natural log) of Eq. (2) over
    the packed batch described by cu_seqlens (int32 [N+1], on the device)."""
    import torch
    _check_tensor(q, "q", torch.bfloat16, 3)
    _check_tensor(k, "k", torch.bfloat16, 3)
    _check_tensor(v, "v", torch.bfloat16, 3)
    _check_tensor(cu_seqlens, "cu_seqlens", torch.int32, 1)
    T, hq, d = q.shape
    hkv = k.shape[1]
    if tuple(k.shape) != (T, hkv, d) or tuple(v.shape) != (T, hkv, d):
        raise ValueError("k and v must be [T, Hkv, d] with q's T and d")
    if max_seqlen is None:
        max_seqlen = validate_cu_seqlens(cu_seqlens, T)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    n = cu_seqlens.numel() - 1
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((hq, T), dtype=torch.float32, device=q.device)
    need = fwd_workspace_size(T, n, max_seqlen, hq, hkv, d)
    if workspace is None:
        workspace = _ws(need, q.device)
    st = lib().attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cu_seqlens.data_ptr(), n, T,
                        int(max_seqlen), hq, hkv, d, int(bool(causal)), float(scale),
                        out.data_ptr(), lse.data_ptr(), workspace.data_ptr(),
                        workspace.numel() * workspace.element_size(),
                        _stream_handle(q.device))
    _check(st, "attn_fwd")
    return out, lse


def _bwd_args(q, k, v, o, lse, dout, cu_seqlens, max_seqlen, scale, dq, dk, dv):
    """Checked shapes and outputs of a backward call (outputs allocated by
    torch when not given)."""
    import torch
    for t, name in ((q, "q"), (k, "k"), (v, "v"), (o, "o"), (dout, "dout")):
        _check_tensor(t, name, torch.bfloat16, 3)
    _check_tensor(lse, "lse", torch.float32, 2)
    _check_tensor(cu_seqlens, "cu_seqlens", torch.int32, 1)
    T, hq, d = q.shape
    hkv = k.shape[1]
    if tuple(o.shape) != (T, hq, d) or tuple(dout.shape) != (T, hq, d):
        raise ValueError("o and dout must match q")
    if tuple(lse.shape) != (hq, T):
        raise ValueError("lse must be [Hq, T]")
    if max_seqlen is None:
        max_seqlen = validate_cu_seqlens(cu_seqlens, T)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if dq is None:
        dq = torch.empty((T, hq, d), dtype=torch.float32, device=q.device)
    if dk is None:
        dk = torch.empty((T, hkv, d), dtype=torch.float32, device=q.device)
    if dv is None:
        dv = torch.empty((T, hkv, d), dtype=torch.float32, device=q.device)
    for t, name, shape in ((dq, "dq", (T, hq, d)), (dk, "dk", (T, hkv, d)),
                           (dv, "dv", (T, hkv, d))):
        _check_tensor(t, name, torch.float32, 3)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} must be {list(shape)}")
    n = cu_seqlens.numel() - 1
    return T, hq, hkv, d, n, int(max_seqlen), float(scale), dq, dk, dv


def attn_bwd(q, k, v, o, lse, dout, cu_seqlens, max_seqlen: Optional[int] = None,
             causal: bool = True, scale: Optional[float] = None, dq=None, dk=None, dv=None,
             workspace=None) -> Tuple:
    """dQ [T, Hq, d], dK, dV [T, Hkv, d] (fp32) of sum(dout * O)."""
    T, hq, hkv, d, n, max_seqlen, scale, dq, dk, dv = _bwd_args(
        q, k, v, o, lse, dout, cu_seqlens, max_seqlen, scale, dq, dk, dv)
    need = bwd_workspace_size(T, n, max_seqlen, hq, hkv, d)
    if workspace is None:
        workspace = _ws(need, q.device)
    st = lib().attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                        dout.data_ptr(), cu_seqlens.data_ptr(), n, T, max_seqlen, hq, hkv, d,
                        int(bool(causal)), scale, dq.data_ptr(), dk.data_ptr(),
                        dv.data_ptr(), workspace.data_ptr(),
                        workspace.numel() * workspace.element_size(), _stream_handle(q.device))
    _check(st, "attn_bwd")
    return dq, dk, dv


def attn_bwd_noalloc(q, k, v, o, lse, dout, cu_seqlens, max_seqlen: Optional[int] = None,
                     causal: bool = True, scale: Optional[float] = None, dq=None, dk=None,
                     dv=None) -> Tuple:
    """attn_bwd without a workspace: the library takes its scratch from a
    static device array of fixed size (PdyError with PDY_ERR_WORKSPACE when
    the sizes need more).  With dq, dk, dv given and max_seqlen known, this
    call allocates nothing.  Calls that overlap on one GPU share that
    scratch and must not run concurrently."""
    T, hq, hkv, d, n, max_seqlen, scale, dq, dk, dv = _bwd_args(
        q, k, v, o, lse, dout, cu_seqlens, max_seqlen, scale, dq, dk, dv)
    st = lib().attn_bwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                lse.data_ptr(), dout.data_ptr(), cu_seqlens.data_ptr(), n, T,
                                max_seqlen, hq, hkv, d, int(bool(causal)), scale,
                                dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                _stream_handle(q.device))
    _check(st, "attn_bwd_noalloc")
    return dq, dk, dv


# ---------------------------------------------------------------------------
# One long sequence split into chunks (context parallelism)
# ---------------------------------------------------------------------------
def fwd_chunk_workspace_size(tq, tk, hq, hkv, d) -> int:
    return int(lib().attn_fwd_chunk_workspace_size(tq, tk, hq, hkv, d))


def bwd_chunk_workspace_size(tq, tk, hq, hkv, d) -> int:
    return int(lib().attn_bwd_chunk_workspace_size(tq, tk, hq, hkv, d))


def _ptr(t):
    return 0 if t is None else t.data_ptr()


def attn_fwd_chunk(q, k, v, q_offset: int, k_offset: int, causal: bool = True,
                   scale: Optional[float] = None, out=None, lse=None, workspace=None):
    """Partial O [Tq, Hq, d] bf16 and LSE [Hq, Tq] fp32 of the query chunk at
    positions q_offset.. over the key/value chunk at positions k_offset.."""
    import torch
    _check_tensor(q, "q", torch.bfloat16, 3)
    _check_tensor(k, "k", torch.bfloat16, 3)
    _check_tensor(v, "v", torch.bfloat16, 3)
    tq, hq, d = q.shape
    tk, hkv = k.shape[0], k.shape[1]
    if tuple(v.shape) != tuple(k.shape) or k.shape[2] != d:
        raise ValueError("k and v must be [Tk, Hkv, d] with q's d")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((hq, tq), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = _ws(fwd_chunk_workspace_size(tq, tk, hq, hkv, d), q.device)
    st = lib().attn_fwd_chunk(q.data_ptr(), _ptr(k) if tk else 0, _ptr(v) if tk else 0, tq, tk,
                              int(q_offset), int(k_offset), hq, hkv, d, int(bool(causal)),
                              float(scale), out.data_ptr(), lse.data_ptr(), workspace.data_ptr(),
                              workspace.numel() * workspace.element_size(),
                              _stream_handle(q.device))
    _check(st, "attn_fwd_chunk")
    return out, lse


def attn_bwd_chunk(q, k, v, o, lse, dout, q_offset: int, k_offset: int, causal: bool = True,
                   scale: Optional[float] = None, dq=None, dk=None, dv=None, workspace=None,
                   accumulate: bool = False):
    """This (query chunk, key chunk) pair's part of dQ [Tq, Hq, d] and dK, dV
    [Tk, Hkv, d] (fp32), given the final o and lse of the query rows; with
    accumulate=True it is added to the given dq, dk, dv."""
    import torch
    for t, name in ((q, "q"), (k, "k"), (v, "v"), (o, "o"), (dout, "dout")):
        _check_tensor(t, name, torch.bfloat16, 3)
    _check_tensor(lse, "lse", torch.float32, 2)
    tq, hq, d = q.shape
    tk, hkv = k.shape[0], k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    dev = q.device if tq else k.device
    if dq is None:
        dq = torch.empty((tq, hq, d), dtype=torch.float32, device=dev)
    if dk is None:
        dk = torch.empty((tk, hkv, d), dtype=torch.float32, device=dev)
    if dv is None:
        dv = torch.empty((tk, hkv, d), dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = _ws(bwd_chunk_workspace_size(tq, tk, hq, hkv, d), dev)
    st = lib().attn_bwd_chunk(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                              lse.data_ptr(), dout.data_ptr(), tq, tk, int(q_offset),
                              int(k_offset), hq, hkv, d, int(bool(causal)), float(scale),
                              dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), int(bool(accumulate)),
                              workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                              _stream_handle(dev))
    _check(st, "attn_bwd_chunk")
    return dq, dk, dv


def attn_merge(o_a, lse_a, o_b, lse_b, out=None, lse=None):
    """Combine two partial (O, LSE) of the same rows; out/lse may be o_a/lse_a."""
    import torch
    _check_tensor(o_a, "o_a", torch.bfloat16, 3)
    _check_tensor(o_b, "o_b", torch.bfloat16, 3)
    _check_tensor(lse_a, "lse_a", torch.float32, 2)
    _check_tensor(lse_b, "lse_b", torch.float32, 2)
    T, hq, d = o_a.shape
    if tuple(o_b.shape) != (T, hq, d) or tuple(lse_a.shape) != (hq, T) or \
            tuple(lse_b.shape) != (hq, T):
        raise ValueError("partials must share shapes [T, Hq, d] and [Hq, T]")
    if out is None:
        out = torch.empty_like(o_a)
    if lse is None:
        lse = torch.empty_like(lse_a)
    st = lib().attn_merge(o_a.data_ptr(), lse_a.data_ptr(), o_b.data_ptr(), lse_b.data_ptr(), T,
                          hq, d, out.data_ptr(), lse.data_ptr(), _stream_handle(o_a.device))
    _check(st, "attn_merge")
    return out, lse
