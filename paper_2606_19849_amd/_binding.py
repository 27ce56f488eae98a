"""ctypes binding of libvico (include/vico.h): argument marshalling only.

Every computation runs in the HIP kernels of libvico.so.  torch supplies the
device buffers and the stream; it is imported before the library is loaded
so that the process holds a single HIP runtime.  If the library is not built
the calls raise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch  # noqa: F401  (load torch's HIP runtime first)

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libvico.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "vico.h")

VICO_DTYPE_BF16 = 0
VICO_DTYPE_F32 = 1
VICO_FULL_HISTORY = -1
VICO_SPLIT_BALANCED = -1

_i32, _i64, _f32, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p

_SIGNATURES = {
    "vico_kv_append": (_i32, [_vp, _vp, _i32, _vp, _vp, _i32, _i64, _i32, _i32, _vp]),
    "vico_chunk_prefill_attn": (_i32, [_vp, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _i64, _i64,
                                       _i32, _i32, _i32, _f32, _vp, _i32, _vp, _i32, _vp, _i64, _vp]),
    "vico_attn_plan": (_i32, [_i32, _i32, _i32, _i64, _i64, _i32, _i32, _i32, _i32,
                              ctypes.POINTER(_i32), ctypes.POINTER(_i64)]),
    "vico_attn_workspace_bytes": (_i64, [_i32, _i32, _i32, _i64, _i64, _i32, _i32, _i32, _i32]),
    "vico_status_str": (ctypes.c_char_p, [_i32]),
    "vico_last_hip_error": (_i32, []),
}

_lib = None


class VicoError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = load_library().vico_status_str(status).decode()
        if status == -6:
            msg += f" (hipError {load_library().vico_last_hip_error()})"
        super().__init__(f"{where}: {msg} [{status}]")


def load_library():
    """Load libvico.so once; raise ImportError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; build it with `python -m paper_2606_19849_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype, fn.argtypes = res, args
        _lib = lib
    return _lib


def header_functions():
    """Names of the functions declared in include/vico.h."""
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vico_\w+)\s*\(", src)))


def _ptr(t):
    if t is None or t.numel() == 0:
        return None
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _check(status: int, where: str):
    if status != 0:
        raise VicoError(status, where)


def _dev_bf16(name, t, ndim=3):
    if t is None:
        return
    if not (t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous() and t.dim() == ndim):
        raise ValueError(f"{name}: expected a contiguous {ndim}-d bfloat16 CUDA tensor, got "
                         f"{tuple(t.shape)} {t.dtype} on {t.device}")


def vico_kv_append(k_chunk, v_chunk, ring_k, ring_v, hist_len: int, stream=None) -> None:
    """ring[(hist_len + j) % R] <- chunk[j] for K and V (vico_kv_append)."""
    for n, t in (("k_chunk", k_chunk), ("v_chunk", v_chunk), ("ring_k", ring_k), ("ring_v", ring_v)):
        _dev_bf16(n, t)
    C, Hkv, D = k_chunk.shape
    st = load_library().vico_kv_append(_ptr(k_chunk), _ptr(v_chunk), C, _ptr(ring_k), _ptr(ring_v),
                                       ring_k.shape[0], int(hist_len), Hkv, D, _stream(stream))
    _check(st, "vico_kv_append")


def vico_attn_plan(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads, head_dim,
                   num_splits=0):
    """(splits, workspace_bytes) the attention call will use (vico_attn_plan)."""
    ns, wb = _i32(0), _i64(0)
    st = load_library().vico_attn_plan(chunk_len, sink_len, ring_slots, int(hist_len), int(window),
                                       num_q_heads, num_kv_heads, head_dim, num_splits,
                                       ctypes.byref(ns), ctypes.byref(wb))
    _check(st, "vico_attn_plan")
    return ns.value, wb.value


def vico_attn_workspace_bytes(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads,
                              head_dim, num_splits=0) -> int:
    b = load_library().vico_attn_workspace_bytes(chunk_len, sink_len, ring_slots, int(hist_len), int(window),
                                                 num_q_heads, num_kv_heads, head_dim, num_splits)
    if b < 0:
        raise VicoError(int(b), "vico_attn_workspace_bytes")
    return b


def vico_chunk_prefill_attn(q, k_chunk, v_chunk, sink_k, sink_v, ring_k, ring_v, hist_len: int, window: int,
                            out, lse=None, workspace=None, num_splits: int = 0, softmax_scale: float = 0.0,
                            stream=None) -> None:
    """Bounded chunk-prefill attention (vico_chunk_prefill_attn); writes `out` (and `lse`)."""
    for n, t in (("q", q), ("k_chunk", k_chunk), ("v_chunk", v_chunk), ("sink_k", sink_k),
                 ("sink_v", sink_v), ("ring_k", ring_k), ("ring_v", ring_v)):
        _dev_bf16(n, t)
    if not (out.is_cuda and out.is_contiguous() and out.dtype in (torch.bfloat16, torch.float32)):
        raise ValueError("out: expected a contiguous bfloat16 or float32 CUDA tensor")
    C, Hq, D = q.shape
    Hkv = k_chunk.shape[1]
    S = 0 if sink_k is None else sink_k.shape[0]
    R = 0 if ring_k is None else ring_k.shape[0]
    if tuple(out.shape) != (C, Hq, D):
        raise ValueError(f"out: shape {tuple(out.shape)} != {(C, Hq, D)}")
    if lse is not None and not (lse.is_cuda and lse.dtype == torch.float32 and lse.is_contiguous()
                                and tuple(lse.shape) == (Hq, C)):
        raise ValueError("lse: expected a contiguous float32 CUDA tensor of shape [num_q_heads, chunk_len]")
    wb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    odt = VICO_DTYPE_F32 if out.dtype == torch.float32 else VICO_DTYPE_BF16
    st = load_library().vico_chunk_prefill_attn(
        _ptr(q), _ptr(k_chunk), _ptr(v_chunk), C, _ptr(sink_k), _ptr(sink_v), S, _ptr(ring_k), _ptr(ring_v), R,
        int(hist_len), int(window), Hq, Hkv, D, float(softmax_scale), _ptr(out), odt, _ptr(lse),
        int(num_splits), _ptr(workspace), wb, _stream(stream))
    _check(st, "vico_chunk_prefill_attn")
