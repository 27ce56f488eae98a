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
VICO_ATTN_BIDIRECTIONAL = 1
VICO_ATTN_APPEND = 2
VICO_NOALLOC_SCRATCH_BYTES = 64 << 20

_i32, _i64, _f32, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p

_SIGNATURES = {
    "vico_kv_append": (_i32, [_vp, _vp, _i32, _vp, _vp, _i32, _i64, _i32, _i32, _vp]),
    "vico_chunk_prefill_attn": (_i32, [_vp, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _i64, _i64,
                                       _i32, _i32, _i32, _f32, _vp, _i32, _vp, _i32, _vp, _i64, _vp]),
    "vico_attn_plan": (_i32, [_i32, _i32, _i32, _i64, _i64, _i32, _i32, _i32, _i32,
                              ctypes.POINTER(_i32), ctypes.POINTER(_i64)]),
    "vico_attn_workspace_bytes": (_i64, [_i32, _i32, _i32, _i64, _i64, _i32, _i32, _i32, _i32]),
    "vico_chunk_prefill_attn_ex": (_i32, [_vp, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _i64, _i64,
                                          _i32, _i32, _i32, _f32, _vp, _i32, _vp, _i32, _i32, _vp, _i64, _vp]),
    "vico_attn_plan_ex": (_i32, [_i32, _i32, _i32, _i64, _i64, _i32, _i32, _i32, _i32, _i32,
                                 ctypes.POINTER(_i32), ctypes.POINTER(_i64)]),
    "vico_acn_window": (_i64, [ctypes.POINTER(_i64), _i32, _i32, _i32]),
    "vico_temporal_drop": (_i32, [_vp, _i32, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp]),
    "vico_temporal_drop_workspace_bytes": (_i64, [_i32, _i32, _i32, _i32]),
    "vico_token_mean": (_i32, [_vp, _i32, _i32, _vp, _vp]),
    "vico_chunk_scores": (_i32, [_vp, _vp, _i32, _i32, _vp, _vp]),
    "vico_topk_chunks": (_i32, [_vp, _i32, _i32, _f32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "vico_gather_plan": (_i32, [_i32, _i32, _i32, _i32, _i32, _i64, _i32, _i32, _i32, _i32,
                                ctypes.POINTER(_i32), ctypes.POINTER(_i64)]),
    "vico_gather_attn": (_i32, [_vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _i64,
                                _i32, _i32, _i32, _f32, _vp, _i32, _vp, _i32, _vp, _i64, _vp]),
    "vico_gather_attn_noalloc": (_i32, [_vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32,
                                        _i64, _i32, _i32, _i32, _f32, _vp, _i32, _vp, _i32, _vp]),
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
                   num_splits=0, flags: int = 0):
    """(splits, workspace_bytes) the attention call will use (vico_attn_plan_ex)."""
    ns, wb = _i32(0), _i64(0)
    st = load_library().vico_attn_plan_ex(chunk_len, sink_len, ring_slots, int(hist_len), int(window),
                                          num_q_heads, num_kv_heads, head_dim, num_splits, int(flags),
                                          ctypes.byref(ns), ctypes.byref(wb))
    _check(st, "vico_attn_plan_ex")
    return ns.value, wb.value


def vico_acn_window(chunk_starts, t: int, acn: int) -> int:
    """Visible history tokens of chunk t under the acn-chunk window (vico_acn_window)."""
    arr = (_i64 * len(chunk_starts))(*[int(x) for x in chunk_starts])
    w = load_library().vico_acn_window(arr, len(chunk_starts), int(t), int(acn))
    if w < 0:
        raise VicoError(int(w), "vico_acn_window")
    return w


def vico_attn_workspace_bytes(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads,
                              head_dim, num_splits=0) -> int:
    b = load_library().vico_attn_workspace_bytes(chunk_len, sink_len, ring_slots, int(hist_len), int(window),
                                                 num_q_heads, num_kv_heads, head_dim, num_splits)
    if b < 0:
        raise VicoError(int(b), "vico_attn_workspace_bytes")
    return b


def vico_chunk_prefill_attn(q, k_chunk, v_chunk, sink_k, sink_v, ring_k, ring_v, hist_len: int, window: int,
                            out, lse=None, workspace=None, num_splits: int = 0, softmax_scale: float = 0.0,
                            stream=None, flags: int = 0) -> None:
    """Bounded chunk-prefill attention (vico_chunk_prefill_attn_ex); writes `out` (and `lse`)."""
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
    st = load_library().vico_chunk_prefill_attn_ex(
        _ptr(q), _ptr(k_chunk), _ptr(v_chunk), C, _ptr(sink_k), _ptr(sink_v), S, _ptr(ring_k), _ptr(ring_v), R,
        int(hist_len), int(window), Hq, Hkv, D, float(softmax_scale), _ptr(out), odt, _ptr(lse),
        int(num_splits), int(flags), _ptr(workspace), wb, _stream(stream))
    _check(st, "vico_chunk_prefill_attn_ex")


def _dev_tensor(name, t, dtype, ndim):
    if not (t.is_cuda and t.dtype == dtype and t.is_contiguous() and t.dim() == ndim):
        raise ValueError(f"{name}: expected a contiguous {ndim}-d {dtype} CUDA tensor, got "
                         f"{tuple(t.shape)} {t.dtype} on {t.device}")


def vico_token_mean(x, out, stream=None) -> None:
    """out[c] = mean over tokens of x[t][c] (vico_token_mean); x bf16 [L, dm], out fp32 [dm]."""
    _dev_tensor("x", x, torch.bfloat16, 2)
    _dev_tensor("out", out, torch.float32, 1)
    L, dm = x.shape
    if out.shape[0] != dm:
        raise ValueError("out: expected [feat_dim]")
    _check(load_library().vico_token_mean(_ptr(x), L, dm, _ptr(out), _stream(stream)), "vico_token_mean")


def vico_chunk_scores(query_feat, chunk_feat, scores, stream=None) -> None:
    """Cosine of the query feature with every chunk feature (vico_chunk_scores)."""
    _dev_tensor("query_feat", query_feat, torch.float32, 1)
    _dev_tensor("chunk_feat", chunk_feat, torch.float32, 2)
    _dev_tensor("scores", scores, torch.float32, 1)
    N, dm = chunk_feat.shape
    if query_feat.shape[0] != dm or scores.shape[0] != N:
        raise ValueError("shape mismatch between query_feat, chunk_feat and scores")
    _check(load_library().vico_chunk_scores(_ptr(query_feat), _ptr(chunk_feat), N, dm, _ptr(scores),
                                            _stream(stream)), "vico_chunk_scores")


def vico_topk_chunks(scores, top_k: int, out_chunks, out_scores, out_count, min_score: float = float("-inf"),
                     chunk_start=None, chunk_len=None, seg_start=None, seg_len=None, stream=None) -> None:
    """Top-k chunks by score with score >= min_score, in stream order (vico_topk_chunks)."""
    _dev_tensor("scores", scores, torch.float32, 1)
    _dev_tensor("out_chunks", out_chunks, torch.int32, 1)
    _dev_tensor("out_scores", out_scores, torch.float32, 1)
    _dev_tensor("out_count", out_count, torch.int32, 1)
    if chunk_start is not None:
        _dev_tensor("chunk_start", chunk_start, torch.int64, 1)
        _dev_tensor("chunk_len", chunk_len, torch.int32, 1)
        _dev_tensor("seg_start", seg_start, torch.int64, 1)
        _dev_tensor("seg_len", seg_len, torch.int32, 1)
    N = scores.shape[0]
    for n, t, want in (("out_chunks", out_chunks, top_k), ("out_scores", out_scores, top_k),
                       ("seg_start", seg_start, top_k), ("seg_len", seg_len, top_k),
                       ("chunk_start", chunk_start, N), ("chunk_len", chunk_len, N)):
        if t is not None and t.shape[0] < want:
            raise ValueError(f"{n}: needs {want} entries")
    st = load_library().vico_topk_chunks(_ptr(scores), N, int(top_k), float(min_score), _ptr(chunk_start),
                                         _ptr(chunk_len), _ptr(out_chunks), _ptr(out_scores), _ptr(seg_start),
                                         _ptr(seg_len), _ptr(out_count), _stream(stream))
    _check(st, "vico_topk_chunks")


def vico_gather_plan(q_len, tail_len, sink_len, store_slots, num_segments, keys_hint, num_q_heads, num_kv_heads,
                     head_dim, num_splits=0):
    """(parts, workspace_bytes) of vico_gather_attn for these arguments."""
    ns, wb = _i32(0), _i64(0)
    st = load_library().vico_gather_plan(q_len, tail_len, sink_len, store_slots, num_segments, int(keys_hint),
                                         num_q_heads, num_kv_heads, head_dim, num_splits,
                                         ctypes.byref(ns), ctypes.byref(wb))
    _check(st, "vico_gather_plan")
    return ns.value, wb.value


def _gather_args(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len, out, lse, keys_hint,
                 softmax_scale):
    """Checked leading arguments shared by vico_gather_attn and its no-alloc variant."""
    for n, t in (("q", q), ("tail_k", tail_k), ("tail_v", tail_v), ("sink_k", sink_k), ("sink_v", sink_v),
                 ("store_k", store_k), ("store_v", store_v)):
        _dev_bf16(n, t)
    if seg_start is not None:
        _dev_tensor("seg_start", seg_start, torch.int64, 1)
        _dev_tensor("seg_len", seg_len, torch.int32, 1)
    if not (out.is_cuda and out.is_contiguous() and out.dtype in (torch.bfloat16, torch.float32)):
        raise ValueError("out: expected a contiguous bfloat16 or float32 CUDA tensor")
    Lq, Hq, D = q.shape
    T, Hkv = tail_k.shape[0], tail_k.shape[1]
    S = 0 if sink_k is None else sink_k.shape[0]
    cap = 0 if store_k is None else store_k.shape[0]
    n_segs = 0 if seg_start is None else seg_start.shape[0]
    if tuple(out.shape) != (Lq, Hq, D):
        raise ValueError(f"out: shape {tuple(out.shape)} != {(Lq, Hq, D)}")
    if lse is not None and not (lse.is_cuda and lse.dtype == torch.float32 and lse.is_contiguous()
                                and tuple(lse.shape) == (Hq, Lq)):
        raise ValueError("lse: expected a contiguous float32 CUDA tensor of shape [num_q_heads, q_len]")
    odt = VICO_DTYPE_F32 if out.dtype == torch.float32 else VICO_DTYPE_BF16
    return (_ptr(q), Lq, _ptr(tail_k), _ptr(tail_v), T, _ptr(sink_k), _ptr(sink_v), S, _ptr(store_k),
            _ptr(store_v), cap, _ptr(seg_start), _ptr(seg_len), n_segs, int(keys_hint), Hq, Hkv, D,
            float(softmax_scale), _ptr(out), odt, _ptr(lse))


def vico_gather_attn(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len, out, lse=None,
                     workspace=None, keys_hint: int = 0, num_splits: int = 0, softmax_scale: float = 0.0,
                     stream=None) -> None:
    """Short-query attention over sink ++ store segments ++ causal tail (vico_gather_attn)."""
    args = _gather_args(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len, out, lse,
                        keys_hint, softmax_scale)
    wb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = load_library().vico_gather_attn(*args, int(num_splits), _ptr(workspace), wb, _stream(stream))
    _check(st, "vico_gather_attn")


def vico_gather_attn_noalloc(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len, out,
                             lse=None, keys_hint: int = 0, num_splits: int = 0, softmax_scale: float = 0.0,
                             stream=None) -> None:
    """vico_gather_attn with the library's fixed device array as workspace
    (vico_gather_attn_noalloc); allocates nothing, here or in the library."""
    args = _gather_args(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len, out, lse,
                        keys_hint, softmax_scale)
    st = load_library().vico_gather_attn_noalloc(*args, int(num_splits), _stream(stream))
    _check(st, "vico_gather_attn_noalloc")


def vico_temporal_drop_workspace_bytes(num_chunks: int, frames_per_chunk: int, tokens_per_frame: int,
                                       feat_dim: int) -> int:
    """Workspace bytes of the single-pass drop (0: that schedule does not apply)."""
    b = load_library().vico_temporal_drop_workspace_bytes(num_chunks, frames_per_chunk, tokens_per_frame, feat_dim)
    if b < 0:
        raise VicoError(int(b), "vico_temporal_drop_workspace_bytes")
    return int(b)


def vico_temporal_drop(frames, tau: float, keep, out_index, out_count, sim=None, out_tokens=None, prev_frame=None,
                       workspace=None, stream=None) -> None:
    """Chunk-level temporal token dropping (vico_temporal_drop); frames bf16 [B, C, n_f, dm].
    With a workspace of vico_temporal_drop_workspace_bytes(B, C, n_f, dm) bytes
    the call takes the single-pass schedule where it applies."""
    _dev_tensor("frames", frames, torch.bfloat16, 4)
    B, C, n_f, dm = frames.shape
    _dev_tensor("keep", keep, torch.uint8, 2)
    _dev_tensor("out_index", out_index, torch.int32, 1)
    _dev_tensor("out_count", out_count, torch.int32, 1)
    if tuple(keep.shape) != (B, n_f) or out_index.shape[0] < B * C * n_f:
        raise ValueError("keep must be [B, n_f] and out_index hold B*C*n_f entries")
    if sim is not None:
        _dev_tensor("sim", sim, torch.float32, 2)
        if tuple(sim.shape) != (B, n_f):
            raise ValueError("sim must be [B, n_f]")
    if out_tokens is not None:
        _dev_tensor("out_tokens", out_tokens, torch.bfloat16, 2)
        if out_tokens.shape[0] < B * C * n_f or out_tokens.shape[1] != dm:
            raise ValueError("out_tokens must hold B*C*n_f rows of dm")
    if prev_frame is not None:
        _dev_tensor("prev_frame", prev_frame, torch.bfloat16, 2)
    if workspace is not None and (not workspace.is_cuda or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous device tensor")
    wb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = load_library().vico_temporal_drop(_ptr(frames), B, C, n_f, dm, float(tau), _ptr(prev_frame), _ptr(keep),
                                           _ptr(sim), _ptr(out_tokens), _ptr(out_index), _ptr(out_count),
                                           _ptr(workspace), wb, _stream(stream))
    _check(st, "vico_temporal_drop")
