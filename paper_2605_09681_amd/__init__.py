"""Forcing-KV hot path on AMD MI355X: Python binding of libfkv.

Thin ctypes layer over the C ABI declared in ``include/fkv.h``; every
function has the C entry point's name and only marshals arguments (torch
tensors supply device memory, ``torch.cuda.current_stream()`` the stream).
All compute runs in the HIP kernels of ``libfkv.so``; there is no CPU
fallback.  If the library has not been built, calls raise
:class:`FkvLibraryMissing`.

Entry points (see ``include/fkv.h`` for the full contract):

* :func:`fkv_compress_static`  -- static structural pruning (Sec. 4.2, Eq. 2)
* :func:`fkv_score_segments`   -- segment similarity (Sec. 4.3, Eq. 3)
* :func:`fkv_select_compact`   -- BottomK + compaction (Sec. 4.3, Eq. 3)
* :func:`fkv_chunk_attention`  -- chunk attention (Eq. 2 / Eq. 4)
* :func:`fkv_chunk_attention_heads` -- the same for a subset of heads
* :func:`fkv_chunk_attention_static` -- the static heads' attention read in
  place from the cache (no compressed copy)
* :func:`fkv_append_frames`    -- rolling-cache write of a finished chunk
* :func:`fkv_fp8_pack`, :func:`fkv_fp8_pack_paged`, :func:`fkv_chunk_attention_fp8`
  -- the FP8 variant of the chunk attention (App. F)
* :func:`fkv_attention_mass`, :func:`fkv_classify_heads` -- offline head
  profiling (Sec. 4.1, Eq. 1)
* :func:`fkv_score_pooled`, :func:`fkv_select_compact_pooled` -- the
  first-block proxy of Sec. 4.3: one similarity row pooled over all heads,
  shared by the dynamic heads of every layer
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfkv.so")

FKV_OK, FKV_ERR_ARG, FKV_ERR_SHAPE, FKV_ERR_CAPACITY, FKV_ERR_DEVICE = range(5)
FKV_BF16, FKV_F32 = 0, 1
FKV_STATIC, FKV_DYNAMIC = 0, 1
FKV_SCOPE_FRAME, FKV_SCOPE_GLOBAL = 0, 1
FKV_MAX_HEADS, FKV_MAX_FRAMES, FKV_MAX_SEGMENTS = 64, 256, 4096

EXPORTED = ("fkv_num_segments", "fkv_kept_tokens_max", "fkv_compress_static",
            "fkv_score_workspace_size", "fkv_score_segments", "fkv_select_compact",
            "fkv_append_frames", "fkv_score_pooled_workspace_size", "fkv_score_pooled",
            "fkv_select_compact_pooled", "fkv_select", "fkv_score_select", "fkv_score_select_noalloc",
            "fkv_score_stats_size", "fkv_score_history",
            "fkv_score_segments_cached",
            "fkv_attention_workspace_size", "fkv_chunk_attention", "fkv_chunk_attention_heads",
            "fkv_chunk_attention_static", "fkv_chunk_attention_paged",
            "fkv_fp8_sizes", "fkv_fp8_pack", "fkv_fp8_pack_paged",
            "fkv_chunk_attention_fp8", "fkv_attention_mass_workspace_size", "fkv_attention_mass",
            "fkv_classify_heads", "fkv_last_error")


class FkvLibraryMissing(RuntimeError):
    pass


class FkvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"fkv status {status}: {message}")
        self.status = status
        self.message = message


class fkv_shape(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("frame_tokens", ctypes.c_int32), ("hist_frames", ctypes.c_int32),
                ("cap_frames", ctypes.c_int32), ("chunk_frames", ctypes.c_int32),
                ("seg_tokens", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class fkv_head(ctypes.Structure):
    _fields_ = [("type", ctypes.c_int32), ("sink_frames", ctypes.c_int32),
                ("recent_frames", ctypes.c_int32), ("keep_k", ctypes.c_int32),
                ("scope", ctypes.c_int32)]


_lib = None


def lib():
    """Load libfkv.so (raises FkvLibraryMissing if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FkvLibraryMissing(
                f"{LIB_PATH} is missing: build it with `python -m paper_2605_09681_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
        S, Hd = ctypes.POINTER(fkv_shape), ctypes.POINTER(fkv_head)
        L.fkv_num_segments.argtypes = [S]
        L.fkv_num_segments.restype = I32
        L.fkv_kept_tokens_max.argtypes = [S, Hd, I32, ctypes.POINTER(I64)]
        L.fkv_kept_tokens_max.restype = ctypes.c_int
        L.fkv_compress_static.argtypes = [S, Hd, P, P, P, P, P, I32, P, P]
        L.fkv_compress_static.restype = ctypes.c_int
        L.fkv_score_workspace_size.argtypes = [S, Hd, ctypes.POINTER(SZ)]
        L.fkv_score_workspace_size.restype = ctypes.c_int
        L.fkv_score_segments.argtypes = [S, Hd, P, P, P, P, P, SZ, P]
        L.fkv_score_segments.restype = ctypes.c_int
        L.fkv_select_compact.argtypes = [S, Hd, P, P, P, P, P, P, P, I32, P, P]
        L.fkv_select_compact.restype = ctypes.c_int
        L.fkv_append_frames.argtypes = [S, P, P, I32, P, P, P, P]
        L.fkv_append_frames.restype = ctypes.c_int
        L.fkv_score_pooled_workspace_size.argtypes = [S, ctypes.POINTER(SZ)]
        L.fkv_score_pooled_workspace_size.restype = ctypes.c_int
        L.fkv_score_pooled.argtypes = [S, P, P, P, P, P, SZ, P]
        L.fkv_score_pooled.restype = ctypes.c_int
        L.fkv_select_compact_pooled.argtypes = [S, Hd, P, P, P, P, P, P, P, I32, P, P]
        L.fkv_select_compact_pooled.restype = ctypes.c_int
        L.fkv_select.argtypes = [S, Hd, P, I32, P, P, P]
        L.fkv_select.restype = ctypes.c_int
        L.fkv_score_select.argtypes = [S, Hd, P, P, P, P, P, P, P, SZ, P]
        L.fkv_score_select.restype = ctypes.c_int
        L.fkv_score_select_noalloc.argtypes = [S, Hd, P, P, P, P, P, P, P]
        L.fkv_score_select_noalloc.restype = ctypes.c_int
        L.fkv_attention_workspace_size.argtypes = [S, ctypes.POINTER(SZ)]
        L.fkv_attention_workspace_size.restype = ctypes.c_int
        L.fkv_chunk_attention.argtypes = [S, P, P, P, I32, P, P, P, F, P, P, P, SZ, P]
        L.fkv_chunk_attention.restype = ctypes.c_int
        L.fkv_score_stats_size.argtypes = [S, Hd, I32, ctypes.POINTER(SZ)]
        L.fkv_score_stats_size.restype = ctypes.c_int
        L.fkv_score_history.argtypes = [S, Hd, I32, P, P, P, SZ, P, SZ, P]
        L.fkv_score_history.restype = ctypes.c_int
        L.fkv_score_segments_cached.argtypes = [S, Hd, I32, P, P, P, P, SZ, P, P, SZ, P]
        L.fkv_score_segments_cached.restype = ctypes.c_int
        L.fkv_chunk_attention_heads.argtypes = [S, P, I32, P, P, P, I32, P, P, P, F, P, P, P, SZ, P]
        L.fkv_chunk_attention_heads.restype = ctypes.c_int
        L.fkv_chunk_attention_static.argtypes = [S, Hd, P, P, P, P, P, P, F, P, P, P, SZ, P]
        L.fkv_chunk_attention_static.restype = ctypes.c_int
        L.fkv_chunk_attention_paged.argtypes = [S, Hd, P, I32, P, P, P, P, P, P, P, P, F, P, P, P, SZ, P]
        L.fkv_chunk_attention_paged.restype = ctypes.c_int
        L.fkv_fp8_sizes.argtypes = [S, I32] + [ctypes.POINTER(SZ)] * 4
        L.fkv_fp8_sizes.restype = ctypes.c_int
        L.fkv_fp8_pack.argtypes = [S, P, P, P, I32, P, P, P, P, P, P, P, P, SZ, P]
        L.fkv_fp8_pack.restype = ctypes.c_int
        L.fkv_fp8_pack_paged.argtypes = [S, Hd, P, P, ctypes.POINTER(I32), P, P, P, P, P, I32, P, P, P, P, P,
                                         SZ, P]
        L.fkv_fp8_pack_paged.restype = ctypes.c_int
        L.fkv_chunk_attention_fp8.argtypes = [S, P, P, P, I32, P, P, F, P, P, P, SZ, P]
        L.fkv_chunk_attention_fp8.restype = ctypes.c_int
        L.fkv_attention_mass_workspace_size.argtypes = [S, I32, ctypes.POINTER(SZ)]
        L.fkv_attention_mass_workspace_size.restype = ctypes.c_int
        L.fkv_attention_mass.argtypes = [S, P, P, I32, P, P, P, F, I32, P, I32, P, SZ, P]
        L.fkv_attention_mass.restype = ctypes.c_int
        L.fkv_classify_heads.argtypes = [P, I32, I32, I32, I32, I32, F, P]
        L.fkv_classify_heads.restype = ctypes.c_int
        L.fkv_last_error.argtypes = []
        L.fkv_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


# ---------------------------------------------------------------------------
# argument marshalling
# ---------------------------------------------------------------------------
def make_shape(n_heads, head_dim, frame_tokens, hist_frames, cap_frames, chunk_frames,
               seg_tokens, dtype) -> fkv_shape:
    dt = {"bf16": FKV_BF16, "f32": FKV_F32, FKV_BF16: FKV_BF16, FKV_F32: FKV_F32}[dtype]
    return fkv_shape(n_heads, head_dim, frame_tokens, hist_frames, cap_frames, chunk_frames,
                     seg_tokens, dt)


def make_heads(budgets: Sequence) -> ctypes.Array:
    """Per-head budgets: objects with type/sink_frames/recent_frames/keep_k/scope
    attributes, or 5-tuples in that order."""
    arr = (fkv_head * len(budgets))()
    for i, b in enumerate(budgets):
        vals = (b.type, b.sink_frames, b.recent_frames, b.keep_k, b.scope) if hasattr(b, "type") else tuple(b)
        arr[i] = fkv_head(*map(int, vals))
    return arr


def _torch_dtype(shape: fkv_shape):
    return torch.bfloat16 if shape.dtype == FKV_BF16 else torch.float32


def _check(t: torch.Tensor, name: str, dtype, size=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if size is not None and tuple(t.shape) != tuple(size):
        raise ValueError(f"{name} must have shape {tuple(size)} (got {tuple(t.shape)})")
    return ctypes.c_void_p(t.data_ptr())


def _slots(frame_slot, H):
    if frame_slot is None:
        import numpy as np
        frame_slot = np.arange(H, dtype="int32")
    arr = (ctypes.c_int32 * max(H, 1))()
    vals = [int(v) for v in (frame_slot.tolist() if hasattr(frame_slot, "tolist") else frame_slot)]
    if len(vals) != H:
        raise ValueError(f"frame_slot needs {H} entries (got {len(vals)})")
    for i, v in enumerate(vals):
        arr[i] = v
    return arr


def _heads(shape: fkv_shape, heads, allow_none: bool = False):
    """The host fkv_head array of a call: the C entry points read exactly
    shape.n_heads entries, so a shorter or longer array is rejected here."""
    if heads is None:
        if allow_none:
            return None
        raise ValueError("heads is None")
    if not isinstance(heads, ctypes.Array) or heads._type_ is not fkv_head:
        raise TypeError("heads must be an fkv_head array (see make_heads)")
    if len(heads) != shape.n_heads:
        raise ValueError(f"heads has {len(heads)} entries, the shape has {shape.n_heads} heads")
    return heads


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _raise(status: int):
    if status != FKV_OK:
        raise FkvError(status, lib().fkv_last_error().decode())


def _lq(shape):
    return shape.chunk_frames * shape.frame_tokens


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------
def fkv_num_segments(shape: fkv_shape) -> int:
    return int(lib().fkv_num_segments(ctypes.byref(shape)))


def fkv_kept_tokens_max(shape: fkv_shape, heads, head: int) -> int:
    out = ctypes.c_int64(0)
    _raise(lib().fkv_kept_tokens_max(ctypes.byref(shape), _heads(shape, heads), int(head), ctypes.byref(out)))
    return int(out.value)


def slab_tokens(shape: fkv_shape, heads) -> int:
    """Smallest slab (tokens per head of Kc/Vc) that fits every head's budget."""
    return max([fkv_kept_tokens_max(shape, heads, h) for h in range(shape.n_heads)] + [0])


def fkv_score_workspace_size(shape: fkv_shape, heads) -> int:
    out = ctypes.c_size_t(0)
    _raise(lib().fkv_score_workspace_size(ctypes.byref(shape), _heads(shape, heads), ctypes.byref(out)))
    return int(out.value)


def fkv_compress_static(shape: fkv_shape, heads, K_hist, V_hist, frame_slot, Kc, Vc, kv_len,
                        stream=None):
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    slab = Kc.shape[1] if Kc.dim() == 3 else -1
    comp = (shape.n_heads, slab, shape.head_dim)
    args = [_check(K_hist, "K_hist", dt, hist), _check(V_hist, "V_hist", dt, hist)]
    sl = _slots(frame_slot, shape.hist_frames)
    args += [_check(Kc, "Kc", dt, comp), _check(Vc, "Vc", dt, comp)]
    kl = _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    _raise(lib().fkv_compress_static(ctypes.byref(shape), _heads(shape, heads), args[0], args[1], sl, args[2],
                                     args[3], int(slab), kl, _stream(stream)))


def fkv_score_segments(shape: fkv_shape, heads, K_hist, frame_slot, K_cur, scores,
                       workspace: Optional[torch.Tensor] = None, stream=None):
    """If ``workspace`` is None a torch uint8 tensor of the required size is
    allocated on the current device (through torch's caching allocator)."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    n_seg = fkv_num_segments(shape)
    kh = _check(K_hist, "K_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    kc = _check(K_cur, "K_cur", dt, (shape.n_heads, _lq(shape), shape.head_dim))
    sc = _check(scores, "scores", torch.float32, (shape.n_heads, n_seg))
    need = fkv_score_workspace_size(shape, heads)
    if workspace is None:   # zero-filled: the scoring workspace starts with arrival counters
        workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=K_hist.device)
    ws = _check(workspace, "workspace", torch.uint8)
    _raise(lib().fkv_score_segments(ctypes.byref(shape), _heads(shape, heads), kh, sl, kc, sc, ws,
                                    workspace.numel(), _stream(stream)))
    return workspace


def fkv_score_stats_size(shape: fkv_shape, heads, pooled: bool = False) -> int:
    """Bytes of the per-frame statistics buffer of incremental rescoring."""
    out = ctypes.c_size_t(0)
    _raise(lib().fkv_score_stats_size(ctypes.byref(shape), _heads(shape, heads, allow_none=bool(pooled)), int(pooled), ctypes.byref(out)))
    return int(out.value)


def fkv_score_history(shape: fkv_shape, heads, K_hist, frame_slot, stats, workspace, pooled: bool = False,
                      stream=None):
    """Per-frame statistics of the history into ``stats`` (float64 device
    tensor of fkv_score_stats_size bytes), once per chunk."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    kh = _check(K_hist, "K_hist", dt, hist)
    st = _check(stats, "stats", torch.float64)
    ws = _check(workspace, "workspace", torch.uint8)
    _raise(lib().fkv_score_history(ctypes.byref(shape), _heads(shape, heads, allow_none=bool(pooled)), int(pooled), kh, _slots(frame_slot, shape.hist_frames),
                                   st, stats.numel() * 8, ws, workspace.numel(), _stream(stream)))


def fkv_score_segments_cached(shape: fkv_shape, heads, K_hist, frame_slot, K_cur, stats, scores, workspace,
                              pooled: bool = False, stream=None):
    """Scores of one AR step from the history statistics plus the pair
    (frame H-1, first frame of K_cur): the result of fkv_score_segments
    (or fkv_score_pooled when pooled) with two frames read per head."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    n_seg = fkv_num_segments(shape)
    kh = _check(K_hist, "K_hist", dt, hist)
    kc = _check(K_cur, "K_cur", dt, (shape.n_heads, _lq(shape), shape.head_dim))
    sc = _check(scores, "scores", torch.float32, (n_seg,) if pooled else (shape.n_heads, n_seg))
    st = _check(stats, "stats", torch.float64)
    ws = _check(workspace, "workspace", torch.uint8)
    _raise(lib().fkv_score_segments_cached(ctypes.byref(shape), _heads(shape, heads, allow_none=bool(pooled)), int(pooled), kh,
                                           _slots(frame_slot, shape.hist_frames), kc, st, stats.numel() * 8, sc,
                                           ws, workspace.numel(), _stream(stream)))


def fkv_append_frames(shape: fkv_shape, K_new, V_new, dst_slot, K_hist, V_hist, stream=None):
    """Writes the frames of K_new / V_new ([n_heads][n*F][d]) into the cache
    slots dst_slot (host ints, one per frame)."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    slots = [int(v) for v in dst_slot]
    n = len(slots)
    new = (shape.n_heads, n * shape.frame_tokens, shape.head_dim)
    kn, vn = _check(K_new, "K_new", dt, new), _check(V_new, "V_new", dt, new)
    kh, vh = _check(K_hist, "K_hist", dt, hist), _check(V_hist, "V_hist", dt, hist)
    arr = (ctypes.c_int32 * max(n, 1))(*slots)
    _raise(lib().fkv_append_frames(ctypes.byref(shape), kn, vn, n, arr, kh, vh, _stream(stream)))


def fkv_score_pooled_workspace_size(shape: fkv_shape) -> int:
    out = ctypes.c_size_t(0)
    _raise(lib().fkv_score_pooled_workspace_size(ctypes.byref(shape), ctypes.byref(out)))
    return int(out.value)


def fkv_score_pooled(shape: fkv_shape, K_hist, frame_slot, K_cur, scores,
                     workspace: Optional[torch.Tensor] = None, stream=None):
    """One similarity row [n_seg] pooled over all heads (the first-block proxy).
    If ``workspace`` is None a torch uint8 tensor of the required size is
    allocated on the current device."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    n_seg = fkv_num_segments(shape)
    kh = _check(K_hist, "K_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    kc = _check(K_cur, "K_cur", dt, (shape.n_heads, _lq(shape), shape.head_dim))
    sc = _check(scores, "scores", torch.float32, (n_seg,))
    need = fkv_score_pooled_workspace_size(shape)
    if workspace is None:   # zero-filled: the scoring workspace starts with arrival counters
        workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=K_hist.device)
    ws = _check(workspace, "workspace", torch.uint8)
    _raise(lib().fkv_score_pooled(ctypes.byref(shape), kh, sl, kc, sc, ws, workspace.numel(),
                                  _stream(stream)))
    return workspace


def fkv_select_compact_pooled(shape: fkv_shape, heads, scores, K_hist, V_hist, frame_slot,
                              kept_seg, Kc, Vc, kv_len, stream=None):
    """fkv_select_compact with one shared score row [n_seg]."""
    _select_compact(shape, heads, scores, K_hist, V_hist, frame_slot, kept_seg, Kc, Vc, kv_len,
                    stream, pooled=True)


def fkv_select(shape: fkv_shape, heads, scores, kept_seg, kv_len, shared_row: bool = False, stream=None):
    """BottomK only: kept_seg and kv_len of the dynamic heads, no copy.
    scores is [n_heads][n_seg], or [n_seg] with shared_row (the pooled proxy)."""
    n_seg = fkv_num_segments(shape)
    sc = _check(scores, "scores", torch.float32, (n_seg,) if shared_row else (shape.n_heads, n_seg))
    ks = _check(kept_seg, "kept_seg", torch.int32, (shape.n_heads, n_seg))
    kl = _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    _raise(lib().fkv_select(ctypes.byref(shape), _heads(shape, heads), sc, int(bool(shared_row)), ks, kl,
                            _stream(stream)))


def fkv_score_select(shape: fkv_shape, heads, K_hist, frame_slot, K_cur, scores, kept_seg, kv_len,
                     workspace: Optional[torch.Tensor] = None, stream=None):
    """fkv_score_segments + fkv_select in one launch.  If ``workspace`` is None
    a zero-filled one is allocated (through torch's caching allocator)."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    n_seg = fkv_num_segments(shape)
    kh = _check(K_hist, "K_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    kc = _check(K_cur, "K_cur", dt, (shape.n_heads, _lq(shape), shape.head_dim))
    sc = _check(scores, "scores", torch.float32, (shape.n_heads, n_seg))
    ks = _check(kept_seg, "kept_seg", torch.int32, (shape.n_heads, n_seg))
    kl = _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    need = fkv_score_workspace_size(shape, heads)
    if workspace is None:
        workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=K_hist.device)
    ws = _check(workspace, "workspace", torch.uint8)
    _raise(lib().fkv_score_select(ctypes.byref(shape), _heads(shape, heads), kh, sl, kc, sc, ks, kl, ws,
                                  workspace.numel(), _stream(stream)))
    return workspace


def fkv_score_select_noalloc(shape: fkv_shape, heads, K_hist, frame_slot, K_cur, scores, kept_seg, kv_len,
                             stream=None):
    """fkv_score_select with the library's own per-GPU scratch as workspace:
    nothing is allocated.  Calls that overlap on one GPU race."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    n_seg = fkv_num_segments(shape)
    kh = _check(K_hist, "K_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    kc = _check(K_cur, "K_cur", dt, (shape.n_heads, _lq(shape), shape.head_dim))
    sc = _check(scores, "scores", torch.float32, (shape.n_heads, n_seg))
    ks = _check(kept_seg, "kept_seg", torch.int32, (shape.n_heads, n_seg))
    kl = _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    _raise(lib().fkv_score_select_noalloc(ctypes.byref(shape), _heads(shape, heads), kh, sl, kc, sc, ks, kl,
                                          _stream(stream)))


def fkv_select_compact(shape: fkv_shape, heads, scores, K_hist, V_hist, frame_slot, kept_seg,
                       Kc, Vc, kv_len, stream=None):
    _select_compact(shape, heads, scores, K_hist, V_hist, frame_slot, kept_seg, Kc, Vc, kv_len,
                    stream, pooled=False)


def _select_compact(shape, heads, scores, K_hist, V_hist, frame_slot, kept_seg, Kc, Vc, kv_len,
                    stream, pooled):
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    n_seg = fkv_num_segments(shape)
    sc = _check(scores, "scores", torch.float32, (n_seg,) if pooled else (shape.n_heads, n_seg))
    kh, vh = _check(K_hist, "K_hist", dt, hist), _check(V_hist, "V_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    ks = _check(kept_seg, "kept_seg", torch.int32, (shape.n_heads, n_seg))
    slab = Kc.shape[1] if Kc.dim() == 3 else -1
    comp = (shape.n_heads, slab, shape.head_dim)
    kc, vc = _check(Kc, "Kc", dt, comp), _check(Vc, "Vc", dt, comp)
    kl = _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    fn = lib().fkv_select_compact_pooled if pooled else lib().fkv_select_compact
    _raise(fn(ctypes.byref(shape), _heads(shape, heads), sc, kh, vh, sl, ks, kc, vc, int(slab), kl, _stream(stream)))


def fkv_attention_workspace_size(shape: fkv_shape) -> int:
    """Bytes of the balanced-schedule workspace on the current device."""
    out = ctypes.c_size_t(0)
    _raise(lib().fkv_attention_workspace_size(ctypes.byref(shape), ctypes.byref(out)))
    return int(out.value)


def _attention_args(shape: fkv_shape, Q, Kc, Vc, kv_len, K_cur, V_cur, O, lse, workspace):
    dt = _torch_dtype(shape)
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    slab = Kc.shape[1] if Kc.dim() == 3 else -1
    comp = (shape.n_heads, slab, shape.head_dim)
    q = _check(Q, "Q", dt, chunk)
    kc, vc = _check(Kc, "Kc", dt, comp), _check(Vc, "Vc", dt, comp)
    kl = _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    kq, vq = _check(K_cur, "K_cur", dt, chunk), _check(V_cur, "V_cur", dt, chunk)
    o = _check(O, "O", dt, chunk)
    ls = None if lse is None else _check(lse, "lse", torch.float32, (shape.n_heads, _lq(shape)))
    ws, nws = None, 0
    if workspace is not None:
        ws, nws = _check(workspace, "workspace", torch.uint8), workspace.numel()
    return q, kc, vc, int(slab), kl, kq, vq, o, ls, ws, nws


def fkv_chunk_attention(shape: fkv_shape, Q, Kc, Vc, kv_len, K_cur, V_cur, scale: float, O,
                        lse: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                        stream=None):
    """``workspace`` (uint8 device tensor of fkv_attention_workspace_size bytes,
    zero-filled before its first use, e.g. torch.zeros) selects the balanced
    schedule; None runs one workgroup per query tile."""
    q, kc, vc, slab, kl, kq, vq, o, ls, ws, nws = _attention_args(shape, Q, Kc, Vc, kv_len, K_cur, V_cur, O,
                                                                  lse, workspace)
    _raise(lib().fkv_chunk_attention(ctypes.byref(shape), q, kc, vc, slab, kl, kq, vq,
                                     ctypes.c_float(scale), o, ls, ws, nws, _stream(stream)))


def fkv_chunk_attention_heads(shape: fkv_shape, heads: Sequence[int], Q, Kc, Vc, kv_len, K_cur, V_cur,
                              scale: float, O, lse: Optional[torch.Tensor] = None,
                              workspace: Optional[torch.Tensor] = None, stream=None):
    """fkv_chunk_attention for the listed heads only (host ints); the other
    heads' rows of O and lse are left untouched."""
    q, kc, vc, slab, kl, kq, vq, o, ls, ws, nws = _attention_args(shape, Q, Kc, Vc, kv_len, K_cur, V_cur, O,
                                                                  lse, workspace)
    ids = [int(h) for h in heads]
    arr = (ctypes.c_int32 * max(len(ids), 1))(*ids)
    _raise(lib().fkv_chunk_attention_heads(ctypes.byref(shape), arr, len(ids), q, kc, vc, slab, kl, kq, vq,
                                           ctypes.c_float(scale), o, ls, ws, nws, _stream(stream)))


def fkv_chunk_attention_static(shape: fkv_shape, heads, K_hist, V_hist, frame_slot, Q, K_cur, V_cur,
                               scale: float, O, lse: Optional[torch.Tensor] = None,
                               workspace: Optional[torch.Tensor] = None, stream=None):
    """Attention of the static heads over their kept frames read in place
    from K_hist / V_hist; only the static heads' rows of O and lse are
    written."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    kh, vh = _check(K_hist, "K_hist", dt, hist), _check(V_hist, "V_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    q = _check(Q, "Q", dt, chunk)
    kq, vq = _check(K_cur, "K_cur", dt, chunk), _check(V_cur, "V_cur", dt, chunk)
    o = _check(O, "O", dt, chunk)
    ls = None if lse is None else _check(lse, "lse", torch.float32, (shape.n_heads, _lq(shape)))
    ws, nws = None, 0
    if workspace is not None:
        ws, nws = _check(workspace, "workspace", torch.uint8), workspace.numel()
    _raise(lib().fkv_chunk_attention_static(ctypes.byref(shape), _heads(shape, heads), kh, vh, sl, q, kq, vq,
                                            ctypes.c_float(scale), o, ls, ws, nws, _stream(stream)))


def fkv_chunk_attention_paged(shape: fkv_shape, heads, K_hist, V_hist, frame_slot, kept_seg, kv_len, Q, K_cur,
                              V_cur, scale: float, O, lse: Optional[torch.Tensor] = None,
                              workspace: Optional[torch.Tensor] = None, head_list: Optional[Sequence[int]] = None,
                              stream=None):
    """Attention of the listed heads (all by default) with every head's kept
    history read in place from K_hist / V_hist: the Eq. 2 frames of static
    heads, the kept segments (kept_seg, kv_len from fkv_select) of dynamic
    heads.  Only the listed heads' rows of O and lse are written."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    n_seg = fkv_num_segments(shape)
    kh, vh = _check(K_hist, "K_hist", dt, hist), _check(V_hist, "V_hist", dt, hist)
    sl = _slots(frame_slot, shape.hist_frames)
    ks = None if kept_seg is None else _check(kept_seg, "kept_seg", torch.int32, (shape.n_heads, n_seg))
    kl = None if kv_len is None else _check(kv_len, "kv_len", torch.int32, (shape.n_heads,))
    q = _check(Q, "Q", dt, chunk)
    kq, vq = _check(K_cur, "K_cur", dt, chunk), _check(V_cur, "V_cur", dt, chunk)
    o = _check(O, "O", dt, chunk)
    ls = None if lse is None else _check(lse, "lse", torch.float32, (shape.n_heads, _lq(shape)))
    ws, nws = None, 0
    if workspace is not None:
        ws, nws = _check(workspace, "workspace", torch.uint8), workspace.numel()
    arr, n = None, 0
    if head_list is not None:
        ids = [int(h) for h in head_list]
        arr, n = (ctypes.c_int32 * max(len(ids), 1))(*ids), len(ids)
    _raise(lib().fkv_chunk_attention_paged(ctypes.byref(shape), _heads(shape, heads), arr, n, kh, vh, sl, ks, kl,
                                           q, kq, vq, ctypes.c_float(scale), o, ls, ws, nws, _stream(stream)))


def fkv_fp8_sizes(shape: fkv_shape, slab: int):
    """(q_bytes, kv_bytes, scale_bytes, workspace_bytes) of the FP8 buffers."""
    out = [ctypes.c_size_t(0) for _ in range(4)]
    _raise(lib().fkv_fp8_sizes(ctypes.byref(shape), int(slab), *[ctypes.byref(o) for o in out]))
    return tuple(int(o.value) for o in out)


def fkv_fp8_pack(shape: fkv_shape, Q, Kc, Vc, kv_len, K_cur, V_cur, Q8, K8, V8T, scales,
                 workspace, stream=None):
    dt = _torch_dtype(shape)
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    slab = Kc.shape[1] if Kc.dim() == 3 else -1
    comp = (shape.n_heads, slab, shape.head_dim)
    qb, kvb, sb, wb = fkv_fp8_sizes(shape, slab)
    args = [_check(Q, "Q", dt, chunk), _check(Kc, "Kc", dt, comp), _check(Vc, "Vc", dt, comp), int(slab),
            _check(kv_len, "kv_len", torch.int32, (shape.n_heads,)), _check(K_cur, "K_cur", dt, chunk),
            _check(V_cur, "V_cur", dt, chunk)]
    for t, name, nb in ((Q8, "Q8", qb), (K8, "K8", kvb), (V8T, "V8T", kvb)):
        args.append(_check(t, name, torch.uint8))
        if t.numel() != nb:
            raise ValueError(f"{name} holds {t.numel()} bytes, {nb} expected")
    args.append(_check(scales, "scales", torch.float32))
    if scales.numel() * 4 != sb:
        raise ValueError(f"scales holds {scales.numel() * 4} bytes, {sb} expected")
    args += [_check(workspace, "workspace", torch.uint8), workspace.numel(), _stream(stream)]
    _raise(lib().fkv_fp8_pack(ctypes.byref(shape), *args))


def fkv_fp8_pack_paged(shape: fkv_shape, heads, K_hist, V_hist, frame_slot, kept_seg, kv_len, Q, K_cur, V_cur,
                       slab: int, Q8, K8, V8T, scales, workspace, stream=None):
    """fkv_fp8_pack with every head's retained history read in place from
    K_hist / V_hist (kept frames of static heads, kept segments of dynamic
    heads); writes the static heads' kv_len."""
    dt = _torch_dtype(shape)
    hist = (shape.n_heads, shape.cap_frames, shape.frame_tokens, shape.head_dim)
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    n_seg = fkv_num_segments(shape)
    qb, kvb, sb, wb = fkv_fp8_sizes(shape, slab)
    args = [_heads(shape, heads), _check(K_hist, "K_hist", dt, hist), _check(V_hist, "V_hist", dt, hist),
            _slots(frame_slot, shape.hist_frames),
            None if kept_seg is None else _check(kept_seg, "kept_seg", torch.int32, (shape.n_heads, n_seg)),
            _check(kv_len, "kv_len", torch.int32, (shape.n_heads,)), _check(Q, "Q", dt, chunk),
            _check(K_cur, "K_cur", dt, chunk), _check(V_cur, "V_cur", dt, chunk), int(slab)]
    for t, name, nb in ((Q8, "Q8", qb), (K8, "K8", kvb), (V8T, "V8T", kvb)):
        args.append(_check(t, name, torch.uint8))
        if t.numel() != nb:
            raise ValueError(f"{name} holds {t.numel()} bytes, {nb} expected")
    args.append(_check(scales, "scales", torch.float32))
    if scales.numel() * 4 != sb:
        raise ValueError(f"scales holds {scales.numel() * 4} bytes, {sb} expected")
    args += [_check(workspace, "workspace", torch.uint8), workspace.numel(), _stream(stream)]
    _raise(lib().fkv_fp8_pack_paged(ctypes.byref(shape), *args))


def fkv_chunk_attention_fp8(shape: fkv_shape, Q8, K8, V8T, slab: int, kv_len, scales, scale: float, O,
                            lse: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                            stream=None):
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    qb, kvb, sb, _ = fkv_fp8_sizes(shape, slab)
    for t, name, nb in ((Q8, "Q8", qb), (K8, "K8", kvb), (V8T, "V8T", kvb)):
        _check(t, name, torch.uint8)
        if t.numel() != nb:
            raise ValueError(f"{name} holds {t.numel()} bytes, {nb} expected")
    ls = None if lse is None else _check(lse, "lse", torch.float32, (shape.n_heads, _lq(shape)))
    ws, nws = None, 0
    if workspace is not None:
        ws, nws = _check(workspace, "workspace", torch.uint8), workspace.numel()
    _raise(lib().fkv_chunk_attention_fp8(
        ctypes.byref(shape), _check(Q8, "Q8", torch.uint8), _check(K8, "K8", torch.uint8),
        _check(V8T, "V8T", torch.uint8), int(slab), _check(kv_len, "kv_len", torch.int32, (shape.n_heads,)),
        _check(scales, "scales", torch.float32), ctypes.c_float(scale), _check(O, "O", torch.bfloat16, chunk),
        ls, ws, nws, _stream(stream)))


def fkv_attention_mass_workspace_size(shape: fkv_shape, n_bins: int) -> int:
    out = ctypes.c_size_t(0)
    _raise(lib().fkv_attention_mass_workspace_size(ctypes.byref(shape), int(n_bins), ctypes.byref(out)))
    return int(out.value)


def fkv_attention_mass(shape: fkv_shape, Q, Kc, kv_len, K_cur, lse, scale: float, mass,
                       accumulate: bool = False, workspace: Optional[torch.Tensor] = None, stream=None):
    """Head-profiling attention mass per key block of F keys (see fkv.h)."""
    dt = _torch_dtype(shape)
    chunk = (shape.n_heads, _lq(shape), shape.head_dim)
    slab = Kc.shape[1] if Kc.dim() == 3 else -1
    m = _check(mass, "mass", torch.float32)
    if mass.dim() != 2 or mass.shape[0] != shape.n_heads:
        raise ValueError("mass must be [n_heads][n_bins]")
    n_bins = mass.shape[1]
    need = fkv_attention_mass_workspace_size(shape, n_bins)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=Q.device)
    _raise(lib().fkv_attention_mass(
        ctypes.byref(shape), _check(Q, "Q", dt, chunk), _check(Kc, "Kc", dt, (shape.n_heads, slab, shape.head_dim)),
        int(slab), _check(kv_len, "kv_len", torch.int32, (shape.n_heads,)), _check(K_cur, "K_cur", dt, chunk),
        _check(lse, "lse", torch.float32, (shape.n_heads, _lq(shape))), ctypes.c_float(scale), int(n_bins), m,
        1 if accumulate else 0, _check(workspace, "workspace", torch.uint8), workspace.numel(), _stream(stream)))
    return workspace


def fkv_classify_heads(mass, hist_frames: int, sink_frames: int = 1, transition_frames: int = 1,
                       alpha: float = 0.8):
    """Eq. 1 on a host mass table [n_heads][n_bins] (numpy float32 or a CPU
    tensor); returns a list of FKV_STATIC / FKV_DYNAMIC."""
    import numpy as np
    m = np.ascontiguousarray(mass.cpu().numpy() if isinstance(mass, torch.Tensor) else mass, dtype=np.float32)
    n_heads, n_bins = m.shape
    out = (ctypes.c_int32 * n_heads)()
    _raise(lib().fkv_classify_heads(m.ctypes.data_as(ctypes.c_void_p), n_heads, n_bins, int(hist_frames),
                                    int(sink_frames), int(transition_frames), ctypes.c_float(alpha), out))
    return list(out)


def fkv_last_error() -> str:
    return lib().fkv_last_error().decode()
