"""CPU oracle of the Forcing-KV hot path (arXiv 2605.09681) -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports it, and the two share no code: the oracle is
plain C in ``fkv_oracle.c`` (fp64 loops, OpenMP over independent rows or
segments), wrapped here with ctypes for numpy arrays.

Per-function citations are in ``fkv_oracle.c``; the pipeline in
:func:`run_layer` follows the paper's order: Eq. 2 for static heads; Eq. 3
(similarity, BottomK), the compression union and Eq. 4 for dynamic heads.

Parity pins: every function here is checked by ``tests/test_oracle_pins.py``
against closed forms, exact rational arithmetic, brute force and library
routines (see that file's docstring for the list).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fkv_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

BF16, F32, F64 = 0, 1, 2
STATIC, DYNAMIC = 0, 1


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (always recompiles)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
           _SRC, "-o", _LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def lib():
    """The compiled oracle.  FKV_ORACLE_LIB may name another build of the same
    source (the mutation tests load deliberately broken copies that way)."""
    global _lib
    if _lib is None:
        path = os.environ.get("FKV_ORACLE_LIB", _LIB)
        if path == _LIB and not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(path)
        P, I, LG, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_long, ctypes.c_double
        L.fkvo_static_frames.argtypes = [I, I, I, P]
        L.fkvo_static_frames.restype = I
        L.fkvo_gather_frames.argtypes = [I, I, I, P, P, P, I, P]
        L.fkvo_gather_frames.restype = LG
        L.fkvo_n_segments.argtypes = [I, I, I]
        L.fkvo_n_segments.restype = I
        L.fkvo_score_head.argtypes = [I, I, I, I, I, P, P, P, P, P]
        L.fkvo_score_head.restype = None
        L.fkvo_append_frames.argtypes = [I, I, I, I, P, P, P]
        L.fkvo_append_frames.restype = None
        L.fkvo_score_pooled.argtypes = [I, I, I, I, I, I, I, LG, P, P, P, P, P]
        L.fkvo_score_pooled.restype = None
        L.fkvo_select_head.argtypes = [I, I, I, I, I, I, I, P, P]
        L.fkvo_select_head.restype = I
        L.fkvo_compact_head.argtypes = [I, I, I, I, I, P, I, P, P, P]
        L.fkvo_compact_head.restype = LG
        L.fkvo_attention_rows.argtypes = [I, I, LG, LG, P, P, P, P, P, D, P, I, P, P]
        L.fkvo_attention_rows.restype = None
        L.fkvo_attention_mass.argtypes = [I, I, LG, LG, I, P, P, P, D, P]
        L.fkvo_attention_mass.restype = None
        L.fkvo_max_threads.argtypes = []
        L.fkvo_max_threads.restype = I
        L.fkvo_set_threads.argtypes = [I]
        L.fkvo_set_threads.restype = None
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dt(arr: np.ndarray) -> int:
    if arr.dtype == np.uint16:
        return BF16
    if arr.dtype == np.float32:
        return F32
    if arr.dtype == np.float64:
        return F64
    raise TypeError(f"oracle takes uint16 (bf16 bits), float32 or float64, got {arr.dtype}")


def _c(a, dtype=None):
    return np.ascontiguousarray(a if dtype is None else np.asarray(a, dtype=dtype))


def max_threads() -> int:
    return lib().fkvo_max_threads()


def set_threads(n: int) -> None:
    """Threads of the oracle's OpenMP regions (timing only)."""
    lib().fkvo_set_threads(int(n))


# ---------------------------------------------------------------------------
# per-head primitives
# ---------------------------------------------------------------------------
def static_frames(H: int, sink: int, recent: int) -> np.ndarray:
    out = np.empty(max(H, 1), np.int32)
    n = lib().fkvo_static_frames(H, sink, recent, _ptr(out))
    return out[:n].copy()


def gather_frames(hist_head: np.ndarray, frame_slot: np.ndarray, frames: np.ndarray) -> np.ndarray:
    """hist_head: [cap][F][d] -> [len(frames)*F][d]."""
    hist_head = _c(hist_head)
    _, F, d = hist_head.shape
    frames = _c(frames, np.int32)
    slot = _c(frame_slot, np.int32)
    out = np.empty((len(frames) * F, d), hist_head.dtype)
    lib().fkvo_gather_frames(hist_head.itemsize, F, d, _ptr(hist_head), _ptr(slot),
                             _ptr(frames), len(frames), _ptr(out))
    return out


def n_segments(H: int, F: int, L: int) -> int:
    return lib().fkvo_n_segments(H, F, L)


def score_head(hist_head: np.ndarray, frame_slot: np.ndarray, cur_head: np.ndarray,
               H: int, L: int):
    """Eq. 3 similarity of every segment.  Returns (fp32 scores, fp64 cosines)."""
    hist_head = _c(hist_head)
    cur_head = _c(cur_head)
    _, F, d = hist_head.shape
    assert cur_head.dtype == hist_head.dtype and cur_head.shape[1] == d
    slot = _c(frame_slot, np.int32)
    n = n_segments(H, F, L)
    s32 = np.empty(max(n, 1), np.float32)
    s64 = np.empty(max(n, 1), np.float64)
    lib().fkvo_score_head(_dt(hist_head), d, F, H, L, _ptr(hist_head), _ptr(slot),
                          _ptr(cur_head), _ptr(s32), _ptr(s64))
    return s32[:n].copy(), s64[:n].copy()


def append_frames(hist_head: np.ndarray, new_frames: np.ndarray, dst_slot: np.ndarray) -> None:
    """Rolling cache: writes new_frames[f] ([n][F][d]) into slot dst_slot[f] of
    hist_head ([cap][F][d]) in place."""
    assert hist_head.flags.c_contiguous and hist_head.flags.writeable
    new_frames = _c(new_frames)
    n, F, d = new_frames.shape
    assert new_frames.dtype == hist_head.dtype and hist_head.shape[1:] == (F, d)
    slot = _c(dst_slot, np.int32)
    assert slot.shape == (n,) and ((slot >= 0) & (slot < hist_head.shape[0])).all()
    lib().fkvo_append_frames(hist_head.dtype.itemsize, F, d, n, _ptr(new_frames), _ptr(slot),
                             _ptr(hist_head))


def score_pooled(hist: np.ndarray, frame_slot: np.ndarray, cur: np.ndarray, H: int, L: int):
    """First-block proxy (Sec. 4.3): one similarity per segment from the keys of
    all heads together.  hist: [n_heads][cap][F][d]; cur: [n_heads][lq][d].
    Returns (fp32 scores, fp64 cosines)."""
    hist = _c(hist)
    cur = _c(cur)
    nh, cap, F, d = hist.shape
    assert cur.dtype == hist.dtype and cur.shape[0] == nh and cur.shape[2] == d
    slot = _c(frame_slot, np.int32)
    n = n_segments(H, F, L)
    s32 = np.empty(max(n, 1), np.float32)
    s64 = np.empty(max(n, 1), np.float64)
    lib().fkvo_score_pooled(_dt(hist), nh, d, F, H, L, cap, cur.shape[1], _ptr(hist), _ptr(slot),
                            _ptr(cur), _ptr(s32), _ptr(s64))
    return s32[:n].copy(), s64[:n].copy()


def select_head(scores: np.ndarray, H: int, F: int, L: int, sink: int, recent: int,
                k: int, scope: int):
    """Eq. 3 BottomK.  Returns (kept [n_seg] ascending, -1 padded; kept count)."""
    n = n_segments(H, F, L)
    s = _c(scores, np.float32)
    assert s.shape == (n,)
    kept = np.empty(max(n, 1), np.int32)
    cnt = lib().fkvo_select_head(H, F, L, sink, recent, k, scope, _ptr(s), _ptr(kept))
    return kept[:n].copy(), cnt


def compact_head(hist_head: np.ndarray, frame_slot: np.ndarray, kept: np.ndarray,
                 H: int, L: int) -> np.ndarray:
    """Concatenated rows of the kept segments: [kv_len][d]."""
    hist_head = _c(hist_head)
    _, F, d = hist_head.shape
    kept = _c(kept, np.int32)
    kept = kept[kept >= 0]
    HF = H * F
    tokens = int(sum(min(g * L + L, HF) - g * L for g in kept))
    out = np.empty((tokens, d), hist_head.dtype)
    n = lib().fkvo_compact_head(hist_head.itemsize, d, F, H, L, _ptr(kept), len(kept),
                                _ptr(hist_head), _ptr(_c(frame_slot, np.int32)), _ptr(out))
    assert n == tokens
    return out


def attention_rows(Q: np.ndarray, Kc: np.ndarray, Vc: np.ndarray, K_cur: np.ndarray,
                   V_cur: np.ndarray, scale: float, rows=None):
    """Eq. 4 attention for one head.  Q/K_cur/V_cur: [Lq][d]; Kc/Vc: [kv_len][d].
    Returns (O [n_rows][d] fp64, lse [n_rows] fp64)."""
    Q, K_cur, V_cur = _c(Q), _c(K_cur), _c(V_cur)
    Kc, Vc = _c(Kc), _c(Vc)
    Lq, d = Q.shape
    kv_len = Kc.shape[0]
    for a in (Kc, Vc, K_cur, V_cur):
        assert a.dtype == Q.dtype and a.shape[1] == d
    rows = np.arange(Lq, dtype=np.int32) if rows is None else _c(rows, np.int32)
    out = np.empty((len(rows), d), np.float64)
    lse = np.empty(len(rows), np.float64)
    kc = Kc if kv_len else np.zeros((1, d), Q.dtype)
    vc = Vc if kv_len else np.zeros((1, d), Q.dtype)
    lib().fkvo_attention_rows(_dt(Q), d, kv_len, Lq, _ptr(Q), _ptr(kc), _ptr(vc),
                              _ptr(K_cur), _ptr(V_cur), float(scale), _ptr(rows),
                              len(rows), _ptr(out), _ptr(lse))
    return out, lse


def attention_mass(Q: np.ndarray, Kc: np.ndarray, K_cur: np.ndarray, F: int, scale: float) -> np.ndarray:
    """Sec. 4.1 attention mass per block of F keys of [Kc; K_cur], summed over
    all query rows (fp64).  Q/K_cur: [Lq][d]; Kc: [kv_len][d]."""
    Q, K_cur, Kc = _c(Q), _c(K_cur), _c(Kc)
    Lq, d = Q.shape
    kv_len = Kc.shape[0]
    n_bins = -(-(kv_len + Lq) // F)
    out = np.empty(max(n_bins, 1), np.float64)
    kc = Kc if kv_len else np.zeros((1, d), Q.dtype)
    lib().fkvo_attention_mass(_dt(Q), d, kv_len, Lq, F, _ptr(Q), _ptr(kc), _ptr(K_cur), float(scale), _ptr(out))
    return out[:n_bins].copy()


def classify_heads(mass: np.ndarray, hist_frames: int, sink_frames: int, transition_frames: int,
                   alpha: float) -> np.ndarray:
    """Eq. 1: a head is static (0) when the mass on the generated chunk plus the
    transition frame(s), over the mass of the whole window without the sink
    frame(s), exceeds alpha; dynamic (1) otherwise.  mass: [n_heads][H + C]
    (history frames in logical order, then the chunk's frames), summed in fp64."""
    mass = np.asarray(mass, np.float64)
    H = hist_frames
    types = []
    for row in mass:
        total = row.sum()
        generate = row[H:].sum()
        transition = row[max(H - transition_frames, 0):H].sum()
        sink = row[:min(sink_frames, H)].sum()
        denom = total - sink
        ratio = (generate + transition) / denom if denom > 0 else np.inf
        types.append(STATIC if ratio > alpha else DYNAMIC)
    return np.array(types, np.int32)


# ---------------------------------------------------------------------------
# whole layer: the hot path in the paper's order
# ---------------------------------------------------------------------------
@dataclass
class LayerResult:
    scores: np.ndarray        # [n_heads][n_seg] fp32 (NaN rows for static heads)
    cos64: np.ndarray         # [n_heads][n_seg] fp64
    kept_seg: np.ndarray      # [n_heads][n_seg] int32, -1 padded (-1 rows for static)
    kv_len: np.ndarray        # [n_heads] int64
    Kc: List[np.ndarray]      # per head [kv_len][d] storage dtype
    Vc: List[np.ndarray]
    rows: Optional[np.ndarray] = None   # query rows attended (shared by all heads)
    O: Optional[np.ndarray] = None      # [n_heads][n_rows][d] fp64
    lse: Optional[np.ndarray] = None    # [n_heads][n_rows] fp64


def run_layer(cfg, inputs, rows=None, attention: bool = True, scale: Optional[float] = None,
              heads=None) -> LayerResult:
    """Compress every head of one layer and (optionally) attend the given query
    rows.  ``cfg``/``inputs`` are the seeded workload records; ``heads``
    overrides the per-head budgets."""
    heads = cfg.heads if heads is None else heads
    H, F, L, d = cfg.hist_frames, cfg.frame_tokens, cfg.seg_tokens, cfg.head_dim
    n_seg = n_segments(H, F, L)
    nh = cfg.n_heads
    scores = np.full((nh, n_seg), np.nan, np.float32)
    cos64 = np.full((nh, n_seg), np.nan, np.float64)
    kept_seg = np.full((nh, n_seg), -1, np.int32)
    kv_len = np.zeros(nh, np.int64)
    Kc, Vc = [], []
    for h in range(nh):
        b = heads[h]
        if b.type == STATIC:
            frames = static_frames(H, b.sink_frames, b.recent_frames)
            kc = gather_frames(inputs.K_hist[h], inputs.frame_slot, frames)
            vc = gather_frames(inputs.V_hist[h], inputs.frame_slot, frames)
        else:
            s32, s64 = score_head(inputs.K_hist[h], inputs.frame_slot, inputs.K_cur[h], H, L)
            scores[h], cos64[h] = s32, s64
            kept, cnt = select_head(s32, H, F, L, b.sink_frames, b.recent_frames,
                                    b.keep_k, b.scope)
            kept_seg[h] = kept
            kc = compact_head(inputs.K_hist[h], inputs.frame_slot, kept[:cnt], H, L)
            vc = compact_head(inputs.V_hist[h], inputs.frame_slot, kept[:cnt], H, L)
        kv_len[h] = kc.shape[0]
        Kc.append(kc)
        Vc.append(vc)
    res = LayerResult(scores, cos64, kept_seg, kv_len, Kc, Vc)
    if attention:
        sc = 1.0 / np.sqrt(d) if scale is None else scale
        rows = np.arange(cfg.lq, dtype=np.int32) if rows is None else np.asarray(rows, np.int32)
        O = np.empty((nh, len(rows), d))
        lse = np.empty((nh, len(rows)))
        for h in range(nh):
            O[h], lse[h] = attention_rows(inputs.Q[h], Kc[h], Vc[h], inputs.K_cur[h],
                                          inputs.V_cur[h], sc, rows)
        res.rows, res.O, res.lse = rows, O, lse
    return res
