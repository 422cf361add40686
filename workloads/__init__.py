"""Seeded synthetic inputs for the Forcing-KV hot path.

This module is the only code shared by the CPU oracle's tests and the HIP
path's tests and benchmark.  It draws random numbers and lays them out; it
holds none of the method's arithmetic (no scoring, selection, compaction or
attention).

Input recipe (stand-in for the real Self Forcing / LongLive activations the
paper measures on, which are not available):

* numpy ``default_rng`` (PCG64), one independent stream per tensor kind,
  seeded from ``SeedSequence([seed, kind, *extra])``.
* Keys follow an AR(1) chain across frames, elementwise per (token, dim):
  ``K_0 ~ N(0,1)``, ``K_t = rho*K_{t-1} + sqrt(1-rho^2)*eps_t``, so every key is
  marginally N(0,1) and adjacent frames have correlation ``rho``.  This mimics
  the high, segment-varying similarity of adjacent frames that motivates
  dynamic similarity pruning (Sec. 3, Observation figure (d); Sec. 4.3).
  The chain runs in fp32; each stored frame is rounded to the storage dtype
  with round-to-nearest-even.  ``K_cur`` (the current chunk's keys) continues
  the chain past the last history frame.
* Queries and values are i.i.d. N(0,1).
* Shapes are Wan-1.3B-style: 12 heads, head_dim 128, 1560 tokens per latent
  frame at 480P (30x52 patches), 8160 at 1080P (68x120), 3-frame chunks and
  a 21-frame history window.

Storage: bf16 tensors are numpy ``uint16`` arrays holding the bf16 bit
patterns; fp32 tensors are ``float32`` arrays.  Layouts (row-major, head_dim
innermost):

* ``K_hist``, ``V_hist``: ``[n_heads][cap_frames][F][d]`` (physical slots)
* ``frame_slot``: ``int32[H]``, logical history frame -> physical slot
* ``Q``, ``K_cur``, ``V_cur``: ``[n_heads][C*F][d]``
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

STATIC = 0
DYNAMIC = 1
SCOPE_FRAME = 0
SCOPE_GLOBAL = 1

_KIND_K, _KIND_V, _KIND_Q, _KIND_MASK, _KIND_RHO = 0, 1, 2, 3, 4


# --------------------------------------------------------------------------
# bf16 storage helpers (bit manipulation only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = u.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def storage_to_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits_to_f32(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)


# --------------------------------------------------------------------------
# configuration records (plain data)
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class HeadBudget:
    """Per-head compression budget, as the boundary takes it."""
    type: int                 # STATIC or DYNAMIC
    sink_frames: int = 0      # leading logical frames always kept
    recent_frames: int = 0    # trailing logical frames always kept
    keep_k: int = 0           # segments kept per selection group (dynamic)
    scope: int = SCOPE_GLOBAL  # selection group: per frame or all candidates


@dataclass(frozen=True)
class LayerConfig:
    name: str
    n_heads: int
    head_dim: int
    frame_tokens: int         # F
    hist_frames: int          # H
    cap_frames: int
    chunk_frames: int         # C
    seg_tokens: int           # L
    dtype: str                # "bf16" | "f32"
    heads: tuple
    rho: object = 0.9         # scalar, per-head tuple, or per-(head, token) array

    @property
    def lq(self) -> int:
        return self.chunk_frames * self.frame_tokens

    @property
    def n_seg(self) -> int:
        ht = self.hist_frames * self.frame_tokens
        return (ht + self.seg_tokens - 1) // self.seg_tokens

    @property
    def esize(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def replace(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


def _split_heads(n_heads, n_static, static_budget, dynamic_budget):
    return tuple([static_budget] * n_static + [dynamic_budget] * (n_heads - n_static))


def tiny_config() -> LayerConfig:
    """2 heads (head0 static, head1 dynamic), d=64, F=64, 4 past frames of one
    segment each, 1-frame query chunk, fp32.  Static keeps frame 0 plus the most
    recent frame; dynamic keeps 2 of 4 segments (no sink)."""
    return LayerConfig(
        name="tiny-f32", n_heads=2, head_dim=64, frame_tokens=64, hist_frames=4,
        cap_frames=4, chunk_frames=1, seg_tokens=64, dtype="f32",
        heads=(HeadBudget(STATIC, 1, 1, 0, SCOPE_GLOBAL),
               HeadBudget(DYNAMIC, 0, 0, 2, SCOPE_GLOBAL)),
        rho=0.9)


def wan_layer_config(resolution: str = "480p", keep_fraction: float = 0.5,
                     seg_tokens: Optional[int] = None, static_recent: int = 6,
                     dtype: str = "bf16") -> LayerConfig:
    """One attention layer at a Wan-1.3B-style shape.

    12 heads, head_dim 128; 480P has 1560 tokens/frame, 1080P 8160.  A 21-frame
    history, a 3-frame query chunk.  Heads 0-5 static (sink frame + last
    ``static_recent`` frames), heads 6-11 dynamic (sink frame + ``keep_fraction``
    of the candidate segments; per-frame groups when segments are shorter than a
    frame, one global group otherwise)."""
    F = {"480p": 1560, "1080p": 8160}[resolution]
    H = 21
    L = F if seg_tokens is None else seg_tokens
    if L < F:
        per_frame = F // L
        k, scope = int(np.floor(per_frame * keep_fraction + 1e-9)), SCOPE_FRAME
    else:
        frames_per_seg = L // F
        n_seg = (H * F + L - 1) // L
        sink_segs = (1 + frames_per_seg - 1) // frames_per_seg  # segments touching frame 0
        k = int(np.floor((n_seg - sink_segs) * keep_fraction + 1e-9))
        scope = SCOPE_GLOBAL
    st = HeadBudget(STATIC, 1, static_recent, 0, SCOPE_GLOBAL)
    dy = HeadBudget(DYNAMIC, 1, 0, k, scope)
    return LayerConfig(
        name=f"wan1.3b-{resolution}-layer", n_heads=12, head_dim=128,
        frame_tokens=F, hist_frames=H, cap_frames=H, chunk_frames=3, seg_tokens=L,
        dtype=dtype, heads=_split_heads(12, 6, st, dy), rho=0.9)


def rollout_head_masks(seed: int, n_layers: int = 30, n_heads: int = 12,
                       n_dynamic: int = 6) -> np.ndarray:
    """Per-layer head-type masks with exactly ``n_dynamic`` dynamic heads per
    layer, drawn by a seeded permutation.  Returns int32 [n_layers][n_heads]."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, _KIND_MASK]))
    out = np.zeros((n_layers, n_heads), np.int32)
    for layer in range(n_layers):
        out[layer, rng.permutation(n_heads)[:n_dynamic]] = DYNAMIC
    return out


def rollout_rhos(seed: int, n_layers: int = 30, n_heads: int = 12,
                 lo: float = 0.8, hi: float = 0.98) -> np.ndarray:
    """Per-(layer, head) AR(1) coefficients drawn uniformly from [lo, hi]."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, _KIND_RHO]))
    return rng.uniform(lo, hi, size=(n_layers, n_heads)).astype(np.float32)


# --------------------------------------------------------------------------
# tensor generation
# --------------------------------------------------------------------------
def _rng(seed: int, kind: int, extra: Sequence[int] = ()) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed), kind, *map(int, extra)]))


def _rho_array(rho, n_heads: int, F: int) -> np.ndarray:
    r = np.asarray(rho, dtype=np.float32)
    if r.ndim == 0:
        r = np.full((n_heads, 1), float(r), np.float32)
    elif r.ndim == 1:
        if r.shape[0] != n_heads:
            raise ValueError("per-head rho needs n_heads entries")
        r = r.reshape(n_heads, 1)
    elif r.shape != (n_heads, F):
        raise ValueError("rho must be scalar, [n_heads] or [n_heads, F]")
    return r.reshape(n_heads, -1, 1)


def ar1_key_frames(seed: int, n_heads: int, n_frames: int, F: int, d: int, rho,
                   dtype: str, extra: Sequence[int] = ()) -> np.ndarray:
    """``n_frames`` consecutive frames of the AR(1) key chain, rounded to the
    storage dtype.  Returns ``[n_heads][n_frames][F][d]``."""
    rng = _rng(seed, _KIND_K, extra)
    r = _rho_array(rho, n_heads, F)            # [h][F or 1][1]
    s = np.sqrt(np.maximum(0.0, 1.0 - r.astype(np.float64) ** 2)).astype(np.float32)
    out = np.empty((n_heads, n_frames, F, d), np.uint16 if dtype == "bf16" else np.float32)
    k = None
    for t in range(n_frames):
        eps = rng.standard_normal((n_heads, F, d), dtype=np.float32)
        k = eps if k is None else (r * k + s * eps).astype(np.float32)
        out[:, t] = to_storage(k, dtype)
    return out


def normal_tensor(seed: int, kind: int, shape, dtype: str, extra: Sequence[int] = (),
                  scale: float = 1.0) -> np.ndarray:
    x = _rng(seed, kind, extra).standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        x = (x * np.float32(scale)).astype(np.float32)
    return to_storage(x, dtype)


@dataclass
class LayerInputs:
    cfg: LayerConfig
    K_hist: np.ndarray
    V_hist: np.ndarray
    K_cur: np.ndarray
    V_cur: np.ndarray
    Q: np.ndarray
    frame_slot: np.ndarray
    extra: dict = field(default_factory=dict)


def make_layer_inputs(cfg: LayerConfig, seed: int = 0, frame_slot=None,
                      q_scale: float = 1.0, extra: Sequence[int] = ()) -> LayerInputs:
    """Generate one layer's history cache, current chunk and queries.

    ``frame_slot`` defaults to the identity map (logical frame t in slot t).
    Unused physical slots are filled with independent N(0,1) noise so that a
    kernel reading a wrong slot produces visibly wrong results."""
    h, d, F, H, cap = cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.cap_frames
    if frame_slot is None:
        frame_slot = np.arange(H, dtype=np.int32)
    frame_slot = np.ascontiguousarray(frame_slot, dtype=np.int32)
    assert frame_slot.shape == (H,)
    chain = ar1_key_frames(seed, h, H + cfg.chunk_frames, F, d, cfg.rho, cfg.dtype, extra)
    sdt = chain.dtype
    K_hist = np.empty((h, cap, F, d), sdt)
    V_hist = np.empty((h, cap, F, d), sdt)
    V_log = normal_tensor(seed, _KIND_V, (h, H, F, d), cfg.dtype, extra)
    for t in range(H):
        K_hist[:, frame_slot[t]] = chain[:, t]
        V_hist[:, frame_slot[t]] = V_log[:, t]
    del V_log
    unused = sorted(set(range(cap)) - set(int(s) for s in frame_slot))
    if unused:
        n = len(unused)
        K_hist[:, unused] = normal_tensor(seed, 10 + _KIND_K, (h, n, F, d), cfg.dtype, extra)
        V_hist[:, unused] = normal_tensor(seed, 10 + _KIND_V, (h, n, F, d), cfg.dtype, extra)
    K_cur = np.ascontiguousarray(chain[:, H:].reshape(h, cfg.lq, d))
    V_cur = normal_tensor(seed, _KIND_V, (h, cfg.lq, d), cfg.dtype, (*extra, 1))
    Q = normal_tensor(seed, _KIND_Q, (h, cfg.lq, d), cfg.dtype, extra, scale=q_scale)
    return LayerInputs(cfg, K_hist, V_hist, K_cur, V_cur, Q, frame_slot)


def ring_frame_slots(chunk_index: int, chunk_frames: int, window: int,
                     pinned_sink: int = 1) -> np.ndarray:
    """Logical -> physical slot map of a fixed-capacity ring-buffer cache.

    Video frame ``v`` is written to slot ``v`` while the cache fills; afterwards
    the first ``pinned_sink`` slots stay pinned to the first video frames and
    the remaining ``window - pinned_sink`` slots are reused in rotation (a write
    pointer, no shifting of cached data).  Before chunk ``i`` the cache holds
    ``H = min(i*chunk_frames, window)`` frames: the sink frames and then the most
    recent ones, oldest first."""
    produced = chunk_index * chunk_frames
    H = min(produced, window)
    if produced <= window:
        return np.arange(H, dtype=np.int32)
    ring = window - pinned_sink
    slots = list(range(pinned_sink))
    first = produced - ring  # oldest non-sink video frame still cached
    for v in range(first, produced):
        slots.append(pinned_sink + (v - pinned_sink) % ring)
    return np.asarray(slots, dtype=np.int32)


def ring_slot(v: int, window: int, pinned_sink: int = 1) -> int:
    """Physical slot of video frame ``v`` in the ring-buffer cache of
    ``ring_frame_slots``: the first ``pinned_sink`` frames keep their slots, the
    others rotate through the remaining ``window - pinned_sink`` slots."""
    if v < pinned_sink:
        return v
    return pinned_sink + (v - pinned_sink) % (window - pinned_sink)


def chunk_write_slots(chunk_index: int, chunk_frames: int, window: int,
                      pinned_sink: int = 1) -> np.ndarray:
    """Slots that receive the frames of chunk ``chunk_index`` once it is done
    (the write pointer of the ring buffer)."""
    assert window - pinned_sink >= chunk_frames, "a chunk must fit in the rotating part"
    v0 = chunk_index * chunk_frames
    return np.array([ring_slot(v, window, pinned_sink) for v in range(v0, v0 + chunk_frames)],
                    dtype=np.int32)


# ---------------------------------------------------------------------------
# comparison policies expressed through the same budgets and selection inputs
# ---------------------------------------------------------------------------
def streaming_llm_heads(n_heads: int, sink_frames: int = 3, recent_frames: int = 4):
    """StreamingLLM-style frame-level cache: every head keeps the same sink
    and recent frames (3 + 4 in the paper's baseline setting)."""
    return tuple(HeadBudget(STATIC, sink_frames, recent_frames) for _ in range(n_heads))


def random_scores(seed: int, n_heads: int, n_seg: int) -> np.ndarray:
    """Scores that turn BottomK into random segment pruning: i.i.d. uniform
    draws (a seeded input, so both sides select the same segments)."""
    return _rng(seed, 9).random((n_heads, n_seg), dtype=np.float32)


def uniform_scores(n_heads: int, H: int, F: int, L: int, keep_k: int) -> np.ndarray:
    """Scores that turn per-frame BottomK (L < F) into uniform pruning: in every
    frame the segments floor(i * n / k), i < k, score 0 and the others 1, so the
    k kept segments are spread evenly over the frame."""
    n = F // L
    row = np.ones(n, np.float32)
    for i in range(min(keep_k, n)):
        row[(i * n) // max(keep_k, 1)] = 0.0
    return np.tile(np.tile(row, H), (n_heads, 1)).astype(np.float32)
