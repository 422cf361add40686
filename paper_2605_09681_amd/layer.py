"""One attention layer's Forcing-KV step, and a multi-layer rollout driver.

:class:`CompressedLayer` owns the per-layer intermediate device buffers
(scores, kept segment ids, compressed K/V slabs, kv_len, the scoring and
attention workspaces) sized from the shape and budgets, and runs one AR step
of one layer.  The four stages of the method:

1. ``fkv_score_segments``  (dynamic heads, Eq. 3 similarity)
2. ``fkv_select_compact``  (dynamic heads, Eq. 3 BottomK + compaction)
3. ``fkv_compress_static`` (static heads, Eq. 2)
4. ``fkv_chunk_attention`` (all heads, Eq. 2 / Eq. 4)

:meth:`CompressedLayer.step` runs them in one of three ways (``step_mode``):

* ``"paged"`` (the default where the shape allows it: bf16, frames and
  segment pieces of at least 64 tokens): ``fkv_score_select`` scores the
  dynamic heads and selects their kept segments in one launch, then ONE
  ``fkv_chunk_attention_paged`` launch attends every head with its kept
  history read in place from the cache -- no compacted copy, no gather;
* ``"paged2"``: the same, with the static heads' attention on a second stream
  (default priority) next to the dynamic heads' scoring and attention;
* ``"compact"``: the static heads attended in place (or gathered first) on a
  side stream while the dynamic heads are scored, compacted into Kc/Vc and
  attended on the current stream.

The individual stages enqueue on the current torch stream; nothing
synchronises with the host.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import torch

from . import (FKV_DYNAMIC, FKV_STATIC, fkv_append_frames, fkv_attention_mass,
               fkv_attention_workspace_size, fkv_chunk_attention, fkv_chunk_attention_heads,
               fkv_chunk_attention_paged, fkv_chunk_attention_static, fkv_classify_heads, fkv_score_select,
               fkv_select,
               fkv_chunk_attention_fp8, fkv_compress_static, fkv_fp8_pack, fkv_fp8_pack_paged, fkv_fp8_sizes,
               fkv_num_segments, fkv_score_pooled, fkv_score_pooled_workspace_size,
               fkv_score_history, fkv_score_segments, fkv_score_segments_cached,
               fkv_score_stats_size, fkv_score_workspace_size, fkv_select_compact,
               fkv_select_compact_pooled, make_heads, make_shape, slab_tokens)


def static_in_place_supported(dtype, frame_tokens: int) -> bool:
    """Whether fkv_chunk_attention_static takes this dtype and frame size."""
    return dtype in ("bf16", 0) and frame_tokens >= 64


def paged_supported(dtype, frame_tokens: int, seg_tokens: int, cap_frames: int) -> bool:
    """Whether fkv_chunk_attention_paged reads dynamic heads of this shape in
    place: bf16, pieces of min(L, F) >= 64 tokens, at most 256 pieces in the
    cache."""
    piece = min(seg_tokens, frame_tokens)
    return (static_in_place_supported(dtype, frame_tokens) and piece >= 64
            and cap_frames * (frame_tokens // piece) <= 256)


class CompressedLayer:
    def __init__(self, n_heads: int, head_dim: int, frame_tokens: int, hist_frames: int,
                 cap_frames: int, chunk_frames: int, seg_tokens: int, dtype: str,
                 budgets: Sequence, device="cuda", slab: Optional[int] = None,
                 balanced: bool = True, overlap: bool = True, in_place: Optional[bool] = None,
                 step_mode: Optional[str] = None):
        if len(budgets) != n_heads:
            raise ValueError(f"{len(budgets)} head budgets for {n_heads} heads")
        self.shape = make_shape(n_heads, head_dim, frame_tokens, hist_frames, cap_frames,
                                chunk_frames, seg_tokens, dtype)
        self.heads = make_heads(budgets)
        self.types = [int(h.type) for h in self.heads]
        self.dtype = torch.bfloat16 if dtype in ("bf16", 0) else torch.float32
        self.device = torch.device(device)
        self.n_seg = fkv_num_segments(self.shape)
        self.slab = slab_tokens(self.shape, self.heads) if slab is None else slab
        self.lq = chunk_frames * frame_tokens
        dev, dt = self.device, self.dtype
        self.scores = torch.zeros((n_heads, self.n_seg), dtype=torch.float32, device=dev)
        self.kept_seg = torch.full((n_heads, self.n_seg), -1, dtype=torch.int32, device=dev)
        self.Kc = torch.zeros((n_heads, self.slab, head_dim), dtype=dt, device=dev)
        self.Vc = torch.zeros((n_heads, self.slab, head_dim), dtype=dt, device=dev)
        self.kv_len = torch.zeros((n_heads,), dtype=torch.int32, device=dev)
        self.ws_bytes = fkv_score_workspace_size(self.shape, self.heads)
        # scoring workspace: zero-filled once (its arrival counters), every call leaves it so
        self.workspace = torch.zeros(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)
        self.attn_workspace = self.attn_workspace2 = None
        if balanced:
            with torch.cuda.device(dev):
                n = fkv_attention_workspace_size(self.shape)
            if n > 0:
                # zero-filled once (arrival counters); every call leaves it so
                self.attn_workspace = torch.zeros(n, dtype=torch.uint8, device=dev)
        self.scale = 1.0 / math.sqrt(head_dim)
        self.has_static = FKV_STATIC in self.types
        self.has_dynamic = FKV_DYNAMIC in self.types
        # side stream for the static heads (only when both head types exist)
        self.side = (torch.cuda.Stream(device=dev) if overlap and self.has_static and self.has_dynamic
                     else None)
        self.static_heads = [h for h, t in enumerate(self.types) if t == FKV_STATIC]
        self.dynamic_heads = [h for h, t in enumerate(self.types) if t == FKV_DYNAMIC]
        if self.side is not None and self.attn_workspace is not None:
            self.attn_workspace2 = torch.zeros_like(self.attn_workspace)
        # static heads attended in place by step() (bf16, frames >= 64 tokens)
        can = static_in_place_supported(dtype, frame_tokens)
        if in_place and not can:
            raise ValueError("in-place static attention needs bf16 and frame_tokens >= 64")
        self.static_in_place = can if in_place is None else bool(in_place)
        can_paged = paged_supported(dtype, frame_tokens, seg_tokens, cap_frames)
        if step_mode is None:
            step_mode = "paged" if can_paged and (in_place is None or in_place) else "compact"
        if step_mode not in ("paged", "paged2", "compact"):
            raise ValueError(f"step_mode {step_mode!r}")
        if step_mode != "compact" and not can_paged:
            raise ValueError("paged steps need bf16, frame and segment pieces of >= 64 tokens and "
                             "cap_frames * F / min(L, F) <= 256")
        self.step_mode = step_mode
        if step_mode == "paged2" and self.side is None and overlap and self.has_static and self.has_dynamic:
            self.side = torch.cuda.Stream(device=dev)

    # individual stages -------------------------------------------------------
    def score(self, K_hist, frame_slot, K_cur):
        fkv_score_segments(self.shape, self.heads, K_hist, frame_slot, K_cur, self.scores,
                           self.workspace)

    def select_compact(self, K_hist, V_hist, frame_slot):
        fkv_select_compact(self.shape, self.heads, self.scores, K_hist, V_hist, frame_slot,
                           self.kept_seg, self.Kc, self.Vc, self.kv_len)

    def compress_static(self, K_hist, V_hist, frame_slot):
        fkv_compress_static(self.shape, self.heads, K_hist, V_hist, frame_slot, self.Kc,
                            self.Vc, self.kv_len)

    def attention(self, Q, K_cur, V_cur, O, lse=None, scale: Optional[float] = None):
        fkv_chunk_attention(self.shape, Q, self.Kc, self.Vc, self.kv_len, K_cur, V_cur,
                            self.scale if scale is None else scale, O, lse, self.attn_workspace)

    def fp8_buffers(self):
        """Packed FP8 inputs of the FP8 attention variant (allocated on first use)."""
        if getattr(self, "_fp8", None) is None:
            qb, kvb, sb, wb = fkv_fp8_sizes(self.shape, self.slab)
            u8 = dict(dtype=torch.uint8, device=self.device)
            self._fp8 = dict(Q8=torch.empty(qb, **u8), K8=torch.empty(kvb, **u8), V8T=torch.empty(kvb, **u8),
                             scales=torch.empty(sb // 4, dtype=torch.float32, device=self.device),
                             ws=torch.empty(max(wb, 1), **u8))
        return self._fp8

    def pack_fp8(self, Q, K_cur, V_cur):
        b = self.fp8_buffers()
        fkv_fp8_pack(self.shape, Q, self.Kc, self.Vc, self.kv_len, K_cur, V_cur, b["Q8"], b["K8"], b["V8T"],
                     b["scales"], b["ws"])

    def attention_fp8_packed(self, O, lse=None, scale: Optional[float] = None):
        b = self.fp8_buffers()
        fkv_chunk_attention_fp8(self.shape, b["Q8"], b["K8"], b["V8T"], self.slab, self.kv_len, b["scales"],
                                self.scale if scale is None else scale, O, lse, self.attn_workspace)

    def attention_fp8(self, Q, K_cur, V_cur, O, lse=None, scale: Optional[float] = None):
        """FP8 variant of :meth:`attention`: pack, then the FP8 kernel."""
        self.pack_fp8(Q, K_cur, V_cur)
        self.attention_fp8_packed(O, lse, scale)

    def pack_fp8_paged(self, K_hist, V_hist, frame_slot, Q, K_cur, V_cur):
        """FP8 packing with every head's retained history read in place from
        the cache (the dynamic heads' kept segments as the selection left them
        in kept_seg / kv_len); writes the static heads' kv_len."""
        b = self.fp8_buffers()
        fkv_fp8_pack_paged(self.shape, self.heads, K_hist, V_hist, frame_slot, self.kept_seg, self.kv_len, Q,
                           K_cur, V_cur, self.slab, b["Q8"], b["K8"], b["V8T"], b["scales"], b["ws"])

    def step_fp8(self, K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse=None, scale: Optional[float] = None):
        """One AR step with the FP8 attention and no compressed copy: scores
        and kept segments of the dynamic heads (one launch), FP8 packing read
        in place from the cache, then the FP8 attention."""
        if self.has_dynamic:
            self.score_select(K_hist, frame_slot, K_cur)
        self.pack_fp8_paged(K_hist, V_hist, frame_slot, Q, K_cur, V_cur)
        self.attention_fp8_packed(O, lse, scale)

    # whole step --------------------------------------------------------------
    def compress(self, K_hist, V_hist, frame_slot, K_cur):
        if self.side is not None:
            main = torch.cuda.current_stream(self.device)
            self.side.wait_stream(main)             # inputs written on the main stream
            with torch.cuda.stream(self.side):
                self.compress_static(K_hist, V_hist, frame_slot)
            for t in (K_hist, V_hist):              # read on the side stream too
                t.record_stream(self.side)
            self.score(K_hist, frame_slot, K_cur)
            self.select_compact(K_hist, V_hist, frame_slot)
            main.wait_stream(self.side)             # attention reads every head's Kc/Vc/kv_len
            return
        if self.has_dynamic:
            self.score(K_hist, frame_slot, K_cur)
            self.select_compact(K_hist, V_hist, frame_slot)
        if self.has_static:
            self.compress_static(K_hist, V_hist, frame_slot)

    def attention_static(self, K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse=None, workspace=None):
        """The static heads' attention read in place from the cache."""
        fkv_chunk_attention_static(self.shape, self.heads, K_hist, V_hist, frame_slot, Q, K_cur, V_cur,
                                   self.scale, O, lse, workspace)

    def score_select(self, K_hist, frame_slot, K_cur):
        """Scores and kept segments of the dynamic heads in one launch (no copy)."""
        fkv_score_select(self.shape, self.heads, K_hist, frame_slot, K_cur, self.scores, self.kept_seg,
                         self.kv_len, self.workspace)

    def attention_paged(self, K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse=None, head_list=None,
                        workspace=None):
        """Attention of the listed heads (all by default), every kept history
        read in place from the cache."""
        fkv_chunk_attention_paged(self.shape, self.heads, K_hist, V_hist, frame_slot, self.kept_seg, self.kv_len,
                                  Q, K_cur, V_cur, self.scale, O, lse,
                                  self.attn_workspace if workspace is None else workspace, head_list)

    def step(self, K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse=None, events=None):
        """One AR step of the layer (see the module docstring for the modes).
        ``events`` (optional) maps a launch name to a pair of torch.cuda.Events
        recorded around that attention launch on the stream it runs on
        ("attention" for one launch, "static_attention" and "dynamic_attention"
        for the two-stream steps), for per-launch timing."""
        def mark(name, i, stream):
            if events is not None and name in events:
                events[name][i].record(stream)
        if self.step_mode == "paged" or (self.step_mode == "paged2" and self.side is None):
            cur = torch.cuda.current_stream(self.device)
            if self.has_dynamic:
                self.score_select(K_hist, frame_slot, K_cur)
            mark("attention", 0, cur)
            self.attention_paged(K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse)
            mark("attention", 1, cur)
            return
        if self.step_mode == "paged2":
            main = torch.cuda.current_stream(self.device)
            self.side.wait_stream(main)
            with torch.cuda.stream(self.side):
                mark("static_attention", 0, self.side)
                self.attention_paged(K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse, self.static_heads,
                                     self.attn_workspace2)
                mark("static_attention", 1, self.side)
            for t in (K_hist, V_hist, Q, K_cur, V_cur, O) + ((lse,) if lse is not None else ()):
                t.record_stream(self.side)
            self.score_select(K_hist, frame_slot, K_cur)
            mark("dynamic_attention", 0, main)
            self.attention_paged(K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse, self.dynamic_heads)
            mark("dynamic_attention", 1, main)
            main.wait_stream(self.side)
            return
        if self.side is None:
            cur = torch.cuda.current_stream(self.device)
            if self.static_in_place and not self.has_dynamic:
                mark("attention", 0, cur)
                self.attention_static(K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse, self.attn_workspace)
                mark("attention", 1, cur)
                return
            self.compress(K_hist, V_hist, frame_slot, K_cur)
            mark("attention", 0, cur)
            self.attention(Q, K_cur, V_cur, O, lse)
            mark("attention", 1, cur)
            return
        main = torch.cuda.current_stream(self.device)
        args = (self.Kc, self.Vc, self.kv_len, K_cur, V_cur, self.scale, O, lse)
        self.side.wait_stream(main)
        with torch.cuda.stream(self.side):
            if self.static_in_place:
                mark("static_attention", 0, self.side)
                self.attention_static(K_hist, V_hist, frame_slot, Q, K_cur, V_cur, O, lse, self.attn_workspace2)
                mark("static_attention", 1, self.side)
            else:
                self.compress_static(K_hist, V_hist, frame_slot)
                mark("static_attention", 0, self.side)
                fkv_chunk_attention_heads(self.shape, self.static_heads, Q, *args[:7], lse=lse,
                                          workspace=self.attn_workspace2)
                mark("static_attention", 1, self.side)
        for t in (K_hist, V_hist, Q, K_cur, V_cur, O) + ((lse,) if lse is not None else ()):
            t.record_stream(self.side)
        self.score(K_hist, frame_slot, K_cur)
        self.select_compact(K_hist, V_hist, frame_slot)
        mark("dynamic_attention", 0, main)
        fkv_chunk_attention_heads(self.shape, self.dynamic_heads, Q, *args[:7], lse=lse,
                                  workspace=self.attn_workspace)
        mark("dynamic_attention", 1, main)
        main.wait_stream(self.side)


class HeadProfiler:
    """Offline head profiling (Sec. 4.1, Eq. 1) of one layer.

    Each :meth:`observe` call attends the chunk's queries over the uncompressed
    cache (every head keeps the whole history, gathered with the static-head
    kernel) and adds the attention mass of every history frame and chunk frame
    to ``mass`` [n_heads][H + C] on the device.  :meth:`classify` applies Eq. 1
    to the accumulated table."""

    def __init__(self, n_heads: int, head_dim: int, frame_tokens: int, hist_frames: int,
                 cap_frames: int, chunk_frames: int, device="cuda"):
        self.H, self.C = hist_frames, chunk_frames
        budgets = [type("B", (), dict(type=FKV_STATIC, sink_frames=0, recent_frames=hist_frames,
                                      keep_k=0, scope=0))() for _ in range(n_heads)]
        self.layer = CompressedLayer(n_heads, head_dim, frame_tokens, hist_frames, cap_frames,
                                     chunk_frames, frame_tokens, "bf16", budgets, device=device)
        dev = self.layer.device
        self.mass = torch.zeros((n_heads, hist_frames + chunk_frames), dtype=torch.float32, device=dev)
        self.lse = torch.empty((n_heads, self.layer.lq), dtype=torch.float32, device=dev)
        self.O = torch.empty((n_heads, self.layer.lq, head_dim), dtype=torch.bfloat16, device=dev)
        self.workspace = None
        self.observed = 0

    def observe(self, Q, K_hist, V_hist, frame_slot, K_cur, V_cur):
        L = self.layer
        L.compress_static(K_hist, V_hist, frame_slot)
        L.attention(Q, K_cur, V_cur, self.O, self.lse)
        self.workspace = fkv_attention_mass(L.shape, Q, L.Kc, L.kv_len, K_cur, self.lse, L.scale, self.mass,
                                            accumulate=self.observed > 0, workspace=self.workspace)
        self.observed += 1

    def classify(self, alpha: float = 0.8, sink_frames: int = 1, transition_frames: int = 1):
        return fkv_classify_heads(self.mass.cpu(), self.H, sink_frames, transition_frames, alpha)


class RolloutStack:
    """A stack of attention layers in a streaming AR rollout.

    Every layer owns a rolling K/V cache of ``window`` frame slots
    ([n_heads][window][F][d]); the caller maps logical history frames to slots
    (``frame_slot``, sink pinned, the others rotating) and writes each finished
    chunk's frames back with :meth:`append`.  Layers run one after another, so
    they share one set of compressed-cache buffers, sized for a full window;
    the history length H = len(frame_slot) may grow from chunk to chunk (0 on
    the first one).  Per layer and AR step :meth:`run_layer` either (step_mode
    "paged", the default where the shape allows it) scores and selects the
    dynamic heads in one launch and then attends every head in one launch with
    its kept history read in place from the cache, or ("compact") runs the
    static heads' attention on a side stream (read in place for bf16 and
    frames of at least 64 tokens, else gathered first) next to the dynamic
    heads' scoring, compaction and attention.  With a shared score row from
    :meth:`score_pooled` -- the first-block proxy of Sec. 4.3 -- the dynamic
    heads of every layer select with one similarity row computed from one
    layer's keys pooled over all heads.  ``budgets`` are per-head objects with
    type/sink_frames/recent_frames/keep_k/scope for the given H.

    Incremental rescoring: :meth:`history` stores a layer's per-frame
    similarity statistics once per chunk (the history is fixed during the
    chunk's AR steps); ``incremental=True`` in :meth:`run_layer` /
    :meth:`score_pooled` then reads only the last history frame and the chunk's
    first frame per head."""

    def __init__(self, n_layers: int, n_heads: int, head_dim: int, frame_tokens: int, window: int,
                 chunk_frames: int, seg_tokens: int, dtype: str = "bf16", device="cuda",
                 overlap: bool = True, step_mode: Optional[str] = None):
        self.n_layers, self.n_heads, self.d = n_layers, n_heads, head_dim
        self.F, self.window, self.C, self.L = frame_tokens, window, chunk_frames, seg_tokens
        self.dtype_name = dtype
        self.dtype = torch.bfloat16 if dtype in ("bf16", 0) else torch.float32
        self.device = torch.device(device)
        dev, dt = self.device, self.dtype
        hist = (n_heads, window, frame_tokens, head_dim)
        self.K_hist = [torch.zeros(hist, dtype=dt, device=dev) for _ in range(n_layers)]
        self.V_hist = [torch.zeros(hist, dtype=dt, device=dev) for _ in range(n_layers)]
        full = self._shape(window)
        self.n_seg_max = fkv_num_segments(full)
        self.slab = window * frame_tokens
        self.Kc = torch.zeros((n_heads, self.slab, head_dim), dtype=dt, device=dev)
        self.Vc = torch.zeros_like(self.Kc)
        self.kv_len = torch.zeros((n_heads,), dtype=torch.int32, device=dev)
        self._scores = torch.zeros((n_heads * max(self.n_seg_max, 1),), dtype=torch.float32, device=dev)
        self._kept = torch.full((n_heads * max(self.n_seg_max, 1),), -1, dtype=torch.int32, device=dev)
        self.pooled_row = torch.zeros((max(self.n_seg_max, 1),), dtype=torch.float32, device=dev)
        # workspaces: the largest history with every head dynamic bounds the scoring workspace
        all_dyn = make_heads([_Budget(FKV_DYNAMIC, 0, 0, 0, 1)] * n_heads)
        # (scoring workspaces are zero-filled once: the one-launch reduction's arrival counters)
        self.score_ws = torch.zeros(max(fkv_score_workspace_size(full, all_dyn), 1), dtype=torch.uint8, device=dev)
        self.pooled_ws = torch.zeros(max(fkv_score_pooled_workspace_size(full), 1), dtype=torch.uint8, device=dev)
        with torch.cuda.device(dev):
            n = fkv_attention_workspace_size(full)
        self.attn_ws = torch.zeros(max(n, 1), dtype=torch.uint8, device=dev) if n > 0 else None
        self.attn_ws2 = torch.zeros_like(self.attn_ws) if (n > 0 and overlap) else None
        self.scale = 1.0 / math.sqrt(head_dim)
        self.side = torch.cuda.Stream(device=dev) if overlap else None
        self.static_in_place = static_in_place_supported(dtype, frame_tokens)
        can_paged = paged_supported(dtype, frame_tokens, seg_tokens, window)
        if step_mode is None:
            step_mode = "paged" if can_paged else "compact"
        if step_mode not in ("paged", "compact") or (step_mode == "paged" and not can_paged):
            raise ValueError(f"step_mode {step_mode!r} is not available for this shape")
        self.step_mode = step_mode
        self._shapes, self._heads = {}, {}
        # per-layer statistics of incremental rescoring (listed heads x window x units x 2)
        units = frame_tokens // min(seg_tokens, frame_tokens)
        self._stats_len = n_heads * window * units * 2
        self._stats, self._pooled_stats = {}, {}

    def _shape(self, H: int):
        return make_shape(self.n_heads, self.d, self.F, H, self.window, self.C, self.L, self.dtype_name)

    def shape(self, H: int):
        if H not in self._shapes:
            self._shapes[H] = self._shape(H)
        return self._shapes[H]

    def _budget_array(self, budgets):
        if len(budgets) != self.n_heads:
            raise ValueError(f"{len(budgets)} head budgets for {self.n_heads} heads")
        key = tuple((int(b.type), int(b.sink_frames), int(b.recent_frames), int(b.keep_k), int(b.scope))
                    for b in budgets)
        if key not in self._heads:
            self._heads[key] = make_heads(budgets)
        return self._heads[key], key

    def views(self, H: int):
        """scores and kept_seg of the current history length, as [n_heads][n_seg] tensors."""
        n_seg = fkv_num_segments(self.shape(H))
        k = self.n_heads * n_seg
        return self._scores[:k].view(self.n_heads, n_seg), self._kept[:k].view(self.n_heads, n_seg)

    def _stats_buf(self, table, layer):
        if layer not in table:
            table[layer] = torch.empty(self._stats_len, dtype=torch.float64, device=self.device)
        return table[layer]

    def history(self, layer: int, budgets, frame_slot, pooled: bool = False):
        """Per-frame statistics of the layer's history (its dynamic heads, or
        every head for the pooled proxy); valid until the history changes."""
        H = len(frame_slot)
        if H == 0:
            return
        shape = self.shape(H)
        heads = None if pooled else self._budget_array(budgets)[0]
        stats = self._stats_buf(self._pooled_stats if pooled else self._stats, layer)
        fkv_score_history(shape, heads, self.K_hist[layer], frame_slot, stats,
                          self.pooled_ws if pooled else self.score_ws, pooled=pooled)

    def score_pooled(self, layer: int, frame_slot, K_cur, incremental: bool = False):
        """The first-block proxy: one score row pooled over all heads of ``layer``
        (from the statistics of :meth:`history` when ``incremental``)."""
        H = len(frame_slot)
        if H == 0:
            return self.pooled_row[:0]
        shape = self.shape(H)
        row = self.pooled_row[:fkv_num_segments(shape)]
        if incremental:
            fkv_score_segments_cached(shape, None, self.K_hist[layer], frame_slot, K_cur,
                                      self._pooled_stats[layer], row, self.pooled_ws, pooled=True)
        else:
            fkv_score_pooled(shape, self.K_hist[layer], frame_slot, K_cur, row, self.pooled_ws)
        return row

    def run_layer(self, layer: int, budgets, frame_slot, Q, K_cur, V_cur, O, lse=None, pooled=None,
                  incremental: bool = False):
        """One AR step of one layer: compress its cache, then chunk attention
        into O -- the static heads (attended in place, or gathered and then
        attended) on the side stream while the dynamic heads are scored,
        compacted and attended on the current stream.  ``pooled`` (a row from :meth:`score_pooled`)
        replaces the layer's own per-head scoring."""
        H = len(frame_slot)
        shape = self.shape(H)
        heads, key = self._budget_array(budgets)
        types = [b[0] for b in key]
        Kh, Vh = self.K_hist[layer], self.V_hist[layer]
        scores, kept = self.views(H)
        has_static, has_dynamic = FKV_STATIC in types, FKV_DYNAMIC in types
        if self.step_mode == "paged":
            # one stream: scores + kept segments, then one attention launch over
            # every head with its kept history read in place (no copy)
            if has_dynamic:
                if pooled is not None:
                    fkv_select(shape, heads, pooled, kept, self.kv_len, shared_row=True)
                elif incremental and H > 0:
                    fkv_score_segments_cached(shape, heads, Kh, frame_slot, K_cur, self._stats[layer], scores,
                                              self.score_ws)
                    fkv_select(shape, heads, scores, kept, self.kv_len)
                else:
                    fkv_score_select(shape, heads, Kh, frame_slot, K_cur, scores, kept, self.kv_len, self.score_ws)
            fkv_chunk_attention_paged(shape, heads, Kh, Vh, frame_slot, kept, self.kv_len, Q, K_cur, V_cur,
                                      self.scale, O, lse, self.attn_ws)
            return
        main = torch.cuda.current_stream(self.device)
        side = self.side if (self.side is not None and has_static and has_dynamic) else None
        att = (self.Kc, self.Vc, self.kv_len, K_cur, V_cur, self.scale, O)
        if side is not None:
            static_ids = [h for h, t in enumerate(types) if t == FKV_STATIC]
            side.wait_stream(main)
            with torch.cuda.stream(side):
                if self.static_in_place:
                    fkv_chunk_attention_static(shape, heads, Kh, Vh, frame_slot, Q, K_cur, V_cur, self.scale, O,
                                               lse, self.attn_ws2)
                else:
                    fkv_compress_static(shape, heads, Kh, Vh, frame_slot, self.Kc, self.Vc, self.kv_len)
                    fkv_chunk_attention_heads(shape, static_ids, Q, *att, lse=lse, workspace=self.attn_ws2)
            for t in (Kh, Vh, Q, K_cur, V_cur, O) + ((lse,) if lse is not None else ()):
                t.record_stream(side)
        elif has_static:
            fkv_compress_static(shape, heads, Kh, Vh, frame_slot, self.Kc, self.Vc, self.kv_len)
        if has_dynamic:
            if pooled is not None:
                fkv_select_compact_pooled(shape, heads, pooled, Kh, Vh, frame_slot, kept, self.Kc, self.Vc,
                                          self.kv_len)
            else:
                if incremental and H > 0:
                    fkv_score_segments_cached(shape, heads, Kh, frame_slot, K_cur, self._stats[layer], scores,
                                              self.score_ws)
                else:
                    fkv_score_segments(shape, heads, Kh, frame_slot, K_cur, scores, self.score_ws)
                fkv_select_compact(shape, heads, scores, Kh, Vh, frame_slot, kept, self.Kc, self.Vc,
                                   self.kv_len)
        if side is not None:
            dynamic_ids = [h for h, t in enumerate(types) if t == FKV_DYNAMIC]
            fkv_chunk_attention_heads(shape, dynamic_ids, Q, *att, lse=lse, workspace=self.attn_ws)
            main.wait_stream(side)
        else:
            fkv_chunk_attention(shape, Q, *att, lse, self.attn_ws)

    def append(self, layer: int, K_new, V_new, dst_slots):
        """Write a finished chunk's frames ([n_heads][n*F][d]) into the layer's cache slots."""
        fkv_append_frames(self.shape(0), K_new, V_new, dst_slots, self.K_hist[layer], self.V_hist[layer])


class _Budget:
    def __init__(self, type, sink_frames, recent_frames, keep_k, scope):
        self.type, self.sink_frames, self.recent_frames, self.keep_k, self.scope = \
            type, sink_frames, recent_frames, keep_k, scope
