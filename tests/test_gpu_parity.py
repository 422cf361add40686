"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Compression (scores, kept segment ids, kv_len, compacted K/V) must be
bit-exact; attention must be within max-abs 2e-2 and relative-L2 1e-2 for
bf16 (1e-4 / 1e-5 for fp32), with the log-normaliser checked too.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import (assert_attention_close, assert_compression_exact, check_layer,
                         dev_inputs, from_dev, make_layer, run_gpu, sample_rows, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2605_09681_amd as fkv
    fkv.lib()
    oracle.lib()


def _print_case(name, **kw):
    print(f"[gpu case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


# ---------------------------------------------------------------------------
# the workloads: tiny fp32, 480P and 1080P layers
# ---------------------------------------------------------------------------
def test_tiny_fp32_full():
    cfg = W.tiny_config()
    _print_case("tiny-fp32", seed=0)
    x = W.make_layer_inputs(cfg, seed=0)
    check_layer(cfg, x)


def test_480p_layer():
    cfg = W.wan_layer_config("480p")
    _print_case("480p", seed=0)
    x = W.make_layer_inputs(cfg, seed=0)
    _, _, _, (max_abs, rel) = check_layer(cfg, x, rows=sample_rows(cfg.lq, 64))
    print(f"480p attention max_abs={max_abs:.2e} rel_l2={rel:.2e}")


def test_480p_sharp_logits():
    """Queries scaled by 6 (logits ~ N(0, 36)): outputs are O(1), so the
    absolute bound is meaningful."""
    cfg = W.wan_layer_config("480p")
    _print_case("480p-sharp", seed=1)
    x = W.make_layer_inputs(cfg, seed=1, q_scale=6.0)
    check_layer(cfg, x, rows=sample_rows(cfg.lq, 32, seed=1))


def test_1080p_layer():
    cfg = W.wan_layer_config("1080p")
    _print_case("1080p", seed=0)
    x = W.make_layer_inputs(cfg, seed=0)
    check_layer(cfg, x, rows=sample_rows(cfg.lq, 8))


# ---------------------------------------------------------------------------
# several tiles with ragged tails, every row checked
# ---------------------------------------------------------------------------
def _small(F=100, L=25, H=7, cap=9, C=2, d=128, dtype="bf16", heads=None, rho=0.85):
    heads = heads or (W.HeadBudget(W.STATIC, 1, 2), W.HeadBudget(W.DYNAMIC, 1, 0, 2, W.SCOPE_FRAME),
                      W.HeadBudget(W.DYNAMIC, 0, 1, 3, W.SCOPE_GLOBAL), W.HeadBudget(W.STATIC, 2, 0))
    return W.LayerConfig("small", len(heads), d, F, H, cap, C, L, dtype, tuple(heads), rho)


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("F,L", [(100, 25), (100, 50), (100, 100), (100, 200), (100, 300)])
def test_small_all_rows(d, F, L):
    heads = (W.HeadBudget(W.STATIC, 1, 2), W.HeadBudget(W.DYNAMIC, 1, 0, 2, W.SCOPE_FRAME if L < F else W.SCOPE_GLOBAL),
             W.HeadBudget(W.DYNAMIC, 0, 1, 3, W.SCOPE_GLOBAL), W.HeadBudget(W.STATIC, 2, 0))
    cfg = _small(F=F, L=L, d=d, heads=heads)
    slot = np.array([3, 0, 8, 1, 5, 2, 7], np.int32)   # a permuted ring; slots 4, 6 hold noise
    _print_case("small", d=d, F=F, L=L)
    x = W.make_layer_inputs(cfg, seed=d + L, frame_slot=slot)
    check_layer(cfg, x)


@pytest.mark.parametrize("d", [128, 64])
def test_small_per_item_schedule(d):
    """Attention without a workspace: one workgroup per (head, query tile)."""
    cfg = _small(F=100, L=25, d=d)
    slot = np.array([3, 0, 8, 1, 5, 2, 7], np.int32)
    _print_case("small-per-item", d=d)
    check_layer(cfg, W.make_layer_inputs(cfg, seed=d + 1, frame_slot=slot), balanced=False)


def test_balanced_many_items():
    """48 heads with ragged budgets and 2 query tiles each: the balanced
    schedule gives workgroups several whole items plus cut ones, every row
    checked."""
    heads = tuple(W.HeadBudget(W.STATIC, h % 2, h % 7) if h % 3 else
                  W.HeadBudget(W.DYNAMIC, 1, h % 2, 1 + h % 9, W.SCOPE_GLOBAL) for h in range(48))
    cfg = W.LayerConfig("many", 48, 64, 128, 12, 12, 4, 128, "bf16", heads, 0.9)
    _print_case("balanced-many")
    check_layer(cfg, W.make_layer_inputs(cfg, seed=21))


def test_schedules_agree_480p():
    """Balanced and per-item schedules on the 480P layer agree to rounding:
    split parts round their probabilities against their own running max and
    sum in another order, so outputs may differ by one bf16 step plus a small
    absolute amount near zero."""
    cfg = W.wan_layer_config("480p")
    _print_case("480p-schedules")
    x = W.make_layer_inputs(cfg, seed=2)
    _, Ob, lb = run_gpu(cfg, x, balanced=True)
    _, Ou, lu = run_gpu(cfg, x, balanced=False)
    ob = W.bf16_bits_to_f32(from_dev(Ob)).astype(np.float64)
    ou = W.bf16_bits_to_f32(from_dev(Ou)).astype(np.float64)
    tol = np.abs(ou) * 2.0 ** -7 + 2e-4
    assert (np.abs(ob - ou) <= tol).all(), float(np.abs(ob - ou).max())
    # Each schedule's normaliser sums probabilities rounded to bf16 against its
    # own running maxima: each is within a relative 2^-9 of the exact sum, so
    # the two lse differ by at most 2 * -log(1 - 2^-9) (+1e-4 for the score
    # accumulation order).  With independent roundings of n_eff >= 1000
    # effective terms, each sum's relative error has standard deviation at most
    # 2^-9 / sqrt(3 * 1000) = 3.6e-5, so the RMS difference stays below 1e-4.
    dl = from_dev(lb).astype(np.float64) - from_dev(lu).astype(np.float64)
    bound = -2 * math.log1p(-2.0 ** -9) + 1e-4
    rms = float(np.sqrt(np.mean(dl ** 2)))
    assert float(np.abs(dl).max()) <= bound and rms <= 1e-4, (float(np.abs(dl).max()), rms)


def test_small_fp32_multitile():
    cfg = _small(F=48, L=16, H=5, cap=6, C=3, d=64, dtype="f32")
    _print_case("small-fp32")
    x = W.make_layer_inputs(cfg, seed=3)
    check_layer(cfg, x)


# ---------------------------------------------------------------------------
# the keep-fraction / segment-length sweep at 480P
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("L", [390, 1560, 4680])
@pytest.mark.parametrize("frac", [0.25, 0.5, 0.75, 1.0])
def test_480p_sweep(L, frac):
    cfg = W.wan_layer_config("480p", keep_fraction=frac, seg_tokens=L)
    _print_case("480p-sweep", L=L, frac=frac)
    x = W.make_layer_inputs(cfg, seed=5)
    check_layer(cfg, x, rows=sample_rows(cfg.lq, 8, seed=L))


def test_480p_many_segments():
    """168 segments per head (an eighth of a frame each, per-frame groups): more
    than the fused select + compact kernel takes, so the selection kernel and
    the copy kernel run separately."""
    cfg = W.wan_layer_config("480p", keep_fraction=0.5, seg_tokens=195)
    assert cfg.hist_frames * cfg.frame_tokens // cfg.seg_tokens == 168
    _print_case("480p-168-segments")
    x = W.make_layer_inputs(cfg, seed=15)
    check_layer(cfg, x, rows=sample_rows(cfg.lq, 8, seed=15))


@pytest.mark.parametrize("case", ["small", "small-d64", "small-f32", "480p", "480p-gather", "1080p"])
def test_pipelined_step(case):
    """CompressedLayer.step: the static heads' attention on a side stream --
    read in place from the cache (bf16), or gathered first (fp32, and the
    480p-gather case) -- while the dynamic heads are scored, compacted and
    attended on the main stream, each stream with its own workspace.  Same
    parity bar as the serial path; the small case interleaves head types."""
    if case.startswith("small"):
        cfg = _small(F=100, L=25, d=64 if case == "small-d64" else 128, dtype="f32" if case == "small-f32" else "bf16")
        x = W.make_layer_inputs(cfg, seed=30, frame_slot=np.array([3, 0, 8, 1, 5, 2, 7], np.int32))
        rows = None
    else:
        cfg = W.wan_layer_config("1080p" if case == "1080p" else "480p")
        slot = np.roll(np.arange(cfg.hist_frames, dtype=np.int32), 3) if case == "1080p" else None
        x = W.make_layer_inputs(cfg, seed=31, frame_slot=slot)
        rows = sample_rows(cfg.lq, 8 if case != "1080p" else 4, seed=31)
    _print_case("pipelined-step", case=case)
    layer = make_layer(cfg, in_place=False if case == "480p-gather" else None, step_mode="compact")
    assert layer.side is not None and (cfg.dtype == "f32" or layer.attn_workspace2 is not None)
    assert layer.static_in_place == (cfg.dtype == "bf16" and case != "480p-gather")
    d = dev_inputs(x)
    O = torch.empty_like(d["Q"])
    lse = torch.empty((cfg.n_heads, cfg.lq), dtype=torch.float32, device="cuda")
    layer.step(d["K_hist"], d["V_hist"], x.frame_slot, d["Q"], d["K_cur"], d["V_cur"], O, lse)
    torch.cuda.synchronize()
    ref = oracle.run_layer(cfg, x, rows=rows, scale=1 / math.sqrt(cfg.head_dim))
    assert_compression_exact(cfg, layer, ref, skip_static=layer.static_in_place)
    assert_attention_close(O, ref, cfg.dtype, lse)


@pytest.mark.parametrize("balanced", [True, False])
def test_attention_heads_subset(balanced):
    """fkv_chunk_attention_heads computes exactly the listed heads (in any
    order) and leaves every other head's rows of O and lse as they were."""
    import paper_2605_09681_amd as fkv
    cfg = _small(F=100, L=25, d=64)
    x = W.make_layer_inputs(cfg, seed=32, frame_slot=np.array([3, 0, 8, 1, 5, 2, 7], np.int32))
    _print_case("attention-heads", balanced=balanced)
    layer = make_layer(cfg, balanced=balanced)
    d = dev_inputs(x)
    layer.compress(d["K_hist"], d["V_hist"], x.frame_slot, d["K_cur"])
    O = torch.full_like(d["Q"], 7.0)
    lse = torch.full((cfg.n_heads, cfg.lq), -3.0, dtype=torch.float32, device="cuda")
    listed = [3, 1]
    fkv.fkv_chunk_attention_heads(layer.shape, listed, d["Q"], layer.Kc, layer.Vc, layer.kv_len, d["K_cur"],
                                  d["V_cur"], layer.scale, O, lse, layer.attn_workspace)
    torch.cuda.synchronize()
    ref = oracle.run_layer(cfg, x, scale=layer.scale)
    Of, lf = from_dev(O), from_dev(lse)
    for h in range(cfg.n_heads):
        if h in listed:
            one = oracle.LayerResult(None, None, None, None, None, None, ref.rows, ref.O[h:h + 1], ref.lse[h:h + 1])
            assert_attention_close(O[h:h + 1], one, "bf16", lse[h:h + 1])
        else:
            assert (W.bf16_bits_to_f32(Of[h]) == 7.0).all() and (lf[h] == -3.0).all(), h


_PERM = np.array([3, 0, 8, 1, 5, 2, 7], np.int32)


@pytest.mark.parametrize("case", ["F100-d128", "F64-d64-per-item", "F80-budgets", "H0", "H2", "H200-cap256", "480p",
                                  "1080p"])
def test_attention_static_in_place(case):
    """fkv_chunk_attention_static reads the static heads' kept frames straight
    from the slot-permuted cache: bit for bit what fkv_compress_static followed
    by fkv_chunk_attention_heads over the static heads gives, the other heads'
    rows of O and lse untouched, and within the attention bar of the oracle.
    Frames of 100 and 80 tokens put frame boundaries inside key tiles; the
    budgets cover a full-history window, a sink longer than the history, an
    empty history window (chunk only) and a one-frame gap."""
    import paper_2605_09681_amd as fkv
    balanced, slot, rows = True, _PERM, None
    if case == "F100-d128":
        cfg = _small(F=100, L=25, d=128)
    elif case == "F64-d64-per-item":
        cfg, balanced = _small(F=64, L=16, d=64), False
    elif case == "F80-budgets":
        S, D = W.STATIC, W.DYNAMIC
        cfg = _small(F=80, L=20, d=128, heads=(
            W.HeadBudget(S, 0, 7), W.HeadBudget(D, 1, 0, 2, W.SCOPE_FRAME), W.HeadBudget(S, 9, 0),
            W.HeadBudget(S, 0, 0), W.HeadBudget(S, 3, 3), W.HeadBudget(S, 0, 1)))
    elif case == "H0":
        cfg, slot = _small(F=100, L=25, H=0, cap=4, d=64), np.zeros(0, np.int32)
    elif case == "H200-cap256":
        # more than 64 kept frames: slot bytes 1..3 of the lane table
        S, D = W.STATIC, W.DYNAMIC
        cfg = _small(F=64, L=32, H=200, cap=256, C=2, d=64, heads=(
            W.HeadBudget(S, 2, 190), W.HeadBudget(D, 1, 0, 1, W.SCOPE_FRAME), W.HeadBudget(S, 0, 200),
            W.HeadBudget(S, 70, 60)))
        slot = np.random.default_rng(7).permutation(256)[:200].astype(np.int32)
    elif case == "H2":
        cfg, slot = _small(F=72, L=24, H=2, cap=3, d=64, heads=(
            W.HeadBudget(W.STATIC, 3, 4), W.HeadBudget(W.DYNAMIC, 1, 0, 1, W.SCOPE_FRAME),
            W.HeadBudget(W.STATIC, 0, 1))), np.array([2, 0], np.int32)
    else:
        cfg = W.wan_layer_config(case)
        slot = np.roll(np.arange(cfg.hist_frames, dtype=np.int32), 5)    # a rotated ring
        rows = sample_rows(cfg.lq, 8 if case == "480p" else 4, seed=33)
    x = W.make_layer_inputs(cfg, seed=33, frame_slot=slot)
    _print_case("attention-static-in-place", case=case, balanced=balanced)
    static = [h for h, b in enumerate(cfg.heads) if b.type == W.STATIC]
    layer = make_layer(cfg, balanced=balanced)
    d = dev_inputs(x)
    fkv.fkv_compress_static(layer.shape, layer.heads, d["K_hist"], d["V_hist"], x.frame_slot, layer.Kc, layer.Vc,
                            layer.kv_len)
    O_ref = torch.full_like(d["Q"], 7.0)
    l_ref = torch.full((cfg.n_heads, cfg.lq), -3.0, dtype=torch.float32, device="cuda")
    fkv.fkv_chunk_attention_heads(layer.shape, static, d["Q"], layer.Kc, layer.Vc, layer.kv_len, d["K_cur"],
                                  d["V_cur"], layer.scale, O_ref, l_ref, layer.attn_workspace)
    O = torch.full_like(d["Q"], 7.0)
    lse = torch.full((cfg.n_heads, cfg.lq), -3.0, dtype=torch.float32, device="cuda")
    fkv.fkv_chunk_attention_static(layer.shape, layer.heads, d["K_hist"], d["V_hist"], x.frame_slot, d["Q"],
                                   d["K_cur"], d["V_cur"], layer.scale, O, lse, layer.attn_workspace)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(O), from_dev(O_ref))
    np.testing.assert_array_equal(from_dev(lse).view(np.uint32), from_dev(l_ref).view(np.uint32))
    ref = oracle.run_layer(cfg, x, rows=rows, scale=layer.scale)
    Of, lf = from_dev(O), from_dev(lse)
    for h in range(cfg.n_heads):
        if h in static:
            one = oracle.LayerResult(None, None, None, None, None, None, ref.rows, ref.O[h:h + 1], ref.lse[h:h + 1])
            assert_attention_close(O[h:h + 1], one, "bf16", lse[h:h + 1])
        else:
            assert (W.bf16_bits_to_f32(Of[h]) == 7.0).all() and (lf[h] == -3.0).all(), h


@pytest.mark.parametrize("dtype,F,L,pooled", [("bf16", 100, 25, False), ("bf16", 100, 100, False),
                                               ("bf16", 100, 300, False), ("f32", 100, 50, False),
                                               ("bf16", 100, 25, True), ("bf16", 100, 200, True),
                                               ("f32", 100, 100, True)])
def test_incremental_rescoring(dtype, F, L, pooled):
    """fkv_score_history once, then fkv_score_segments_cached for three
    different chunks K_cur: every score bit-exact with the oracle's full
    scoring of that step (per dynamic head, or pooled over all heads), for
    segments shorter than, equal to and longer than a frame."""
    import paper_2605_09681_amd as fkv
    cfg = _small(F=F, L=L, d=64, dtype=dtype)
    if L >= F:
        cfg = cfg.replace(heads=tuple(W.HeadBudget(b.type, b.sink_frames, b.recent_frames, b.keep_k, W.SCOPE_GLOBAL)
                                      for b in cfg.heads))
    slot = np.array([3, 0, 8, 1, 5, 2, 7], np.int32)
    x = W.make_layer_inputs(cfg, seed=40 + L, frame_slot=slot)
    _print_case("incremental", dtype=dtype, F=F, L=L, pooled=pooled)
    shape = fkv.make_shape(cfg.n_heads, cfg.head_dim, F, cfg.hist_frames, cfg.cap_frames, cfg.chunk_frames, L, dtype)
    heads = fkv.make_heads(cfg.heads)
    ws_bytes = fkv.fkv_score_pooled_workspace_size(shape) if pooled else fkv.fkv_score_workspace_size(shape, heads)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")   # scoring workspaces start zero-filled
    stats = torch.empty(fkv.fkv_score_stats_size(shape, heads, pooled) // 8, dtype=torch.float64, device="cuda")
    Kh = to_dev(x.K_hist, dtype)
    fkv.fkv_score_history(shape, heads, Kh, slot, stats, ws, pooled=pooled)
    n_seg = fkv.fkv_num_segments(shape)
    dyn = [h for h, b in enumerate(cfg.heads) if b.type == W.DYNAMIC]
    for step in range(3):
        Kq = W.normal_tensor(41, step, (cfg.n_heads, cfg.lq, cfg.head_dim), dtype) if step else x.K_cur
        scores = torch.full((n_seg,) if pooled else (cfg.n_heads, n_seg), 9.0, dtype=torch.float32, device="cuda")
        fkv.fkv_score_segments_cached(shape, heads, Kh, slot, to_dev(Kq, dtype), stats, scores, ws, pooled=pooled)
        torch.cuda.synchronize()
        got = from_dev(scores)
        if pooled:
            want, _ = oracle.score_pooled(x.K_hist, slot, Kq, cfg.hist_frames, L)
            np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32), err_msg=f"step {step}")
        else:
            for h in range(cfg.n_heads):
                if h in dyn:
                    want, _ = oracle.score_head(x.K_hist[h], slot, Kq[h], cfg.hist_frames, L)
                    np.testing.assert_array_equal(got[h].view(np.uint32), want.view(np.uint32),
                                                  err_msg=f"step {step} head {h}")
                else:
                    assert (got[h] == 9.0).all(), h


def test_480p_no_pruning_equals_full_attention():
    """Keep everything (dynamic f = 1, static recent = H): both head types
    reduce to full attention over the uncompressed cache."""
    cfg = W.wan_layer_config("480p", keep_fraction=1.0, static_recent=21)
    _print_case("480p-full")
    x = W.make_layer_inputs(cfg, seed=6)
    layer, O, lse = run_gpu(cfg, x)
    rows = sample_rows(cfg.lq, 16, seed=6)
    kv = from_dev(layer.kv_len)
    assert (kv == 21 * cfg.frame_tokens).all()
    full = [oracle.attention_rows(x.Q[h], x.K_hist[h].reshape(-1, 128), x.V_hist[h].reshape(-1, 128),
                                  x.K_cur[h], x.V_cur[h], 1 / math.sqrt(128), rows) for h in range(12)]
    ref = oracle.LayerResult(None, None, None, None, None, None, rows,
                             np.stack([f[0] for f in full]), np.stack([f[1] for f in full]))
    assert_attention_close(O, ref, "bf16", lse)


def test_ragged_budgets():
    """Per-head budgets drawn from a seed: sink 0..2, recent 0..6, k and scope
    per dynamic head -- ragged kv_len across heads."""
    rng = np.random.default_rng(11)
    heads = []
    for h in range(12):
        if rng.random() < 0.5:
            heads.append(W.HeadBudget(W.STATIC, int(rng.integers(0, 3)), int(rng.integers(0, 7))))
        else:
            scope = W.SCOPE_FRAME if rng.random() < 0.5 else W.SCOPE_GLOBAL
            k = int(rng.integers(0, 5 if scope == W.SCOPE_FRAME else 21))
            heads.append(W.HeadBudget(W.DYNAMIC, int(rng.integers(0, 3)), int(rng.integers(0, 3)), k, scope))
    cfg = W.wan_layer_config("480p", seg_tokens=390).replace(heads=tuple(heads))
    _print_case("ragged")
    x = W.make_layer_inputs(cfg, seed=11)
    check_layer(cfg, x, rows=sample_rows(cfg.lq, 8, seed=11))


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------
def test_first_step_empty_history():
    """H = 0 (the first AR step): nothing to compress, attention over the chunk only."""
    cfg = _small(H=0, cap=4)
    _print_case("H=0")
    x = W.make_layer_inputs(cfg, seed=7)
    layer, O, ref, _ = check_layer(cfg, x)
    assert (from_dev(layer.kv_len) == 0).all()


@pytest.mark.parametrize("H", [1, 2])
def test_short_history(H):
    """Sink and recent windows overlapping or exceeding a 1-2 frame history."""
    heads = (W.HeadBudget(W.STATIC, 3, 4), W.HeadBudget(W.DYNAMIC, 1, 0, 5, W.SCOPE_FRAME),
             W.HeadBudget(W.DYNAMIC, 2, 2, 1, W.SCOPE_GLOBAL), W.HeadBudget(W.STATIC, 0, 1))
    cfg = _small(H=H, cap=3, heads=heads)
    _print_case("short", H=H)
    check_layer(cfg, W.make_layer_inputs(cfg, seed=8 + H))


def test_empty_budgets():
    """recent = sink = 0 and k = 0 (the ablations that drop one head type's
    cache): kv_len = 0, attention over the chunk alone."""
    heads = (W.HeadBudget(W.STATIC, 0, 0), W.HeadBudget(W.DYNAMIC, 0, 0, 0, W.SCOPE_GLOBAL),
             W.HeadBudget(W.DYNAMIC, 0, 0, 0, W.SCOPE_FRAME), W.HeadBudget(W.STATIC, 1, 0))
    cfg = _small(heads=heads)
    _print_case("empty-budgets")
    layer, _, _, _ = check_layer(cfg, W.make_layer_inputs(cfg, seed=9))
    assert from_dev(layer.kv_len).tolist() == [0, 0, 0, 100]


@pytest.mark.parametrize("F,L,H", [(64, 16, 6), (64, 4, 10)])
def test_select_crafted_scores(F, L, H):
    """fkv_select_compact on crafted scores: ties, signed zeros and NaNs, with
    24 segments (selection inside the compaction kernel) and 160 segments
    (separate selection kernel)."""
    _print_case("crafted", F=F, L=L, H=H)
    heads = (W.HeadBudget(W.DYNAMIC, 0, 0, 5, W.SCOPE_GLOBAL), W.HeadBudget(W.DYNAMIC, 1, 1, 2, W.SCOPE_FRAME),
             W.HeadBudget(W.DYNAMIC, 0, 0, 7, W.SCOPE_GLOBAL), W.HeadBudget(W.DYNAMIC, 0, 2, 3, W.SCOPE_GLOBAL))
    cfg = W.LayerConfig("crafted", 4, 64, F, H, H, 1, L, "bf16", heads)
    x = W.make_layer_inputs(cfg, seed=10)
    n = H * F // L
    rng = np.random.default_rng(10)
    # NaNs of both signs (the sign bit must not order them), signed zeros, infinities
    palette = np.array([0.5, 0.0, -0.0, np.nan, -np.nan, 0.25, 0.5, -1.0, np.inf, -np.inf], np.float32)
    scores = palette[rng.integers(0, len(palette), (4, n))].astype(np.float32)
    scores[0] = 0.75                                    # all equal
    layer = make_layer(cfg)
    d = dev_inputs(x)
    layer.scores.copy_(torch.from_numpy(scores))
    layer.select_compact(d["K_hist"], d["V_hist"], x.frame_slot)
    torch.cuda.synchronize()
    kept = from_dev(layer.kept_seg)
    for h, b in enumerate(heads):
        want, cnt = oracle.select_head(scores[h], H, F, L, b.sink_frames, b.recent_frames, b.keep_k, b.scope)
        np.testing.assert_array_equal(kept[h], want, err_msg=f"head {h}")
        kc = oracle.compact_head(x.K_hist[h], x.frame_slot, want[:cnt], H, L)
        assert int(from_dev(layer.kv_len)[h]) == kc.shape[0]
        np.testing.assert_array_equal(from_dev(layer.Kc)[h, :kc.shape[0]], kc)
    assert kept[0, :5].tolist() == [0, 1, 2, 3, 4]


def test_determinism():
    """Two runs give bit-identical scores, kept sets, compacted K/V and output."""
    cfg = W.wan_layer_config("480p", seg_tokens=390)
    _print_case("determinism")
    x = W.make_layer_inputs(cfg, seed=12)
    a = run_gpu(cfg, x)
    b = run_gpu(cfg, x)
    for name in ("scores", "kept_seg", "kv_len", "Kc", "Vc"):
        np.testing.assert_array_equal(from_dev(getattr(a[0], name)), from_dev(getattr(b[0], name)), err_msg=name)
    np.testing.assert_array_equal(from_dev(a[1]), from_dev(b[1]))
    np.testing.assert_array_equal(from_dev(a[2]), from_dev(b[2]))


@pytest.mark.parametrize("mode", ["paged", "paged2", "compact"])
def test_determinism_pipelined_step(mode):
    """Every step mode gives the same bits on repeated runs: the one-launch
    scoring reduces in a fixed order, the two-stream steps touch disjoint heads
    on their streams, each with its own workspace, and nothing depends on how
    they interleave."""
    cfg = W.wan_layer_config("480p")
    _print_case("determinism-step", mode=mode)
    x = W.make_layer_inputs(cfg, seed=13)
    d = dev_inputs(x)
    layer = make_layer(cfg, step_mode=mode)
    assert layer.static_in_place and layer.side is not None
    outs = []
    for _ in range(3):
        O = torch.empty_like(d["Q"])
        lse = torch.empty((cfg.n_heads, cfg.lq), dtype=torch.float32, device="cuda")
        layer.step(d["K_hist"], d["V_hist"], x.frame_slot, d["Q"], d["K_cur"], d["V_cur"], O, lse)
        torch.cuda.synchronize()
        outs.append((from_dev(O), from_dev(lse), from_dev(layer.scores), from_dev(layer.kept_seg)))
    for run in outs[1:]:
        for a, b in zip(run, outs[0]):
            np.testing.assert_array_equal(a.view(np.uint8), b.view(np.uint8))


def test_api_errors_on_gpu():
    """Host-side validation rejects a short slab before anything runs."""
    import paper_2605_09681_amd as fkv
    cfg = W.wan_layer_config("480p")
    layer = make_layer(cfg, slab=100)
    x = W.make_layer_inputs(_small(), seed=0)
    with pytest.raises(fkv.FkvError) as e:
        fkv.fkv_compress_static(layer.shape, layer.heads,
                                torch.zeros((12, 21, 1560, 128), dtype=torch.bfloat16, device="cuda"),
                                torch.zeros((12, 21, 1560, 128), dtype=torch.bfloat16, device="cuda"),
                                np.arange(21, dtype=np.int32), layer.Kc, layer.Vc, layer.kv_len)
    assert e.value.status == fkv.FKV_ERR_CAPACITY


def test_attention_workspace_capacity_on_gpu():
    """A balanced-schedule workspace one byte short is rejected before any
    launch by every bf16 attention entry point, the in-place static one
    included; the output is left untouched."""
    import paper_2605_09681_amd as fkv
    cfg = _small(F=100, L=25, d=64)
    x = W.make_layer_inputs(cfg, seed=3, frame_slot=_PERM)
    layer = make_layer(cfg)
    d = dev_inputs(x)
    need = fkv.fkv_attention_workspace_size(layer.shape)
    short = torch.zeros(need - 1, dtype=torch.uint8, device="cuda")
    O = torch.full_like(d["Q"], 5.0)
    calls = (
        lambda: fkv.fkv_chunk_attention(layer.shape, d["Q"], layer.Kc, layer.Vc, layer.kv_len, d["K_cur"],
                                        d["V_cur"], layer.scale, O, workspace=short),
        lambda: fkv.fkv_chunk_attention_heads(layer.shape, [0, 3], d["Q"], layer.Kc, layer.Vc, layer.kv_len,
                                              d["K_cur"], d["V_cur"], layer.scale, O, workspace=short),
        lambda: fkv.fkv_chunk_attention_static(layer.shape, layer.heads, d["K_hist"], d["V_hist"], x.frame_slot,
                                               d["Q"], d["K_cur"], d["V_cur"], layer.scale, O, workspace=short),
    )
    for call in calls:
        with pytest.raises(fkv.FkvError) as e:
            call()
        assert e.value.status == fkv.FKV_ERR_CAPACITY
    torch.cuda.synchronize()
    assert (W.bf16_bits_to_f32(from_dev(O)) == 5.0).all()


# ---------------------------------------------------------------------------
# streaming rollout with a ring-buffer cache (sampled units)
# ---------------------------------------------------------------------------
def test_rollout_ring_buffer_sampled():
    """A 10-chunk rollout at 480P with a rolling 21-frame cache (sink pinned in
    slot 0): the cache is written through the ring map, each chunk's step is
    checked on a sampled layer.  Per-layer head masks and rho are seeded."""
    F, C, window = 1560, 3, 21
    masks = W.rollout_head_masks(0, n_layers=2)
    rhos = W.rollout_rhos(0, n_layers=2)
    for chunk in (1, 4, 7, 9):
        slots = W.ring_frame_slots(chunk, C, window)
        H = len(slots)
        layer_idx = chunk % 2
        heads = tuple(W.HeadBudget(W.DYNAMIC, 1, 0, (H - 1) // 2, W.SCOPE_GLOBAL) if m == W.DYNAMIC
                      else W.HeadBudget(W.STATIC, 1, 6) for m in masks[layer_idx])
        cfg = W.wan_layer_config("480p").replace(hist_frames=H, heads=heads, rho=tuple(rhos[layer_idx]))
        _print_case("rollout", chunk=chunk, H=H)
        x = W.make_layer_inputs(cfg, seed=100 + chunk, frame_slot=slots, extra=(chunk, layer_idx))
        check_layer(cfg, x, rows=sample_rows(cfg.lq, 4, seed=chunk))


# ---------------------------------------------------------------------------
# the first-block proxy (Sec. 4.3): one similarity row pooled over all heads,
# reused by the dynamic heads of another layer
# ---------------------------------------------------------------------------
def _pooled_gpu(cfg, x):
    import paper_2605_09681_amd as fkv
    shape = fkv.make_shape(cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames,
                           cfg.cap_frames, cfg.chunk_frames, cfg.seg_tokens, cfg.dtype)
    d = dev_inputs(x)
    scores = torch.full((fkv.fkv_num_segments(shape),), float("nan"), dtype=torch.float32, device="cuda")
    fkv.fkv_score_pooled(shape, d["K_hist"], x.frame_slot, d["K_cur"], scores)
    torch.cuda.synchronize()
    return from_dev(scores)


def test_pooled_scores_480p():
    cfg = W.wan_layer_config("480p")
    _print_case("pooled-480p", seed=13)
    x = W.make_layer_inputs(cfg, seed=13)
    got = _pooled_gpu(cfg, x)
    want, _ = oracle.score_pooled(x.K_hist, x.frame_slot, x.K_cur, cfg.hist_frames, cfg.seg_tokens)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("F,L", [(100, 25), (100, 100), (100, 300)])
def test_pooled_scores_small(dtype, F, L):
    cfg = _small(F=F, L=L, d=64, dtype=dtype)
    slot = np.array([3, 0, 8, 1, 5, 2, 7], np.int32)
    _print_case("pooled-small", dtype=dtype, F=F, L=L)
    x = W.make_layer_inputs(cfg, seed=L + 1, frame_slot=slot)
    got = _pooled_gpu(cfg, x)
    want, _ = oracle.score_pooled(x.K_hist, x.frame_slot, x.K_cur, cfg.hist_frames, L)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


def test_pooled_scores_reused_by_another_layer():
    """Scores pooled from one layer's keys select the segments of a second
    layer with other head types and budgets (fkv_select_compact_pooled):
    kept ids, kv_len and compacted K/V bit-exact, then attention."""
    import paper_2605_09681_amd as fkv
    first = W.wan_layer_config("480p", seg_tokens=390)
    _print_case("pooled-reuse")
    x0 = W.make_layer_inputs(first, seed=14)
    pooled = _pooled_gpu(first, x0)
    heads = tuple(W.HeadBudget(W.DYNAMIC, 1, 0, 2, W.SCOPE_FRAME) if h % 3 else W.HeadBudget(W.STATIC, 1, 6)
                  for h in range(12))
    cfg = first.replace(heads=heads)
    x = W.make_layer_inputs(cfg, seed=15)
    layer = make_layer(cfg)
    d = dev_inputs(x)
    fkv.fkv_select_compact_pooled(layer.shape, layer.heads, torch.from_numpy(pooled).cuda(), d["K_hist"],
                                  d["V_hist"], x.frame_slot, layer.kept_seg, layer.Kc, layer.Vc, layer.kv_len)
    layer.compress_static(d["K_hist"], d["V_hist"], x.frame_slot)
    O = torch.empty_like(d["Q"])
    layer.attention(d["Q"], d["K_cur"], d["V_cur"], O)
    torch.cuda.synchronize()
    kept, kv = from_dev(layer.kept_seg), from_dev(layer.kv_len)
    Kc, Vc = from_dev(layer.Kc), from_dev(layer.Vc)
    H, F, L = cfg.hist_frames, cfg.frame_tokens, cfg.seg_tokens
    rows = sample_rows(cfg.lq, 4, seed=15)
    outs = []
    for h, b in enumerate(heads):
        if b.type == W.DYNAMIC:
            want, cnt = oracle.select_head(pooled, H, F, L, b.sink_frames, b.recent_frames, b.keep_k, b.scope)
            np.testing.assert_array_equal(kept[h], want, err_msg=f"head {h}")
            kc = oracle.compact_head(x.K_hist[h], x.frame_slot, want[:cnt], H, L)
            vc = oracle.compact_head(x.V_hist[h], x.frame_slot, want[:cnt], H, L)
        else:
            frames = oracle.static_frames(H, b.sink_frames, b.recent_frames)
            kc = oracle.gather_frames(x.K_hist[h], x.frame_slot, frames)
            vc = oracle.gather_frames(x.V_hist[h], x.frame_slot, frames)
        assert int(kv[h]) == kc.shape[0]
        np.testing.assert_array_equal(Kc[h, :kc.shape[0]], kc)
        np.testing.assert_array_equal(Vc[h, :kc.shape[0]], vc)
        outs.append(oracle.attention_rows(x.Q[h], kc, vc, x.K_cur[h], x.V_cur[h], 1 / math.sqrt(128), rows))
    ref = oracle.LayerResult(None, None, None, None, None, None, rows,
                             np.stack([o[0] for o in outs]), np.stack([o[1] for o in outs]))
    assert_attention_close(O, ref, "bf16")


# ---------------------------------------------------------------------------
# rolling cache maintained on the GPU through fkv_append_frames
# ---------------------------------------------------------------------------
def test_append_frames_bit_exact():
    import paper_2605_09681_amd as fkv
    cfg = _small(H=5, cap=7, C=3, d=64)
    _print_case("append")
    x = W.make_layer_inputs(cfg, seed=31)
    layer = make_layer(cfg)
    d = dev_inputs(x)
    dst = [6, 2, 4]
    fkv.fkv_append_frames(layer.shape, d["K_cur"], d["V_cur"], dst, d["K_hist"], d["V_hist"])
    torch.cuda.synchronize()
    K, V = x.K_hist.copy(), x.V_hist.copy()
    F = cfg.frame_tokens
    for h in range(cfg.n_heads):
        oracle.append_frames(K[h], x.K_cur[h].reshape(3, F, -1), np.array(dst, np.int32))
        oracle.append_frames(V[h], x.V_cur[h].reshape(3, F, -1), np.array(dst, np.int32))
    np.testing.assert_array_equal(from_dev(d["K_hist"]), K)
    np.testing.assert_array_equal(from_dev(d["V_hist"]), V)


def test_gpu_rollout_with_rolling_cache():
    """Eight chunks of a streaming rollout (window 7 frames, sink pinned,
    2-frame chunks): the cache lives on the GPU and is advanced by
    fkv_append_frames; the oracle keeps its own copy through its own append.
    Every chunk's step (compression bit-exact, attention on every row) is
    checked, across the point where the ring starts to rotate."""
    import paper_2605_09681_amd as fkv
    window, C, F, d, nh = 7, 2, 64, 64, 4
    n_chunks = 8
    heads = (W.HeadBudget(W.STATIC, 1, 2), W.HeadBudget(W.DYNAMIC, 1, 0, 1, W.SCOPE_FRAME),
             W.HeadBudget(W.DYNAMIC, 1, 0, 2, W.SCOPE_GLOBAL), W.HeadBudget(W.STATIC, 1, 1))
    keys = W.ar1_key_frames(40, nh, n_chunks * C, F, d, 0.9, "bf16")       # [nh][frames][F][d]
    vals = W.normal_tensor(40, 7, (nh, n_chunks * C, F, d), "bf16")
    qs = W.normal_tensor(40, 8, (nh, n_chunks * C * F, d), "bf16")
    K_o = np.zeros((nh, window, F, d), np.uint16)
    V_o = np.zeros((nh, window, F, d), np.uint16)
    K_g = torch.zeros((nh, window, F, d), dtype=torch.bfloat16, device="cuda")
    V_g = torch.zeros_like(K_g)
    for i in range(n_chunks):
        slots = W.ring_frame_slots(i, C, window)
        H = len(slots)
        cfg = W.LayerConfig("roll", nh, d, F, H, window, C, 16, "bf16", heads, 0.9)
        Kq = np.ascontiguousarray(keys[:, i * C:(i + 1) * C].reshape(nh, C * F, d))
        Vq = np.ascontiguousarray(vals[:, i * C:(i + 1) * C].reshape(nh, C * F, d))
        Q = np.ascontiguousarray(qs[:, i * C * F:(i + 1) * C * F])
        x = W.LayerInputs(cfg, K_o.copy(), V_o.copy(), Kq, Vq, Q, slots)
        _print_case("gpu-rollout", chunk=i, H=H)
        layer = make_layer(cfg)
        Kq_d, Vq_d, Q_d = to_dev(Kq, "bf16"), to_dev(Vq, "bf16"), to_dev(Q, "bf16")
        O = torch.empty_like(Q_d)
        lse = torch.empty((nh, C * F), dtype=torch.float32, device="cuda")
        layer.step(K_g, V_g, slots, Q_d, Kq_d, Vq_d, O, lse)
        torch.cuda.synchronize()
        ref = oracle.run_layer(cfg, x, scale=1 / math.sqrt(d))
        assert_compression_exact(cfg, layer, ref, skip_static=layer.static_in_place)
        assert_attention_close(O, ref, "bf16", lse)
        dst = W.chunk_write_slots(i, C, window)
        fkv.fkv_append_frames(layer.shape, Kq_d, Vq_d, dst.tolist(), K_g, V_g)
        for h in range(nh):
            oracle.append_frames(K_o[h], Kq[h].reshape(C, F, d), dst)
            oracle.append_frames(V_o[h], Vq[h].reshape(C, F, d), dst)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(K_g), K_o)
    np.testing.assert_array_equal(from_dev(V_g), V_o)


# ---------------------------------------------------------------------------
# comparison policies through the same kernels
# ---------------------------------------------------------------------------
def test_streaming_llm_budgets():
    """3 sink + 4 recent frames on every head (frame-level StreamingLLM)."""
    cfg = W.wan_layer_config("480p").replace(heads=W.streaming_llm_heads(12))
    _print_case("streaming-llm")
    layer, _, _, _ = check_layer(cfg, W.make_layer_inputs(cfg, seed=16), rows=sample_rows(cfg.lq, 8, seed=16))
    assert (from_dev(layer.kv_len) == 7 * cfg.frame_tokens).all()


@pytest.mark.parametrize("policy", ["random", "uniform"])
def test_random_and_uniform_segment_pruning(policy):
    """BottomK fed with seeded random scores (random pruning) or an evenly
    spaced pattern (uniform pruning) instead of similarities."""
    cfg = W.wan_layer_config("480p", seg_tokens=260, keep_fraction=0.7)   # 6 segments per frame
    _print_case("pruning-policy", policy=policy)
    x = W.make_layer_inputs(cfg, seed=17)
    n_seg = cfg.hist_frames * 6
    dyn = [h for h, b in enumerate(cfg.heads) if b.type == W.DYNAMIC]
    k = cfg.heads[dyn[0]].keep_k
    scores = (W.random_scores(17, 12, n_seg) if policy == "random"
              else W.uniform_scores(12, cfg.hist_frames, cfg.frame_tokens, 260, k))
    layer = make_layer(cfg)
    d = dev_inputs(x)
    layer.scores.copy_(torch.from_numpy(scores))
    layer.select_compact(d["K_hist"], d["V_hist"], x.frame_slot)
    torch.cuda.synchronize()
    kept, kv, Kc = from_dev(layer.kept_seg), from_dev(layer.kv_len), from_dev(layer.Kc)
    for h in dyn:
        b = cfg.heads[h]
        want, cnt = oracle.select_head(scores[h], cfg.hist_frames, cfg.frame_tokens, 260, b.sink_frames,
                                       b.recent_frames, b.keep_k, b.scope)
        np.testing.assert_array_equal(kept[h], want)
        kc = oracle.compact_head(x.K_hist[h], x.frame_slot, want[:cnt], cfg.hist_frames, 260)
        assert int(kv[h]) == kc.shape[0]
        np.testing.assert_array_equal(Kc[h, :kc.shape[0]], kc)
        if policy == "uniform":   # kept segments within every non-sink frame: 0, 1, 3, 4 of 6 (k = 4)
            sel = want[:cnt]
            assert sorted(set((sel[sel >= 6] % 6).tolist())) == sorted({(i * 6) // k for i in range(k)})


# ---------------------------------------------------------------------------
# the layer-stack rollout driver
# ---------------------------------------------------------------------------
def _stack_budgets(mask_row, H, F, L):
    """Per-head budgets of one layer for history length H: static heads keep the
    sink and the last two frames, dynamic heads the sink plus half of the
    candidate segments (one global group)."""
    n_seg = (H * F + L - 1) // L
    k = max((n_seg - (F + L - 1) // L) // 2, 0)
    return tuple(W.HeadBudget(W.DYNAMIC, 1, 0, k, W.SCOPE_GLOBAL) if m == W.DYNAMIC else
                 W.HeadBudget(W.STATIC, 1, 2) for m in mask_row)


@pytest.mark.parametrize("pooled,incremental", [(False, False), (True, False), (False, True), (True, True)])
def test_rollout_stack(pooled, incremental):
    """RolloutStack: 3 layers with their own head masks and rolling caches
    (window 7, sink pinned, 2-frame chunks) over 6 chunks of 2 AR steps, across
    the ring wrap, sharing one set of compressed buffers.  Every layer's step is
    checked against the oracle (compression bit-exact, attention on every row);
    with pooled=True the dynamic heads of every layer select with the score row
    pooled over all heads of layer 0 (the first-block proxy); with
    incremental=True the scores come from per-chunk history statistics plus
    the pair touching the chunk (fkv_score_history once per chunk,
    fkv_score_segments_cached every step)."""
    import paper_2605_09681_amd as fkv
    from paper_2605_09681_amd.layer import RolloutStack
    from types import SimpleNamespace
    n_layers, nh, d, F, window, C, L = 3, 4, 64, 64, 7, 2, 32
    n_chunks, n_steps = 6, 2
    masks = W.rollout_head_masks(21, n_layers=n_layers, n_heads=nh, n_dynamic=2)
    stack = RolloutStack(n_layers, nh, d, F, window, C, L)
    K_o = np.zeros((n_layers, nh, window, F, d), np.uint16)
    V_o = np.zeros_like(K_o)
    for i in range(n_chunks):
        slots = W.ring_frame_slots(i, C, window)
        H = len(slots)
        if incremental:
            if pooled:
                stack.history(0, None, slots, pooled=True)
            else:
                for layer in range(n_layers):
                    stack.history(layer, _stack_budgets(masks[layer], H, F, L), slots)
        for step in range(n_steps):
            ex = (i, step)
            Kq = W.normal_tensor(22, 1, (nh, C * F, d), "bf16", extra=ex)
            Vq = W.normal_tensor(22, 2, (nh, C * F, d), "bf16", extra=ex)
            Q = W.normal_tensor(22, 3, (nh, C * F, d), "bf16", extra=ex)
            Kq_d, Vq_d, Q_d = to_dev(Kq, "bf16"), to_dev(Vq, "bf16"), to_dev(Q, "bf16")
            row = None
            if pooled and H > 0:
                row_d = stack.score_pooled(0, slots, Kq_d, incremental=incremental)
                row_want, _ = oracle.score_pooled(K_o[0], slots, Kq, H, L)
                torch.cuda.synchronize()
                np.testing.assert_array_equal(from_dev(row_d).view(np.uint32), row_want.view(np.uint32))
                row = row_d
            for layer in range(n_layers):
                _print_case("rollout-stack", pooled=pooled, incremental=incremental, chunk=i, step=step, layer=layer)
                heads = _stack_budgets(masks[layer], H, F, L)
                O = torch.empty_like(Q_d)
                lse = torch.empty((nh, C * F), dtype=torch.float32, device="cuda")
                stack.run_layer(layer, heads, slots, Q_d, Kq_d, Vq_d, O, lse, pooled=row, incremental=incremental)
                torch.cuda.synchronize()
                cfg = W.LayerConfig("stack", nh, d, F, H, window, C, L, "bf16", heads)
                x = W.LayerInputs(cfg, K_o[layer], V_o[layer], Kq, Vq, Q, slots)
                scores, kept = stack.views(H)
                got = SimpleNamespace(kv_len=stack.kv_len, scores=scores, kept_seg=kept, Kc=stack.Kc, Vc=stack.Vc)
                assert stack.static_in_place   # static heads attended in place: Kc/Vc rows not written
                if row is None:
                    ref = oracle.run_layer(cfg, x, scale=1 / math.sqrt(d))
                    assert_compression_exact(cfg, got, ref, skip_static=True)
                else:
                    ref = oracle.run_layer(cfg, x, scale=1 / math.sqrt(d), attention=False)
                    kept_d, kv_d = from_dev(kept), from_dev(stack.kv_len)
                    Kc_d, Vc_d = from_dev(stack.Kc), from_dev(stack.Vc)
                    for h, b in enumerate(heads):
                        if b.type == W.DYNAMIC:
                            want, cnt = oracle.select_head(row_want, H, F, L, b.sink_frames, b.recent_frames,
                                                           b.keep_k, b.scope)
                            np.testing.assert_array_equal(kept_d[h], want)
                            kc = oracle.compact_head(K_o[layer][h], slots, want[:cnt], H, L)
                            vc = oracle.compact_head(V_o[layer][h], slots, want[:cnt], H, L)
                            assert int(kv_d[h]) == kc.shape[0]
                            np.testing.assert_array_equal(Kc_d[h, :kc.shape[0]], kc)
                            np.testing.assert_array_equal(Vc_d[h, :vc.shape[0]], vc)
                    rows = np.arange(C * F, dtype=np.int32)
                    Kc_l = [Kc_d[h, :int(kv_d[h])] if b.type == W.DYNAMIC else ref.Kc[h] for h, b in enumerate(heads)]
                    Vc_l = [Vc_d[h, :int(kv_d[h])] if b.type == W.DYNAMIC else ref.Vc[h] for h, b in enumerate(heads)]
                    att = [oracle.attention_rows(Q[h], Kc_l[h], Vc_l[h], Kq[h], Vq[h], 1 / math.sqrt(d), rows)
                           for h in range(nh)]
                    ref = oracle.LayerResult(None, None, None, None, None, None, rows,
                                             np.stack([a[0] for a in att]), np.stack([a[1] for a in att]))
                assert_attention_close(O, ref, "bf16", lse)
        dst = W.chunk_write_slots(i, C, window)
        for layer in range(n_layers):
            stack.append(layer, Kq_d, Vq_d, dst.tolist())
            for h in range(nh):
                oracle.append_frames(K_o[layer][h], Kq[h].reshape(C, F, d), dst)
                oracle.append_frames(V_o[layer][h], Vq[h].reshape(C, F, d), dst)
    torch.cuda.synchronize()
    for layer in range(n_layers):
        np.testing.assert_array_equal(from_dev(stack.K_hist[layer]), K_o[layer])
        np.testing.assert_array_equal(from_dev(stack.V_hist[layer]), V_o[layer])
