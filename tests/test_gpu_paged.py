"""The one-launch scoring (fkv_score_segments / fkv_score_select, per-frame
sums reduced by the last workgroup of each head) and attention with every
head's kept history read in place from the cache (fkv_select +
fkv_chunk_attention_paged), through the C ABI:

* fkv_score_select writes the scores, kept segments and kv_len that
  fkv_score_segments followed by fkv_select writes, and both match the
  oracle bit for bit (Eq. 3 similarity and BottomK);
* incremental rescoring (fkv_score_history + fkv_score_segments_cached)
  equals the full pass bit for bit, per head and pooled;
* fkv_chunk_attention_paged gives O and lse bit-identical to compaction
  (fkv_compress_static + fkv_select_compact) followed by fkv_chunk_attention
  of the same heads -- all heads, or a listed subset with every other head's
  rows untouched -- and within the attention bar of the oracle;
* the paged step modes of CompressedLayer against the oracle.

Cases: the 480P layer with one-frame, quarter-frame (per-frame groups) and
three-frame segments, a 20-frame history whose last three-frame segment holds
two frames, 1080P, and small multi-tile shapes whose 64-token pieces put
piece boundaries inside key tiles; rotated rings throughout.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import (assert_attention_close, assert_compression_exact, dev_inputs, from_dev, make_layer,
                         sample_rows)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2605_09681_amd as fkv
    fkv.lib()
    torch.cuda.set_device(0)


def _print_case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _case(name):
    """(cfg, frame_slot, rows) of a named case; rows None = every row."""
    S, D = W.STATIC, W.DYNAMIC
    if name.startswith("480p") or name == "1080p":
        res = "1080p" if name == "1080p" else "480p"
        L = {"480p": None, "480p-L390": 390, "480p-L4680": 4680, "480p-H20-L4680": 4680, "1080p": None}[name]
        cfg = W.wan_layer_config(res, seg_tokens=L)
        if name == "480p-H20-L4680":
            cfg = cfg.replace(hist_frames=20, cap_frames=21)
        slot = np.roll(np.arange(cfg.cap_frames, dtype=np.int32), 4)[:cfg.hist_frames]
        rows = sample_rows(cfg.lq, 8 if res == "480p" else 4, seed=len(name))
        return cfg, slot, rows
    if name == "small-F128-L64":
        heads = (W.HeadBudget(S, 1, 2), W.HeadBudget(D, 1, 0, 1, W.SCOPE_FRAME), W.HeadBudget(D, 0, 1, 4, W.SCOPE_GLOBAL),
                 W.HeadBudget(S, 0, 3), W.HeadBudget(D, 1, 1, 0, W.SCOPE_FRAME), W.HeadBudget(D, 2, 0, 9, W.SCOPE_GLOBAL))
        cfg = W.LayerConfig("small-paged", len(heads), 128, 128, 7, 9, 2, 64, "bf16", heads, 0.85)
        return cfg, np.array([3, 0, 8, 1, 5, 2, 7], np.int32), None
    if name == "small-F96-L192-d64":
        heads = (W.HeadBudget(D, 1, 0, 2, W.SCOPE_GLOBAL), W.HeadBudget(S, 1, 1), W.HeadBudget(D, 0, 0, 1, W.SCOPE_GLOBAL),
                 W.HeadBudget(D, 0, 2, 3, W.SCOPE_GLOBAL))
        cfg = W.LayerConfig("small-paged64", len(heads), 64, 96, 9, 11, 3, 192, "bf16", heads, 0.8)
        return cfg, np.array([10, 3, 0, 8, 1, 5, 2, 7, 4], np.int32), None
    if name == "H1":
        heads = (W.HeadBudget(S, 1, 1), W.HeadBudget(D, 1, 0, 1, W.SCOPE_GLOBAL), W.HeadBudget(D, 0, 0, 1, W.SCOPE_GLOBAL))
        cfg = W.LayerConfig("h1", 3, 128, 64, 1, 3, 2, 64, "bf16", heads, 0.9)
        return cfg, np.array([2], np.int32), None
    raise KeyError(name)


CASES = ["480p", "480p-L390", "480p-L4680", "480p-H20-L4680", "1080p", "small-F128-L64", "small-F96-L192-d64", "H1"]


@pytest.mark.parametrize("case", CASES)
def test_score_select_equals_score_then_select(case):
    import paper_2605_09681_amd as fkv
    cfg, slot, _ = _case(case)
    _print_case("score-select", case=case)
    x = W.make_layer_inputs(cfg, seed=51, frame_slot=slot)
    d = dev_inputs(x)
    layer = make_layer(cfg)
    n_seg = layer.n_seg
    fkv.fkv_score_segments(layer.shape, layer.heads, d["K_hist"], slot, d["K_cur"], layer.scores, layer.workspace)
    kept_a = torch.full((cfg.n_heads, n_seg), -7, dtype=torch.int32, device="cuda")
    kv_a = torch.full((cfg.n_heads,), -7, dtype=torch.int32, device="cuda")
    fkv.fkv_select(layer.shape, layer.heads, layer.scores, kept_a, kv_a)
    scores_a = layer.scores.clone()
    scores_b = torch.full_like(layer.scores, 5.0)
    kept_b = torch.full_like(kept_a, -7)
    kv_b = torch.full_like(kv_a, -7)
    fkv.fkv_score_select(layer.shape, layer.heads, d["K_hist"], slot, d["K_cur"], scores_b, kept_b, kv_b,
                         layer.workspace)
    torch.cuda.synchronize()
    dyn = [h for h, b in enumerate(cfg.heads) if b.type == W.DYNAMIC]
    st = [h for h, b in enumerate(cfg.heads) if b.type == W.STATIC]
    np.testing.assert_array_equal(from_dev(scores_b)[dyn].view(np.uint32), from_dev(scores_a)[dyn].view(np.uint32))
    np.testing.assert_array_equal(from_dev(kept_b)[dyn], from_dev(kept_a)[dyn])
    np.testing.assert_array_equal(from_dev(kv_b)[dyn], from_dev(kv_a)[dyn])
    assert (from_dev(scores_b)[st] == 5.0).all() and (from_dev(kept_b)[st] == -7).all() and \
        (from_dev(kv_b)[st] == -7).all(), "static heads' rows must stay untouched"
    ref = oracle.run_layer(cfg, x, attention=False)
    for h in dyn:
        np.testing.assert_array_equal(from_dev(scores_b)[h].view(np.uint32), ref.scores[h].view(np.uint32),
                                      err_msg=f"scores head {h}")
        np.testing.assert_array_equal(from_dev(kept_b)[h], ref.kept_seg[h], err_msg=f"kept head {h}")
        assert int(from_dev(kv_b)[h]) == ref.kv_len[h]


@pytest.mark.parametrize("case", ["480p", "480p-L390", "480p-L4680", "small-F128-L64", "small-F96-L192-d64"])
@pytest.mark.parametrize("pooled", [False, True])
def test_incremental_scores_equal_full_pass(case, pooled):
    """History statistics + cached step scores are the full pass's scores bit
    for bit, over three different chunk keys (per head, or pooled)."""
    import paper_2605_09681_amd as fkv
    cfg, slot, _ = _case(case)
    _print_case("incremental-vs-full", case=case, pooled=pooled)
    x = W.make_layer_inputs(cfg, seed=52, frame_slot=slot)
    d = dev_inputs(x)
    shape = fkv.make_shape(cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.cap_frames,
                           cfg.chunk_frames, cfg.seg_tokens, cfg.dtype)
    heads = fkv.make_heads(cfg.heads)
    n_seg = fkv.fkv_num_segments(shape)
    wsb = fkv.fkv_score_pooled_workspace_size(shape) if pooled else fkv.fkv_score_workspace_size(shape, heads)
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    stats = torch.empty(fkv.fkv_score_stats_size(shape, heads, pooled) // 8, dtype=torch.float64, device="cuda")
    fkv.fkv_score_history(shape, heads, d["K_hist"], slot, stats, ws, pooled=pooled)
    sh = (n_seg,) if pooled else (cfg.n_heads, n_seg)
    dyn = [h for h, b in enumerate(cfg.heads) if b.type == W.DYNAMIC]
    for step in range(3):
        Kq = d["K_cur"] if step == 0 else torch.randn_like(d["K_cur"], dtype=torch.float32).to(torch.bfloat16)
        full = torch.zeros(sh, dtype=torch.float32, device="cuda")
        inc = torch.ones(sh, dtype=torch.float32, device="cuda")
        if pooled:
            fkv.fkv_score_pooled(shape, d["K_hist"], slot, Kq, full, ws)
        else:
            fkv.fkv_score_segments(shape, heads, d["K_hist"], slot, Kq, full, ws)
        fkv.fkv_score_segments_cached(shape, heads, d["K_hist"], slot, Kq, stats, inc, ws, pooled=pooled)
        torch.cuda.synchronize()
        a, b = from_dev(full), from_dev(inc)
        if not pooled:
            a, b = a[dyn], b[dyn]
        np.testing.assert_array_equal(b.view(np.uint32), a.view(np.uint32), err_msg=f"step {step}")


def _compact_reference(layer, d, slot, heads_list=None):
    """O and lse through the compacting path: gather + select/compact, then
    attention of the listed heads (all by default) over Kc / Vc."""
    import paper_2605_09681_amd as fkv
    layer.score(d["K_hist"], slot, d["K_cur"])
    layer.select_compact(d["K_hist"], d["V_hist"], slot)
    layer.compress_static(d["K_hist"], d["V_hist"], slot)
    O = torch.full_like(d["Q"], 7.0)
    lse = torch.full((layer.shape.n_heads, layer.lq), -3.0, dtype=torch.float32, device="cuda")
    if heads_list is None:
        layer.attention(d["Q"], d["K_cur"], d["V_cur"], O, lse)
    else:
        fkv.fkv_chunk_attention_heads(layer.shape, heads_list, d["Q"], layer.Kc, layer.Vc, layer.kv_len,
                                      d["K_cur"], d["V_cur"], layer.scale, O, lse, layer.attn_workspace)
    return O, lse


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("subset", ["all", "dynamic", "mixed"])
def test_paged_attention_bit_identical_to_compaction(case, subset):
    import paper_2605_09681_amd as fkv
    cfg, slot, rows = _case(case)
    if case == "1080p" and subset != "all":
        pytest.skip("1080P: the all-heads launch covers it")
    _print_case("paged-attention", case=case, subset=subset)
    x = W.make_layer_inputs(cfg, seed=53, frame_slot=slot)
    d = dev_inputs(x)
    dyn = [h for h, b in enumerate(cfg.heads) if b.type == W.DYNAMIC]
    listed = None if subset == "all" else dyn if subset == "dynamic" else \
        sorted(dyn[::2] + [h for h, b in enumerate(cfg.heads) if b.type == W.STATIC][:1], reverse=True)
    ref_layer = make_layer(cfg, step_mode="compact")
    O_ref, l_ref = _compact_reference(ref_layer, d, slot, listed)
    layer = make_layer(cfg)
    assert layer.step_mode == "paged"
    layer.score_select(d["K_hist"], slot, d["K_cur"])
    O = torch.full_like(d["Q"], 7.0)
    lse = torch.full((cfg.n_heads, cfg.lq), -3.0, dtype=torch.float32, device="cuda")
    fkv.fkv_chunk_attention_paged(layer.shape, layer.heads, d["K_hist"], d["V_hist"], slot, layer.kept_seg,
                                  layer.kv_len, d["Q"], d["K_cur"], d["V_cur"], layer.scale, O, lse,
                                  layer.attn_workspace, listed)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(O), from_dev(O_ref))
    np.testing.assert_array_equal(from_dev(lse).view(np.uint32), from_dev(l_ref).view(np.uint32))
    ref = oracle.run_layer(cfg, x, rows=rows, scale=layer.scale)
    Of, lf = from_dev(O), from_dev(lse)
    for h in range(cfg.n_heads):
        if listed is None or h in listed:
            one = oracle.LayerResult(None, None, None, None, None, None, ref.rows, ref.O[h:h + 1], ref.lse[h:h + 1])
            assert_attention_close(O[h:h + 1], one, "bf16", lse[h:h + 1])
        else:
            assert (W.bf16_bits_to_f32(Of[h]) == 7.0).all() and (lf[h] == -3.0).all(), h


@pytest.mark.parametrize("case", ["480p", "480p-L390", "small-F128-L64", "H1"])
@pytest.mark.parametrize("mode", ["paged", "paged2"])
def test_paged_step_modes(case, mode):
    cfg, slot, rows = _case(case)
    _print_case("paged-step", case=case, mode=mode)
    x = W.make_layer_inputs(cfg, seed=54, frame_slot=slot)
    d = dev_inputs(x)
    layer = make_layer(cfg, step_mode=mode)
    O = torch.empty_like(d["Q"])
    lse = torch.empty((cfg.n_heads, cfg.lq), dtype=torch.float32, device="cuda")
    layer.step(d["K_hist"], d["V_hist"], slot, d["Q"], d["K_cur"], d["V_cur"], O, lse)
    torch.cuda.synchronize()
    ref = oracle.run_layer(cfg, x, rows=rows, scale=1 / math.sqrt(cfg.head_dim))
    assert_compression_exact(cfg, layer, ref, skip_static=True, skip_dynamic_copy=True)
    assert_attention_close(O, ref, "bf16", lse)


def test_paged_step_480p_every_row():
    """The default step at the 480P shape, every query row of every head
    against the oracle (rotated ring slots): the balanced schedule cuts nearly
    every (head, query tile) item at this size, so this checks every cut
    item's in-kernel merge at full size, not only on sampled rows."""
    cfg, slot, _ = _case("480p")
    _print_case("paged-step-every-row", case="480p")
    x = W.make_layer_inputs(cfg, seed=56, frame_slot=slot)
    d = dev_inputs(x)
    layer = make_layer(cfg, step_mode="paged")
    O = torch.empty_like(d["Q"])
    lse = torch.empty((cfg.n_heads, cfg.lq), dtype=torch.float32, device="cuda")
    layer.step(d["K_hist"], d["V_hist"], slot, d["Q"], d["K_cur"], d["V_cur"], O, lse)
    torch.cuda.synchronize()
    ref = oracle.run_layer(cfg, x, rows=None, scale=1 / math.sqrt(cfg.head_dim))
    assert len(ref.rows) == cfg.lq
    assert_compression_exact(cfg, layer, ref, skip_static=True, skip_dynamic_copy=True)
    max_abs, rel = assert_attention_close(O, ref, "bf16", lse)
    print(f"480p every row: max_abs={max_abs:.2e} rel_l2={rel:.2e}", flush=True)


def test_paged_empty_history_and_select_only():
    """H = 0: fkv_score_select and fkv_select give every dynamic head kv_len 0
    and the paged launch attends the chunk alone; a pooled score row selects
    through fkv_select(shared_row) like fkv_select_compact_pooled."""
    import paper_2605_09681_amd as fkv
    S, D = W.STATIC, W.DYNAMIC
    heads = (W.HeadBudget(S, 1, 1), W.HeadBudget(D, 1, 0, 1, W.SCOPE_GLOBAL), W.HeadBudget(D, 0, 0, 2, W.SCOPE_FRAME))
    cfg = W.LayerConfig("h0", 3, 128, 128, 0, 4, 2, 64, "bf16", heads, 0.9)
    _print_case("paged-h0")
    x = W.make_layer_inputs(cfg, seed=55, frame_slot=np.zeros(0, np.int32))
    d = dev_inputs(x)
    layer = make_layer(cfg)
    layer.kv_len.fill_(999)
    O = torch.empty_like(d["Q"])
    lse = torch.empty((cfg.n_heads, cfg.lq), dtype=torch.float32, device="cuda")
    layer.step(d["K_hist"], d["V_hist"], x.frame_slot, d["Q"], d["K_cur"], d["V_cur"], O, lse)
    torch.cuda.synchronize()
    assert (from_dev(layer.kv_len)[[1, 2]] == 0).all()
    ref = oracle.run_layer(cfg, x, scale=layer.scale)
    assert_attention_close(O, ref, "bf16", lse)
    # pooled row through fkv_select(shared_row=True) == fkv_select_compact_pooled's selection
    cfg2, slot2, _ = _case("480p-L390")
    x2 = W.make_layer_inputs(cfg2, seed=56, frame_slot=slot2)
    d2 = dev_inputs(x2)
    L2 = make_layer(cfg2, step_mode="compact")
    row = torch.empty((L2.n_seg,), dtype=torch.float32, device="cuda")
    fkv.fkv_score_pooled(L2.shape, d2["K_hist"], slot2, d2["K_cur"], row)
    kept = torch.full_like(L2.kept_seg, -9)
    kv = torch.full_like(L2.kv_len, -9)
    fkv.fkv_select(L2.shape, L2.heads, row, kept, kv, shared_row=True)
    fkv.fkv_select_compact_pooled(L2.shape, L2.heads, row, d2["K_hist"], d2["V_hist"], slot2, L2.kept_seg, L2.Kc,
                                  L2.Vc, L2.kv_len)
    torch.cuda.synchronize()
    dyn = [h for h, b in enumerate(cfg2.heads) if b.type == W.DYNAMIC]
    np.testing.assert_array_equal(from_dev(kept)[dyn], from_dev(L2.kept_seg)[dyn])
    np.testing.assert_array_equal(from_dev(kv)[dyn], from_dev(L2.kv_len)[dyn])
