"""Long-horizon streaming rollouts with the rolling cache (the rolling-cache
paragraph at the end of Sec. 4; the 30 s / 60 s settings of the long-video
experiments): 60 AR chunks through RolloutStack and fkv_append_frames, the
ring of rotating slots wrapping many times, every step checked against the
oracle, which keeps its own copy of every layer's cache through its own
append.

* small shape (4 heads, F = 64, window 7, 2-frame chunks; half-frame
  segments through the compacting step, one- and two-frame segments through
  the paged step): every chunk of every layer, selection (and compaction)
  bit-exact and attention on every query row; layer 1 scores incrementally
  (history statistics once per chunk);
* 480P shape (12 heads, F = 1560, window 21, 3-frame chunks: 180 frames, the
  20 rotating slots wrap 8 times): kept segments and kv_len of every chunk of
  every layer bit-exact; the paged step's attention (kept history read in
  place) on sampled rows at sampled (chunk, layer) units; both layers' caches
  bit-exact at the end.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import assert_attention_close, assert_compression_exact, from_dev, sample_rows, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2605_09681_amd as fkv
    fkv.lib()
    torch.cuda.set_device(0)


def _print(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _budgets(mask_row, H, F, L, recent_static):
    """Static heads keep the sink and `recent_static` recent frames; dynamic
    heads the sink plus half of the other segments (one global group)."""
    n_seg = (H * F + L - 1) // L
    k = max((n_seg - (F + L - 1) // L) // 2, 0)
    return tuple(W.HeadBudget(W.DYNAMIC, 1, 0, k, W.SCOPE_GLOBAL) if m == W.DYNAMIC else
                 W.HeadBudget(W.STATIC, 1, recent_static) for m in mask_row)


def _wraps(n_chunks, C, window, sink=1):
    """How many times the write pointer returns to the first rotating slot:
    video frame v >= sink goes to slot sink + (v - sink) % (window - sink), so
    it wraps at v = sink + j * (window - sink), j >= 1."""
    frames = n_chunks * C
    return (frames - 1 - sink) // (window - sink)


@pytest.mark.parametrize("L", [32, 64, 128])
def test_long_rollout_60_chunks_small_every_step(L):
    """L = 32: the compacting step (pieces below 64 tokens); L = 64 and 128 (one
    and two frames per segment): the paged step, every head read in place."""
    from paper_2605_09681_amd.layer import RolloutStack
    from types import SimpleNamespace
    n_layers, nh, d, F, window, C = 2, 4, 64, 64, 7, 2
    n_chunks = 60
    assert _wraps(n_chunks, C, window) >= 8
    masks = W.rollout_head_masks(31, n_layers=n_layers, n_heads=nh, n_dynamic=2)
    stack = RolloutStack(n_layers, nh, d, F, window, C, L)
    assert stack.step_mode == ("compact" if L < 64 else "paged")
    paged = stack.step_mode == "paged"
    keys = W.ar1_key_frames(61, nh, n_chunks * C, F, d, 0.9, "bf16")     # [nh][frames][F][d]
    vals = W.normal_tensor(61, 7, (nh, n_chunks * C, F, d), "bf16")
    qs = W.normal_tensor(61, 8, (nh, n_chunks * C * F, d), "bf16")
    K_o = np.zeros((n_layers, nh, window, F, d), np.uint16)
    V_o = np.zeros_like(K_o)
    for i in range(n_chunks):
        slots = W.ring_frame_slots(i, C, window)
        H = len(slots)
        Kq = np.ascontiguousarray(keys[:, i * C:(i + 1) * C].reshape(nh, C * F, d))
        Vq = np.ascontiguousarray(vals[:, i * C:(i + 1) * C].reshape(nh, C * F, d))
        Q = np.ascontiguousarray(qs[:, i * C * F:(i + 1) * C * F])
        Kq_d, Vq_d, Q_d = to_dev(Kq, "bf16"), to_dev(Vq, "bf16"), to_dev(Q, "bf16")
        for layer in range(n_layers):
            _print("long-rollout-small", L=L, chunk=i, layer=layer, H=H)
            heads = _budgets(masks[layer], H, F, L, 2)
            incremental = layer == 1 and H > 0
            if incremental:
                stack.history(layer, heads, slots)
            O = torch.empty_like(Q_d)
            lse = torch.empty((nh, C * F), dtype=torch.float32, device="cuda")
            stack.run_layer(layer, heads, slots, Q_d, Kq_d, Vq_d, O, lse, incremental=incremental)
            torch.cuda.synchronize()
            cfg = W.LayerConfig("long", nh, d, F, H, window, C, L, "bf16", heads)
            x = W.LayerInputs(cfg, K_o[layer], V_o[layer], Kq, Vq, Q, slots)
            ref = oracle.run_layer(cfg, x, scale=1 / math.sqrt(d))
            scores, kept = stack.views(H)
            got = SimpleNamespace(kv_len=stack.kv_len, scores=scores, kept_seg=kept, Kc=stack.Kc, Vc=stack.Vc)
            assert_compression_exact(cfg, got, ref, skip_static=stack.static_in_place or paged,
                                     skip_dynamic_copy=paged)
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


def _chunk_inputs(i, nh, C, F, d, rho):
    """One chunk's keys (an AR(1) chain over its frames), values and queries,
    generated on the device from a seed and rounded to bf16."""
    g = torch.Generator(device="cuda").manual_seed(7000 + i)
    k = torch.randn(nh, C, F, d, device="cuda", generator=g)
    a = math.sqrt(1 - rho * rho)
    for f in range(1, C):
        k[:, f] = rho * k[:, f - 1] + a * k[:, f]
    Kq = k.reshape(nh, C * F, d).to(torch.bfloat16)
    Vq = torch.randn(nh, C * F, d, device="cuda", generator=g).to(torch.bfloat16)
    Q = torch.randn(nh, C * F, d, device="cuda", generator=g).to(torch.bfloat16)
    return Kq, Vq, Q


def test_long_rollout_60_chunks_480p_sampled():
    from paper_2605_09681_amd.layer import RolloutStack
    from types import SimpleNamespace
    n_layers, nh, d, F, window, C, L = 2, 12, 128, 1560, 21, 3, 1560
    n_chunks = 60
    assert _wraps(n_chunks, C, window) >= 8
    sampled = {(7, 1), (15, 0), (29, 1), (44, 0), (59, 1)}
    masks = W.rollout_head_masks(0, n_layers=n_layers)
    stack = RolloutStack(n_layers, nh, d, F, window, C, L)
    paged = stack.step_mode == "paged"
    assert paged
    K_o = np.zeros((n_layers, nh, window, F, d), np.uint16)
    V_o = np.zeros_like(K_o)
    for i in range(n_chunks):
        slots = W.ring_frame_slots(i, C, window)
        H = len(slots)
        Kq_d, Vq_d, Q_d = _chunk_inputs(i, nh, C, F, d, 0.9)
        Kq, Vq = from_dev(Kq_d), from_dev(Vq_d)
        for layer in range(n_layers):
            heads = _budgets(masks[layer], H, F, L, 6)
            full = (i, layer) in sampled
            _print("long-rollout-480p", chunk=i, layer=layer, H=H, full=full)
            O = torch.empty_like(Q_d)
            lse = torch.empty((nh, C * F), dtype=torch.float32, device="cuda")
            stack.run_layer(layer, heads, slots, Q_d, Kq_d, Vq_d, O, lse)
            torch.cuda.synchronize()
            cfg = W.LayerConfig("long480", nh, d, F, H, window, C, L, "bf16", heads)
            Q = from_dev(Q_d) if full else None
            x = W.LayerInputs(cfg, K_o[layer], V_o[layer], Kq, Vq, Q, slots)
            scores, kept = stack.views(H)
            if full:
                rows = sample_rows(cfg.lq, 4, seed=i)
                ref = oracle.run_layer(cfg, x, rows=rows, scale=1 / math.sqrt(d))
                got = SimpleNamespace(kv_len=stack.kv_len, scores=scores, kept_seg=kept, Kc=stack.Kc,
                                      Vc=stack.Vc)
                assert_compression_exact(cfg, got, ref, skip_static=True, skip_dynamic_copy=paged)
                assert_attention_close(O, ref, "bf16", lse)
            else:
                # selection only: scores, kept segment ids and kv_len of the dynamic heads
                dyn = [h for h, b in enumerate(heads) if b.type == W.DYNAMIC]
                kv, kp, sc = from_dev(stack.kv_len), from_dev(kept), from_dev(scores)
                for h in dyn:
                    b = heads[h]
                    s32, _ = oracle.score_head(K_o[layer][h], slots, Kq[h], H, L)
                    want, cnt = oracle.select_head(s32, H, F, L, b.sink_frames, b.recent_frames, b.keep_k,
                                                   b.scope)
                    np.testing.assert_array_equal(sc[h].view(np.uint32), s32.view(np.uint32),
                                                  err_msg=f"scores chunk {i} layer {layer} head {h}")
                    np.testing.assert_array_equal(kp[h], want, err_msg=f"kept chunk {i} layer {layer} head {h}")
                    assert int(kv[h]) == sum(min(g * L + L, H * F) - g * L for g in want[:cnt])
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
