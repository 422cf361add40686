"""fkv_score_select_noalloc -- scoring + selection with the library's own
per-GPU scratch instead of a caller workspace (for callers that cannot
allocate) -- writes exactly what fkv_score_select writes with a workspace,
through the C ABI, on two calls in a row on the same GPU, the second with a
smaller input (the scratch keeps the last call's contents; its arrival
counters must be back at zero)."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import dev_inputs, from_dev, make_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2605_09681_amd as fkv
    fkv.lib()
    torch.cuda.set_device(0)


def _cases():
    S, D = W.STATIC, W.DYNAMIC
    big = W.wan_layer_config("480p")
    big_slot = np.roll(np.arange(21, dtype=np.int32), 2)
    heads = (W.HeadBudget(D, 1, 0, 1, W.SCOPE_FRAME), W.HeadBudget(S, 1, 2), W.HeadBudget(D, 0, 1, 3, W.SCOPE_GLOBAL))
    small = W.LayerConfig("small-noalloc", 3, 64, 96, 5, 7, 2, 48, "bf16", heads, 0.85)
    small_slot = np.array([6, 0, 3, 1, 5], np.int32)
    return [("480p", big, big_slot), ("small", small, small_slot)]


def test_noalloc_equals_workspace_call_twice():
    import paper_2605_09681_amd as fkv
    for name, cfg, slot in _cases():
        print(f"[case] noalloc {name}", flush=True)
        x = W.make_layer_inputs(cfg, seed=71, frame_slot=slot)
        d = dev_inputs(x)
        layer = make_layer(cfg, step_mode="compact")
        n = (cfg.n_heads, layer.n_seg)
        ref_s = torch.full(n, 3.0, dtype=torch.float32, device="cuda")
        ref_k = torch.full(n, -5, dtype=torch.int32, device="cuda")
        ref_l = torch.full((cfg.n_heads,), -5, dtype=torch.int32, device="cuda")
        fkv.fkv_score_select(layer.shape, layer.heads, d["K_hist"], slot, d["K_cur"], ref_s, ref_k, ref_l,
                             layer.workspace)
        got_s = torch.full(n, 3.0, dtype=torch.float32, device="cuda")
        got_k = torch.full(n, -5, dtype=torch.int32, device="cuda")
        got_l = torch.full((cfg.n_heads,), -5, dtype=torch.int32, device="cuda")
        fkv.fkv_score_select_noalloc(layer.shape, layer.heads, d["K_hist"], slot, d["K_cur"], got_s, got_k, got_l)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(from_dev(got_s).view(np.uint32), from_dev(ref_s).view(np.uint32), err_msg=name)
        np.testing.assert_array_equal(from_dev(got_k), from_dev(ref_k), err_msg=name)
        np.testing.assert_array_equal(from_dev(got_l), from_dev(ref_l), err_msg=name)
        dyn = [h for h, b in enumerate(cfg.heads) if b.type == W.DYNAMIC]
        assert (from_dev(got_l)[dyn] > 0).all(), name
