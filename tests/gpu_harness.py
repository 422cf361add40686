"""Helpers for the GPU parity tests: host <-> device marshalling of the seeded
workloads, running the HIP path through the C ABI, and comparing with the
oracle."""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
import workloads as W

# Attention acceptance (bf16 inputs, fp32 accumulation, normalised output):
# max abs error 2e-2, plus the stronger relative L2 bound 1e-2 (N(0,1) data
# gives outputs of only ~1e-2, so the absolute bound alone is weak).
BF16_MAX_ABS = 2e-2
BF16_REL_L2 = 1e-2
# fp32 path: fp32 accumulation over at most a few thousand keys.
F32_MAX_ABS = 1e-4
F32_REL_L2 = 1e-5
# Log-normaliser of the bf16 path: 2e-3 for the bf16 score products and fp32
# accumulation, plus the normaliser's own rounding -- it is the sum of the
# bf16-rounded probabilities that weight V (each within a relative 2^-9 of
# the exact one, so the sum is too), which moves lse by at most
# -log(1 - 2^-9) = 1.96e-3 from the exact log-sum-exp.
BF16_LSE_ABS = 2e-3 - math.log1p(-2.0 ** -9)


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def from_dev(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dev_inputs(x: W.LayerInputs):
    dt = x.cfg.dtype
    return dict(K_hist=to_dev(x.K_hist, dt), V_hist=to_dev(x.V_hist, dt), K_cur=to_dev(x.K_cur, dt),
                V_cur=to_dev(x.V_cur, dt), Q=to_dev(x.Q, dt))


def make_layer(cfg: W.LayerConfig, heads=None, slab=None, balanced=True, in_place=None, step_mode=None):
    from paper_2605_09681_amd.layer import CompressedLayer
    return CompressedLayer(cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames,
                           cfg.cap_frames, cfg.chunk_frames, cfg.seg_tokens, cfg.dtype,
                           cfg.heads if heads is None else heads, slab=slab, balanced=balanced,
                           in_place=in_place, step_mode=step_mode)


def run_gpu(cfg: W.LayerConfig, x: W.LayerInputs, heads=None, with_lse=True, scale=None,
            balanced=True):
    """Run one layer step on the GPU; returns (layer, O, lse) with device tensors.
    balanced selects the attention schedule (workspace given or not)."""
    layer = make_layer(cfg, heads, balanced=balanced)
    d = dev_inputs(x)
    O = torch.empty_like(d["Q"])
    lse = torch.empty((cfg.n_heads, cfg.lq), dtype=torch.float32, device="cuda") if with_lse else None
    layer.compress(d["K_hist"], d["V_hist"], x.frame_slot, d["K_cur"])
    layer.attention(d["Q"], d["K_cur"], d["V_cur"], O, lse, scale=scale)
    torch.cuda.synchronize()
    return layer, O, lse


def sample_rows(lq: int, n_random: int = 48, seed: int = 0) -> np.ndarray:
    """First rows, the ragged tail of the last 256-row tile, and random rows."""
    rng = np.random.default_rng(seed)
    tail_start = (lq // 256) * 256
    rows = set(range(min(16, lq))) | set(range(max(0, min(tail_start, lq - 40)), lq))
    rows |= set(rng.integers(0, lq, n_random).tolist())
    return np.array(sorted(rows), dtype=np.int32)


def assert_compression_exact(cfg, layer, ref: oracle.LayerResult, heads=None, skip_static=False,
                             skip_dynamic_copy=False):
    """skip_static: the static heads were attended in place, so their rows of
    kv_len / Kc / Vc were never written.  skip_dynamic_copy: the dynamic heads
    were attended in place (scores, kept_seg and kv_len written, no Kc / Vc)."""
    heads = cfg.heads if heads is None else heads
    kv_len = from_dev(layer.kv_len).astype(np.int64)
    checked = [h for h, b in enumerate(heads) if not (skip_static and b.type == W.STATIC)]
    np.testing.assert_array_equal(kv_len[checked], ref.kv_len[checked], err_msg="kv_len")
    scores = from_dev(layer.scores)
    kept = from_dev(layer.kept_seg)
    Kc, Vc = from_dev(layer.Kc), from_dev(layer.Vc)
    for h, b in enumerate(heads):
        if h not in checked:
            continue
        if b.type == W.DYNAMIC and ref.scores.shape[1] > 0:
            np.testing.assert_array_equal(scores[h].view(np.uint32), ref.scores[h].view(np.uint32),
                                          err_msg=f"scores head {h}")
            np.testing.assert_array_equal(kept[h], ref.kept_seg[h], err_msg=f"kept_seg head {h}")
        if skip_dynamic_copy and b.type == W.DYNAMIC:
            continue
        n = int(ref.kv_len[h])
        np.testing.assert_array_equal(Kc[h, :n], ref.Kc[h], err_msg=f"Kc head {h}")
        np.testing.assert_array_equal(Vc[h, :n], ref.Vc[h], err_msg=f"Vc head {h}")


def attention_errors(O_dev: torch.Tensor, ref: oracle.LayerResult, dtype: str):
    O = W.storage_to_f32(from_dev(O_dev), dtype).astype(np.float64)[:, ref.rows]
    diff = O - ref.O
    max_abs = float(np.abs(diff).max())
    rel = float(np.linalg.norm(diff) / max(np.linalg.norm(ref.O), 1e-300))
    return max_abs, rel


def assert_attention_close(O_dev, ref, dtype, lse_dev=None):
    max_abs, rel = attention_errors(O_dev, ref, dtype)
    lim_abs, lim_rel = (BF16_MAX_ABS, BF16_REL_L2) if dtype == "bf16" else (F32_MAX_ABS, F32_REL_L2)
    assert max_abs <= lim_abs, f"attention max abs error {max_abs:.3e} > {lim_abs}"
    assert rel <= lim_rel, f"attention relative L2 error {rel:.3e} > {lim_rel}"
    if lse_dev is not None:
        lse = from_dev(lse_dev).astype(np.float64)[:, ref.rows]
        lse_tol = BF16_LSE_ABS if dtype == "bf16" else 1e-5
        err = float(np.abs(lse - ref.lse).max())
        assert err <= lse_tol, f"lse max abs error {err:.3e} > {lse_tol}"
    return max_abs, rel


def check_layer(cfg, x, heads=None, rows=None, scale=None, balanced=True):
    """Full parity check of one layer step: compression bit-exact on every
    head, attention on the given query rows (all rows by default)."""
    heads = cfg.heads if heads is None else heads
    layer, O, lse = run_gpu(cfg, x, heads=heads, scale=scale, balanced=balanced)
    ref = oracle.run_layer(cfg, x, rows=rows, heads=heads,
                           scale=(1 / math.sqrt(cfg.head_dim)) if scale is None else scale)
    assert_compression_exact(cfg, layer, ref, heads)
    errs = assert_attention_close(O, ref, cfg.dtype, lse)
    return layer, O, ref, errs
