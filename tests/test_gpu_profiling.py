"""GPU parity of offline head profiling (Sec. 4.1, Eq. 1) through the C ABI.

The attention mass per key frame (fkv_attention_mass after the full-cache
attention) is compared with the oracle's exact fp64 mass; the bound covers
fp32 summation of probabilities whose scores come from bf16 products
(relative 1e-4 of the frame's mass plus 1e-5 of the total mass Lq).  The
classification itself is host code compared exactly in the CPU suite; here the
whole profiling pass must give the oracle's head types on synthetic heads
built to be static-like or dynamic-like.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2605_09681_amd as fkv
    fkv.lib()
    oracle.lib()


def _case(name, **kw):
    print(f"[gpu case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _oracle_mass(x, H, F, scale):
    out = []
    for h in range(x.Q.shape[0]):
        full = x.K_hist[h][x.frame_slot[:H]].reshape(H * F, -1) if H else np.zeros((0, x.Q.shape[2]), x.Q.dtype)
        out.append(oracle.attention_mass(x.Q[h], full, x.K_cur[h], F, scale))
    return np.stack(out)


def _profile(cfg, xs):
    from paper_2605_09681_amd.layer import HeadProfiler
    prof = HeadProfiler(cfg.n_heads, cfg.head_dim, cfg.frame_tokens, cfg.hist_frames, cfg.cap_frames,
                        cfg.chunk_frames)
    for x in xs:
        d = {k: to_dev(getattr(x, k), "bf16") for k in ("Q", "K_hist", "V_hist", "K_cur", "V_cur")}
        prof.observe(d["Q"], d["K_hist"], d["V_hist"], x.frame_slot, d["K_cur"], d["V_cur"])
    torch.cuda.synchronize()
    return prof


def _check_mass(got, want, lq):
    err = np.abs(got.astype(np.float64) - want)
    tol = 1e-4 * want + 1e-5 * lq
    assert (err <= tol).all(), (float(err.max()), float((err / tol).max()))


@pytest.mark.parametrize("F,H,C,d", [(100, 7, 2, 128), (37, 5, 2, 64), (64, 3, 1, 128), (100, 0, 2, 128),
                                     (20, 9, 3, 64)])
def test_mass_small(F, H, C, d):
    heads = tuple(W.HeadBudget(W.STATIC, 0, H) for _ in range(4))
    cap = max(H, 1) + 2
    cfg = W.LayerConfig("mass", 4, d, F, H, cap, C, F, "bf16", heads, 0.85)
    slot = np.random.default_rng(F + H).permutation(cap)[:H].astype(np.int32)
    _case("mass", F=F, H=H, C=C, d=d)
    x = W.make_layer_inputs(cfg, seed=F * 7 + H, frame_slot=slot)
    prof = _profile(cfg, [x])
    _check_mass(from_dev(prof.mass), _oracle_mass(x, H, F, 1 / math.sqrt(d)), cfg.lq)


def test_mass_accumulates_over_observations():
    heads = tuple(W.HeadBudget(W.STATIC, 0, 4) for _ in range(3))
    cfg = W.LayerConfig("mass-acc", 3, 128, 96, 4, 5, 2, 96, "bf16", heads, 0.9)
    _case("mass-acc")
    xs = [W.make_layer_inputs(cfg, seed=s) for s in (1, 2, 3)]
    prof = _profile(cfg, xs)
    want = sum(_oracle_mass(x, 4, 96, 1 / math.sqrt(128)) for x in xs)
    _check_mass(from_dev(prof.mass), want, 3 * cfg.lq)


def test_mass_480p_shape():
    """Two heads of the 480P layer shape (21 history frames of 1560 tokens, a
    3-frame chunk): every query row, every frame."""
    heads = tuple(W.HeadBudget(W.STATIC, 0, 21) for _ in range(2))
    cfg = W.wan_layer_config("480p").replace(n_heads=2, heads=heads)
    _case("mass-480p")
    x = W.make_layer_inputs(cfg, seed=4)
    prof = _profile(cfg, [x])
    _check_mass(from_dev(prof.mass), _oracle_mass(x, 21, cfg.frame_tokens, 1 / math.sqrt(128)), cfg.lq)


def test_profiling_classifies_synthetic_heads():
    """Heads whose queries copy the current chunk's keys concentrate their mass
    locally (static); heads whose queries copy an old frame spread it (dynamic).
    The GPU profiling pass must reproduce the oracle's Eq. 1 decisions, which
    must be the intended ones."""
    F, H, C, d, nh = 64, 6, 2, 128, 6
    heads = tuple(W.HeadBudget(W.STATIC, 0, H) for _ in range(nh))
    cfg = W.LayerConfig("classify", nh, d, F, H, H, C, F, "bf16", heads, 0.8)
    intended = [W.STATIC, W.DYNAMIC, W.STATIC, W.DYNAMIC, W.DYNAMIC, W.STATIC]
    xs = []
    for s in range(2):
        x = W.make_layer_inputs(cfg, seed=50 + s)
        rng = np.random.default_rng(60 + s)
        for h, t in enumerate(intended):
            src = (W.bf16_bits_to_f32(x.K_cur[h]) if t == W.STATIC
                   else np.tile(W.bf16_bits_to_f32(x.K_hist[h][x.frame_slot[1 + h % 3]]), (C, 1)))
            q = 2.0 * src + 0.2 * rng.standard_normal(src.shape).astype(np.float32)
            x.Q[h] = W.f32_to_bf16_bits(q.astype(np.float32))
        xs.append(x)
    _case("classify")
    prof = _profile(cfg, xs)
    got = prof.classify(alpha=0.8, sink_frames=1, transition_frames=1)
    ref_mass = sum(_oracle_mass(x, H, F, 1 / math.sqrt(d)) for x in xs)
    want = oracle.classify_heads(ref_mass, H, 1, 1, 0.8).tolist()
    assert got == want == intended, (got, want, intended)
