"""Pins of the head-profiling oracle (Sec. 4.1, Eq. 1): the attention mass per
key frame and the static/dynamic decision, against torch's softmax, closed
forms and hand-made mass tables."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W


def _keys(rng, n, d):
    return W.f32_to_bf16_bits(rng.standard_normal((n, d)).astype(np.float32))


def test_mass_matches_torch_softmax(oracle_lib):
    rng = np.random.default_rng(0)
    F, H, C, d = 5, 4, 2, 16
    Q, Kc, Kq = _keys(rng, C * F, d), _keys(rng, H * F, d), _keys(rng, C * F, d)
    mass = oracle.attention_mass(Q, Kc, Kq, F, 0.3)
    q = torch.from_numpy(W.bf16_bits_to_f32(Q).astype(np.float64))
    k = torch.from_numpy(W.bf16_bits_to_f32(np.concatenate([Kc, Kq])).astype(np.float64))
    p = torch.softmax(0.3 * q @ k.T, dim=1).sum(dim=0).numpy()
    np.testing.assert_allclose(mass, p.reshape(-1, F).sum(axis=1), rtol=1e-12, atol=1e-12)


def test_mass_closed_forms(oracle_lib):
    rng = np.random.default_rng(1)
    F, d, Lq = 4, 8, 6
    Kc, Kq = _keys(rng, 3 * F + 2, d), _keys(rng, Lq, d)        # a partial last history block
    # rows sum to one: the total mass is the number of query rows
    Q = _keys(rng, Lq, d)
    m = oracle.attention_mass(Q, Kc, Kq, F, 0.5)
    assert abs(m.sum() - Lq) < 1e-12
    # Q = 0: uniform attention, every key gets Lq / Lk
    m0 = oracle.attention_mass(np.zeros((Lq, d), np.uint16), Kc, Kq, F, 0.5)
    Lk = Kc.shape[0] + Lq
    sizes = np.diff(np.minimum(np.arange(0, -(-Lk // F) + 1) * F, Lk))
    np.testing.assert_allclose(m0, Lq * sizes / Lk, rtol=1e-13)


def test_classify_closed_forms():
    # H = 4 history frames + C = 2 chunk frames; sink 1, transition 1, alpha 0.8
    rows = np.array([
        [0.0, 0.0, 0.0, 1.0, 2.0, 3.0],   # all mass on transition + chunk: ratio 1 -> static
        [5.0, 1.0, 1.0, 1.0, 1.0, 1.0],   # sink excluded: (1+1+1)/(5) = 0.6 -> dynamic
        [9.0, 0.0, 0.5, 0.5, 1.0, 2.0],   # (0.5+3)/(4) = 0.875 -> static
        [0.0, 1.0, 0.0, 1.0, 2.0, 0.0],   # (1+2)/4 = 0.75 -> dynamic
        [0.0, 1.0, 0.0, 1.0, 3.0, 0.0],   # (1+3)/5 = 0.8, not above alpha -> dynamic
    ])
    got = oracle.classify_heads(rows, hist_frames=4, sink_frames=1, transition_frames=1, alpha=0.8)
    assert got.tolist() == [W.STATIC, W.DYNAMIC, W.STATIC, W.DYNAMIC, W.DYNAMIC]
    # a lower alpha turns the 0.75 and 0.8 heads static; no history: ratio 1 -> static
    got = oracle.classify_heads(rows, 4, 1, 1, 0.5)
    assert got.tolist() == [W.STATIC, W.STATIC, W.STATIC, W.STATIC, W.STATIC]
    assert oracle.classify_heads(np.array([[1.0, 2.0]]), 0, 1, 1, 0.8).tolist() == [W.STATIC]


def test_mass_separates_local_from_spread_heads(oracle_lib):
    """A head whose queries match the current chunk's keys is classified
    static; one whose queries match an old frame is dynamic."""
    rng = np.random.default_rng(2)
    F, H, C, d = 8, 6, 2, 32
    hist = rng.standard_normal((H * F, d)).astype(np.float32)
    cur = rng.standard_normal((C * F, d)).astype(np.float32)
    local_q = cur + 0.1 * rng.standard_normal(cur.shape).astype(np.float32)
    spread_q = np.tile(hist[F:2 * F], (C, 1)) + 0.1 * rng.standard_normal(cur.shape).astype(np.float32)
    b = W.f32_to_bf16_bits
    m = np.stack([oracle.attention_mass(b(q), b(hist), b(cur), F, 0.5) for q in (local_q, spread_q)])
    assert oracle.classify_heads(m, H, 1, 1, 0.8).tolist() == [W.STATIC, W.DYNAMIC]
