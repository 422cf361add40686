"""Pins of the FP8 oracle (``oracle/fp8.py``) against facts it does not derive
from itself: torch's float8_e4m3fn conversion (a library routine that also
rounds to nearest even), the E4M3 code table, exact rational means, the
rounding bound of a 3-bit mantissa, and the shift invariance of softmax that
licenses subtracting the key mean."""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import fp8
import workloads as W


def _torch_encode(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_torch_for_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = fp8.e4m3_decode(codes)
    nan = np.isnan(ref)
    assert (np.isnan(got) == nan).all() and nan.sum() == 2   # S.1111.111
    np.testing.assert_array_equal(got[~nan], ref[~nan])
    assert got[0x7E] == 448.0 and got[0x01] == 2.0 ** -9 and got[0x38] == 1.0


def test_encode_matches_torch_on_values_and_midpoints():
    vals = fp8.e4m3_decode(np.arange(0, 0x7F, dtype=np.uint8))      # every finite magnitude
    mids = (vals[:-1] + vals[1:]) / 2                                # exact ties
    rng = np.random.default_rng(0)
    rand = np.exp(rng.uniform(np.log(1e-4), np.log(440.0), 20000))
    x = np.concatenate([vals, mids, rand, rng.uniform(-3, 3, 5000)]).astype(np.float32)
    x = np.concatenate([x, -x])
    np.testing.assert_array_equal(fp8.e4m3_encode(x), _torch_encode(x))


def test_encode_round_trip_and_error_bound():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], np.uint8)
    back = fp8.e4m3_encode(fp8.e4m3_decode(codes).astype(np.float32))
    same = (back == codes) | ((codes == 0x80) & (back == 0x80))
    assert same.all()
    rng = np.random.default_rng(1)
    x = rng.uniform(2.0 ** -6, 448, 100000).astype(np.float32)     # normal range
    rel = np.abs(fp8.e4m3_decode(fp8.e4m3_encode(x)) - x) / x
    assert rel.max() <= 2.0 ** -4 * (1 + 1e-7)                      # half an ulp of a 3-bit mantissa
    y = rng.uniform(0, 2.0 ** -6, 10000).astype(np.float32)         # subnormals: absolute half quantum
    assert np.abs(fp8.e4m3_decode(fp8.e4m3_encode(y)) - y).max() <= 2.0 ** -10


def _head(seed, n_hist=40, lq=24, d=16, bias=0.0):
    rng = np.random.default_rng(seed)
    K = W.bf16_bits_to_f32(W.f32_to_bf16_bits((rng.standard_normal((n_hist + lq, d)) + bias).astype(np.float32)))
    V = W.bf16_bits_to_f32(W.f32_to_bf16_bits((rng.standard_normal((n_hist + lq, d)) * np.linspace(0.1, 4, d)).astype(np.float32)))
    Q = W.bf16_bits_to_f32(W.f32_to_bf16_bits(rng.standard_normal((lq, d)).astype(np.float32)))
    return Q, K, V


def test_quantize_head_definitions():
    Q, K, V = _head(2, bias=3.0)
    h = fp8.quantize_head(Q, K, V)
    # mean: exact rational mean rounded once to fp32
    for c in range(K.shape[1]):
        m = sum(Fraction(float(v)) for v in K[:, c]) / K.shape[0]
        assert np.float32(float(m)) == h.mu_k[c] or abs(float(m) - float(h.mu_k[c])) <= 2 ** -24 * abs(float(m))
    # the largest magnitude of each scaled tensor (per channel for V) lands on +-448
    assert (np.abs(fp8.e4m3_decode(h.k8)).max() == 448.0)
    assert (np.abs(fp8.e4m3_decode(h.q8)).max() == 448.0)
    assert (np.abs(fp8.e4m3_decode(h.v8)).max(axis=0) == 448.0).all()
    # dequantised values within the E4M3 rounding bound of the originals
    q, k, v = fp8.dequantized(h)
    Kt = (K - h.mu_k).astype(np.float64)
    for orig, deq, s in ((Q.astype(np.float64), q, float(h.s_q)), (Kt, k, float(h.s_k)),
                         (V.astype(np.float64), v, h.s_v.astype(np.float64)[None, :])):
        err = np.abs(deq - orig)
        bound = np.maximum(np.abs(orig) * 2.0 ** -4 * 1.0001, 2.0 ** -10 * np.broadcast_to(s, orig.shape) * 1.0001)
        assert (err <= bound + 1e-12).all()
    # an all-zero tensor quantises to zeros with zero scales
    z = fp8.quantize_head(np.zeros((4, 8), np.float32), np.zeros((6, 8), np.float32), np.zeros((6, 8), np.float32))
    assert z.s_q == 0 and z.s_k == 0 and (z.s_v == 0).all() and not z.k8.any()


def test_key_smoothing_leaves_attention_unchanged(oracle_lib):
    """Adding the per-channel key mean back changes every logit of a row by
    the same q . mu, so the fp64 attention of the dequantised values is the
    same with or without it."""
    Q, K, V = _head(3, bias=2.0)
    h = fp8.quantize_head(Q, K, V)
    q, k, v = fp8.dequantized(h)
    n_hist = K.shape[0] - Q.shape[0]
    a = oracle.attention_rows(q, k[:n_hist], v[:n_hist], k[n_hist:], v[n_hist:], 0.25)[0]
    k2 = k + h.mu_k.astype(np.float64)[None, :]
    b = oracle.attention_rows(q, k2[:n_hist], v[:n_hist], k2[n_hist:], v[n_hist:], 0.25)[0]
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_dequantized_attention_error_matches_rounding_model(oracle_lib):
    """The output error of quantising V alone follows the same law as the
    probability rounding the kernel adds (a weighted average of relative
    errors uniform in +-2^-4): measured against p_rounding_sigma evaluated for
    V's relative errors, the normalised error has unit-order spread, and the
    whole quantisation stays within a few percent (relative L2) of the exact
    attention."""
    Q, K, V = _head(4, n_hist=600, lq=16, d=32)
    h = fp8.quantize_head(Q, K, V)
    q, k, v = fp8.dequantized(h)
    n = K.shape[0] - Q.shape[0]
    rows = np.arange(16, dtype=np.int32)
    Kf, Vf = K.astype(np.float64), V.astype(np.float64)
    only_v = oracle.attention_rows(Q.astype(np.float64), Kf[:n], v[:n], Kf[n:], v[n:], 0.17)[0]
    exact = oracle.attention_rows(Q, K[:n], V[:n], K[n:], V[n:], 0.17)[0]
    sig = fp8.p_rounding_sigma(Q, Kf, Vf, 0.17, rows, p_bias_log2=12.0)   # all normal: relative model
    z = (only_v - exact) / sig
    assert 0.3 < np.sqrt((z ** 2).mean()) < 2.0 and np.abs(z).max() < 7
    deq = oracle.attention_rows(q, k[:n], v[:n], k[n:], v[n:], 0.17)[0]
    assert np.linalg.norm(exact - deq) / np.linalg.norm(exact) < 0.1
