"""FP8 variant of the chunk attention (App. F: the method combined with FP8
attention) -- TEST INFRASTRUCTURE, like the rest of ``oracle/``.

Plain numpy definitions of what the FP8 path computes, in this order:

1. Per head, the attention inputs are quantised to OCP FP8 E4M3 (the "fn"
   variant: no infinities, max 448, NaN = S.1111.111) with round-to-nearest-
   even:
   * keys [Kc[0:kv_len]; K_cur] are first smoothed by subtracting their
     per-channel mean mu (exact fp64 sum, one rounding to fp32) -- softmax is
     unchanged because q . mu is the same for every key of a row -- then
     scaled by inv_k = fp32(448 / amax|K - mu|);
   * queries are scaled by inv_q = fp32(448 / amax|Q|);
   * values [Vc[0:kv_len]; V_cur] per channel c by inv_v[c] = fp32(448 / amax_c|V|);
   every scaled value is one fp32 multiply (after one fp32 subtract for keys)
   and then rounded to E4M3.  Dequantisation scales are s = fp32(amax / 448);
   an all-zero tensor (or channel) has inv = s = 0.
2. Attention on the dequantised values, exactly (fp64), with the caller's
   softmax scale.

The GPU kernel additionally rounds the probabilities to E4M3 before the value
product; that rounding is the only difference it may have from step 2, and the
tests bound it.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

E4M3_MAX = 448.0


def e4m3_encode(x) -> np.ndarray:
    """Round float32 values to E4M3 codes (uint8), nearest-even, saturating at
    +-448.  Normal numbers 2^(e-7) * (1 + m/8) for e = 1..15 (e = 15 only up to
    m = 6); subnormals m * 2^-9."""
    x = np.asarray(x, dtype=np.float32)
    a = np.abs(x).astype(np.float64)
    sign = (np.signbit(x)).astype(np.uint8) << 7
    # quantum of the binade holding a: 2^(floor(log2 a) - 3), at least 2^-9
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.maximum(e, -6.0)
    q = np.exp2(e - 3.0)
    n = np.round(a / q)                       # numpy rounds halves to even
    v = n * q
    v = np.minimum(v, E4M3_MAX)
    # encode v (now exactly representable)
    code = np.zeros(a.shape, np.uint8)
    nz = v > 0
    ev = np.floor(np.log2(np.where(nz, v, 1.0)))
    sub = nz & (ev < -6)
    norm = nz & ~sub
    m_sub = np.round(v / 2.0 ** -9).astype(np.int64)
    code[sub] = m_sub[sub].astype(np.uint8)
    E = (ev + 7).astype(np.int64)
    M = np.round((v / np.exp2(ev) - 1.0) * 8).astype(np.int64)
    code[norm] = ((E[norm] << 3) | M[norm]).astype(np.uint8)
    return code | sign


def e4m3_decode(code) -> np.ndarray:
    """Values (float64) of E4M3 codes; NaN codes decode to NaN."""
    c = np.asarray(code, dtype=np.uint8).astype(np.int64)
    s = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 7
    v = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    v = np.where((c & 0x7F) == 0x7F, np.nan, v)
    return s * v


def _scale_pair(amax: np.ndarray):
    amax = np.asarray(amax, np.float32)
    with np.errstate(divide="ignore"):
        inv = np.where(amax > 0, np.float32(E4M3_MAX) / amax, np.float32(0)).astype(np.float32)
    s = (amax / np.float32(E4M3_MAX)).astype(np.float32)
    return inv, s


@dataclass
class Fp8Head:
    q8: np.ndarray      # [Lq][d] uint8
    k8: np.ndarray      # [kv_len + Lq][d] uint8 (history rows, then chunk rows)
    v8: np.ndarray      # [kv_len + Lq][d] uint8
    s_q: np.float32
    s_k: np.float32
    mu_k: np.ndarray    # [d] float32
    s_v: np.ndarray     # [d] float32
    inv_q: np.float32 = np.float32(0)
    inv_k: np.float32 = np.float32(0)
    inv_v: np.ndarray = None  # [d] float32


def quantize_head(Q, K, V) -> Fp8Head:
    """Step 1 for one head.  Q: [Lq][d]; K, V: [n_keys][d] (history rows then
    chunk rows), all float32 (bf16 values widened exactly)."""
    Q = np.asarray(Q, np.float32)
    K = np.asarray(K, np.float32)
    V = np.asarray(V, np.float32)
    n = K.shape[0]
    mu = (K.astype(np.float64).sum(axis=0) / n).astype(np.float32)
    Kt = (K - mu).astype(np.float32)                     # one fp32 subtract
    inv_k, s_k = _scale_pair(np.abs(Kt).max())
    inv_q, s_q = _scale_pair(np.abs(Q).max())
    inv_v, s_v = _scale_pair(np.abs(V).max(axis=0))
    k8 = e4m3_encode((Kt * inv_k).astype(np.float32))
    q8 = e4m3_encode((Q * inv_q).astype(np.float32))
    v8 = e4m3_encode((V * inv_v[None, :]).astype(np.float32))
    return Fp8Head(q8, k8, v8, np.float32(s_q), np.float32(s_k), mu, s_v.astype(np.float32),
                   np.float32(inv_q), np.float32(inv_k), inv_v.astype(np.float32))


def dequantized(h: Fp8Head):
    """(q, k, v) float64 values the FP8 kernel multiplies (k without mu)."""
    return (e4m3_decode(h.q8) * float(h.s_q), e4m3_decode(h.k8) * float(h.s_k),
            e4m3_decode(h.v8) * h.s_v.astype(np.float64)[None, :])


def p_rounding_sigma(q, k, v, scale: float, rows, p_bias_log2: float = 6.0) -> np.ndarray:
    """Standard deviation, per output element, of the error that rounding every
    probability to E4M3 adds to a softmax-weighted average normalised by the
    same rounded probabilities.  The probabilities are taken as
    p'_k = 2^p_bias_log2 * exp(z_k - max z) (the kernel's scaling, whose lagging
    running maximum only makes its values larger, i.e. rounded more finely);
    a normal E4M3 value has relative error within +-2^-4, a subnormal one
    (below 2^-6) absolute error within +-2^-10, both taken as uniform:
        sigma_d = sqrt(sum_k var_k (v_kd - o_d)^2) / sum_k p'_k.
    q: [Lq][d]; k, v: [n_keys][d] (float64, dequantised); returns [n_rows][d]."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    out = np.empty((len(rows), v.shape[1]))
    for i, r in enumerate(rows):
        z = scale * (k @ q[r])
        p = np.exp(z - z.max()) * 2.0 ** p_bias_log2
        o = (p @ v) / p.sum()
        out[i] = np.sqrt((p_rounding_var(p)[:, None] * (v - o[None, :]) ** 2).sum(axis=0)) / p.sum()
    return out


def p_rounding_var(p) -> np.ndarray:
    """Variance of the E4M3 rounding error of each (scaled) probability."""
    p = np.asarray(p, np.float64)
    return np.where(p >= 2.0 ** -6, (2.0 ** -4 * p) ** 2, (2.0 ** -10) ** 2) / 3.0
