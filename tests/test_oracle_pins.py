"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

The paper prints no worked example for any step of the hot path, so the
oracle is pinned by:

* Eq. 2 static kept set: hand-listed closed-form cases (overlapping sink and
  recent windows, empty history, the paper's one-anchor-frame rule), and the
  frame gather against numpy fancy indexing.
* Sec. 4.3 first-block proxy (pooled over heads): exact rational arithmetic,
  the closed form (a - b) / (a + b) of a repeating and a sign-alternating
  head, reduction to the per-head score for one or 2^k identical heads, torch
  cosine of the concatenation over heads.
* Eq. 3 similarity: exact rational arithmetic (``fractions`` + 80-digit
  ``decimal``, rounded to fp32 by hand) on tiny bf16 and fp32 inputs for
  segments shorter than, equal to and longer than a frame; closed forms
  (identical -> 1, negated -> -1, positively scaled -> 1, orthogonal -> 0, zero
  -> 0); a partner/index test where exactly one adjacent-frame transition is
  negated, including the last history frame against the current chunk; slot
  permutation invariance; agreement with torch's fp64 cosine_similarity; the
  AR(1) statistic E[s] = rho.
* Eq. 3 BottomK: brute force over all subsets on tiny inputs with ties, signed
  zeros and NaNs (the kept subset is the unique one whose keys all precede the
  evicted keys); crafted all-equal / +-0 / NaN cases; kept-count formula;
  budgets k = 0 and k >= group size (the "w/o dynamic-head cache" ablation
  and no pruning).
* Compaction: against numpy slicing of the logical token sequence.
* Eq. 4 attention: torch's fp64 scaled_dot_product_attention (the library
  routine for the plain definition); Q = 0 gives the mean of V; a single key
  returns its value; the two-key closed form (a logistic weight);
  duplicating every key/value pair changes nothing; the log-normaliser
  against scipy's logsumexp; attention over the compressed cache equals
  full attention with evicted keys masked out; keeping everything equals
  full attention over the uncompressed history.
"""
import itertools
import math
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

import oracle
import workloads as W

getcontext().prec = 80


# ---------------------------------------------------------------------------
# helpers (exact arithmetic)
# ---------------------------------------------------------------------------
def _f32_neighbours(c: Decimal):
    f = np.float32(float(c))
    if Decimal(float(f)) > c:
        hi, lo = f, np.nextafter(f, np.float32(-np.inf))
    else:
        lo, hi = f, np.nextafter(f, np.float32(np.inf))
    return lo, hi


def round_decimal_to_f32(c: Decimal):
    """Correctly rounded (nearest-even) fp32 of an exact decimal value, and a
    flag telling whether c lies within 1e-12 (relative) of a rounding midpoint,
    where an fp64 computation may legitimately round the other way."""
    if c == 0:
        return np.float32(0.0), False
    lo, hi = _f32_neighbours(c)
    mid = (Decimal(float(lo)) + Decimal(float(hi))) / 2
    if c < mid:
        r = lo
    elif c > mid:
        r = hi
    else:
        r = lo if (lo.view(np.uint32) & 1) == 0 else hi
    near = abs(c - mid) <= abs(c) * Decimal("1e-12")
    return np.float32(r), near


def exact_cos_f32(a: np.ndarray, b: np.ndarray):
    fa = [Fraction(float(x)) for x in a.ravel()]
    fb = [Fraction(float(x)) for x in b.ravel()]
    dot = sum(x * y for x, y in zip(fa, fb))
    na = sum(x * x for x in fa)
    nb = sum(y * y for y in fb)
    if na * nb == 0:
        return np.float32(0.0), False
    prod = na * nb
    c = (Decimal(dot.numerator) / Decimal(dot.denominator)) / \
        (Decimal(prod.numerator) / Decimal(prod.denominator)).sqrt()
    return round_decimal_to_f32(c)


def logical_tokens(hist_head, frame_slot, H):
    """[H*F][d] logical history via numpy fancy indexing."""
    return np.asarray(hist_head)[np.asarray(frame_slot[:H])].reshape(H * hist_head.shape[1], -1)


def to_f(x, dtype):
    return W.storage_to_f32(x, dtype).astype(np.float64)


# ---------------------------------------------------------------------------
# Eq. 2: static kept set
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("H,sink,recent,expect", [
    (4, 1, 1, [0, 3]),                      # tiny config: frame 0 + most recent frame
    (21, 1, 6, [0, 15, 16, 17, 18, 19, 20]),  # 480P static heads
    (21, 1, 1, [0, 20]),                    # paper's rule: sink + transition anchor frame
    (21, 3, 4, [0, 1, 2, 17, 18, 19, 20]),  # StreamingLLM-style 3 sink + 4 recent
    (0, 1, 6, []),                          # first AR step: nothing cached
    (3, 2, 2, [0, 1, 2]),                   # overlapping windows, each frame once
    (5, 0, 0, []),                          # "w/o static-head cache"
    (2, 5, 0, [0, 1]),                      # sink larger than the history
    (6, 0, 9, [0, 1, 2, 3, 4, 5]),          # recent larger than the history
    (7, 2, 0, [0, 1]),
])
def test_static_frames_closed_form(oracle_lib, H, sink, recent, expect):
    got = oracle.static_frames(H, sink, recent)
    assert got.tolist() == expect


def test_static_frames_count_formula(oracle_lib):
    for H in range(0, 12):
        for sink in range(0, 6):
            for recent in range(0, 8):
                a, b = min(sink, H), min(recent, H)
                overlap = max(0, a - (H - b))
                assert len(oracle.static_frames(H, sink, recent)) == a + b - overlap


def test_gather_frames_matches_fancy_indexing(oracle_lib):
    rng = np.random.default_rng(1)
    hist = rng.standard_normal((6, 5, 8), dtype=np.float32)
    slot = np.array([3, 0, 5, 1, 2], np.int32)
    frames = np.array([0, 2, 4], np.int32)
    got = oracle.gather_frames(hist, slot, frames)
    np.testing.assert_array_equal(got, hist[slot[frames]].reshape(-1, 8))


# ---------------------------------------------------------------------------
# Eq. 3: segment similarity
# ---------------------------------------------------------------------------
def _tiny_stream(dtype, H, F, d, C, seed, rho=0.7):
    frames = W.ar1_key_frames(seed, 1, H + C, F, d, rho, dtype)[0]
    hist = np.ascontiguousarray(frames[:H])
    cur = np.ascontiguousarray(frames[H:].reshape(C * F, d))
    return hist, cur


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("F,L", [(4, 1), (4, 2), (4, 4), (4, 8), (4, 12), (6, 3)])
def test_score_exact_rational(oracle_lib, dtype, F, L):
    H, d, C = 5, 6, 2
    for seed in range(3):
        hist, cur = _tiny_stream(dtype, H, F, d, C, seed)
        slot = np.arange(H, dtype=np.int32)
        s32, s64 = oracle.score_head(hist, slot, cur, H, L)
        tok = logical_tokens(to_f(hist, dtype), slot, H)
        nxt = np.concatenate([tok[F:], to_f(cur, dtype)[:F]])  # token x -> x + F
        n = -(-H * F // L)
        assert s32.shape == (n,)
        for g in range(n):
            x0, x1 = g * L, min(g * L + L, H * F)
            want, near = exact_cos_f32(tok[x0:x1], nxt[x0:x1])
            if not near:
                assert s32[g].view(np.uint32) == want.view(np.uint32), (g, s32[g], want)


def test_score_closed_forms(oracle_lib):
    rng = np.random.default_rng(7)
    H, F, d = 4, 5, 16
    base = W.f32_to_bf16_bits(rng.standard_normal((F, d), dtype=np.float32))
    basef = W.bf16_bits_to_f32(base)
    slot = np.arange(H, dtype=np.int32)

    def score(frames_f32, cur_f32):
        hist = W.f32_to_bf16_bits(np.stack(frames_f32))
        cur = W.f32_to_bf16_bits(cur_f32)
        return oracle.score_head(hist, slot, cur, H, F)[0]

    # identical frames -> exactly 1
    s = score([basef] * H, basef)
    assert (s == np.float32(1.0)).all()
    # positive scaling by powers of two (exact in bf16) -> exactly 1
    s = score([basef, 2 * basef, 8 * basef, 0.25 * basef], 0.5 * basef)
    assert (s == np.float32(1.0)).all()
    # negation -> exactly -1
    s = score([basef, -basef, basef, -basef], basef)
    assert (s == np.float32(-1.0)).all()
    # orthogonal pair (disjoint supports) -> exactly 0
    a = np.zeros((F, d), np.float32); a[:, : d // 2] = basef[:, : d // 2]
    b = np.zeros((F, d), np.float32); b[:, d // 2:] = basef[:, d // 2:]
    s = score([a, b, a, b], a)
    assert (s == 0.0).all()
    # a zero segment -> 0 (no division by zero)
    z = np.zeros((F, d), np.float32)
    s = score([basef, z, basef, basef], basef)
    assert s[0] == 0.0 and s[1] == 0.0 and s[2] == 1.0 and s[3] == 1.0


@pytest.mark.parametrize("L", [3, 6, 12])
def test_score_partner_is_next_frame(oracle_lib, L):
    """Only the transition 2 -> 3 (and the last frame -> current chunk) is a
    negation; every other adjacent pair is identical.  Catches a partner taken
    from the previous frame, a missing shift, or a wrong current-chunk row."""
    rng = np.random.default_rng(3)
    H, F, d = 6, 6, 8
    X = W.bf16_bits_to_f32(W.f32_to_bf16_bits(rng.standard_normal((F, d), dtype=np.float32)))
    frames = [X, X, X, -X, -X, -X]
    cur = np.concatenate([X, 2 * X])               # first chunk frame = -(last frame)
    hist = W.f32_to_bf16_bits(np.stack(frames))
    s = oracle.score_head(hist, np.arange(H, dtype=np.int32), W.f32_to_bf16_bits(cur), H, L)[0]
    tok_frame = lambda g: (g * L) // F
    for g, v in enumerate(s):
        if L <= F:
            t = tok_frame(g)
            expect = -1.0 if t in (2, 5) else 1.0
            assert v == np.float32(expect), (g, v)
        else:  # segment of L/F frames: mixed transitions give intermediate values
            frames_in = range(tok_frame(g), min(tok_frame(g) + L // F, H))
            n_neg = sum(1 for t in frames_in if t in (2, 5))
            expect = (len(frames_in) - 2 * n_neg) / len(frames_in)
            assert abs(float(v) - expect) < 1e-6, (g, v, expect)


def test_score_slot_permutation_invariant(oracle_lib):
    H, F, d, L = 5, 4, 8, 2
    hist, cur = _tiny_stream("bf16", H, F, d, 1, seed=11)
    ident = oracle.score_head(hist, np.arange(H, dtype=np.int32), cur, H, L)[0]
    perm = np.array([4, 0, 6, 2, 5], np.int32)          # logical -> physical
    phys = np.zeros((7, F, d), np.uint16)
    phys[perm] = hist
    s = oracle.score_head(phys, perm, cur, H, L)[0]
    np.testing.assert_array_equal(s.view(np.uint32), ident.view(np.uint32))


def test_score_matches_torch_cosine(oracle_lib):
    H, F, d, L = 6, 10, 32, 5
    hist, cur = _tiny_stream("bf16", H, F, d, 1, seed=5, rho=0.5)
    slot = np.arange(H, dtype=np.int32)
    _, s64 = oracle.score_head(hist, slot, cur, H, L)
    tok = torch.from_numpy(logical_tokens(to_f(hist, "bf16"), slot, H))
    nxt = torch.cat([tok[F:], torch.from_numpy(to_f(cur, "bf16"))[:F]])
    a = tok.reshape(-1, L * d)
    b = nxt.reshape(-1, L * d)
    ref = torch.nn.functional.cosine_similarity(a, b, dim=1, eps=0.0).numpy()
    np.testing.assert_allclose(s64, ref, rtol=0, atol=1e-13)


def test_score_ar1_statistic(oracle_lib):
    """E[s] = rho for AR(1) keys; sd about (1 - rho^2)/sqrt(L d)."""
    rho, H, F, d = 0.9, 8, 64, 64
    hist, cur = _tiny_stream("f32", H, F, d, 1, seed=2, rho=rho)
    s = oracle.score_head(hist, np.arange(H, dtype=np.int32), cur, H, F)[0]
    sd = (1 - rho ** 2) / math.sqrt(F * d)
    assert abs(float(s.mean()) - rho) < 4 * sd / math.sqrt(H) + 2e-3


# ---------------------------------------------------------------------------
# rolling cache: chunk frames written through the ring write pointer
# ---------------------------------------------------------------------------
def test_append_frames_matches_assignment(oracle_lib):
    rng = np.random.default_rng(4)
    hist = rng.standard_normal((6, 3, 4), dtype=np.float32)
    want = hist.copy()
    new = rng.standard_normal((2, 3, 4), dtype=np.float32)
    slot = np.array([4, 1], np.int32)
    oracle.append_frames(hist, new, slot)
    want[slot] = new
    np.testing.assert_array_equal(hist, want)


@pytest.mark.parametrize("window,C,pinned", [(7, 2, 1), (21, 3, 1), (6, 3, 0), (9, 3, 2)])
def test_ring_cache_holds_sink_and_latest_frames(oracle_lib, window, C, pinned):
    """Writing each finished chunk through the write pointer keeps, in the
    logical order of ring_frame_slots, the pinned sink frames followed by the
    most recent frames: frame v is stamped with the value v."""
    F, d = 2, 3
    hist = np.full((window, F, d), -1.0, np.float32)
    for i in range(12):
        slots = W.ring_frame_slots(i, C, window, pinned)
        produced = i * C
        H = len(slots)
        if H:
            got = hist[slots][:, 0, 0].astype(int).tolist()
            n_sink = min(pinned, H)
            expect = list(range(n_sink)) + list(range(produced - (H - n_sink), produced))
            assert got == expect, (i, got, expect)
        chunk = np.arange(produced, produced + C, dtype=np.float32)[:, None, None] * np.ones((1, F, d), np.float32)
        oracle.append_frames(hist, chunk, W.chunk_write_slots(i, C, window, pinned))


# ---------------------------------------------------------------------------
# Sec. 4.3 first-block proxy: one similarity from the keys of all heads
# ---------------------------------------------------------------------------
def _tiny_heads(dtype, n_heads, H, F, d, C, seed, rho=0.7):
    frames = W.ar1_key_frames(seed, n_heads, H + C, F, d, rho, dtype)
    hist = np.ascontiguousarray(frames[:, :H])
    cur = np.ascontiguousarray(frames[:, H:].reshape(n_heads, C * F, d))
    return hist, cur


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("F,L", [(4, 2), (4, 4), (4, 8)])
def test_pooled_score_exact_rational(oracle_lib, dtype, F, L):
    """Cosine over the concatenation of all heads' segment keys, in exact
    rational arithmetic, rounded to fp32 by hand."""
    nh, H, d, C = 3, 4, 5, 1
    for seed in range(2):
        hist, cur = _tiny_heads(dtype, nh, H, F, d, C, seed)
        slot = np.arange(H, dtype=np.int32)
        s32, _ = oracle.score_pooled(hist, slot, cur, H, L)
        toks = [logical_tokens(to_f(hist[h], dtype), slot, H) for h in range(nh)]
        nxts = [np.concatenate([toks[h][F:], to_f(cur[h], dtype)[:F]]) for h in range(nh)]
        for g in range(-(-H * F // L)):
            x0, x1 = g * L, min(g * L + L, H * F)
            a = np.concatenate([t[x0:x1] for t in toks])
            b = np.concatenate([t[x0:x1] for t in nxts])
            want, near = exact_cos_f32(a, b)
            if not near:
                assert s32[g].view(np.uint32) == want.view(np.uint32), (g, s32[g], want)


def test_pooled_score_closed_forms(oracle_lib):
    """Head A repeats its frame (cosine 1, squared norm a per frame), head B
    alternates sign (cosine -1, squared norm b): the pooled cosine is
    (a - b) / (a + b).  With one head the pooled score is that head's score;
    with 2 or 4 identical heads it equals the per-head score bit for bit."""
    rng = np.random.default_rng(17)
    H, F, d = 4, 3, 8
    X = W.bf16_bits_to_f32(W.f32_to_bf16_bits(rng.standard_normal((F, d), dtype=np.float32)))
    Y = W.bf16_bits_to_f32(W.f32_to_bf16_bits(rng.standard_normal((F, d), dtype=np.float32)))
    slot = np.arange(H, dtype=np.int32)
    hist = W.f32_to_bf16_bits(np.stack([np.stack([X] * H), np.stack([Y, -Y, Y, -Y])]))
    cur = W.f32_to_bf16_bits(np.stack([X, Y]))
    s32, s64 = oracle.score_pooled(hist, slot, cur, H, F)
    a, b = float((X.astype(np.float64) ** 2).sum()), float((Y.astype(np.float64) ** 2).sum())
    np.testing.assert_allclose(s64, (a - b) / (a + b), rtol=1e-15, atol=0)

    h1, c1 = _tiny_heads("bf16", 1, H, F, d, 1, seed=3)
    for L in (1, 3, 6):
        one = oracle.score_pooled(h1, slot, c1, H, L)[0]
        per = oracle.score_head(h1[0], slot, c1[0], H, L)[0]
        np.testing.assert_array_equal(one.view(np.uint32), per.view(np.uint32))
        for n in (2, 4):
            rep = oracle.score_pooled(np.repeat(h1, n, 0), slot, np.repeat(c1, n, 0), H, L)[0]
            np.testing.assert_array_equal(rep.view(np.uint32), per.view(np.uint32))


def test_pooled_score_matches_torch_cosine(oracle_lib):
    nh, H, F, d, L = 4, 5, 6, 16, 3
    hist, cur = _tiny_heads("bf16", nh, H, F, d, 1, seed=9, rho=0.6)
    perm = np.array([2, 0, 4, 1, 3], np.int32)
    phys = np.zeros((nh, 5, F, d), np.uint16)
    phys[:, perm] = hist
    _, s64 = oracle.score_pooled(phys, perm, cur, H, L)
    slot = np.arange(H, dtype=np.int32)
    toks = [torch.from_numpy(logical_tokens(to_f(hist[h], "bf16"), slot, H)) for h in range(nh)]
    nxts = [torch.cat([toks[h][F:], torch.from_numpy(to_f(cur[h], "bf16"))[:F]]) for h in range(nh)]
    a = torch.cat([t.reshape(-1, L * d) for t in toks], dim=1)
    b = torch.cat([t.reshape(-1, L * d) for t in nxts], dim=1)
    ref = torch.nn.functional.cosine_similarity(a, b, dim=1, eps=0.0).numpy()
    np.testing.assert_allclose(s64, ref, rtol=0, atol=1e-13)


# ---------------------------------------------------------------------------
# Eq. 3: BottomK selection
# ---------------------------------------------------------------------------
def _key(s, g):
    s = float(s)
    return (1, 0.0, g) if math.isnan(s) else (0, s + 0.0, g)


def _brute_select(scores, H, F, L, sink, recent, k, scope):
    n = -(-H * F // L)
    forced, groups = set(), {}
    for g in range(n):
        x0, x1 = g * L, min(g * L + L, H * F)
        touches_sink = x0 < sink * F
        touches_recent = x1 > (H - recent) * F
        if touches_sink or touches_recent:
            forced.add(g)
        else:
            groups.setdefault(x0 // F if scope == W.SCOPE_FRAME else 0, []).append(g)
    kept = set(forced)
    for members in groups.values():
        kk = min(k, len(members))
        found = []
        for sub in itertools.combinations(members, kk):
            rest = [g for g in members if g not in sub]
            if all(_key(scores[a], a) < _key(scores[b], b) for a in sub for b in rest):
                found.append(sub)
        assert len(found) == 1
        kept |= set(found[0])
    return sorted(kept)


@pytest.mark.parametrize("scope,F,L", [(W.SCOPE_GLOBAL, 4, 4), (W.SCOPE_GLOBAL, 4, 8),
                                       (W.SCOPE_FRAME, 4, 1), (W.SCOPE_FRAME, 6, 2),
                                       (W.SCOPE_GLOBAL, 6, 2)])
def test_select_brute_force(oracle_lib, scope, F, L):
    rng = np.random.default_rng(0)
    palette = np.array([0.5, -0.0, 0.0, 0.25, np.nan, -1.0, 0.5, 1.0, -np.nan], np.float32)
    for trial in range(60):
        H = int(rng.integers(1, 6))
        n = -(-H * F // L)
        scores = palette[rng.integers(0, len(palette), n)]
        sink, recent = int(rng.integers(0, 3)), int(rng.integers(0, 3))
        k = int(rng.integers(0, 5))
        kept, cnt = oracle.select_head(scores, H, F, L, sink, recent, k, scope)
        want = _brute_select(scores, H, F, L, sink, recent, k, scope)
        assert kept[:cnt].tolist() == want, (trial, scores, sink, recent, k)
        assert (kept[cnt:] == -1).all()


def test_select_crafted(oracle_lib):
    H, F, L = 6, 4, 4  # one segment per frame, global group
    eq = np.full(6, 0.75, np.float32)
    kept, cnt = oracle.select_head(eq, H, F, L, 0, 0, 3, W.SCOPE_GLOBAL)
    assert kept[:cnt].tolist() == [0, 1, 2]           # ties -> lowest indices
    pm = np.array([0.0, -0.0, 0.0, -0.0, 1.0, 1.0], np.float32)
    kept, cnt = oracle.select_head(pm, H, F, L, 0, 0, 2, W.SCOPE_GLOBAL)
    assert kept[:cnt].tolist() == [0, 1]              # -0 == +0
    nan = np.array([np.nan, 0.9, np.nan, 0.1, 0.5, 0.2], np.float32)
    kept, cnt = oracle.select_head(nan, H, F, L, 0, 0, 4, W.SCOPE_GLOBAL)
    assert kept[:cnt].tolist() == [1, 3, 4, 5]        # NaN evicted first
    kept, cnt = oracle.select_head(nan, H, F, L, 0, 0, 5, W.SCOPE_GLOBAL)
    assert kept[:cnt].tolist() == [0, 1, 3, 4, 5]     # then NaN by index
    signed = np.array([np.nan, 0.9, -np.nan, 0.1, 0.5, 0.2], np.float32)
    assert np.signbit(signed[2]) and not np.signbit(signed[0])
    kept, cnt = oracle.select_head(signed, H, F, L, 0, 0, 5, W.SCOPE_GLOBAL)
    assert kept[:cnt].tolist() == [0, 1, 3, 4, 5]     # the NaN's sign does not order it
    low = np.array([0.9, 0.1, 0.8, 0.2, 0.7, 0.3], np.float32)
    kept, cnt = oracle.select_head(low, H, F, L, 1, 1, 2, W.SCOPE_GLOBAL)
    assert kept[:cnt].tolist() == [0, 1, 3, 5]        # sink 0, recent 5, two least similar


def test_select_counts(oracle_lib):
    rng = np.random.default_rng(4)
    for H, F, L, scope in [(21, 1560, 1560, 1), (21, 1560, 390, 0), (21, 1560, 4680, 1),
                           (20, 1560, 4680, 1), (7, 10, 5, 0), (7, 10, 5, 1)]:
        n = -(-H * F // L)
        s = rng.standard_normal(n).astype(np.float32)
        for sink in (0, 1, 3):
            for recent in (0, 1, 2):
                for k in (0, 1, 2, 50):
                    kept, cnt = oracle.select_head(s, H, F, L, sink, recent, k, scope)
                    forced = [g for g in range(n)
                              if g * L < sink * F or min(g * L + L, H * F) > (H - recent) * F]
                    cands = [g for g in range(n) if g not in forced]
                    if scope == 0:
                        per = {}
                        for g in cands:
                            per[(g * L) // F] = per.get((g * L) // F, 0) + 1
                        want = len(forced) + sum(min(k, m) for m in per.values())
                    else:
                        want = len(forced) + min(k, len(cands))
                    assert cnt == want
                    assert set(forced) <= set(kept[:cnt].tolist())
                    assert (np.diff(kept[:cnt]) > 0).all()


# ---------------------------------------------------------------------------
# compaction
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("F,L,H", [(4, 4, 5), (4, 2, 5), (4, 8, 5), (6, 12, 5), (6, 3, 4)])
def test_compact_matches_slicing(oracle_lib, F, L, H):
    rng = np.random.default_rng(9)
    d, cap = 8, H + 2
    hist = rng.integers(0, 65535, (cap, F, d)).astype(np.uint16)
    slot = rng.permutation(cap)[:H].astype(np.int32)
    n = -(-H * F // L)
    for _ in range(5):
        kept = np.sort(rng.permutation(n)[: int(rng.integers(0, n + 1))]).astype(np.int32)
        got = oracle.compact_head(hist, slot, kept, H, L)
        tok = hist[slot].reshape(H * F, d)
        want = (np.concatenate([tok[g * L: min(g * L + L, H * F)] for g in kept])
                if len(kept) else np.zeros((0, d), np.uint16))
        np.testing.assert_array_equal(got, want)


# ---------------------------------------------------------------------------
# Eq. 4: attention
# ---------------------------------------------------------------------------
def _rand(rng, shape, dtype, scale=1.0):
    return W.to_storage((rng.standard_normal(shape) * scale).astype(np.float32), dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attention_matches_torch_sdpa(oracle_lib, dtype):
    rng = np.random.default_rng(12)
    d, Lq, kv = 32, 9, 23
    Q, Kc, Vc = _rand(rng, (Lq, d), dtype, 2.0), _rand(rng, (kv, d), dtype), _rand(rng, (kv, d), dtype)
    Kcur, Vcur = _rand(rng, (Lq, d), dtype), _rand(rng, (Lq, d), dtype)
    scale = 0.3
    O, lse = oracle.attention_rows(Q, Kc, Vc, Kcur, Vcur, scale)
    q = torch.from_numpy(to_f(Q, dtype))[None, None]
    k = torch.from_numpy(np.concatenate([to_f(Kc, dtype), to_f(Kcur, dtype)]))[None, None]
    v = torch.from_numpy(np.concatenate([to_f(Vc, dtype), to_f(Vcur, dtype)]))[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale)[0, 0].numpy()
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)
    z = scale * (to_f(Q, dtype) @ k[0, 0].numpy().T)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=0, atol=1e-12)


def test_attention_special_cases(oracle_lib):
    rng = np.random.default_rng(13)
    d = 16
    # Q = 0: uniform weights -> mean of all values
    Q = np.zeros((3, d), np.float32)
    Kc, Vc = _rand(rng, (5, d), "f32"), _rand(rng, (5, d), "f32")
    Kcur, Vcur = _rand(rng, (3, d), "f32"), _rand(rng, (3, d), "f32")
    O, lse = oracle.attention_rows(Q, Kc, Vc, Kcur, Vcur, 1.0)
    mean = np.concatenate([Vc, Vcur]).astype(np.float64).mean(0)
    np.testing.assert_allclose(O, np.broadcast_to(mean, O.shape), atol=1e-14)
    np.testing.assert_allclose(lse, math.log(8.0), atol=1e-14)
    # a single key (empty history, one-token chunk) returns its value
    q1, k1, v1 = _rand(rng, (1, d), "f32"), _rand(rng, (1, d), "f32"), _rand(rng, (1, d), "f32")
    O, _ = oracle.attention_rows(q1, np.zeros((0, d), np.float32), np.zeros((0, d), np.float32), k1, v1, 0.7)
    np.testing.assert_array_equal(O[0], v1[0].astype(np.float64))
    # two keys: weight of key 1 is the logistic function of the logit gap
    k2 = _rand(rng, (1, d), "f32"); v2 = _rand(rng, (1, d), "f32")
    O, _ = oracle.attention_rows(q1, k2, v2, k1, v1, 0.5)
    z2 = 0.5 * float(q1[0].astype(np.float64) @ k2[0].astype(np.float64))
    z1 = 0.5 * float(q1[0].astype(np.float64) @ k1[0].astype(np.float64))
    w2 = 1.0 / (1.0 + math.exp(z1 - z2))
    np.testing.assert_allclose(O[0], w2 * v2[0] + (1 - w2) * v1[0], atol=1e-14)


def test_attention_duplicate_keys_invariant(oracle_lib):
    rng = np.random.default_rng(14)
    d, Lq, kv = 16, 5, 7
    Q, Kc, Vc = _rand(rng, (Lq, d), "bf16"), _rand(rng, (kv, d), "bf16"), _rand(rng, (kv, d), "bf16")
    Kcur, Vcur = _rand(rng, (Lq, d), "bf16"), _rand(rng, (Lq, d), "bf16")
    O1, _ = oracle.attention_rows(Q, Kc, Vc, Kcur, Vcur, 0.25)
    # duplicate the history AND the chunk keys: every weight doubles, output unchanged
    O2, _ = oracle.attention_rows(Q, np.concatenate([Kc, Kcur, Kc]), np.concatenate([Vc, Vcur, Vc]),
                                  Kcur, Vcur, 0.25)
    np.testing.assert_allclose(O1, O2, atol=1e-13)


def _layer(cfg, seed=0):
    return W.make_layer_inputs(cfg, seed=seed)


def _small_cfg(**kw):
    base = dict(name="small", n_heads=2, head_dim=16, frame_tokens=6, hist_frames=5, cap_frames=6,
                chunk_frames=2, seg_tokens=3, dtype="bf16",
                heads=(W.HeadBudget(W.STATIC, 1, 1), W.HeadBudget(W.DYNAMIC, 1, 0, 1, W.SCOPE_FRAME)),
                rho=0.8)
    base.update(kw)
    return W.LayerConfig(**base)


def test_compressed_attention_equals_masked_full_attention(oracle_lib):
    cfg = _small_cfg()
    x = _layer(cfg, seed=3)
    res = oracle.run_layer(cfg, x)
    H, F, L, d = cfg.hist_frames, cfg.frame_tokens, cfg.seg_tokens, cfg.head_dim
    for h in range(cfg.n_heads):
        tok = logical_tokens(to_f(x.K_hist[h], "bf16"), x.frame_slot, H)
        vtok = logical_tokens(to_f(x.V_hist[h], "bf16"), x.frame_slot, H)
        keep = np.zeros(H * F, bool)
        if cfg.heads[h].type == W.STATIC:
            for t in oracle.static_frames(H, cfg.heads[h].sink_frames, cfg.heads[h].recent_frames):
                keep[t * F:(t + 1) * F] = True
        else:
            for g in res.kept_seg[h][res.kept_seg[h] >= 0]:
                keep[g * L: min(g * L + L, H * F)] = True
        q = torch.from_numpy(to_f(x.Q[h], "bf16"))[None, None]
        k = torch.from_numpy(np.concatenate([tok, to_f(x.K_cur[h], "bf16")]))[None, None]
        v = torch.from_numpy(np.concatenate([vtok, to_f(x.V_cur[h], "bf16")]))[None, None]
        mask = torch.from_numpy(np.concatenate([keep, np.ones(cfg.lq, bool)]))[None, None, None]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask,
                                                               scale=1 / math.sqrt(d))[0, 0].numpy()
        np.testing.assert_allclose(res.O[h], ref, atol=1e-12)


@pytest.mark.parametrize("L,scope", [(3, W.SCOPE_FRAME), (6, W.SCOPE_GLOBAL), (12, W.SCOPE_GLOBAL)])
def test_no_pruning_equals_full_attention(oracle_lib, L, scope):
    """Keep 100% (dynamic k >= group size, static recent = H): the compressed
    cache is the whole history in order and attention is full attention."""
    H = 5
    cfg = _small_cfg(seg_tokens=L, heads=(W.HeadBudget(W.STATIC, 1, H),
                                          W.HeadBudget(W.DYNAMIC, 1, 0, 99, scope)))
    x = _layer(cfg, seed=4)
    res = oracle.run_layer(cfg, x)
    F, d = cfg.frame_tokens, cfg.head_dim
    for h in range(cfg.n_heads):
        full_k = logical_tokens(x.K_hist[h], x.frame_slot, H)
        full_v = logical_tokens(x.V_hist[h], x.frame_slot, H)
        np.testing.assert_array_equal(res.Kc[h], full_k)
        np.testing.assert_array_equal(res.Vc[h], full_v)
        O, _ = oracle.attention_rows(x.Q[h], full_k, full_v, x.K_cur[h], x.V_cur[h], 1 / math.sqrt(d))
        np.testing.assert_array_equal(res.O[h], O)


def test_empty_budgets_attend_chunk_only(oracle_lib):
    """k = 0 and recent = 0 with no sink (the ablation rows dropping a head
    type's cache): attention covers the current chunk alone."""
    cfg = _small_cfg(heads=(W.HeadBudget(W.STATIC, 0, 0), W.HeadBudget(W.DYNAMIC, 0, 0, 0, W.SCOPE_FRAME)))
    x = _layer(cfg, seed=5)
    res = oracle.run_layer(cfg, x)
    assert (res.kv_len == 0).all()
    for h in range(2):
        q = torch.from_numpy(to_f(x.Q[h], "bf16"))[None, None]
        k = torch.from_numpy(to_f(x.K_cur[h], "bf16"))[None, None]
        v = torch.from_numpy(to_f(x.V_cur[h], "bf16"))[None, None]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=0.25)[0, 0].numpy()
        np.testing.assert_allclose(res.O[h], ref, atol=1e-12)
