// select_common.h -- the BottomK keep rule of dynamic heads (Sec. 4.3, Eq. 3),
// shared by the stand-alone selection kernel and the fused select + compact
// kernel so that both decide every segment identically.
//
// Candidates are ordered by the key (isNaN(s), s, g): a NaN score sorts after
// every number, -0 and +0 are equal, and the lower segment index wins a tie.
// The key is a strict total order, so the ranks inside a selection group are
// a permutation and exactly kk = min(k, |group|) members are kept.  Segments
// that touch the sink frames or the most recent frames are forced and always
// kept; they are not members of any group.
#pragma once

#include "fkv_internal.h"

namespace fkv {
namespace sel {

// The key (isNaN(s), s, g) as one unsigned 64-bit integer whose order is the
// key's: the high word maps the score's bits monotonically (-0 taken as +0,
// negative scores bit-inverted, the sign bit set on the others, every NaN
// 0xffffffff), the low word is the index g >= 0.  Comparing two keys is one
// integer compare -- no branches or lane-mask logic per candidate.
__device__ __forceinline__ uint64_t sort_key(float s, int g) {
    uint32_t b = __float_as_uint(s);
    b = b == 0x80000000u ? 0u : b;
    b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
    b = __builtin_isnan(s) ? 0xffffffffu : b;
    return ((uint64_t)b << 32) | (uint32_t)g;
}

__device__ __forceinline__ bool key_less(float sa, int ga, float sb, int gb) {
    return sort_key(sa, ga) < sort_key(sb, gb);
}

// Logical frames [first, last] that segment g covers.  F and L divide one
// another (the host checks it), so this is small 32-bit arithmetic: a
// segment is a 1/(F/L) share of one frame, or L/F whole frames (the last
// segment of the history possibly fewer).
template <class A>
__device__ __forceinline__ void seg_frames(const A &a, int g, int *first, int *last) {
    if (a.L <= a.F) {
        *first = *last = g / (a.F / a.L);
    } else {
        const int m = a.L / a.F;
        *first = g * m;
        *last = min(*first + m, a.H) - 1;
    }
}

// The keep rule of list entry li: sink and recent frames, selection scope and
// k.  Read once per selection (each field is a load from the launch
// arguments), ahead of the work that needs it.
struct Rule {
    int sink, recent, scope, k;
};
template <class A>
__device__ __forceinline__ Rule rule_of(const A &a, int li) {
    return Rule{a.sink[li], a.recent[li], a.scope[li], a.k[li]};
}

// Does segment g intersect logical frames [0, sink) or [H - recent, H)?
template <class A>
__device__ __forceinline__ bool is_forced(const A &a, const Rule &r, int g) {
    int first, last;
    seg_frames(a, g, &first, &last);
    return first < r.sink || last >= a.H - r.recent;
}

// Tokens of segment g (only the last segment of the history can be short).
template <class A>
__device__ __forceinline__ int seg_tokens(const A &a, int g) {
    if (a.L <= a.F) return a.L;
    int first, last;
    seg_frames(a, g, &first, &last);
    return (last - first + 1) * a.F;
}

// The helpers take any argument block with the fields F, L, H and n_seg (and,
// for rule_of, the per-list-entry arrays sink, recent, scope and k):
// SelectArgs, SelectCopyArgs, ScoreArgs.

// Keep decision of a non-forced segment g, given the keys of all n_seg
// segments in LDS (sort_key, the largest key for a forced segment): its rank
// inside its group (one frame's segments for FKV_SCOPE_FRAME, all segments
// otherwise) is below kk.
template <class A>
__device__ __forceinline__ bool keep_by_rank(const A &a, const Rule &r, const uint64_t *keys, int g) {
    int lo = 0, hi = a.n_seg;
    if (r.scope == FKV_SCOPE_FRAME) {
        const int spf = a.F / a.L;
        lo = (g / spf) * spf;
        hi = lo + spf;
    }
    const int kk = r.k;
    const uint64_t kg = keys[g];
    int rank = 0;
    // eight candidates per step, their LDS reads issued together (one read
    // latency per step rather than per candidate); indices past the group are
    // clamped to its last member and not counted.  Neither g itself (equal
    // key) nor a forced segment (largest key) precedes g.
    for (int g0 = lo; g0 < hi && rank < kk; g0 += 8) {
        uint64_t kv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) kv[i] = keys[min(g0 + i, hi - 1)];
#pragma unroll
        for (int i = 0; i < 8; ++i) rank += (int)((g0 + i < hi) & (kv[i] < kg));
    }
    return rank < kk;
}

// n_seg <= 64: one wave decides head h's keep set, lane g holding candidate
// g; a candidate's rank counts the smaller keys of its group, read from the
// other lanes with v_readlane one candidate at a time (no LDS round trip, no
// barrier), then a ballot and a masked bit count give the output positions.
// Same rule and result as the general path below.
template <class A>
__device__ __forceinline__ void select_one_wave(const A &a, const Rule &r, int h, const float *s,
                                                int32_t *kept_seg, int32_t *kv_len, int lane) {
    const int n = a.n_seg;
    const int g = lane;
    const bool valid = g < n;
    const bool f = valid && is_forced(a, r, g);
    const uint64_t key = valid && !f ? sort_key(s[g], g) : ~0ull;
    int lo = 0, hi = n;
    if (r.scope == FKV_SCOPE_FRAME) {
        const int spf = a.F / a.L;
        lo = (g / spf) * spf;
        hi = lo + spf;
    }
    const uint32_t klo = (uint32_t)key, khi = (uint32_t)(key >> 32);
    int rank = 0;
    for (int j = 0; j < n; ++j) {
        const uint64_t kj = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)khi, j) << 32) |
                            (uint32_t)__builtin_amdgcn_readlane((int)klo, j);
        rank += (int)((j >= lo) & (j < hi) & (kj < key));
    }
    const bool kp = valid && (f || rank < r.k);
    const uint64_t mask = __ballot(kp);
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
    if (kp) kept_seg[(int64_t)h * n + below] = g;
    if (valid && g >= __popcll(mask)) kept_seg[(int64_t)h * n + g] = -1;
    int tokens = kp ? seg_tokens(a, g) : 0;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) tokens += __shfl_xor(tokens, off);
    if (lane == 0) kv_len[h] = tokens;
}

// One workgroup decides head h's keep set (rule r) from its scores
// s[0..n_seg) in LDS and writes kept_seg[h] (ascending, -1 padded) and
// kv_len[h]; with at most 64 segments its first wave does it alone
// (select_one_wave).  keys (n_seg), forced and keep (n_seg bytes each) are
// LDS scratch.  Every thread of the workgroup calls it (it contains
// barriers); nthreads is the workgroup size.
template <class A>
__device__ __forceinline__ void select_from_lds(const A &a, const Rule &r, int h, const float *s,
                                                uint64_t *keys, unsigned char *forced, unsigned char *keep,
                                                int32_t *kept_seg, int32_t *kv_len, int tid,
                                                int nthreads) {
    const int n = a.n_seg;
    if (n <= 64) {
        if (tid < 64) select_one_wave(a, r, h, s, kept_seg, kv_len, tid);
        return;
    }
    for (int g = tid; g < n; g += nthreads) {
        const bool f = is_forced(a, r, g);
        forced[g] = f ? 1 : 0;
        keys[g] = f ? ~0ull : sort_key(s[g], g);
    }
    __syncthreads();
    for (int g = tid; g < n; g += nthreads)
        keep[g] = (forced[g] || keep_by_rank(a, r, keys, g)) ? 1 : 0;
    __syncthreads();
    if (tid < 64) {
        int base = 0;
        int tokens = 0;
        for (int c0 = 0; c0 < n; c0 += 64) {
            const int g = c0 + tid;
            const bool kp = g < n && keep[g];
            const uint64_t mask = __ballot(kp);
            const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
            if (kp) {
                kept_seg[(int64_t)h * n + base + below] = g;
                tokens += seg_tokens(a, g);
            }
            base += __popcll(mask);
        }
        for (int p = base + tid; p < n; p += 64) kept_seg[(int64_t)h * n + p] = -1;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) tokens += __shfl_xor(tokens, off);
        if (tid == 0) kv_len[h] = tokens;
    }
}

}  // namespace sel
}  // namespace fkv
