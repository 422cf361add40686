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

__device__ __forceinline__ bool key_less(float sa, int ga, float sb, int gb) {
    const bool na = __builtin_isnan(sa), nb = __builtin_isnan(sb);
    if (na != nb) return nb;          // a finite/inf score precedes a NaN
    if (!na) {
        if (sa < sb) return true;     // -0 and +0 compare equal here
        if (sa > sb) return false;
    }
    return ga < gb;
}

// Logical frames [first, last] that segment g covers.  F and L divide one
// another (the host checks it), so this is small 32-bit arithmetic: a
// segment is a 1/(F/L) share of one frame, or L/F whole frames (the last
// segment of the history possibly fewer).
__device__ __forceinline__ void seg_frames(const SelectArgs &a, int g, int *first, int *last) {
    if (a.L <= a.F) {
        *first = *last = g / (a.F / a.L);
    } else {
        const int m = a.L / a.F;
        *first = g * m;
        *last = min(*first + m, a.H) - 1;
    }
}

// Does segment g intersect logical frames [0, sink) or [H - recent, H)?
__device__ __forceinline__ bool is_forced(const SelectArgs &a, int li, int g) {
    int first, last;
    seg_frames(a, g, &first, &last);
    return first < a.sink[li] || last >= a.H - a.recent[li];
}

// Tokens of segment g (only the last segment of the history can be short).
__device__ __forceinline__ int seg_tokens(const SelectArgs &a, int g) {
    if (a.L <= a.F) return a.L;
    int first, last;
    seg_frames(a, g, &first, &last);
    return (last - first + 1) * a.F;
}

// Keep decision of a non-forced segment g with score sg, given the scores s[]
// and forced flags of all n_seg segments (in LDS): its rank inside its group
// (one frame's segments for FKV_SCOPE_FRAME, all segments otherwise) is below
// kk.
__device__ __forceinline__ bool keep_by_rank(const SelectArgs &a, int li, const float *s,
                                             const unsigned char *forced, int g) {
    int lo = 0, hi = a.n_seg;
    if (a.scope[li] == FKV_SCOPE_FRAME) {
        const int spf = a.F / a.L;
        lo = (g / spf) * spf;
        hi = lo + spf;
    }
    const int kk = a.k[li];
    const float sg = s[g];
    int rank = 0;
    for (int g2 = lo; g2 < hi && rank < kk; ++g2)
        rank += (!forced[g2] && g2 != g && key_less(s[g2], g2, sg, g)) ? 1 : 0;
    return rank < kk;
}

}  // namespace sel
}  // namespace fkv
