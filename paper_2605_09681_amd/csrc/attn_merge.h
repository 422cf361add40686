// attn_merge.h -- the combination of a cut work item's partial results, shared
// by the bf16 and FP8 attention kernels: under the balanced schedule
// (attn_common.h) an item whose key tiles are split over several workgroups
// is computed in parts, each part stores its normalised output with its row
// maxima and sums in a slot of the attention workspace (device-scope stores,
// handover.h), and the workgroup whose part arrives last on the item's counter
// combines them.
#pragma once

#include "attn_common.h"
#include "handover.h"

namespace fkv {
namespace attn {

// Combines the parts of a cut item (list entry li, query tile qt; first tile
// ibase of the concatenated sequence, T tiles), for the 32 rows of wave block
// w.  With part maxima m_j, sums l_j and normalised outputs o_j of a row,
//   M = max_j m_j,  w_j = 2^(m_j - M) l_j,  L = sum_j w_j,  O = sum_j w_j o_j / L,
// and lse = ln 2 * M + ln L, the parts taken in schedule order.  Thread t of
// the NT that share the block handles row t % 32 and the block's uint2
// elements i * NT + t -- every element gets the same arithmetic whichever
// thread does it.  The parts were written in this launch by other
// workgroups, so they are read with device-scope loads; every other part is
// complete when its workgroup arrives, so nothing waits.
template <int D, int NT>
__device__ __forceinline__ void merge_rows(const AttnArgs &a, const Schedule &sc, int li, int qt, int64_t ibase,
                                           int T, int w, int t) {
    constexpr int MB = D / 32;             // 32-row blocks of O^T
    constexpr int kML = BM * D / 2;        // float offset of m within a slot
    constexpr int kVecs = MB * 4 * 64;     // uint2s (4 values) of one wave block's accumulators
    constexpr int kPer = kVecs / NT;
    const int h = a.heads.head[li];
    const int b0 = sc.owner(ibase), b1 = sc.owner(ibase + T - 1);
    // the item is b0's last segment unless b0's range starts with it, and the
    // first segment of every later workgroup up to b1
    const int s0 = sc.start(b0) == ibase ? 2 * b0 : 2 * b0 + 1;
    const int r = t & 31, row = w * 32 + r;
    const int qrow = qt * BM + row;
    float M = -__builtin_inff(), L = 0.f;
    float x[kPer][4] = {};
    for (int b = b0; b <= b1; ++b) {
        const float *p = a.part + (size_t)(b == b0 ? s0 : 2 * b) * slot_floats<D>();
        const float m = get_shared(p + kML + row), l = get_shared(p + kML + BM + row);
        uint2 v[kPer];
#pragma unroll
        for (int i = 0; i < kPer; ++i) v[i] = get_shared((const uint2 *)p + (size_t)w * kVecs + i * NT + t);
        const float Mn = fmaxf(M, m);
        const float s = __builtin_amdgcn_exp2f(M - Mn), wg = __builtin_amdgcn_exp2f(m - Mn) * l;
        M = Mn;
        L = L * s + wg;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            x[i][0] = x[i][0] * s + wg * bf16_lo(v[i].x);
            x[i][1] = x[i][1] * s + wg * bf16_hi(v[i].x);
            x[i][2] = x[i][2] * s + wg * bf16_lo(v[i].y);
            x[i][3] = x[i][3] * s + wg * bf16_hi(v[i].y);
        }
    }
    if (qrow >= a.Lq) return;
    if (a.lse && t < 32) a.lse[(size_t)h * a.Lq + qrow] = fmaf(M, 0.69314718055994530942f, logf(L));
    const float inv = 1.f / L;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int q = i * NT + t;
        const int mb = q / (4 * 64), g = (q / 64) % 4;
        const int d0 = 32 * mb + 8 * g + 4 * ((t & 63) >> 5);
        *(uint2 *)((uint16_t *)a.O + ((size_t)h * a.Lq + qrow) * D + d0) =
            pack_bf16x4(x[i][0] * inv, x[i][1] * inv, x[i][2] * inv, x[i][3] * inv);
    }
}

}  // namespace attn
}  // namespace fkv
