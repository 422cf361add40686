// k_select.hip -- BottomK keep-set selection of dynamic heads (Sec. 4.3, Eq. 3).
//
// One workgroup per dynamic head.  The head's scores are staged in LDS; every
// thread takes candidate segments and computes each one's rank inside its
// selection group (the number of group members with a smaller key (isNaN(s),
// s, g)); a candidate is kept when its rank is below kk = min(k, |group|).
// Because the key is a strict total order (the index breaks every tie), the
// ranks of a group are a permutation and exactly kk members are kept.  Forced
// segments (touching the sink frames or the most recent frames) are always
// kept.  Wave 0 then walks the segments in ascending order 64 at a time,
// turning the keep flags into output positions with a ballot and a masked bit
// count (mbcnt), and writes kept_seg and kv_len.
#include "fkv_internal.h"

namespace fkv {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool key_less(float sa, int ga, float sb, int gb) {
    const bool na = __builtin_isnan(sa), nb = __builtin_isnan(sb);
    if (na != nb) return nb;          // a finite/inf score precedes a NaN
    if (!na) {
        if (sa < sb) return true;     // -0 and +0 compare equal here
        if (sa > sb) return false;
    }
    return ga < gb;
}

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
    __shared__ float s[FKV_MAX_SEGMENTS];
    __shared__ unsigned char keep[FKV_MAX_SEGMENTS];
    __shared__ unsigned char forced[FKV_MAX_SEGMENTS];

    const int li = blockIdx.x;
    const int h = a.heads.head[li];
    const int n = a.n_seg;
    const int tid = threadIdx.x;
    const int64_t HF = (int64_t)a.H * a.F;
    const int sink = a.sink[li], recent = a.recent[li];
    const int kk = a.k[li];                       // min(k, |group|), from the host
    const bool per_frame = a.scope[li] == FKV_SCOPE_FRAME;
    const int segs_per_frame = per_frame ? a.F / a.L : 0;

    for (int g = tid; g < n; g += kThreads) {
        s[g] = a.scores[(int64_t)h * a.score_stride + g];
        const int64_t x0 = (int64_t)g * a.L;
        const int64_t x1 = x0 + a.L < HF ? x0 + a.L : HF;
        const int first = (int)(x0 / a.F), last = (int)((x1 - 1) / a.F);
        forced[g] = (first < sink || last >= a.H - recent) ? 1 : 0;
    }
    __syncthreads();

    for (int g = tid; g < n; g += kThreads) {
        bool kp = forced[g];
        if (!kp) {
            int lo = 0, hi = n;
            if (per_frame) {
                lo = (g / segs_per_frame) * segs_per_frame;
                hi = lo + segs_per_frame;
            }
            const float sg = s[g];
            int rank = 0;
            for (int g2 = lo; g2 < hi && rank < kk; ++g2)
                rank += (!forced[g2] && g2 != g && key_less(s[g2], g2, sg, g)) ? 1 : 0;
            kp = rank < kk;
        }
        keep[g] = kp ? 1 : 0;
    }
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
                a.kept_seg[(int64_t)h * n + base + below] = g;
                const int64_t x0 = (int64_t)g * a.L;
                tokens += (int)((x0 + a.L < HF ? x0 + a.L : HF) - x0);
            }
            base += __popcll(mask);
        }
        for (int p = base + tid; p < n; p += 64) a.kept_seg[(int64_t)h * n + p] = -1;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) tokens += __shfl_xor(tokens, off);
        if (tid == 0) a.kv_len[h] = tokens;
    }
}

}  // namespace

hipError_t launch_select(const SelectArgs &a, hipStream_t s) {
    if (a.heads.n == 0) return hipSuccess;
    hipLaunchKernelGGL(select_kernel, dim3(a.heads.n), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
