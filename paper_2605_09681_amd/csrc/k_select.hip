// k_select.hip -- BottomK keep-set selection of dynamic heads (Sec. 4.3, Eq. 3),
// the stand-alone kernel used when a head has more segments than the fused
// select + compact kernel handles (k_copy.hip).
//
// One workgroup per dynamic head.  The head's scores are staged in LDS; every
// thread takes candidate segments and applies the keep rule of
// select_common.h (rank inside the selection group below kk, forced segments
// always kept).  Wave 0 then walks the segments in ascending order 64 at a
// time, turning the keep flags into output positions with a ballot and a
// masked bit count (mbcnt), and writes kept_seg and kv_len.
#include "select_common.h"

namespace fkv {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
    __shared__ float s[FKV_MAX_SEGMENTS];
    __shared__ unsigned char keep[FKV_MAX_SEGMENTS];
    __shared__ unsigned char forced[FKV_MAX_SEGMENTS];

    const int li = blockIdx.x;
    const int h = a.heads.head[li];
    const int n = a.n_seg;
    const int tid = threadIdx.x;

    for (int g = tid; g < n; g += kThreads) {
        s[g] = a.scores[(int64_t)h * a.score_stride + g];
        forced[g] = sel::is_forced(a, li, g) ? 1 : 0;
    }
    __syncthreads();

    for (int g = tid; g < n; g += kThreads)
        keep[g] = (forced[g] || sel::keep_by_rank(a, li, s, forced, g)) ? 1 : 0;
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
                tokens += sel::seg_tokens(a, g);
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
