// k_select.hip -- BottomK keep-set selection of dynamic heads (Sec. 4.3, Eq. 3),
// the stand-alone kernel used when a head has more segments than the fused
// select + compact kernel handles (k_copy.hip).
//
// One workgroup per dynamic head.  The head's scores are staged in LDS; every
// thread takes candidate segments and applies the keep rule of
// select_common.h (rank inside the selection group below kk, forced segments
// always kept).  Wave 0 then walks the segments in ascending order 64 at a
// time, turning the keep flags into output positions with a ballot and a
// masked bit count (mbcnt), and writes kept_seg and kv_len
// (sel::select_from_lds, which the fused score + select kernel also runs).
#include "select_common.h"

namespace fkv {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
    __shared__ uint64_t keys[FKV_MAX_SEGMENTS];
    __shared__ float s[FKV_MAX_SEGMENTS];
    __shared__ unsigned char keep[FKV_MAX_SEGMENTS];
    __shared__ unsigned char forced[FKV_MAX_SEGMENTS];

    const int li = blockIdx.x;
    const int h = a.heads.head[li];
    const int tid = threadIdx.x;
    const sel::Rule rule = sel::rule_of(a, li);
    for (int g = tid; g < a.n_seg; g += kThreads) s[g] = a.scores[(int64_t)h * a.score_stride + g];
    __syncthreads();
    sel::select_from_lds(a, rule, h, s, keys, forced, keep, a.kept_seg, a.kv_len, tid, kThreads);
}

}  // namespace

hipError_t launch_select(const SelectArgs &a, hipStream_t s) {
    if (a.heads.n == 0) return hipSuccess;
    hipLaunchKernelGGL(select_kernel, dim3(a.heads.n), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
