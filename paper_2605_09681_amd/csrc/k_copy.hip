// k_copy.hip -- structured frame gather for static heads (Sec. 4.2, Eq. 2),
// kept-segment compaction for dynamic heads (Sec. 4.3: the compressed cache is
// the union of the kept segments of every history frame), and the write of a
// finished chunk's frames into the rolling cache's slots.
//
// Both are pure HBM copies: each byte of a retained K/V row is read once and
// written once with 16-byte vector accesses.  A workgroup moves one tile of one
// "piece" (a contiguous run of tokens inside one logical frame, so one slot
// lookup per workgroup) for K and V together; all loads of a thread are issued
// before its stores.
#include "fkv_internal.h"

namespace fkv {
namespace {

constexpr int kThreads = 256;
constexpr int kVPT = 4;                      // 16-byte vectors per thread per tensor
constexpr int kTile = kThreads * kVPT;       // vectors per workgroup per tensor

__device__ __forceinline__ void copy_tile(const u32x4 *__restrict__ srcK,
                                          const u32x4 *__restrict__ srcV,
                                          u32x4 *__restrict__ dstK,
                                          u32x4 *__restrict__ dstV, int64_t n_vecs,
                                          int64_t first) {
    u32x4 k[kVPT], v[kVPT];
#pragma unroll
    for (int i = 0; i < kVPT; ++i) {
        const int64_t idx = first + (int64_t)i * kThreads;
        if (idx < n_vecs) {
            k[i] = __builtin_nontemporal_load(srcK + idx);
            v[i] = __builtin_nontemporal_load(srcV + idx);
        }
    }
#pragma unroll
    for (int i = 0; i < kVPT; ++i) {
        const int64_t idx = first + (int64_t)i * kThreads;
        if (idx < n_vecs) {
            dstK[idx] = k[i];
            dstV[idx] = v[i];
        }
    }
}

// grid: x = tile within a frame, y = kept frame y of the head, z = static head list index.
__global__ __launch_bounds__(kThreads) void static_copy_kernel(StaticCopyArgs a) {
    const int li = blockIdx.z;
    const int h = a.heads.head[li];
    const int n_kept = a.n_kept[li];
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) a.kv_len[h] = n_kept * a.F;
    const int y = blockIdx.y;
    if (y >= n_kept) return;
    // Kept frames are [0, n_first) followed by [n_first + gap, ...): the sink
    // frames, then the most recent frames (the transition anchor frames).
    const int t = y < a.n_first[li] ? y : y + a.gap[li];
    const int64_t frame_bytes = (int64_t)a.F * a.row_bytes;
    const int64_t src_off = ((int64_t)h * a.cap + a.slots.slot[t]) * frame_bytes;
    const int64_t dst_off = (int64_t)h * a.slab * a.row_bytes + (int64_t)y * frame_bytes;
    copy_tile((const u32x4 *)(a.K_hist + src_off), (const u32x4 *)(a.V_hist + src_off),
              (u32x4 *)(a.Kc + dst_off), (u32x4 *)(a.Vc + dst_off), a.frame_vecs,
              (int64_t)blockIdx.x * kTile + threadIdx.x);
}

// grid: x = tile within a piece, y = kept piece p of the head, z = dynamic head list index.
// Piece p is sub-piece f = p % m of the q = p / m -th kept segment (m pieces per
// segment, one per frame when segments span frames).  The destination is
// p * piece_tokens because only the last segment of the history can be short
// and it sorts last.
__global__ __launch_bounds__(kThreads) void dyn_copy_kernel(DynCopyArgs a) {
    const int li = blockIdx.z;
    const int h = a.heads.head[li];
    const int p = blockIdx.y;
    const int q = p / a.pieces_per_seg;
    const int f = p - q * a.pieces_per_seg;
    if (q >= a.n_seg) return;
    const int g = a.kept_seg[(int64_t)h * a.n_seg + q];
    if (g < 0 || g >= a.n_seg) return;
    const int64_t start = (int64_t)g * a.L + (int64_t)f * a.piece_tokens;  // logical token
    if (start >= (int64_t)a.H * a.F) return;                              // short last segment
    const int t = (int)(start / a.F);
    const int64_t pos = start - (int64_t)t * a.F;
    const int64_t src_off = (((int64_t)h * a.cap + a.slots.slot[t]) * a.F + pos) * a.row_bytes;
    const int64_t dst_off = ((int64_t)h * a.slab + (int64_t)p * a.piece_tokens) * a.row_bytes;
    copy_tile((const u32x4 *)(a.K_hist + src_off), (const u32x4 *)(a.V_hist + src_off),
              (u32x4 *)(a.Kc + dst_off), (u32x4 *)(a.Vc + dst_off), a.piece_vecs,
              (int64_t)blockIdx.x * kTile + threadIdx.x);
}

// grid: x = tile within a frame, y = new frame f, z = head.
__global__ __launch_bounds__(kThreads) void append_kernel(AppendArgs a) {
    const int f = blockIdx.y, h = blockIdx.z;
    const int64_t src = ((int64_t)h * a.n_frames + f) * a.frame_vecs;
    const int64_t dst = ((int64_t)h * a.cap + a.slots.slot[f]) * a.frame_vecs;
    copy_tile((const u32x4 *)a.K_new + src, (const u32x4 *)a.V_new + src, (u32x4 *)a.K_hist + dst,
              (u32x4 *)a.V_hist + dst, a.frame_vecs, (int64_t)blockIdx.x * kTile + threadIdx.x);
}

}  // namespace

hipError_t launch_static_copy(const StaticCopyArgs &a, int max_kept, hipStream_t s) {
    if (a.heads.n == 0) return hipSuccess;
    const int64_t tiles = (a.frame_vecs + kTile - 1) / kTile;
    dim3 grid((unsigned)(tiles > 0 ? tiles : 1), (unsigned)(max_kept > 0 ? max_kept : 1),
              (unsigned)a.heads.n);
    hipLaunchKernelGGL(static_copy_kernel, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_dyn_copy(const DynCopyArgs &a, int max_pieces, hipStream_t s) {
    if (a.heads.n == 0 || max_pieces <= 0) return hipSuccess;
    const int64_t tiles = (a.piece_vecs + kTile - 1) / kTile;
    dim3 grid((unsigned)tiles, (unsigned)max_pieces, (unsigned)a.heads.n);
    hipLaunchKernelGGL(dyn_copy_kernel, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_append(const AppendArgs &a, int n_heads, hipStream_t s) {
    if (a.n_frames == 0) return hipSuccess;
    const unsigned tiles = (unsigned)((a.frame_vecs + kTile - 1) / kTile);
    hipLaunchKernelGGL(append_kernel, dim3(tiles, (unsigned)a.n_frames, (unsigned)n_heads), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
