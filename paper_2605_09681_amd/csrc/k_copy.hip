// k_copy.hip -- structured frame gather for static heads (Sec. 4.2, Eq. 2),
// kept-segment compaction for dynamic heads (Sec. 4.3: the compressed cache is
// the union of the kept segments of every history frame), and the write of a
// finished chunk's frames into the rolling cache's slots.
//
// For heads with at most kFusedSelectMaxSeg segments the BottomK selection
// runs inside the compaction kernel: every copy workgroup re-derives its
// head's keep set from the scores (a few hundred comparisons, far cheaper than
// a separate launch), finds the segment of its kept position with a ballot,
// and copies it; one workgroup per head also writes kept_seg and kv_len.
//
// Both are pure HBM copies: each byte of a retained K/V row is read once and
// written once with 16-byte vector accesses.  A workgroup moves one tile of one
// "piece" (a contiguous run of tokens inside one logical frame, so one slot
// lookup per workgroup) for K and V together; all loads of a thread are issued
// before its stores.
#include "select_common.h"

namespace fkv {
namespace {

constexpr int kThreads = 256;
constexpr int kVPT = 4;                      // 16-byte vectors per thread per tensor
constexpr int kTile = kThreads * kVPT;       // vectors per workgroup per tensor

// Values every lane of the workgroup shares, read from memory: moving them to
// scalar registers keeps the base addresses scalar.
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Per-lane indices are 32-bit offsets from workgroup-uniform bases (a piece
// or frame holds far fewer than 2^32 vectors), so the accesses address off a
// scalar base register: few VGPRs, high occupancy.
// Copies tile `tile` (kTile vectors) of an n_vecs-vector run of K and V.
// Full tiles (all but a run's last) take a branch without per-vector bounds
// checks, which keeps the register count and the instruction count low.
__device__ __forceinline__ void copy_tile(const u32x4 *__restrict__ srcK,
                                          const u32x4 *__restrict__ srcV,
                                          u32x4 *__restrict__ dstK,
                                          u32x4 *__restrict__ dstV, int64_t n_vecs, int tile) {
    const uint32_t n = (uint32_t)n_vecs;
    const uint32_t f = (uint32_t)tile * kTile + threadIdx.x;
    auto at = [](const u32x4 *base, uint32_t idx) {  // byte offset idx*16 as a 32-bit value
        return (const u32x4 *)((const char *)base + idx * 16u);
    };
    auto atw = [](u32x4 *base, uint32_t idx) { return (u32x4 *)((char *)base + idx * 16u); };
    u32x4 k[kVPT], v[kVPT];
    if ((uint32_t)(tile + 1) * kTile <= n) {
#pragma unroll
        for (int i = 0; i < kVPT; ++i) {
            k[i] = __builtin_nontemporal_load(at(srcK, f + i * kThreads));
            v[i] = __builtin_nontemporal_load(at(srcV, f + i * kThreads));
        }
#pragma unroll
        for (int i = 0; i < kVPT; ++i) {
            *atw(dstK, f + i * kThreads) = k[i];
            *atw(dstV, f + i * kThreads) = v[i];
        }
        return;
    }
    // the run's last, partial tile: one vector of K and V at a time
    for (int i = 0; i < kVPT; ++i) {
        const uint32_t idx = f + (uint32_t)i * kThreads;
        if (idx < n) {
            const u32x4 a = __builtin_nontemporal_load(at(srcK, idx));
            const u32x4 b = __builtin_nontemporal_load(at(srcV, idx));
            *atw(dstK, idx) = a;
            *atw(dstV, idx) = b;
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
    const int64_t src_off = ((int64_t)h * a.cap + uniform(a.slots.slot[t])) * frame_bytes;
    const int64_t dst_off = (int64_t)h * a.slab * a.row_bytes + (int64_t)y * frame_bytes;
    copy_tile((const u32x4 *)(a.K_hist + src_off), (const u32x4 *)(a.V_hist + src_off),
              (u32x4 *)(a.Kc + dst_off), (u32x4 *)(a.Vc + dst_off), a.frame_vecs, blockIdx.x);
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
    const int g = uniform(a.kept_seg[(int64_t)h * a.n_seg + q]);
    if (g < 0 || g >= a.n_seg) return;
    const int64_t start = (int64_t)g * a.L + (int64_t)f * a.piece_tokens;  // logical token
    if (start >= (int64_t)a.H * a.F) return;                              // short last segment
    const int t = (int)(start / a.F);
    const int64_t pos = start - (int64_t)t * a.F;
    const int64_t src_off = (((int64_t)h * a.cap + uniform(a.slots.slot[t])) * a.F + pos) * a.row_bytes;
    const int64_t dst_off = ((int64_t)h * a.slab + (int64_t)p * a.piece_tokens) * a.row_bytes;
    copy_tile((const u32x4 *)(a.K_hist + src_off), (const u32x4 *)(a.V_hist + src_off),
              (u32x4 *)(a.Kc + dst_off), (u32x4 *)(a.Vc + dst_off), a.piece_vecs, blockIdx.x);
}

// grid as dyn_copy_kernel; n_seg <= kFusedSelectMaxSeg.  Every wave derives
// the keep set on its own, in registers: lane l holds the scores of segments
// l and 64 + l, the forced flags are two ballot masks, and each candidate's
// rank inside its group is counted over the group's members read with
// cross-lane permutes -- no LDS arrays and no barrier before the copy.
__global__ __launch_bounds__(kThreads) void select_copy_kernel(SelectCopyArgs A) {
    static_assert(kFusedSelectMaxSeg <= 128, "two 64-bit masks");
    const SelectArgs &a = A.sel;
    const DynCopyArgs &c = A.copy;
    const int li = blockIdx.z;
    const int h = a.heads.head[li];
    const int n = a.n_seg;
    const int lane = threadIdx.x & 63;
    const bool two = n > 64;  // uniform: a second block of segments 64..127

    const sel::Rule rule = sel::rule_of(a, li);
    const float *srow = a.scores + (int64_t)h * a.score_stride;
    const float s0 = lane < n ? srow[lane] : 0.f;
    const float s1 = two && 64 + lane < n ? srow[64 + lane] : 0.f;
    const uint64_t F0 = __ballot(lane < n && sel::is_forced(a, rule, lane));
    const uint64_t F1 = two ? __ballot(64 + lane < n && sel::is_forced(a, rule, 64 + lane)) : 0;
    const bool per_frame = rule.scope == FKV_SCOPE_FRAME;
    const int spf = per_frame ? a.F / a.L : 0;
    const int cnt = per_frame ? spf : n;  // group size, the same for every lane
    const int kk = rule.k;
    // keep flag of segment g (score sg): forced, or fewer than kk group
    // members precede it in the order (isNaN(s), s, g).  Every lane runs the
    // same trip count with all lanes active (the permutes read other lanes);
    // a lane past n works on segment 0 and its answer is dropped.
    auto keep = [&](int g, float sg) -> bool {
        const bool valid = g < n;
        const int gc = valid ? g : 0;
        const bool fg = gc < 64 ? (F0 >> gc) & 1 : (F1 >> (gc - 64)) & 1;
        const int lo = per_frame ? (gc / spf) * spf : 0;
        int rank = 0;
        for (int j = 0; j < cnt; ++j) {
            const int g2 = lo + j;
            const float v0 = __shfl(s0, g2 & 63);
            const float v1 = two ? __shfl(s1, g2 & 63) : 0.f;
            const float v = g2 >= 64 ? v1 : v0;
            const bool f2 = g2 < 64 ? (F0 >> g2) & 1 : (F1 >> (g2 - 64)) & 1;
            rank += (int)(!f2 & (g2 != gc) & sel::key_less(v, g2, sg, gc));
        }
        return valid && (fg || rank < kk);
    };
    const uint64_t m0 = __ballot(keep(lane, s0));
    const uint64_t m1 = two ? __ballot(keep(64 + lane, s1)) : 0;
    const int c0 = __popcll(m0);
    const int n_kept = c0 + __popcll(m1);
    auto below = [&](uint64_t m) {
        return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
    };

    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x < 64) {
        int tokens = 0;
        if ((m0 >> lane) & 1) {
            a.kept_seg[(int64_t)h * n + below(m0)] = lane;
            tokens += sel::seg_tokens(a, lane);
        }
        if ((m1 >> lane) & 1) {
            a.kept_seg[(int64_t)h * n + c0 + below(m1)] = 64 + lane;
            tokens += sel::seg_tokens(a, 64 + lane);
        }
        for (int p = n_kept + lane; p < n; p += 64) a.kept_seg[(int64_t)h * n + p] = -1;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) tokens += __shfl_xor(tokens, off);
        if (lane == 0) a.kv_len[h] = tokens;
    }

    const int p = blockIdx.y;
    const int q = p / c.pieces_per_seg;
    const int f = p - q * c.pieces_per_seg;
    if (q >= n_kept) return;
    // the segment at kept position q: the set bit of its mask with q bits below
    const bool in0 = q < c0;
    const uint64_t m = in0 ? m0 : m1;
    const int qq = in0 ? q : q - c0;
    const uint64_t hit = __ballot(((m >> lane) & 1) && below(m) == qq);
    const int g = uniform((in0 ? 0 : 64) + (int)__builtin_ctzll(hit));
    const int64_t start = (int64_t)g * c.L + (int64_t)f * c.piece_tokens;  // logical token
    if (start >= (int64_t)c.H * c.F) return;                              // short last segment
    const int t = (int)(start / c.F);
    const int64_t pos = start - (int64_t)t * c.F;
    const int64_t src_off = (((int64_t)h * c.cap + uniform(c.slots.slot[t])) * c.F + pos) * c.row_bytes;
    const int64_t dst_off = ((int64_t)h * c.slab + (int64_t)p * c.piece_tokens) * c.row_bytes;
    copy_tile((const u32x4 *)(c.K_hist + src_off), (const u32x4 *)(c.V_hist + src_off),
              (u32x4 *)(c.Kc + dst_off), (u32x4 *)(c.Vc + dst_off), c.piece_vecs, blockIdx.x);
}

// grid: x = tile within a frame, y = new frame f, z = head.
__global__ __launch_bounds__(kThreads) void append_kernel(AppendArgs a) {
    const int f = blockIdx.y, h = blockIdx.z;
    const int64_t src = ((int64_t)h * a.n_frames + f) * a.frame_vecs;
    const int64_t dst = ((int64_t)h * a.cap + uniform(a.slots.slot[f])) * a.frame_vecs;
    copy_tile((const u32x4 *)a.K_new + src, (const u32x4 *)a.V_new + src, (u32x4 *)a.K_hist + dst,
              (u32x4 *)a.V_hist + dst, a.frame_vecs, blockIdx.x);
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

hipError_t launch_select_copy(const SelectCopyArgs &a, int max_pieces, hipStream_t s) {
    const int64_t tiles = (a.copy.piece_vecs + kTile - 1) / kTile;
    dim3 grid((unsigned)tiles, (unsigned)max_pieces, (unsigned)a.sel.heads.n);
    hipLaunchKernelGGL(select_copy_kernel, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_append(const AppendArgs &a, int n_heads, hipStream_t s) {
    if (a.n_frames == 0) return hipSuccess;
    const unsigned tiles = (unsigned)((a.frame_vecs + kTile - 1) / kTile);
    hipLaunchKernelGGL(append_kernel, dim3(tiles, (unsigned)a.n_frames, (unsigned)n_heads), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
