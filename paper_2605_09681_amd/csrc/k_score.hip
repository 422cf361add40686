// k_score.hip -- segment-wise cosine similarity of adjacent frames for dynamic
// heads (Sec. 4.3, Eq. 3), per head or pooled over all heads.
//
// Segment g of the history is compared with the same token range one frame
// later.  Splitting every frame into units of U = min(L, F) tokens (a unit is
// a segment when L <= F, a whole frame otherwise), each score is a sum of
// per-(frame t, unit u) quantities:
//   SQ[t][u]  = sum over the unit's elements of K_t^2          (t = 0..H, frame H
//               being the first frame of the current chunk)
//   DOT[t][u] = sum over the unit's elements of K_t * K_{t+1}   (t = 0..H-1)
// with dot = sum DOT, na = sum SQ[t], nb = sum SQ[t+1] over the frames of the
// segment.
//
// Pass 1 (score_partials_kernel) streams the cache once: a workgroup owns a
// 256-vector column chunk of one unit of one head and walks the frames t = 0..H
// in order, keeping the previous frame's elements in registers, so every key
// byte is read from HBM exactly once (16-byte coalesced loads, loads of the next
// frames in flight while the current one is reduced).  Every product is exact
// in fp64 (a bf16*bf16 or fp32*fp32 product has at most 48 significant bits);
// sums are fp64.  Each wave reduces its per-frame sums with DPP row operations
// and writes them to the workspace.
// Pass 2 (score_finalize_kernel) sums the partials of each segment in a fixed
// order, forms dot / sqrt(na*nb) in fp64 (0 when na*nb == 0) and rounds once
// to fp32 (nearest even).  The result is deterministic run to run.
//
// The first-block proxy of Sec. 4.3 (scores pooled over heads) runs the same
// two passes over every head and sums the partials of all heads of a segment
// before the cosine.
//
// Incremental rescoring.  During the AR steps of one chunk the history does not
// change; only K_cur does, and with it only SQ[H] and DOT[H-1].  The history
// pass streams frames 0..H-1 once and reduces each frame's partials into a
// per-frame statistics buffer (SQ(t), and DOT(t) for t < H-1); each step then
// streams frames H-1..H only (2 frames per head instead of H+1) and the
// finalize takes every other term from the statistics.
#include "fkv_internal.h"

namespace fkv {
namespace {

constexpr int kThreads = kScoreThreads;
constexpr int kWaves = kScoreWaves;
// Frames in flight per thread.  Four keep the pass within 64 VGPRs (the
// launch bound below), so its waves fit on a CU next to the two 224-VGPR
// waves per SIMD of a running attention workgroup: in the two-stream layer
// step the scoring of the dynamic heads then runs beside the static heads'
// attention instead of waiting for CUs (8 frames took 88 VGPRs).
constexpr int kDepth = 4;
// Frames per part when a long range is split over several workgroup columns:
// more waves in flight per CU hide the fp64 products and reductions behind the
// loads.  At 480P (22 frames) 6-frame parts (4 columns, 3 frames read twice)
// took the partials pass from 19.0 to 16.7 us with 8 frames in flight (11- and
// 8-frame parts: 17.6 and 17.8 us); with 4 in flight 4-, 6-, 8- and 11-frame
// parts are within 3% of each other.
#ifndef FKV_SCORE_PART_FRAMES
#define FKV_SCORE_PART_FRAMES 6
#endif
constexpr int kScorePartFrames = FKV_SCORE_PART_FRAMES;

// One DPP step on a double (both 32-bit halves moved with the same control);
// lanes without a source, or outside row_mask, contribute 0.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ double dpp_d(double v) {
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROW_MASK, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROW_MASK, 0xF, true);
    return __hiloint2double(hi, lo);
}

// Sum over the 64 lanes of a wave, in a fixed order: inclusive scans inside each
// 16-lane row (row_shr 1, 2, 4, 8), then row 0's total into row 1 and row 2's
// into row 3 (row_bcast:15), then rows 0+1 into rows 2 and 3 (row_bcast:31).
// Lane 63 ends with the total.  VALU only (no LDS crossbar traffic).
__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_d<0x111>(v);
    v += dpp_d<0x112>(v);
    v += dpp_d<0x114>(v);
    v += dpp_d<0x118>(v);
    v += dpp_d<0x142, 0xA>(v);
    v += dpp_d<0x143, 0xC>(v);
    return v;  // valid in lane 63
}

// Widen the 16-byte vector to fp64 elements (exact).
template <bool F32>
struct Vec;

template <>
struct Vec<false> {  // 8 bf16
    static constexpr int N = 8;
    __device__ static __forceinline__ void widen(const u32x4 &v, double *x) {
        const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] = (double)__uint_as_float(w[i] << 16);
            x[2 * i + 1] = (double)__uint_as_float(w[i] & 0xffff0000u);
        }
    }
};

template <>
struct Vec<true> {  // 4 fp32
    static constexpr int N = 4;
    __device__ static __forceinline__ void widen(const u32x4 &v, double *x) {
        x[0] = (double)__uint_as_float(v[0]);
        x[1] = (double)__uint_as_float(v[1]);
        x[2] = (double)__uint_as_float(v[2]);
        x[3] = (double)__uint_as_float(v[3]);
    }
};

// Workspace layout: ws[(((li*(H+1) + t)*units + u)*chunks + c)*kWaves + w][2]
// with [0] = SQ of frame t and [1] = DOT of frames (t, t+1).
__device__ __forceinline__ int64_t ws_index(const ScoreArgs &a, int li, int t, int u, int c, int w) {
    return ((((int64_t)li * (a.H + 1) + t) * a.units_per_frame + u) * a.chunks_per_unit + c) * kWaves + w;
}

// Statistics layout: stats[((li*H + t)*units + u)][2], [0] = SQ(t), [1] = DOT(t, t+1)
// (DOT(H-1) is not part of the history and never stored).
__device__ __forceinline__ int64_t stats_index(const ScoreArgs &a, int li, int t, int u) {
    return ((int64_t)li * a.H + t) * a.units_per_frame + u;
}

template <bool F32>
__global__ __launch_bounds__(kThreads, 8) void score_partials_kernel(ScoreArgs a) {
    using V = Vec<F32>;
    const int c = blockIdx.x, u = blockIdx.y, li = blockIdx.z / a.n_parts, part = blockIdx.z % a.n_parts;
    const int h = a.heads.head[li];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t v = (int64_t)c * kThreads + tid;       // vector within the unit
    const bool active = v < a.unit_vecs;
    const int64_t frame_vecs = a.frame_bytes / 16;
    const int64_t off = (int64_t)u * a.unit_vecs + v;   // vector within a frame
    const u32x4 *hist = (const u32x4 *)a.K_hist + (int64_t)h * a.cap * frame_vecs;
    const u32x4 *cur = (const u32x4 *)a.K_cur + (int64_t)h * a.cur_vecs;
    const int H = a.H;
    // This workgroup streams frames [tb, te] of the range [t_begin, t_end]:
    // parts overlap by one frame, whose SQ the later part writes and whose DOT
    // with the previous frame the earlier part writes, so every per-frame
    // partial is computed exactly as by a single pass.
    const bool last_part = part == a.n_parts - 1;
    const int tb = a.t_begin + part * a.part_frames;
    const int te = last_part ? a.t_end : tb + a.part_frames;

    auto load = [&](int t) -> u32x4 {
        u32x4 r = u32x4{0, 0, 0, 0};
        if (active && t <= te) {
            const u32x4 *base = t < H ? hist + (int64_t)a.slots.slot[t] * frame_vecs : cur;
            r = __builtin_nontemporal_load(base + off);
        }
        return r;
    };

    u32x4 ring[kDepth];
#pragma unroll
    for (int i = 0; i < kDepth; ++i) ring[i] = load(tb + i);

    double prev[V::N];
#pragma unroll
    for (int i = 0; i < V::N; ++i) prev[i] = 0.0;

    for (int t0 = tb; t0 <= te; t0 += kDepth) {
#pragma unroll
        for (int i = 0; i < kDepth; ++i) {
            const int t = t0 + i;
            if (t > te) break;
            double x[V::N];
            V::widen(ring[i], x);
            ring[i] = load(t + kDepth);
            double sq = 0.0, dot = 0.0;
#pragma unroll
            for (int e = 0; e < V::N; ++e) {
                sq = fma(x[e], x[e], sq);
                dot = fma(prev[e], x[e], dot);
                prev[e] = x[e];
            }
            sq = wave_sum(sq);
            dot = wave_sum(dot);
            if (lane == 63) {
                if (t < te || last_part) a.ws[ws_index(a, li, t, u, c, w) * 2 + 0] = sq;
                if (t > tb) a.ws[ws_index(a, li, t - 1, u, c, w) * 2 + 1] = dot;
            }
        }
    }
}

// One workgroup per (segment, listed head), or per segment when the score is
// pooled over all listed heads: every thread sums a strided slice of the
// segment's partials, then a fixed-order tree over the workgroup; the result
// does not depend on timing.
__global__ __launch_bounds__(kThreads) void score_finalize_kernel(ScoreArgs a) {
    __shared__ double red[3][kThreads];
    const int g = blockIdx.x;
    const int tid = threadIdx.x;
    const int nparts = a.chunks_per_unit * kWaves;
    int t0, t1, u;
    if (a.L <= a.F) {  // one unit = one segment inside frame t0
        t0 = g / a.units_per_frame;
        u = g - t0 * a.units_per_frame;
        t1 = t0 + 1;
    } else {           // the segment spans frames [t0, t1), one unit each
        const int m = a.L / a.F;
        t0 = g * m;
        t1 = min(t0 + m, a.H);
        u = 0;
    }
    const int li0 = a.pooled ? 0 : blockIdx.y;
    const int nli = a.pooled ? a.heads.n : 1;
    double dot = 0.0, na = 0.0, nb = 0.0;
    if (!a.cached) {
        const int per_head = (t1 - t0) * nparts;
        const int n = nli * per_head;
        for (int i = tid; i < n; i += kThreads) {
            const int li = li0 + i / per_head, j = i % per_head;
            const int t = t0 + j / nparts, k = j % nparts;
            const double *pa = a.ws + ws_index(a, li, t, u, 0, 0) * 2;
            const double *pb = a.ws + ws_index(a, li, t + 1, u, 0, 0) * 2;
            na += pa[2 * k];
            dot += pa[2 * k + 1];
            nb += pb[2 * k];
        }
    } else {
        // every term from the statistics, except the pair (H-1, H): DOT(H-1)
        // and SQ(H) come from this step's partials
        const int per_head = t1 - t0;
        for (int i = tid; i < nli * per_head; i += kThreads) {
            const int li = li0 + i / per_head, t = t0 + i % per_head;
            const double *st = a.stats + stats_index(a, li, t, u) * 2;
            na += st[0];
            if (t + 1 < a.H) {
                dot += st[1];
                nb += st[2 * a.units_per_frame];  // SQ(t + 1)
            }
        }
        if (t1 == a.H) {
            for (int i = tid; i < nli * nparts; i += kThreads) {
                const int li = li0 + i / nparts, k = i % nparts;
                dot += a.ws[ws_index(a, li, a.H - 1, u, 0, 0) * 2 + 2 * k + 1];
                nb += a.ws[ws_index(a, li, a.H, u, 0, 0) * 2 + 2 * k];
            }
        }
    }
    red[0][tid] = dot;
    red[1][tid] = na;
    red[2][tid] = nb;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (tid < w) {
            red[0][tid] += red[0][tid + w];
            red[1][tid] += red[1][tid + w];
            red[2][tid] += red[2][tid + w];
        }
        __syncthreads();
    }
    if (tid == 0) {
        const double prod = red[1][0] * red[2][0];
        const double cosv = prod == 0.0 ? 0.0 : red[0][0] / sqrt(prod);
        const int64_t row = a.pooled ? 0 : (int64_t)a.heads.head[li0] * a.n_seg;
        a.scores[row + g] = (float)cosv;
    }
}

// History statistics: one wave per (unit u, frame t < H, listed head li) sums
// the frame's partials in a fixed order (lanes stride over the parts, then the
// DPP tree) into SQ(t) and, for t < H-1, DOT(t).
__global__ __launch_bounds__(64) void score_stats_kernel(ScoreArgs a) {
    const int u = blockIdx.x, t = blockIdx.y, li = blockIdx.z;
    const int lane = threadIdx.x;
    const int nparts = a.chunks_per_unit * kWaves;
    const double *p = a.ws + ws_index(a, li, t, u, 0, 0) * 2;
    const bool has_dot = t + 1 < a.H;
    double sq = 0.0, dot = 0.0;
    for (int k = lane; k < nparts; k += 64) {
        sq += p[2 * k];
        if (has_dot) dot += p[2 * k + 1];
    }
    sq = wave_sum(sq);
    dot = wave_sum(dot);
    if (lane == 63) {
        double *st = a.stats + stats_index(a, li, t, u) * 2;
        st[0] = sq;
        if (has_dot) st[1] = dot;
    }
}

}  // namespace

size_t score_workspace_doubles(int n_dyn, int H, int units_per_frame, int chunks_per_unit) {
    return (size_t)n_dyn * (H + 1) * units_per_frame * chunks_per_unit * kWaves * 2;
}

namespace {

// Frames per part of a streamed range of `frames` frames (kScorePartFrames,
// or the whole range when it is short).
int split_parts(int frames, int *part_frames) {
    if (frames <= kScorePartFrames + 1) {
        *part_frames = frames;
        return 1;
    }
    *part_frames = kScorePartFrames;
    return (frames - 1 + kScorePartFrames - 1) / kScorePartFrames;  // parts share a boundary frame
}

hipError_t launch_partials(const ScoreArgs &a0, bool f32, hipStream_t s) {
    ScoreArgs a = a0;
    a.n_parts = split_parts(a.t_end - a.t_begin + 1, &a.part_frames);
    dim3 grid((unsigned)a.chunks_per_unit, (unsigned)a.units_per_frame, (unsigned)(a.heads.n * a.n_parts));
    if (f32)
        hipLaunchKernelGGL(score_partials_kernel<true>, grid, dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(score_partials_kernel<false>, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score_history(const ScoreArgs &a, bool f32, hipStream_t s) {
    if (a.heads.n == 0 || a.H == 0) return hipSuccess;
    ScoreArgs h = a;
    h.t_begin = 0;
    h.t_end = a.H - 1;
    hipError_t e = launch_partials(h, f32, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_stats_kernel, dim3(a.units_per_frame, a.H, a.heads.n), dim3(64), 0, s, h);
    return hipGetLastError();
}

hipError_t launch_score_cached(const ScoreArgs &a, bool f32, hipStream_t s) {
    if (a.heads.n == 0 || a.H == 0) return hipSuccess;
    ScoreArgs c = a;
    c.t_begin = a.H - 1;
    c.t_end = a.H;
    c.cached = 1;
    hipError_t e = launch_partials(c, f32, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_finalize_kernel, dim3(a.n_seg, a.pooled ? 1 : a.heads.n), dim3(kThreads), 0, s, c);
    return hipGetLastError();
}

hipError_t launch_score(const ScoreArgs &a, bool f32, hipStream_t s) {
    if (a.heads.n == 0 || a.H == 0) return hipSuccess;
    ScoreArgs f = a;  // the full pass: frames 0..H, finalize from the partials
    f.t_begin = 0;
    f.t_end = a.H;
    f.cached = 0;
    hipError_t e = launch_partials(f, f32, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_finalize_kernel, dim3(a.n_seg, a.pooled ? 1 : a.heads.n), dim3(kThreads), 0, s, f);
    return hipGetLastError();
}

}  // namespace fkv
