// k_score.hip -- segment-wise cosine similarity of adjacent frames for dynamic
// heads (Sec. 4.3, Eq. 3), per head or pooled over all heads, optionally
// followed by the BottomK selection, in ONE kernel launch.
//
// Segment g of the history is compared with the same token range one frame
// later.  Splitting every frame into units of U = min(L, F) tokens (a unit is
// a segment when L <= F, a whole frame otherwise), each score is a sum of
// per-(frame t, unit u) quantities
//   SQ(t, u)  = sum over the unit's elements of K_t^2           (t = 0..H, frame H
//               being the first frame of the current chunk)
//   DOT(t, u) = sum over the unit's elements of K_t * K_{t+1}   (t = 0..H-1)
// with dot = sum DOT, na = sum SQ(t), nb = sum SQ(t+1) over the frames of the
// segment.  Every product is exact in fp64 (a bf16*bf16 or fp32*fp32 product
// has at most 48 significant bits); every sum is fp64 in a fixed order, and
// the cosine dot / sqrt(na*nb) (0 when na*nb == 0) is rounded once to fp32.
//
// Streaming.  Workgroup (cg, u, li) owns column group cg -- 2 x 64 adjacent
// 16-byte vectors -- of unit u of listed head li, and streams those columns of
// every frame once: its four waves split the frames into four contiguous
// runs, every lane loads two frames of its run at once,
// so no key byte is read twice and every load is a full 1 KB-per-wave
// coalesced access.  A lane widens each frame's elements to fp64 once and
// accumulates, per frame, its columns' squares and products with the previous
// frame's widened elements (vector 0 then vector 1, elements in order); the
// wave reduces each sum over its 64 lanes with DPP row scans in a fixed order
// and writes one partial per (frame, column group).  The product across a run
// boundary uses the next run's first frame, which its wave leaves in LDS.
//
// Finish.  Each workgroup stores its per-frame sums as one block and arrives
// on one of its head's kGroups first-level counters (device-scope stores,
// loads and counters; see put_shared).  The last arrival of a group sums its
// members' blocks (in increasing order) into the group's sums and arrives on
// the head's counter; the last of those sums the kGroups group sums in order
// -- a fixed tree for every (unit, frame, quantity) -- and then, by mode:
//   full:    the head's scores (and, with `select`, its BottomK selection);
//   history: per-frame statistics SQ(t), DOT(t) into `stats`, kept across the
//            AR steps of a chunk (the history does not change, only K_cur);
//   cached:  frames H-1 and H only were streamed; the scores take DOT(H-1) and
//            SQ(H) from this pass and every other term from `stats`.
// Because the history pass and the full pass reduce every (frame, unit) sum
// with the same lanes, the same DPP order and the same column-group tree, the
// cached scores equal the full pass's bit for bit.  Pooled scores (the
// first-block proxy of Sec. 4.3): each head's finisher stores its per-frame
// sums, and the last head to finish sums them over the heads (in list order)
// before the cosine.
//
// The counters live at the start of the workspace; the caller zero-fills the
// workspace once and every call returns the counters to zero.  Partials and
// sums pass between workgroups through device-scope stores and loads
// (handover.h).
#include "handover.h"
#include "select_common.h"

namespace fkv {
namespace {

constexpr int kThreads = kScoreThreads;  // 4 waves
constexpr int kWaves = kScoreWaves;
constexpr int kV = 2;                    // 16-byte vectors per lane and frame
constexpr int kCols = 64 * kV;           // vectors (columns) per workgroup
// Frames a lane loads at once, next to the widened current and previous frame
// (32 + 32 VGPRs for bf16), within 96 VGPRs: five waves per SIMD, so every
// workgroup of a 480P layer is resident at once.  (Four frames at once with
// each element widened where it is used measured 7% slower at 480P.)
constexpr int kMaxF = 2;
// Arrival counters: device-scope atomics on one address serialise at the
// memory side, so each counter has a 256-byte line of its own and a head's
// workgroups arrive in two levels -- kGroups first-level counters (workgroup
// w on counter w % kGroups), whose last arrivals then meet on the head's
// counter.  Per listed head: kGroups + 1 counters; one more for pooling.
constexpr int kGroups = 16;
constexpr int kCounterStride = 64;       // uint32 per counter (256 bytes)
constexpr int kCountersPerHead = kGroups + 1;

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

// Element e of a 16-byte vector widened to fp64 (exact): 8 bf16 or 4 fp32.
template <bool F32>
struct Vec;

template <>
struct Vec<false> {  // 8 bf16
    static constexpr int N = 8;
    __device__ static __forceinline__ double at(const u32x4 &v, int e) {
        const uint32_t w = v[e >> 1];
        return (double)__uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    }
};

template <>
struct Vec<true> {  // 4 fp32
    static constexpr int N = 4;
    __device__ static __forceinline__ double at(const u32x4 &v, int e) { return (double)__uint_as_float(v[e]); }
};

// A lane's columns of one frame widened to fp64 (exact), vector 0 then vector
// 1, elements in order: each element is converted once, and the frame serves
// as the current frame (its squares, its product with the previous frame) and
// then as the previous frame of the next.
template <bool F32>
struct Wide {
    static constexpr int N = kV * Vec<F32>::N;
    double v[N];
    __device__ __forceinline__ void set(const u32x4 (&x)[kV]) {
#pragma unroll
        for (int j = 0; j < kV; ++j)
#pragma unroll
            for (int e = 0; e < Vec<F32>::N; ++e) v[j * Vec<F32>::N + e] = Vec<F32>::at(x[j], e);
    }
    // sum of squares, elements in order
    __device__ __forceinline__ double sq() const {
        double acc = 0.0;
#pragma unroll
        for (int k = 0; k < N; ++k) acc = fma(v[k], v[k], acc);
        return acc;
    }
    // sum of products with frame b, elements in order
    __device__ __forceinline__ double dot(const Wide &b) const {
        double acc = 0.0;
#pragma unroll
        for (int k = 0; k < N; ++k) acc = fma(v[k], b.v[k], acc);
        return acc;
    }
};

// Partial row of (unit u, streamed frame f, quantity q: 0 = SQ, 1 = DOT).
__device__ __forceinline__ int row_of(const ScoreArgs &a, int u, int f, int q) {
    return (u * a.n_frames + f) * 2 + q;
}

// Per-(unit, frame) sums of one head as the scores read them, with the frame
// given as a logical frame t: T holds this pass's rows (streamed frames
// [t_begin, t_begin + n_frames)), stats the history statistics (cached mode).
template <bool SHARED>
struct Terms {
    const ScoreArgs &a;
    const double *T;      // rows of this head (LDS, or per-head sums written by other workgroups)
    const double *stats;  // [H][units][2] of this head (cached mode)
    __device__ __forceinline__ double row(int r) const { return SHARED ? get_shared(T + r) : T[r]; }
    __device__ __forceinline__ double sq(int t, int u) const {
        if (a.mode == kScoreModeCached && t < a.H) return stats[((int64_t)t * a.units + u) * 2];
        return row(row_of(a, u, t - a.t_begin, 0));
    }
    __device__ __forceinline__ double dot(int t, int u) const {
        if (a.mode == kScoreModeCached && t < a.H - 1) return stats[((int64_t)t * a.units + u) * 2 + 1];
        return row(row_of(a, u, t - a.t_begin, 1));
    }
};

// Segment g -> its unit and frames [t0, t1).
__device__ __forceinline__ void seg_span(const ScoreArgs &a, int g, int *u, int *t0, int *t1) {
    if (a.L <= a.F) {
        *t0 = g / a.units;
        *u = g - *t0 * a.units;
        *t1 = *t0 + 1;
    } else {
        const int m = a.L / a.F;
        *t0 = g * m;
        *t1 = min(*t0 + m, a.H);
        *u = 0;
    }
}

__device__ __forceinline__ float cosine(double dot, double na, double nb) {
    const double prod = na * nb;
    return (float)(prod == 0.0 ? 0.0 : dot / sqrt(prod));
}

// The last workgroup to arrive of arrival group g of listed head li: for every
// row (u, f, q) the sum of the group's members' partials -- members are the
// workgroups wi = u * n_cg + cg with wi % kGroups == g, cg = c0, c0 + kGroups,
// ... -- into the group sums G[li][g][row] (0 where the group has no member in
// the row's unit).  Four adjacent lanes share a row: lane j of the quad sums
// members j, j + 4, j + 8, ... in order, loading eight at a time, and the
// quad adds its four sums as (s0 + s1) + (s2 + s3) -- a fixed order, so
// every pass over the same members gives the same sum.
__device__ void group_sum(const ScoreArgs &a, int li, int g) {
    const int blk = a.n_frames * 2, n_rows = a.units * blk;
    const double *part = a.part + (int64_t)li * n_rows * a.n_cg;   // [u][cg][f][q]
    double *G = a.group + ((int64_t)li * kGroups + g) * n_rows;
    // n_rows * 4 and kThreads are multiples of 4: a quad is active or
    // inactive as a whole in every iteration
    for (int x = threadIdx.x; x < n_rows * 4; x += kThreads) {
        const int r = x >> 2, j = x & 3;
        const int u = r / blk, rp = r - u * blk;
        const double *p = part + (int64_t)u * a.n_cg * blk + rp;
        const int c0 = (g - (u * a.n_cg) % kGroups + kGroups) % kGroups;
        const int nm = c0 < a.n_cg ? (a.n_cg - 1 - c0) / kGroups + 1 : 0;   // members in the unit
        double acc = 0.0;
        for (int k0 = j; k0 < nm; k0 += 4 * 8) {
            double v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int k = k0 + 4 * i;
                v[i] = k < nm ? get_shared(p + (int64_t)(c0 + k * kGroups) * blk) : 0.0;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) acc += v[i];
        }
        acc += __shfl_xor(acc, 1);
        acc += __shfl_xor(acc, 2);
        if (j == 0) put_shared(G + r, acc);
    }
}

// The last workgroup of listed head li: the head's per-row sums T (LDS,
// lds_rows doubles) from the group sums, groups in order, then the finish by
// mode.
__device__ void finish_head(const ScoreArgs &a, int li, double *T, uint64_t *s_keys, float *s_scores,
                            unsigned char *s_forced, unsigned char *s_keep) {
    const int tid = threadIdx.x;
    const int h = a.heads.head[li];
    // the keep rule is read here, its loads overlapping the group sums' loads
    const sel::Rule rule = sel::rule_of(a, li);
    const int n_rows = a.units * a.n_frames * 2;
    const double *G = a.group + (int64_t)li * kGroups * n_rows;
    // groups 0 .. min(n_wg, kGroups) - 1 have members and wrote every row; the
    // others were not written by this call
    const int n_groups = min(a.units * a.n_cg, kGroups);
    for (int r = tid; r < n_rows; r += kThreads) {
        double v[kGroups];
#pragma unroll
        for (int g = 0; g < kGroups; ++g) v[g] = g < n_groups ? get_shared(G + (int64_t)g * n_rows + r) : 0.0;
        double acc = 0.0;
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
            if (g < n_groups) acc += v[g];
        T[r] = acc;
    }
    __syncthreads();

    if (a.mode == kScoreModeHistory) {
        // SQ(t) for t < H, DOT(t) for t < H - 1 (t_begin = 0)
        double *st = a.stats + (int64_t)li * a.H * a.units * 2;
        for (int i = tid; i < a.H * a.units; i += kThreads) {
            const int t = i / a.units, u = i - t * a.units;
            st[(int64_t)i * 2] = T[row_of(a, u, t, 0)];
            if (t + 1 < a.H) st[(int64_t)i * 2 + 1] = T[row_of(a, u, t, 1)];
        }
        return;
    }
    if (a.pooled) {
        double *tot = a.totals + (int64_t)li * n_rows;
        for (int r = tid; r < n_rows; r += kThreads) put_shared(tot + r, T[r]);
        return;  // the caller counts finished heads; the last one scores
    }
    const Terms<false> tm{a, T, a.stats + (int64_t)li * a.H * a.units * 2};
    for (int g = tid; g < a.n_seg; g += kThreads) {
        int u, t0, t1;
        seg_span(a, g, &u, &t0, &t1);
        double dot = 0.0, na = 0.0, nb = 0.0;
        for (int t = t0; t < t1; ++t) {
            dot += tm.dot(t, u);
            na += tm.sq(t, u);
            nb += tm.sq(t + 1, u);
        }
        const float sc = cosine(dot, na, nb);
        a.scores[(int64_t)h * a.n_seg + g] = sc;
        if (a.select) s_scores[g] = sc;
    }
    if (a.select) {
        __syncthreads();
        sel::select_from_lds(a, rule, h, s_scores, s_keys, s_forced, s_keep, a.kept_seg, a.kv_len, tid, kThreads);
    }
}

// The last head to finish (pooled): one score per segment from every listed
// head's per-frame sums, summed over the heads in list order.
__device__ void finish_pooled(const ScoreArgs &a) {
    const int n_rows = a.units * a.n_frames * 2;
    for (int g = threadIdx.x; g < a.n_seg; g += kThreads) {
        int u, t0, t1;
        seg_span(a, g, &u, &t0, &t1);
        double dot = 0.0, na = 0.0, nb = 0.0;
        for (int li = 0; li < a.heads.n; ++li) {
            const Terms<true> tm{a, a.totals + (int64_t)li * n_rows, a.stats + (int64_t)li * a.H * a.units * 2};
            for (int t = t0; t < t1; ++t) {
                dot += tm.dot(t, u);
                na += tm.sq(t, u);
                nb += tm.sq(t + 1, u);
            }
        }
        a.scores[g] = cosine(dot, na, nb);
    }
}

template <bool F32>
__global__ __launch_bounds__(kThreads, 5) void score_kernel(ScoreArgs a) {
    extern __shared__ double dyn[];            // finisher rows (lds_rows), this workgroup's sums (2 n_frames),
                                               // then (selecting) n_seg keys, n_seg floats, 2 n_seg bytes
    __shared__ u32x4 edge[kWaves][kV][64];     // first frame of each wave's run
    __shared__ uint32_t flag;

    const int cg = blockIdx.x, u = blockIdx.y, li = blockIdx.z;
    const int h = a.heads.head[li];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int nf = a.n_frames;
    const int nw = min(kWaves, nf);            // waves with frames
    const int fa = w < nw ? (w * nf) / nw : nf;
    const int fb = w < nw ? ((w + 1) * nf) / nw : nf;

    int col[kV];
    bool ok[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) {
        col[j] = cg * kCols + j * 64 + lane;
        ok[j] = col[j] < a.unit_vecs;
    }
    const u32x4 *hist = (const u32x4 *)a.K_hist + (int64_t)h * a.cap * a.frame_vecs + (int64_t)u * a.unit_vecs;
    const u32x4 *cur = (const u32x4 *)a.K_cur + (int64_t)h * a.cur_head_vecs + (int64_t)u * a.unit_vecs;
    auto load = [&](int f, u32x4 (&x)[kV]) {
        const int t = a.t_begin + f;
        const u32x4 *base = t < a.H ? hist + (int64_t)a.slots.slot[t] * a.frame_vecs : cur;
#pragma unroll
        for (int j = 0; j < kV; ++j) x[j] = ok[j] ? __builtin_nontemporal_load(base + col[j]) : u32x4{0, 0, 0, 0};
    };
    // per-frame sums of this workgroup, staged in LDS and stored as one block
    double *wg_part = dyn + a.lds_rows;       // 2 * nf doubles after the finisher's rows
    auto put = [&](int f, int q, double v) {
        if (lane == 63) wg_part[f * 2 + q] = v;
    };

    Wide<F32> prev{};
    constexpr int MF = kMaxF;
    for (int f0 = fa; f0 < fb; f0 += MF) {
        const int nb = min(MF, fb - f0);
        u32x4 x[MF][kV];
#pragma unroll
        for (int i = 0; i < MF; ++i)
            if (i < nb) load(f0 + i, x[i]);
        if (f0 == fa) {
#pragma unroll
            for (int j = 0; j < kV; ++j) edge[w][j][lane] = x[0][j];
        }
#pragma unroll
        for (int i = 0; i < MF; ++i) {
            if (i < nb) {
                const int f = f0 + i;
                Wide<F32> cur;
                cur.set(x[i]);
                put(f, 0, wave_sum(cur.sq()));
                if (f > fa) put(f - 1, 1, wave_sum(prev.dot(cur)));
                prev = cur;
            }
        }
    }
    __syncthreads();
    // the product across the run boundary: this run's last frame with the next run's first
    if (w + 1 < nw) {
        u32x4 nx[kV];
#pragma unroll
        for (int j = 0; j < kV; ++j) nx[j] = edge[w + 1][j][lane];
        Wide<F32> next;
        next.set(nx);
        put(fb - 1, 1, wave_sum(prev.dot(next)));
    }

    __syncthreads();
    {
        double *blk = a.part + (((int64_t)li * a.units + u) * a.n_cg + cg) * (nf * 2);
        for (int r = tid; r < nf * 2; r += kThreads) put_shared(blk + r, wg_part[r]);
    }
    // two-level arrival of the head's workgroups
    const int n_wg = a.units * a.n_cg, wi = u * a.n_cg + cg, g1 = wi % kGroups;
    uint32_t *cnt = a.counters + (int64_t)li * kCountersPerHead * kCounterStride;
    if (!arrive_last(cnt + g1 * kCounterStride, (uint32_t)((n_wg - g1 + kGroups - 1) / kGroups), &flag)) return;
    group_sum(a, li, g1);
    if (!arrive_last(cnt + kGroups * kCounterStride, (uint32_t)min(n_wg, kGroups), &flag)) return;
    double *T = dyn;
    uint64_t *s_keys = (uint64_t *)(dyn + a.lds_rows + nf * 2);
    float *s_scores = (float *)(s_keys + a.n_seg);
    unsigned char *s_forced = (unsigned char *)(s_scores + a.n_seg);
    finish_head(a, li, T, s_keys, s_scores, s_forced, s_forced + a.n_seg);
    if (a.pooled && a.mode != kScoreModeHistory) {
        uint32_t *pc = a.counters + (int64_t)a.heads.n * kCountersPerHead * kCounterStride;
        if (!arrive_last(pc, (uint32_t)a.heads.n, &flag)) return;
        finish_pooled(a);
    }
}

}  // namespace

int score_column_groups(int64_t unit_vecs) { return (int)((unit_vecs + kCols - 1) / kCols); }

size_t score_workspace_bytes(int n_list, int H, int units, int n_cg) {
    if (n_list == 0 || H == 0) return 0;
    const size_t rows = (size_t)units * (H + 1) * 2;  // the full pass streams H + 1 frames
    const size_t counters = ((size_t)n_list * kCountersPerHead + 1) * kCounterStride * sizeof(uint32_t);
    const size_t b = counters + ((size_t)n_list * rows * n_cg + (size_t)n_list * rows * (kGroups + 1)) * sizeof(double);
    return (b + 255) & ~(size_t)255;
}

// The workspace of score_workspace_bytes split into counters, partials, sums.
void score_workspace_layout(ScoreArgs &a, void *ws, int n_list, int H, int units, int n_cg) {
    const size_t rows = (size_t)units * (H + 1) * 2;
    const size_t counters = ((size_t)n_list * kCountersPerHead + 1) * kCounterStride * sizeof(uint32_t);
    a.counters = (uint32_t *)ws;
    a.part = (double *)((char *)ws + counters);
    a.totals = a.part + (size_t)n_list * rows * n_cg;
    a.group = a.totals + (size_t)n_list * rows;
}

hipError_t launch_score(const ScoreArgs &a0, bool f32, hipStream_t s) {
    ScoreArgs a = a0;
    if (a.heads.n == 0 || a.n_frames <= 0) return hipSuccess;
    a.lds_rows = a.units * a.n_frames * 2;
    size_t lds = (size_t)(a.lds_rows + a.n_frames * 2) * sizeof(double);   // + this workgroup's sums
    if (a.select) lds += (size_t)a.n_seg * (sizeof(uint64_t) + sizeof(float) + 2);
    lds = (lds + 15) & ~(size_t)15;
    const dim3 grid((unsigned)a.n_cg, (unsigned)a.units, (unsigned)a.heads.n);
    if (f32)
        hipLaunchKernelGGL(score_kernel<true>, grid, dim3(kThreads), lds, s, a);
    else
        hipLaunchKernelGGL(score_kernel<false>, grid, dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace fkv
