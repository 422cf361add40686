// fkv_api.hip -- the C ABI of libfkv: host-side validation, launch planning
// and error reporting for the Forcing-KV hot path kernels.
//
// Every entry point checks all of its arguments before it touches the HIP
// runtime, so a non-OK status means nothing was enqueued or written.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "fkv_internal.h"

namespace {

thread_local char g_err[512] = "";

fkv_status fail(fkv_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

fkv_status ok() {
    g_err[0] = '\0';
    return FKV_OK;
}

size_t elem_size(const fkv_shape *s) { return s->dtype == FKV_BF16 ? 2 : 4; }

fkv_status check_shape(const fkv_shape *s) {
    if (!s) return fail(FKV_ERR_ARG, "shape is NULL");
    if (s->dtype != FKV_BF16 && s->dtype != FKV_F32)
        return fail(FKV_ERR_ARG, "dtype %d is not FKV_BF16 or FKV_F32", s->dtype);
    if (s->n_heads < 1 || s->n_heads > FKV_MAX_HEADS)
        return fail(FKV_ERR_SHAPE, "n_heads %d outside [1, %d]", s->n_heads, FKV_MAX_HEADS);
    if (s->head_dim != 64 && s->head_dim != 128)
        return fail(FKV_ERR_SHAPE, "head_dim %d is not 64 or 128", s->head_dim);
    if (s->frame_tokens < 1) return fail(FKV_ERR_SHAPE, "frame_tokens %d < 1", s->frame_tokens);
    if (s->cap_frames < 1 || s->cap_frames > FKV_MAX_FRAMES)
        return fail(FKV_ERR_SHAPE, "cap_frames %d outside [1, %d]", s->cap_frames, FKV_MAX_FRAMES);
    if (s->hist_frames < 0 || s->hist_frames > s->cap_frames)
        return fail(FKV_ERR_SHAPE, "hist_frames %d outside [0, cap_frames=%d]", s->hist_frames,
                    s->cap_frames);
    if (s->chunk_frames < 1) return fail(FKV_ERR_SHAPE, "chunk_frames %d < 1", s->chunk_frames);
    if (s->seg_tokens < 1) return fail(FKV_ERR_SHAPE, "seg_tokens %d < 1", s->seg_tokens);
    if (s->frame_tokens % s->seg_tokens != 0 && s->seg_tokens % s->frame_tokens != 0)
        return fail(FKV_ERR_SHAPE, "seg_tokens %d neither divides nor is a multiple of frame_tokens %d",
                    s->seg_tokens, s->frame_tokens);
    const int64_t hist_tokens = (int64_t)s->hist_frames * s->frame_tokens;
    const int64_t lq = (int64_t)s->chunk_frames * s->frame_tokens;
    const int64_t cap_tokens = (int64_t)s->cap_frames * s->frame_tokens;
    if (cap_tokens + lq > (int64_t)1 << 30)
        return fail(FKV_ERR_SHAPE, "cache + chunk of %lld tokens per head is too large",
                    (long long)(cap_tokens + lq));
    // Kernels address a frame, a segment piece and the chunk of one head
    // through 32-bit byte offsets and raw buffer ranges: keep each below 2^31.
    const int64_t row_bytes = (int64_t)s->head_dim * (s->dtype == FKV_BF16 ? 2 : 4);
    if ((int64_t)s->frame_tokens * row_bytes >= (int64_t)1 << 31)
        return fail(FKV_ERR_SHAPE, "a frame of %d tokens spans 2^31 bytes or more", s->frame_tokens);
    if (lq * row_bytes >= (int64_t)1 << 31)
        return fail(FKV_ERR_SHAPE, "a chunk of %lld tokens spans 2^31 bytes or more", (long long)lq);
    if (cap_tokens * row_bytes >= (int64_t)1 << 31)
        return fail(FKV_ERR_SHAPE, "a head's cache of %lld tokens spans 2^31 bytes or more",
                    (long long)cap_tokens);
    const int64_t n_seg = (hist_tokens + s->seg_tokens - 1) / s->seg_tokens;
    if (n_seg > FKV_MAX_SEGMENTS)
        return fail(FKV_ERR_SHAPE, "%lld segments exceed %d", (long long)n_seg, FKV_MAX_SEGMENTS);
    return FKV_OK;
}

fkv_status check_heads(const fkv_shape *s, const fkv_head *heads) {
    if (!heads) return fail(FKV_ERR_ARG, "heads is NULL");
    for (int h = 0; h < s->n_heads; ++h) {
        const fkv_head &b = heads[h];
        if (b.type != FKV_STATIC && b.type != FKV_DYNAMIC)
            return fail(FKV_ERR_ARG, "head %d: type %d is not FKV_STATIC or FKV_DYNAMIC", h, b.type);
        if (b.sink_frames < 0 || b.recent_frames < 0 || b.keep_k < 0)
            return fail(FKV_ERR_ARG, "head %d: negative budget (sink %d, recent %d, keep_k %d)", h,
                        b.sink_frames, b.recent_frames, b.keep_k);
        if (b.scope != FKV_SCOPE_FRAME && b.scope != FKV_SCOPE_GLOBAL)
            return fail(FKV_ERR_ARG, "head %d: scope %d is not FKV_SCOPE_FRAME or FKV_SCOPE_GLOBAL", h,
                        b.scope);
        if (b.type == FKV_DYNAMIC && b.scope == FKV_SCOPE_FRAME && s->seg_tokens >= s->frame_tokens)
            return fail(FKV_ERR_SHAPE, "head %d: per-frame selection needs seg_tokens %d < frame_tokens %d",
                        h, s->seg_tokens, s->frame_tokens);
    }
    return FKV_OK;
}

fkv_status check_slots(const fkv_shape *s, const int32_t *slots) {
    if (s->hist_frames == 0) return FKV_OK;
    if (!slots) return fail(FKV_ERR_ARG, "frame_slot is NULL");
    for (int t = 0; t < s->hist_frames; ++t)
        if (slots[t] < 0 || slots[t] >= s->cap_frames)
            return fail(FKV_ERR_ARG, "frame_slot[%d] = %d outside [0, cap_frames=%d)", t, slots[t],
                        s->cap_frames);
    return FKV_OK;
}

// --------------------------------------------------------------- budgets
struct StaticPlan {
    int n_first, gap, n_kept;
};

// Kept frames [0, min(sink,H)) U [max(H-recent,0), H): y < n_first -> y, else y + gap.
StaticPlan static_plan(int H, const fkv_head &b) {
    const int a = std::min(b.sink_frames, H);
    const int lo = std::max(H - b.recent_frames, 0);
    StaticPlan p;
    if (lo <= a) {  // the two windows meet: the whole history is kept
        p.n_first = H;
        p.gap = 0;
        p.n_kept = H;
    } else {
        p.n_first = a;
        p.gap = lo - a;
        p.n_kept = a + (H - lo);
    }
    return p;
}

struct DynPlan {
    int kk;            // kept candidates per group
    int n_kept;        // kept segments (exact)
    int64_t max_tokens;  // largest possible kv_len
};

DynPlan dyn_plan(const fkv_shape *s, const fkv_head &b) {
    const int H = s->hist_frames, F = s->frame_tokens, L = s->seg_tokens;
    const int64_t HF = (int64_t)H * F;
    const int n_seg = (int)((HF + L - 1) / L);
    std::vector<int64_t> cand_tokens;
    int n_forced = 0;
    int64_t forced_tokens = 0;
    for (int g = 0; g < n_seg; ++g) {
        const int64_t x0 = (int64_t)g * L, x1 = std::min(x0 + L, HF);
        const int first = (int)(x0 / F), last = (int)((x1 - 1) / F);
        if (first < b.sink_frames || last >= H - b.recent_frames) {
            ++n_forced;
            forced_tokens += x1 - x0;
        } else {
            cand_tokens.push_back(x1 - x0);
        }
    }
    DynPlan p;
    const int n_cand = (int)cand_tokens.size();
    if (b.scope == FKV_SCOPE_FRAME) {
        // every candidate frame holds F/L full segments
        const int per = F / L;
        p.kk = std::min(b.keep_k, per);
        const int cand_frames = n_cand / per;
        p.n_kept = n_forced + cand_frames * p.kk;
        p.max_tokens = forced_tokens + (int64_t)cand_frames * p.kk * L;
    } else {
        p.kk = std::min(b.keep_k, n_cand);
        p.n_kept = n_forced + p.kk;
        std::sort(cand_tokens.begin(), cand_tokens.end(), [](int64_t x, int64_t y) { return x > y; });
        int64_t t = forced_tokens;
        for (int i = 0; i < p.kk; ++i) t += cand_tokens[i];
        p.max_tokens = t;
    }
    return p;
}

fkv_status device_status(hipError_t e, const char *what) {
    if (e != hipSuccess)
        return fail(FKV_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

template <typename T>
T *as(void *p) { return (T *)p; }

// Workgroups of the balanced attention schedule on the current device: its
// compute-unit count rounded down to a multiple of 8 (one workgroup fills a CU).
fkv_status balanced_blocks(int *blocks) {
    static int cached[64];  // per device id, 0 = not queried yet
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(FKV_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
    int n = (dev >= 0 && dev < 64) ? __atomic_load_n(&cached[dev], __ATOMIC_RELAXED) : 0;
    if (n == 0) {
        int cus = 0;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return fail(FKV_ERR_DEVICE, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
        n = std::max(8, cus / 8 * 8);
        if (dev >= 0 && dev < 64) __atomic_store_n(&cached[dev], n, __ATOMIC_RELAXED);
    }
    *blocks = n;
    return FKV_OK;
}

// Attention workspace (bf16 balanced schedule): 2 * blocks partial-result
// slots, then one arrival counter per (head, query tile) item.
size_t attention_workspace_bytes(const fkv_shape *s, int blocks) {
    const int64_t lq = (int64_t)s->chunk_frames * s->frame_tokens;
    const int64_t n_items = (int64_t)s->n_heads * ((lq + fkv::kAttnRowsBf16 - 1) / fkv::kAttnRowsBf16);
    return 2 * (size_t)blocks * fkv::attention_part_bytes(s->head_dim) + fkv::attention_counter_bytes(n_items);
}

// Scoring geometry: units of U = min(L, F) tokens per frame, their 16-byte
// vectors, and the column groups (workgroups) per unit.
void score_geometry(const fkv_shape *s, int *units, int64_t *unit_vecs, int *n_cg) {
    const int U = std::min(s->seg_tokens, s->frame_tokens);
    *units = s->frame_tokens / U;
    *unit_vecs = (int64_t)U * s->head_dim * elem_size(s) / 16;
    *n_cg = fkv::score_column_groups(*unit_vecs);
}

size_t score_bytes(const fkv_shape *shape, int n_list) {
    if (n_list == 0 || shape->hist_frames == 0) return 0;
    int units, n_cg;
    int64_t uv;
    score_geometry(shape, &units, &uv, &n_cg);
    return fkv::score_workspace_bytes(n_list, shape->hist_frames, units, n_cg);
}

}  // namespace

extern "C" {

int32_t fkv_num_segments(const fkv_shape *shape) {
    if (check_shape(shape) != FKV_OK) return 0;
    const int64_t ht = (int64_t)shape->hist_frames * shape->frame_tokens;
    return (int32_t)((ht + shape->seg_tokens - 1) / shape->seg_tokens);
}

fkv_status fkv_kept_tokens_max(const fkv_shape *shape, const fkv_head *heads, int32_t head,
                               int64_t *tokens) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (!tokens) return fail(FKV_ERR_ARG, "tokens is NULL");
    if (head < 0 || head >= shape->n_heads)
        return fail(FKV_ERR_ARG, "head %d outside [0, %d)", head, shape->n_heads);
    const fkv_head &b = heads[head];
    if (b.type == FKV_STATIC)
        *tokens = (int64_t)static_plan(shape->hist_frames, b).n_kept * shape->frame_tokens;
    else
        *tokens = shape->hist_frames == 0 ? 0 : dyn_plan(shape, b).max_tokens;
    return ok();
}

fkv_status fkv_compress_static(const fkv_shape *shape, const fkv_head *heads, const void *K_hist,
                               const void *V_hist, const int32_t *frame_slot, void *Kc, void *Vc,
                               int32_t slab, int32_t *kv_len, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (!K_hist || !V_hist || !kv_len) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (slab < 0) return fail(FKV_ERR_ARG, "slab %d < 0", slab);
    if (slab > 0 && (!Kc || !Vc)) return fail(FKV_ERR_ARG, "NULL Kc/Vc with slab %d", slab);
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;

    fkv::StaticCopyArgs a;
    memset(&a, 0, sizeof a);
    int max_kept = 0;
    for (int h = 0; h < shape->n_heads; ++h) {
        if (heads[h].type != FKV_STATIC) continue;
        const StaticPlan p = static_plan(shape->hist_frames, heads[h]);
        const int64_t need = (int64_t)p.n_kept * shape->frame_tokens;
        if (need > slab)
            return fail(FKV_ERR_CAPACITY, "head %d keeps %lld tokens but slab is %d", h,
                        (long long)need, slab);
        const int li = a.heads.n++;
        a.heads.head[li] = h;
        a.n_first[li] = p.n_first;
        a.gap[li] = p.gap;
        a.n_kept[li] = p.n_kept;
        max_kept = std::max(max_kept, p.n_kept);
    }
    if (a.heads.n == 0) return ok();
    const size_t es = elem_size(shape);
    a.K_hist = (const uint8_t *)K_hist;
    a.V_hist = (const uint8_t *)V_hist;
    a.Kc = (uint8_t *)Kc;
    a.Vc = (uint8_t *)Vc;
    a.kv_len = kv_len;
    a.slab = slab;
    a.row_bytes = (int64_t)shape->head_dim * es;
    a.frame_vecs = (int64_t)shape->frame_tokens * a.row_bytes / 16;
    a.F = shape->frame_tokens;
    a.cap = shape->cap_frames;
    for (int t = 0; t < shape->hist_frames; ++t) a.slots.slot[t] = frame_slot[t];
    (void)hipGetLastError();
    return device_status(fkv::launch_static_copy(a, max_kept, (hipStream_t)stream),
                         "fkv_compress_static launch");
}


fkv_status fkv_score_workspace_size(const fkv_shape *shape, const fkv_head *heads, size_t *bytes) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (!bytes) return fail(FKV_ERR_ARG, "bytes is NULL");
    int n_dyn = 0;
    for (int h = 0; h < shape->n_heads; ++h) n_dyn += heads[h].type == FKV_DYNAMIC;
    *bytes = score_bytes(shape, n_dyn);
    return ok();
}

}  // extern "C"

namespace {

// Scoring of the heads in `list` (per head, or pooled into one row), in one
// launch: the full pass, the history statistics or the cached scores, with an
// optional BottomK selection of every listed head (per-head scores only).
struct SelectOut {
    const fkv_head *heads;
    int32_t *kept_seg, *kv_len;
};

fkv_status score_impl(const fkv_shape *shape, const fkv::HeadList &list, bool pooled, const void *K_hist,
                      const int32_t *frame_slot, const void *K_cur, float *scores, void *workspace,
                      void *stream, const char *what, fkv::ScoreMode mode = fkv::kScoreModeFull,
                      double *stats = nullptr, const SelectOut *select = nullptr) {
    fkv::ScoreArgs a;
    memset(&a, 0, sizeof a);
    a.heads = list;
    a.pooled = pooled ? 1 : 0;
    a.stats = stats;
    const size_t es = elem_size(shape);
    a.K_hist = (const uint8_t *)K_hist;
    a.K_cur = (const uint8_t *)K_cur;
    a.scores = scores;
    a.frame_vecs = (int64_t)shape->frame_tokens * shape->head_dim * es / 16;
    a.cur_head_vecs = (int64_t)shape->chunk_frames * a.frame_vecs;
    a.F = shape->frame_tokens;
    a.L = shape->seg_tokens;
    a.H = shape->hist_frames;
    a.cap = shape->cap_frames;
    a.n_seg = fkv_num_segments(shape);
    int64_t uv;
    score_geometry(shape, &a.units, &uv, &a.n_cg);
    a.unit_vecs = (int32_t)uv;
    a.mode = mode;
    a.t_begin = mode == fkv::kScoreModeCached ? a.H - 1 : 0;
    a.n_frames = mode == fkv::kScoreModeFull ? a.H + 1 : mode == fkv::kScoreModeHistory ? a.H : 2;
    fkv::score_workspace_layout(a, workspace, list.n, a.H, a.units, a.n_cg);
    for (int t = 0; t < shape->hist_frames; ++t) a.slots.slot[t] = frame_slot[t];
    if (select) {
        a.select = 1;
        a.kept_seg = select->kept_seg;
        a.kv_len = select->kv_len;
        for (int li = 0; li < list.n; ++li) {
            const fkv_head &b = select->heads[list.head[li]];
            a.sink[li] = b.sink_frames;
            a.recent[li] = b.recent_frames;
            a.scope[li] = b.scope;
            a.k[li] = dyn_plan(shape, b).kk;
        }
    }
    (void)hipGetLastError();
    return device_status(fkv::launch_score(a, shape->dtype == FKV_F32, (hipStream_t)stream), what);
}

// Heads of an incremental-rescoring call: every dynamic head, or every head
// when the score is pooled (heads may then be NULL).
fkv_status stats_heads(const fkv_shape *shape, const fkv_head *heads, int32_t pooled, fkv::HeadList *list) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (pooled != 0 && pooled != 1) return fail(FKV_ERR_ARG, "pooled %d is neither 0 nor 1", pooled);
    if (!pooled && (st = check_heads(shape, heads)) != FKV_OK) return st;
    memset(list, 0, sizeof *list);
    for (int h = 0; h < shape->n_heads; ++h)
        if (pooled || heads[h].type == FKV_DYNAMIC) list->head[list->n++] = h;
    return FKV_OK;
}

size_t stats_bytes(const fkv_shape *shape, int n_list) {
    int units, n_cg;
    int64_t uv;
    score_geometry(shape, &units, &uv, &n_cg);
    return (size_t)n_list * shape->hist_frames * units * 2 * sizeof(double);
}

// Shared checks of the two incremental calls; need = 0 means there is nothing
// to do (no listed head, or no history yet).
fkv_status stats_call_checks(const fkv_shape *shape, const fkv::HeadList &list, const int32_t *frame_slot,
                             const void *K_hist, const double *stats, size_t stats_size, void *workspace,
                             size_t workspace_bytes, size_t *need) {
    fkv_status st;
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    *need = score_bytes(shape, list.n);
    if (*need == 0) return FKV_OK;
    if (!K_hist) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (!stats) return fail(FKV_ERR_ARG, "stats is NULL");
    const size_t sb = stats_bytes(shape, list.n);
    if (stats_size < sb) return fail(FKV_ERR_CAPACITY, "stats of %zu bytes, %zu needed", stats_size, sb);
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < *need)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, *need);
    return FKV_OK;
}


}  // namespace

extern "C" {

fkv_status fkv_score_segments(const fkv_shape *shape, const fkv_head *heads, const void *K_hist,
                              const int32_t *frame_slot, const void *K_cur, float *scores,
                              void *workspace, size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    size_t need = 0;
    if ((st = fkv_score_workspace_size(shape, heads, &need)) != FKV_OK) return st;
    if (need == 0) return ok();  // no dynamic head, or nothing cached yet
    if (!K_hist || !K_cur || !scores) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < need)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    for (int h = 0; h < shape->n_heads; ++h)
        if (heads[h].type == FKV_DYNAMIC) list.head[list.n++] = h;
    return score_impl(shape, list, false, K_hist, frame_slot, K_cur, scores, workspace, stream,
                      "fkv_score_segments launch");
}

fkv_status fkv_score_stats_size(const fkv_shape *shape, const fkv_head *heads, int32_t pooled, size_t *bytes) {
    fkv::HeadList list;
    fkv_status st;
    if ((st = stats_heads(shape, heads, pooled, &list)) != FKV_OK) return st;
    if (!bytes) return fail(FKV_ERR_ARG, "bytes is NULL");
    *bytes = stats_bytes(shape, list.n);
    return ok();
}

fkv_status fkv_score_history(const fkv_shape *shape, const fkv_head *heads, int32_t pooled, const void *K_hist,
                             const int32_t *frame_slot, double *stats, size_t stats_size, void *workspace,
                             size_t workspace_bytes, void *stream) {
    fkv::HeadList list;
    fkv_status st;
    if ((st = stats_heads(shape, heads, pooled, &list)) != FKV_OK) return st;
    size_t need = 0;
    if ((st = stats_call_checks(shape, list, frame_slot, K_hist, stats, stats_size, workspace, workspace_bytes,
                                &need)) != FKV_OK)
        return st;
    if (need == 0) return ok();
    return score_impl(shape, list, pooled, K_hist, frame_slot, K_hist, nullptr, workspace, stream,
                      "fkv_score_history launch", fkv::kScoreModeHistory, stats);
}

fkv_status fkv_score_segments_cached(const fkv_shape *shape, const fkv_head *heads, int32_t pooled,
                                     const void *K_hist, const int32_t *frame_slot, const void *K_cur,
                                     const double *stats, size_t stats_size, float *scores, void *workspace,
                                     size_t workspace_bytes, void *stream) {
    fkv::HeadList list;
    fkv_status st;
    if ((st = stats_heads(shape, heads, pooled, &list)) != FKV_OK) return st;
    size_t need = 0;
    if ((st = stats_call_checks(shape, list, frame_slot, K_hist, stats, stats_size, workspace, workspace_bytes,
                                &need)) != FKV_OK)
        return st;
    if (need == 0) return ok();
    if (!K_cur || !scores) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    return score_impl(shape, list, pooled, K_hist, frame_slot, K_cur, scores, workspace, stream,
                      "fkv_score_segments_cached launch", fkv::kScoreModeCached, const_cast<double *>(stats));
}

fkv_status fkv_score_pooled_workspace_size(const fkv_shape *shape, size_t *bytes) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (!bytes) return fail(FKV_ERR_ARG, "bytes is NULL");
    *bytes = score_bytes(shape, shape->n_heads);
    return ok();
}

fkv_status fkv_score_pooled(const fkv_shape *shape, const void *K_hist, const int32_t *frame_slot,
                            const void *K_cur, float *scores, void *workspace, size_t workspace_bytes,
                            void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    const size_t need = score_bytes(shape, shape->n_heads);
    if (need == 0) return ok();  // nothing cached yet
    if (!K_hist || !K_cur || !scores) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < need)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    for (int h = 0; h < shape->n_heads; ++h) list.head[list.n++] = h;
    return score_impl(shape, list, true, K_hist, frame_slot, K_cur, scores, workspace, stream,
                      "fkv_score_pooled launch");
}

}  // extern "C"

namespace {

// BottomK of the dynamic heads only (no copy): kept_seg and kv_len.
fkv_status select_impl(const fkv_shape *shape, const fkv_head *heads, const float *scores, bool shared_row,
                       int32_t *kept_seg, int32_t *kv_len, void *stream, const char *what) {
    const int n_seg = fkv_num_segments(shape);
    fkv::SelectArgs sa;
    memset(&sa, 0, sizeof sa);
    for (int h = 0; h < shape->n_heads; ++h) {
        if (heads[h].type != FKV_DYNAMIC) continue;
        const int li = sa.heads.n++;
        sa.heads.head[li] = h;
        sa.sink[li] = heads[h].sink_frames;
        sa.recent[li] = heads[h].recent_frames;
        sa.scope[li] = heads[h].scope;
        sa.k[li] = shape->hist_frames > 0 ? dyn_plan(shape, heads[h]).kk : 0;
    }
    if (sa.heads.n == 0) return ok();
    sa.scores = scores;
    sa.score_stride = shared_row ? 0 : n_seg;
    sa.kept_seg = kept_seg;
    sa.kv_len = kv_len;
    sa.F = shape->frame_tokens;
    sa.L = shape->seg_tokens;
    sa.H = shape->hist_frames;
    sa.n_seg = n_seg;
    (void)hipGetLastError();
    return device_status(fkv::launch_select(sa, (hipStream_t)stream), what);
}

}  // namespace

extern "C" {

fkv_status fkv_select(const fkv_shape *shape, const fkv_head *heads, const float *scores, int32_t shared_row,
                      int32_t *kept_seg, int32_t *kv_len, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (shared_row != 0 && shared_row != 1) return fail(FKV_ERR_ARG, "shared_row %d is neither 0 nor 1", shared_row);
    if (!kv_len) return fail(FKV_ERR_ARG, "kv_len is NULL");
    if (fkv_num_segments(shape) > 0 && (!scores || !kept_seg)) return fail(FKV_ERR_ARG, "NULL scores or kept_seg");
    return select_impl(shape, heads, scores, shared_row != 0, kept_seg, kv_len, stream, "fkv_select launch");
}

fkv_status fkv_score_select(const fkv_shape *shape, const fkv_head *heads, const void *K_hist,
                            const int32_t *frame_slot, const void *K_cur, float *scores, int32_t *kept_seg,
                            int32_t *kv_len, void *workspace, size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    if (!kv_len) return fail(FKV_ERR_ARG, "kv_len is NULL");
    size_t need = 0;
    if ((st = fkv_score_workspace_size(shape, heads, &need)) != FKV_OK) return st;
    if (need == 0)  // no dynamic head, or nothing cached: every dynamic head keeps nothing
        return select_impl(shape, heads, nullptr, false, kept_seg, kv_len, stream, "fkv_score_select launch");
    if (!K_hist || !K_cur || !scores || !kept_seg) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < need)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    for (int h = 0; h < shape->n_heads; ++h)
        if (heads[h].type == FKV_DYNAMIC) list.head[list.n++] = h;
    const SelectOut out{heads, kept_seg, kv_len};
    return score_impl(shape, list, false, K_hist, frame_slot, K_cur, scores, workspace, stream,
                      "fkv_score_select launch", fkv::kScoreModeFull, nullptr, &out);
}

}  // extern "C"

// ------------------------------------------------- scoring that allocates nothing
// fkv_score_select_noalloc's workspace: a device array of the library (one
// copy per GPU, held until the process ends), zero at load like every scoring
// workspace, and left with its arrival counters at zero by every call.
static constexpr size_t kNoallocScratchBytes = (size_t)FKV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

namespace {

// The array's device address on the current device.  In host code `scratch`
// is only a stand-in symbol, never a device address: the address comes from
// hipGetSymbolAddress, once per device with that device current.
fkv_status scratch_address(void **out) {
    static std::mutex mu;
    static void *addr[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(FKV_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= 64) return fail(FKV_ERR_DEVICE, "device %d outside [0, 64)", dev);
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(FKV_ERR_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        addr[dev] = p;
    }
    *out = addr[dev];
    return FKV_OK;
}

}  // namespace

extern "C" {

fkv_status fkv_score_select_noalloc(const fkv_shape *shape, const fkv_head *heads, const void *K_hist,
                                    const int32_t *frame_slot, const void *K_cur, float *scores,
                                    int32_t *kept_seg, int32_t *kv_len, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    if (!kv_len) return fail(FKV_ERR_ARG, "kv_len is NULL");
    size_t need = 0;
    if ((st = fkv_score_workspace_size(shape, heads, &need)) != FKV_OK) return st;
    if (need > kNoallocScratchBytes)
        return fail(FKV_ERR_CAPACITY, "scoring needs %zu bytes of scratch, the library holds %zu", need,
                    kNoallocScratchBytes);
    if (need == 0)  // no dynamic head, or nothing cached: every dynamic head keeps nothing
        return select_impl(shape, heads, nullptr, false, kept_seg, kv_len, stream, "fkv_score_select_noalloc launch");
    if (!K_hist || !K_cur || !scores || !kept_seg) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    void *ws = nullptr;
    if ((st = scratch_address(&ws)) != FKV_OK) return st;
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    for (int h = 0; h < shape->n_heads; ++h)
        if (heads[h].type == FKV_DYNAMIC) list.head[list.n++] = h;
    const SelectOut out{heads, kept_seg, kv_len};
    return score_impl(shape, list, false, K_hist, frame_slot, K_cur, scores, ws, stream,
                      "fkv_score_select_noalloc launch", fkv::kScoreModeFull, nullptr, &out);
}

}  // extern "C"

namespace {

fkv_status select_compact_impl(const fkv_shape *shape, const fkv_head *heads, const float *scores,
                               bool shared_row, const void *K_hist, const void *V_hist,
                               const int32_t *frame_slot, int32_t *kept_seg, void *Kc, void *Vc,
                               int32_t slab, int32_t *kv_len, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (!K_hist || !V_hist || !kv_len) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (slab < 0) return fail(FKV_ERR_ARG, "slab %d < 0", slab);
    if (slab > 0 && (!Kc || !Vc)) return fail(FKV_ERR_ARG, "NULL Kc/Vc with slab %d", slab);
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    const int n_seg = fkv_num_segments(shape);
    if (n_seg > 0 && (!scores || !kept_seg)) return fail(FKV_ERR_ARG, "NULL scores or kept_seg");

    fkv::SelectArgs sa;
    memset(&sa, 0, sizeof sa);
    int max_pieces = 0;
    const int m = shape->seg_tokens > shape->frame_tokens ? shape->seg_tokens / shape->frame_tokens : 1;
    for (int h = 0; h < shape->n_heads; ++h) {
        if (heads[h].type != FKV_DYNAMIC) continue;
        DynPlan p = {0, 0, 0};
        if (shape->hist_frames > 0) p = dyn_plan(shape, heads[h]);
        if (p.max_tokens > slab)
            return fail(FKV_ERR_CAPACITY, "head %d may keep %lld tokens but slab is %d", h,
                        (long long)p.max_tokens, slab);
        const int li = sa.heads.n++;
        sa.heads.head[li] = h;
        sa.sink[li] = heads[h].sink_frames;
        sa.recent[li] = heads[h].recent_frames;
        sa.scope[li] = heads[h].scope;
        sa.k[li] = p.kk;
        max_pieces = std::max(max_pieces, p.n_kept * m);
    }
    if (sa.heads.n == 0) return ok();
    (void)hipGetLastError();
    sa.scores = scores;
    sa.score_stride = shared_row ? 0 : n_seg;
    sa.kept_seg = kept_seg;
    sa.kv_len = kv_len;
    sa.F = shape->frame_tokens;
    sa.L = shape->seg_tokens;
    sa.H = shape->hist_frames;
    sa.n_seg = n_seg;
    fkv::DynCopyArgs ca;
    memset(&ca, 0, sizeof ca);
    const size_t es = elem_size(shape);
    ca.K_hist = (const uint8_t *)K_hist;
    ca.V_hist = (const uint8_t *)V_hist;
    ca.Kc = (uint8_t *)Kc;
    ca.Vc = (uint8_t *)Vc;
    ca.kept_seg = kept_seg;
    ca.slab = slab;
    ca.row_bytes = (int64_t)shape->head_dim * es;
    ca.piece_tokens = std::min(shape->seg_tokens, shape->frame_tokens);
    ca.pieces_per_seg = m;
    ca.piece_vecs = (int64_t)ca.piece_tokens * ca.row_bytes / 16;
    ca.F = shape->frame_tokens;
    ca.L = shape->seg_tokens;
    ca.H = shape->hist_frames;
    ca.cap = shape->cap_frames;
    ca.n_seg = n_seg;
    ca.heads = sa.heads;
    for (int t = 0; t < shape->hist_frames; ++t) ca.slots.slot[t] = frame_slot[t];
    // One launch when every copy workgroup can re-derive its head's keep set;
    // otherwise the selection kernel, then the copy.  With nothing cached
    // (H = 0, the first AR step) or nothing kept, only the selection kernel
    // runs: it writes kv_len = 0 and the -1 padding of kept_seg.
    if (n_seg > 0 && n_seg <= fkv::kFusedSelectMaxSeg && max_pieces > 0) {
        fkv::SelectCopyArgs sc;
        sc.sel = sa;
        sc.copy = ca;
        return device_status(fkv::launch_select_copy(sc, max_pieces, (hipStream_t)stream),
                             "fkv_select_compact launch");
    }
    fkv_status rs = device_status(fkv::launch_select(sa, (hipStream_t)stream), "fkv_select_compact select launch");
    if (rs != FKV_OK || n_seg == 0) return rs;
    return device_status(fkv::launch_dyn_copy(ca, max_pieces, (hipStream_t)stream),
                         "fkv_select_compact copy launch");
}

}  // namespace

extern "C" {

fkv_status fkv_select_compact(const fkv_shape *shape, const fkv_head *heads, const float *scores,
                              const void *K_hist, const void *V_hist, const int32_t *frame_slot,
                              int32_t *kept_seg, void *Kc, void *Vc, int32_t slab, int32_t *kv_len,
                              void *stream) {
    return select_compact_impl(shape, heads, scores, false, K_hist, V_hist, frame_slot, kept_seg, Kc, Vc,
                               slab, kv_len, stream);
}

fkv_status fkv_select_compact_pooled(const fkv_shape *shape, const fkv_head *heads, const float *scores,
                                     const void *K_hist, const void *V_hist, const int32_t *frame_slot,
                                     int32_t *kept_seg, void *Kc, void *Vc, int32_t slab,
                                     int32_t *kv_len, void *stream) {
    return select_compact_impl(shape, heads, scores, true, K_hist, V_hist, frame_slot, kept_seg, Kc, Vc,
                               slab, kv_len, stream);
}

fkv_status fkv_append_frames(const fkv_shape *shape, const void *K_new, const void *V_new, int32_t n_frames,
                             const int32_t *dst_slot, void *K_hist, void *V_hist, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (n_frames < 0 || n_frames > shape->cap_frames)
        return fail(FKV_ERR_ARG, "n_frames %d outside [0, cap_frames=%d]", n_frames, shape->cap_frames);
    if (n_frames == 0) return ok();
    if (!K_new || !V_new || !K_hist || !V_hist) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (!dst_slot) return fail(FKV_ERR_ARG, "dst_slot is NULL");
    bool used[FKV_MAX_FRAMES] = {};
    for (int f = 0; f < n_frames; ++f) {
        const int sl = dst_slot[f];
        if (sl < 0 || sl >= shape->cap_frames)
            return fail(FKV_ERR_ARG, "dst_slot[%d] = %d outside [0, %d)", f, sl, shape->cap_frames);
        if (used[sl]) return fail(FKV_ERR_ARG, "dst_slot[%d] = %d is given twice", f, sl);
        used[sl] = true;
    }
    fkv::AppendArgs a;
    memset(&a, 0, sizeof a);
    a.K_new = (const uint8_t *)K_new;
    a.V_new = (const uint8_t *)V_new;
    a.K_hist = (uint8_t *)K_hist;
    a.V_hist = (uint8_t *)V_hist;
    a.frame_vecs = (int64_t)shape->frame_tokens * shape->head_dim * elem_size(shape) / 16;
    a.n_frames = n_frames;
    a.cap = shape->cap_frames;
    for (int f = 0; f < n_frames; ++f) a.slots.slot[f] = dst_slot[f];
    (void)hipGetLastError();
    return device_status(fkv::launch_append(a, shape->n_heads, (hipStream_t)stream), "fkv_append_frames launch");
}

fkv_status fkv_attention_workspace_size(const fkv_shape *shape, size_t *bytes) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (!bytes) return fail(FKV_ERR_ARG, "bytes is NULL");
    *bytes = 0;
    if (shape->dtype != FKV_BF16) return ok();
    int blocks = 0;
    if ((st = balanced_blocks(&blocks)) != FKV_OK) return st;
    *bytes = attention_workspace_bytes(shape, blocks);
    return ok();
}

}  // extern "C"

namespace {

// Identity head list (every head of the shape, in order).
fkv::HeadList all_heads(int n_heads) {
    fkv::HeadList l;
    memset(&l, 0, sizeof l);
    l.n = n_heads;
    for (int h = 0; h < n_heads; ++h) l.head[h] = h;
    return l;
}

// Heads attended in place: the kept history is read from the cache through the
// frame-slot map instead of from a compressed copy -- the kept frames of a
// static head (from its budget), the kept segments of a dynamic head (kept_seg
// and kv_len as fkv_select writes them).
struct PagedHistory {
    const void *K_hist, *V_hist;
    const int32_t *frame_slot;
    const fkv_head *heads;
    const int32_t *kept_seg;   // dynamic heads only
};

// Can the paged kernel read dynamic heads of this shape in place?  Pieces of
// min(L, F) >= 64 tokens (a key tile spans at most two), and a page-table
// entry slot * (F / piece) + unit below 256 for every cache slot.
fkv_status check_paged_dynamic(const fkv_shape *s) {
    const int P = std::min(s->seg_tokens, s->frame_tokens);
    if (P < fkv::kAttnKeysPerTile)
        return fail(FKV_ERR_SHAPE, "in-place dynamic heads need min(seg_tokens, frame_tokens) = %d >= %d", P,
                    fkv::kAttnKeysPerTile);
    if ((int64_t)s->cap_frames * (s->frame_tokens / P) > 256)
        return fail(FKV_ERR_SHAPE, "in-place dynamic heads need cap_frames * (F / min(L, F)) = %lld <= 256",
                    (long long)s->cap_frames * (s->frame_tokens / P));
    return FKV_OK;
}

fkv_status chunk_attention_impl(const fkv_shape *shape, const fkv::HeadList &list, const void *Q,
                                const void *Kc, const void *Vc, int32_t slab, const int32_t *kv_len,
                                const void *K_cur, const void *V_cur, float scale, void *O, float *lse,
                                void *workspace, size_t workspace_bytes, void *stream,
                                const PagedHistory *paged = nullptr) {
    fkv_status st;
    if (!Q || !K_cur || !V_cur || !O || (!kv_len && !paged)) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (slab < 0) return fail(FKV_ERR_ARG, "slab %d < 0", slab);
    if (slab > 0 && (!Kc || !Vc)) return fail(FKV_ERR_ARG, "NULL Kc/Vc with slab %d", slab);
    if (!(scale > 0.f) || !isfinite(scale)) return fail(FKV_ERR_ARG, "scale %g must be positive and finite", (double)scale);
    const bool bf16 = shape->dtype == FKV_BF16;
    int blocks = 0;
    if (bf16 && workspace) {
        if ((st = balanced_blocks(&blocks)) != FKV_OK) return st;
        const size_t need = attention_workspace_bytes(shape, blocks);
        if (workspace_bytes < need)
            return fail(FKV_ERR_CAPACITY, "attention workspace of %zu bytes, %zu needed", workspace_bytes, need);
    }
    if (list.n == 0) return ok();

    fkv::AttnArgs a;
    memset(&a, 0, sizeof a);
    a.Q = Q;
    a.Kc = Kc ? Kc : K_cur;
    a.Vc = Vc ? Vc : V_cur;
    a.K_cur = K_cur;
    a.V_cur = V_cur;
    a.O = O;
    a.lse = lse;
    a.kv_len = kv_len;
    a.slab = slab;
    a.n_heads = shape->n_heads;
    a.heads = list;
    a.Lq = shape->chunk_frames * shape->frame_tokens;
    a.scale = scale;
    a.scale_log2 = scale * 1.4426950408889634f;
    const int rows = bf16 ? fkv::kAttnRowsBf16 : fkv::kAttnRowsF32;
    a.n_qtiles = (a.Lq + rows - 1) / rows;
    a.n_items = list.n * a.n_qtiles;
    a.items_per_xcd = (a.n_items + 7) / 8;
    a.n_blocks = blocks;
    a.part = (float *)workspace;
    if (workspace)
        a.item_counters = (uint32_t *)((char *)workspace + 2 * (size_t)blocks * fkv::attention_part_bytes(shape->head_dim));
    if (paged) {
        a.paged = 1;
        a.K_hist = paged->K_hist;
        a.V_hist = paged->V_hist;
        a.F = shape->frame_tokens;
        a.cap = shape->cap_frames;
        // a dynamic head's kv_len is clamped to the history, so its pieces never
        // leave the cached frames whatever kv_len holds
        a.slab = (int64_t)shape->hist_frames * shape->frame_tokens;
        a.kept_seg = paged->kept_seg;
        a.pg_L = shape->seg_tokens;
        a.pg_nseg = fkv_num_segments(shape);
        // one piece length for the launch: a frame, or min(L, F) when a dynamic
        // head is read in place (static frames are then split into pieces too)
        bool dyn = false;
        for (int li = 0; li < list.n; ++li)
            dyn |= paged->heads[list.head[li]].type == FKV_DYNAMIC && shape->hist_frames > 0;
        a.pg_P = dyn ? std::min(shape->seg_tokens, shape->frame_tokens) : shape->frame_tokens;
        a.pg_ppf = shape->frame_tokens / a.pg_P;
        {   // M = floor(2^64 / P) + 1 (P >= 64, not a power of two in general)
            const unsigned __int128 m = (((unsigned __int128)1) << 64) / (uint64_t)a.pg_P + 1;
            a.pg_magic_hi = (uint32_t)(uint64_t)(m >> 32);
            a.pg_magic_lo = (uint32_t)(uint64_t)m;
        }
        for (int li = 0; li < list.n; ++li) {
            const int h = list.head[li];
            if (paged->heads[h].type == FKV_DYNAMIC && shape->hist_frames > 0) {
                a.st_kept[li] = -1;
                continue;
            }
            // static heads, and dynamic heads with nothing cached (no history, kv_len unread)
            const StaticPlan p = paged->heads[h].type == FKV_DYNAMIC ? StaticPlan{0, 0, 0}
                                                                     : static_plan(shape->hist_frames, paged->heads[h]);
            a.st_first[li] = p.n_first;
            a.st_gap[li] = p.gap;
            a.st_kept[li] = p.n_kept;
        }
        for (int t = 0; t < shape->hist_frames; ++t) a.slots.slot[t] = paged->frame_slot[t];
    }
    (void)hipGetLastError();
    hipError_t e = bf16 ? fkv::launch_attention_bf16(a, shape->head_dim, (hipStream_t)stream)
                        : fkv::launch_attention_f32(a, shape->head_dim, (hipStream_t)stream);
    return device_status(e, "fkv_chunk_attention launch");
}

}  // namespace

extern "C" {

fkv_status fkv_chunk_attention(const fkv_shape *shape, const void *Q, const void *Kc, const void *Vc,
                               int32_t slab, const int32_t *kv_len, const void *K_cur,
                               const void *V_cur, float scale, void *O, float *lse, void *workspace,
                               size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    return chunk_attention_impl(shape, all_heads(shape->n_heads), Q, Kc, Vc, slab, kv_len, K_cur, V_cur,
                                scale, O, lse, workspace, workspace_bytes, stream);
}

fkv_status fkv_chunk_attention_heads(const fkv_shape *shape, const int32_t *head_list, int32_t n_list,
                                     const void *Q, const void *Kc, const void *Vc, int32_t slab,
                                     const int32_t *kv_len, const void *K_cur, const void *V_cur,
                                     float scale, void *O, float *lse, void *workspace,
                                     size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (n_list < 0 || n_list > shape->n_heads) return fail(FKV_ERR_ARG, "n_list %d outside [0, %d]", n_list, shape->n_heads);
    if (n_list > 0 && !head_list) return fail(FKV_ERR_ARG, "head_list is NULL");
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    bool seen[FKV_MAX_HEADS] = {};
    for (int i = 0; i < n_list; ++i) {
        const int h = head_list[i];
        if (h < 0 || h >= shape->n_heads) return fail(FKV_ERR_ARG, "head_list[%d] = %d outside [0, %d)", i, h, shape->n_heads);
        if (seen[h]) return fail(FKV_ERR_ARG, "head %d listed twice", h);
        seen[h] = true;
        list.head[list.n++] = h;
    }
    return chunk_attention_impl(shape, list, Q, Kc, Vc, slab, kv_len, K_cur, V_cur, scale, O, lse,
                                workspace, workspace_bytes, stream);
}

fkv_status fkv_chunk_attention_static(const fkv_shape *shape, const fkv_head *heads, const void *K_hist,
                                      const void *V_hist, const int32_t *frame_slot, const void *Q,
                                      const void *K_cur, const void *V_cur, float scale, void *O, float *lse,
                                      void *workspace, size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (shape->dtype != FKV_BF16) return fail(FKV_ERR_SHAPE, "in-place static attention needs bf16");
    if (shape->frame_tokens < fkv::kAttnKeysPerTile)
        return fail(FKV_ERR_SHAPE, "in-place static attention needs frame_tokens %d >= %d",
                    shape->frame_tokens, fkv::kAttnKeysPerTile);
    if (shape->hist_frames > 0 && (!K_hist || !V_hist)) return fail(FKV_ERR_ARG, "NULL K_hist/V_hist");
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    for (int h = 0; h < shape->n_heads; ++h)
        if (heads[h].type == FKV_STATIC) list.head[list.n++] = h;
    const PagedHistory paged{K_hist, V_hist, frame_slot, heads, nullptr};
    return chunk_attention_impl(shape, list, Q, nullptr, nullptr, 0, nullptr, K_cur, V_cur, scale, O, lse,
                                workspace, workspace_bytes, stream, &paged);
}

fkv_status fkv_chunk_attention_paged(const fkv_shape *shape, const fkv_head *heads, const int32_t *head_list,
                                     int32_t n_list, const void *K_hist, const void *V_hist,
                                     const int32_t *frame_slot, const int32_t *kept_seg, const int32_t *kv_len,
                                     const void *Q, const void *K_cur, const void *V_cur, float scale, void *O,
                                     float *lse, void *workspace, size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    if (shape->dtype != FKV_BF16) return fail(FKV_ERR_SHAPE, "in-place attention needs bf16");
    if (shape->frame_tokens < fkv::kAttnKeysPerTile)
        return fail(FKV_ERR_SHAPE, "in-place attention needs frame_tokens %d >= %d", shape->frame_tokens,
                    fkv::kAttnKeysPerTile);
    if (n_list < 0 || n_list > shape->n_heads)
        return fail(FKV_ERR_ARG, "n_list %d outside [0, %d]", n_list, shape->n_heads);
    fkv::HeadList list;
    memset(&list, 0, sizeof list);
    bool seen[FKV_MAX_HEADS] = {};
    const int n = head_list ? n_list : shape->n_heads;
    for (int i = 0; i < n; ++i) {
        const int h = head_list ? head_list[i] : i;
        if (h < 0 || h >= shape->n_heads)
            return fail(FKV_ERR_ARG, "head_list[%d] = %d outside [0, %d)", i, h, shape->n_heads);
        if (seen[h]) return fail(FKV_ERR_ARG, "head %d listed twice", h);
        seen[h] = true;
        list.head[list.n++] = h;
    }
    bool any_dynamic = false;
    for (int i = 0; i < list.n; ++i) any_dynamic |= heads[list.head[i]].type == FKV_DYNAMIC;
    if (any_dynamic) {
        if ((st = check_paged_dynamic(shape)) != FKV_OK) return st;
        if (!kv_len) return fail(FKV_ERR_ARG, "kv_len is NULL");
        if (shape->hist_frames > 0 && !kept_seg) return fail(FKV_ERR_ARG, "kept_seg is NULL");
    }
    if (shape->hist_frames > 0 && (!K_hist || !V_hist)) return fail(FKV_ERR_ARG, "NULL K_hist/V_hist");
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    const PagedHistory paged{K_hist, V_hist, frame_slot, heads, kept_seg};
    return chunk_attention_impl(shape, list, Q, nullptr, nullptr, 0, kv_len, K_cur, V_cur, scale, O, lse,
                                workspace, workspace_bytes, stream, &paged);
}

fkv_status fkv_fp8_sizes(const fkv_shape *shape, int32_t slab, size_t *q_bytes, size_t *kv_bytes,
                         size_t *scale_bytes, size_t *workspace_bytes) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (shape->dtype != FKV_BF16) return fail(FKV_ERR_SHAPE, "the FP8 path takes bf16 inputs");
    if (slab < 0) return fail(FKV_ERR_ARG, "slab %d < 0", slab);
    if ((int64_t)slab > (int64_t)shape->cap_frames * shape->frame_tokens)
        return fail(FKV_ERR_ARG, "slab %d exceeds the cache's %lld tokens", slab,
                    (long long)shape->cap_frames * shape->frame_tokens);
    if (!q_bytes || !kv_bytes || !scale_bytes || !workspace_bytes) return fail(FKV_ERR_ARG, "NULL size pointer");
    const int64_t lq = (int64_t)shape->chunk_frames * shape->frame_tokens;
    const int64_t rows = (slab + lq + 63) / 64 * 64;
    const int d = shape->head_dim;
    *q_bytes = (size_t)shape->n_heads * lq * d;
    *kv_bytes = (size_t)shape->n_heads * rows * d;
    *scale_bytes = (size_t)shape->n_heads * fkv::fp8_scale_floats(d) * sizeof(float);
    const int chunks = (int)((slab + lq + fkv::kFp8ChunkRows - 1) / fkv::kFp8ChunkRows) +
                       (int)((lq + fkv::kFp8ChunkRows - 1) / fkv::kFp8ChunkRows);
    *workspace_bytes = (fkv::fp8_stats_doubles(shape->n_heads, chunks, d) * sizeof(double) + 255) & ~(size_t)255;
    return ok();
}

fkv_status fkv_fp8_pack(const fkv_shape *shape, const void *Q, const void *Kc, const void *Vc, int32_t slab,
                        const int32_t *kv_len, const void *K_cur, const void *V_cur, void *Q8, void *K8,
                        void *V8T, float *scales, void *workspace, size_t workspace_bytes, void *stream) {
    fkv_status st;
    size_t qb, kvb, sb, wb;
    if ((st = fkv_fp8_sizes(shape, slab, &qb, &kvb, &sb, &wb)) != FKV_OK) return st;
    if (!Q || !K_cur || !V_cur || !kv_len || !Q8 || !K8 || !V8T || !scales)
        return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (slab > 0 && (!Kc || !Vc)) return fail(FKV_ERR_ARG, "NULL Kc/Vc with slab %d", slab);
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < wb)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, wb);
    fkv::Fp8PackArgs a;
    memset(&a, 0, sizeof a);
    a.Q = (const uint16_t *)Q;
    a.Kc = (const uint16_t *)(Kc ? Kc : K_cur);
    a.Vc = (const uint16_t *)(Vc ? Vc : V_cur);
    a.K_cur = (const uint16_t *)K_cur;
    a.V_cur = (const uint16_t *)V_cur;
    a.kv_len = kv_len;
    a.slab = slab;
    a.n_heads = shape->n_heads;
    a.Lq = shape->chunk_frames * shape->frame_tokens;
    a.d = shape->head_dim;
    a.rows = ((int64_t)slab + a.Lq + 63) / 64 * 64;
    a.Q8 = (uint8_t *)Q8;
    a.K8 = (uint8_t *)K8;
    a.V8T = (uint8_t *)V8T;
    a.scales = scales;
    a.ws = (double *)workspace;
    a.chunk_rows = fkv::kFp8ChunkRows;
    a.n_kchunks = (int)(((int64_t)slab + a.Lq + fkv::kFp8ChunkRows - 1) / fkv::kFp8ChunkRows);
    a.n_qchunks = (a.Lq + fkv::kFp8ChunkRows - 1) / fkv::kFp8ChunkRows;
    (void)hipGetLastError();
    return device_status(fkv::launch_fp8_pack(a, (hipStream_t)stream), "fkv_fp8_pack launch");
}

fkv_status fkv_fp8_pack_paged(const fkv_shape *shape, const fkv_head *heads, const void *K_hist,
                              const void *V_hist, const int32_t *frame_slot, const int32_t *kept_seg,
                              int32_t *kv_len, const void *Q, const void *K_cur, const void *V_cur, int32_t slab,
                              void *Q8, void *K8, void *V8T, float *scales, void *workspace,
                              size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if ((st = check_heads(shape, heads)) != FKV_OK) return st;
    size_t qb, kvb, sb, wb;
    if ((st = fkv_fp8_sizes(shape, slab, &qb, &kvb, &sb, &wb)) != FKV_OK) return st;
    if (!Q || !K_cur || !V_cur || !kv_len || !Q8 || !K8 || !V8T || !scales)
        return fail(FKV_ERR_ARG, "NULL tensor pointer");
    const int H = shape->hist_frames;
    bool any_dynamic = false;
    for (int h = 0; h < shape->n_heads; ++h) any_dynamic |= heads[h].type == FKV_DYNAMIC;
    if (H > 0 && (!K_hist || !V_hist)) return fail(FKV_ERR_ARG, "NULL K_hist/V_hist");
    if (H > 0 && any_dynamic && !kept_seg) return fail(FKV_ERR_ARG, "kept_seg is NULL");
    if ((st = check_slots(shape, frame_slot)) != FKV_OK) return st;
    for (int h = 0; h < shape->n_heads; ++h) {
        int64_t kept = 0;
        if ((st = fkv_kept_tokens_max(shape, heads, h, &kept)) != FKV_OK) return st;
        if (kept > slab)
            return fail(FKV_ERR_CAPACITY, "slab %d below head %d's %lld retained tokens", slab, h, (long long)kept);
    }
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < wb)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, wb);
    fkv::Fp8PackArgs a;
    memset(&a, 0, sizeof a);
    a.Q = (const uint16_t *)Q;
    a.Kc = a.K_cur = (const uint16_t *)K_cur;
    a.Vc = a.V_cur = (const uint16_t *)V_cur;
    a.kv_len = kv_len;
    a.slab = slab;
    a.n_heads = shape->n_heads;
    a.Lq = shape->chunk_frames * shape->frame_tokens;
    a.d = shape->head_dim;
    a.rows = ((int64_t)slab + a.Lq + 63) / 64 * 64;
    a.Q8 = (uint8_t *)Q8;
    a.K8 = (uint8_t *)K8;
    a.V8T = (uint8_t *)V8T;
    a.scales = scales;
    a.ws = (double *)workspace;
    a.chunk_rows = fkv::kFp8ChunkRows;
    a.n_kchunks = (int)(((int64_t)slab + a.Lq + fkv::kFp8ChunkRows - 1) / fkv::kFp8ChunkRows);
    a.n_qchunks = (a.Lq + fkv::kFp8ChunkRows - 1) / fkv::kFp8ChunkRows;
    a.paged = 1;
    a.K_hist = (const uint16_t *)(H > 0 ? K_hist : K_cur);
    a.V_hist = (const uint16_t *)(H > 0 ? V_hist : V_cur);
    a.F = shape->frame_tokens;
    a.L = shape->seg_tokens;
    a.H = H;
    a.cap = shape->cap_frames;
    a.n_seg = fkv_num_segments(shape);
    auto magic = [](int P, uint32_t *hi, uint32_t *lo) {   // floor(2^64 / P) + 1; P = 1 as 0, 0
        if (P == 1) {
            *hi = *lo = 0;
            return;
        }
        const unsigned __int128 m = (((unsigned __int128)1) << 64) / (uint64_t)P + 1;
        *hi = (uint32_t)(uint64_t)(m >> 32);
        *lo = (uint32_t)(uint64_t)m;
    };
    magic(a.F, &a.mf_hi, &a.mf_lo);
    magic(a.L, &a.ml_hi, &a.ml_lo);
    a.kept_seg = kept_seg;
    a.kv_out = kv_len;
    for (int h = 0; h < shape->n_heads; ++h) {
        if (heads[h].type == FKV_DYNAMIC && H > 0) {
            a.st_kept[h] = -1;
            continue;
        }
        // static heads, and dynamic heads with nothing cached
        const StaticPlan p = heads[h].type == FKV_DYNAMIC ? StaticPlan{0, 0, 0} : static_plan(H, heads[h]);
        a.st_first[h] = p.n_first;
        a.st_gap[h] = p.gap;
        a.st_kept[h] = p.n_kept;
    }
    for (int t = 0; t < H; ++t) a.slots.slot[t] = frame_slot[t];
    (void)hipGetLastError();
    return device_status(fkv::launch_fp8_pack(a, (hipStream_t)stream), "fkv_fp8_pack_paged launch");
}

fkv_status fkv_chunk_attention_fp8(const fkv_shape *shape, const void *Q8, const void *K8, const void *V8T,
                                   int32_t slab, const int32_t *kv_len, const float *scales, float scale,
                                   void *O, float *lse, void *workspace, size_t workspace_bytes,
                                   void *stream) {
    fkv_status st;
    size_t qb, kvb, sb, wb;
    if ((st = fkv_fp8_sizes(shape, slab, &qb, &kvb, &sb, &wb)) != FKV_OK) return st;
    if (!Q8 || !K8 || !V8T || !kv_len || !scales || !O) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (!(scale > 0.f) || !isfinite(scale)) return fail(FKV_ERR_ARG, "scale %g must be positive and finite", (double)scale);
    int blocks = 0;
    if (workspace) {
        if ((st = balanced_blocks(&blocks)) != FKV_OK) return st;
        const size_t need = attention_workspace_bytes(shape, blocks);
        if (workspace_bytes < need)
            return fail(FKV_ERR_CAPACITY, "attention workspace of %zu bytes, %zu needed", workspace_bytes, need);
    }
    fkv::AttnArgs a;
    memset(&a, 0, sizeof a);
    a.Q = Q8;
    a.Kc = K8;
    a.Vc = V8T;
    a.O = O;
    a.lse = lse;
    a.kv_len = kv_len;
    a.slab = slab;
    a.n_heads = shape->n_heads;
    a.heads = all_heads(shape->n_heads);
    a.Lq = shape->chunk_frames * shape->frame_tokens;
    a.scale = scale;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.n_qtiles = (a.Lq + fkv::kAttnRowsBf16 - 1) / fkv::kAttnRowsBf16;
    a.n_items = a.n_heads * a.n_qtiles;
    a.items_per_xcd = (a.n_items + 7) / 8;
    a.n_blocks = blocks;
    a.part = (float *)workspace;
    if (workspace)
        a.item_counters = (uint32_t *)((char *)workspace + 2 * (size_t)blocks * fkv::attention_part_bytes(shape->head_dim));
    a.fp8_scales = scales;
    a.fp8_rows = ((int64_t)slab + a.Lq + 63) / 64 * 64;
    (void)hipGetLastError();
    return device_status(fkv::launch_attention_fp8(a, shape->head_dim, (hipStream_t)stream),
                         "fkv_chunk_attention_fp8 launch");
}

fkv_status fkv_attention_mass_workspace_size(const fkv_shape *shape, int32_t n_bins, size_t *bytes) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (!bytes) return fail(FKV_ERR_ARG, "bytes is NULL");
    if (n_bins < 1) return fail(FKV_ERR_ARG, "n_bins %d < 1", n_bins);
    const int lq = shape->chunk_frames * shape->frame_tokens;
    const size_t n_qtiles = (size_t)((lq + fkv::kAttnRowsBf16 - 1) / fkv::kAttnRowsBf16);
    *bytes = ((size_t)shape->n_heads * n_qtiles * 8 * n_bins * sizeof(float) + 255) & ~(size_t)255;
    return ok();
}

fkv_status fkv_attention_mass(const fkv_shape *shape, const void *Q, const void *Kc, int32_t slab,
                              const int32_t *kv_len, const void *K_cur, const float *lse, float scale,
                              int32_t n_bins, float *mass, int32_t accumulate, void *workspace,
                              size_t workspace_bytes, void *stream) {
    fkv_status st;
    if ((st = check_shape(shape)) != FKV_OK) return st;
    if (shape->dtype != FKV_BF16) return fail(FKV_ERR_SHAPE, "the attention mass takes bf16 inputs");
    if (!Q || !K_cur || !kv_len || !lse || !mass) return fail(FKV_ERR_ARG, "NULL tensor pointer");
    if (slab < 0) return fail(FKV_ERR_ARG, "slab %d < 0", slab);
    if (slab > 0 && !Kc) return fail(FKV_ERR_ARG, "NULL Kc with slab %d", slab);
    if (!(scale > 0.f) || !isfinite(scale)) return fail(FKV_ERR_ARG, "scale %g must be positive and finite", (double)scale);
    if (accumulate != 0 && accumulate != 1) return fail(FKV_ERR_ARG, "accumulate must be 0 or 1");
    const int64_t lq = (int64_t)shape->chunk_frames * shape->frame_tokens;
    const int64_t need_bins = (slab + lq + shape->frame_tokens - 1) / shape->frame_tokens;
    if (n_bins < need_bins)
        return fail(FKV_ERR_CAPACITY, "n_bins %d below ceil((slab + C*F) / F) = %lld", n_bins, (long long)need_bins);
    size_t need = 0;
    if ((st = fkv_attention_mass_workspace_size(shape, n_bins, &need)) != FKV_OK) return st;
    if (!workspace) return fail(FKV_ERR_ARG, "workspace is NULL");
    if (workspace_bytes < need)
        return fail(FKV_ERR_CAPACITY, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    fkv::AttnArgs a;
    memset(&a, 0, sizeof a);
    a.Q = Q;
    a.Kc = Kc ? Kc : K_cur;
    a.K_cur = K_cur;
    a.kv_len = kv_len;
    a.lse = (float *)lse;
    a.slab = slab;
    a.n_heads = shape->n_heads;
    a.heads = all_heads(shape->n_heads);
    a.Lq = (int32_t)lq;
    a.scale = scale;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.n_qtiles = (a.Lq + fkv::kAttnRowsBf16 - 1) / fkv::kAttnRowsBf16;
    a.n_items = a.n_heads * a.n_qtiles;
    a.part = (float *)workspace;
    a.mass_F = shape->frame_tokens;
    a.mass_bins = n_bins;
    a.mass_acc = accumulate;
    a.mass_out = mass;
    (void)hipGetLastError();
    return device_status(fkv::launch_attention_mass(a, shape->head_dim, (hipStream_t)stream),
                         "fkv_attention_mass launch");
}

fkv_status fkv_classify_heads(const float *mass, int32_t n_heads, int32_t n_bins, int32_t hist_frames,
                              int32_t sink_frames, int32_t transition_frames, float alpha, int32_t *head_type) {
    if (!mass || !head_type) return fail(FKV_ERR_ARG, "NULL pointer");
    if (n_heads < 1 || n_bins < 1) return fail(FKV_ERR_ARG, "n_heads %d, n_bins %d", n_heads, n_bins);
    if (hist_frames < 0 || hist_frames > n_bins)
        return fail(FKV_ERR_ARG, "hist_frames %d outside [0, n_bins=%d]", hist_frames, n_bins);
    if (sink_frames < 0 || transition_frames < 0) return fail(FKV_ERR_ARG, "negative frame count");
    if (!isfinite(alpha)) return fail(FKV_ERR_ARG, "alpha is not finite");
    for (int h = 0; h < n_heads; ++h) {
        const float *m = mass + (size_t)h * n_bins;
        double total = 0.0, generate = 0.0, transition = 0.0, sink = 0.0;
        for (int b = 0; b < n_bins; ++b) total += m[b];
        for (int b = hist_frames; b < n_bins; ++b) generate += m[b];
        for (int b = std::max(hist_frames - transition_frames, 0); b < hist_frames; ++b) transition += m[b];
        for (int b = 0; b < std::min(sink_frames, hist_frames); ++b) sink += m[b];
        const double denom = total - sink;
        const bool is_static = denom > 0.0 ? (generate + transition) / denom > (double)alpha : true;
        head_type[h] = is_static ? FKV_STATIC : FKV_DYNAMIC;
    }
    return ok();
}

const char *fkv_last_error(void) { return g_err; }

}  // extern "C"
