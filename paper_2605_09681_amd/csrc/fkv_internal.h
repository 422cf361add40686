// fkv_internal.h -- kernel argument blocks and launchers shared by the HIP
// translation units of libfkv (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fkv.h"

namespace fkv {

// Native 16-byte vector (usable with the nontemporal load/store builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Per-call tables passed by value in the kernel argument segment: the host
// has validated every entry, so kernels index with them without re-checking.
struct SlotTable {
    int32_t slot[FKV_MAX_FRAMES];  // logical history frame -> physical slot
};

struct HeadList {
    int32_t n;                      // number of heads in the list
    int32_t head[FKV_MAX_HEADS];    // head index into the [n_heads] tensors
};

// ---------------------------------------------------------------- static copy
struct StaticCopyArgs {
    const uint8_t *K_hist, *V_hist;
    uint8_t *Kc, *Vc;
    int32_t *kv_len;
    int64_t slab;                   // tokens per head in Kc/Vc
    int64_t frame_vecs;             // 16-byte vectors per frame (F*d*esize/16)
    int64_t row_bytes;              // d * esize
    int32_t F, cap;
    HeadList heads;
    int32_t n_first[FKV_MAX_HEADS]; // kept frames y < n_first are frame y
    int32_t gap[FKV_MAX_HEADS];     // kept frames y >= n_first are frame y + gap
    int32_t n_kept[FKV_MAX_HEADS];  // kept frame count
    SlotTable slots;
};

// --------------------------------------------------------------- dynamic copy
struct DynCopyArgs {
    const uint8_t *K_hist, *V_hist;
    uint8_t *Kc, *Vc;
    const int32_t *kept_seg;        // [n_heads][n_seg]
    int64_t slab;
    int64_t piece_vecs;             // 16-byte vectors per piece
    int64_t row_bytes;
    int32_t F, L, H, cap, n_seg;
    int32_t piece_tokens;           // min(L, F)
    int32_t pieces_per_seg;         // max(1, L / F)
    HeadList heads;
    SlotTable slots;
};

// ------------------------------------------------------------ cache append
struct AppendArgs {
    const uint8_t *K_new, *V_new;   // [n_heads][n_frames*F][d]
    uint8_t *K_hist, *V_hist;       // [n_heads][cap][F][d]
    int64_t frame_vecs;             // 16-byte vectors per frame
    int32_t n_frames, cap;
    SlotTable slots;                // destination slot of new frame f
};

// ---------------------------------------------------------------- selection
struct SelectArgs {
    const float *scores;            // head h's row at scores + h * score_stride
    int64_t score_stride;           // n_seg, or 0 when all heads share one row
    int32_t *kept_seg;              // [n_heads][n_seg]
    int32_t *kv_len;                // [n_heads]
    int32_t F, L, H, n_seg;
    HeadList heads;
    int32_t sink[FKV_MAX_HEADS], recent[FKV_MAX_HEADS], scope[FKV_MAX_HEADS];
    int32_t k[FKV_MAX_HEADS];       // kk = min(keep_k, |group|) per head
};

// Fused selection + compaction: used when a head has at most kFusedSelectMaxSeg
// segments, so that every copy workgroup can re-derive its head's keep set.
constexpr int kFusedSelectMaxSeg = 128;
struct SelectCopyArgs {
    SelectArgs sel;
    DynCopyArgs copy;
};

// ------------------------------------------------------------------ scoring
// One kernel per scoring call (k_score.hip).  Workgroup (cg, u, li) streams
// column group cg of unit u of listed head li over the frames [t_begin,
// t_begin + n_frames) and writes its per-frame partial sums; the last
// workgroup of a head to arrive (a counter in the workspace) reduces the
// head's partials in a fixed order and finishes: statistics, scores, and
// optionally the BottomK selection.
enum ScoreMode : int32_t { kScoreModeFull = 0, kScoreModeHistory = 1, kScoreModeCached = 2 };

struct ScoreArgs {
    const uint8_t *K_hist, *K_cur;
    float *scores;                  // [n_heads][n_seg], or [n_seg] when pooled
    uint32_t *counters;             // [heads.n + 1] arrivals per listed head, then finished heads
    double *part;                   // [li][row][n_cg] partial sums, row = (u*n_frames + f)*2 + q
    double *totals;                 // [li][row] per-head sums (pooled finish)
    double *group;                  // [li][arrival group][row] sums of each arrival group's partials
    double *stats;                  // incremental rescoring: [li][H][units][2] = SQ(t), DOT(t, t+1)
    int64_t frame_vecs;             // 16-byte vectors per frame (F*d*esize/16)
    int64_t cur_head_vecs;          // 16-byte vectors per head of K_cur (C*F*d*esize/16)
    int32_t F, L, H, cap, n_seg;
    int32_t units;                  // units per frame, F / U with U = min(L, F)
    int32_t unit_vecs;              // 16-byte vectors per unit
    int32_t n_cg;                   // column groups (workgroups) per unit
    int32_t mode;                   // ScoreMode
    int32_t pooled;                 // 1: one score row over all listed heads
    int32_t t_begin, n_frames;      // streamed frames (frame H is the first frame of K_cur)
    int32_t select;                 // 1: also the BottomK selection (the fields at the end)
    int32_t lds_rows;               // doubles of dynamic LDS for the finishing workgroup's row sums
    HeadList heads;
    SlotTable slots;
    // BottomK parameters per listed head (fused selection)
    int32_t *kept_seg, *kv_len;
    int32_t sink[FKV_MAX_HEADS], recent[FKV_MAX_HEADS], scope[FKV_MAX_HEADS];
    int32_t k[FKV_MAX_HEADS];       // kk = min(keep_k, |group|) per listed head
};

// ---------------------------------------------------------------- attention
struct AttnArgs {
    const void *Q, *Kc, *Vc, *K_cur, *V_cur;
    void *O;
    float *lse;
    const int32_t *kv_len;
    int64_t slab;
    int32_t n_heads, Lq;
    int32_t n_qtiles;               // ceil(Lq / BM)
    int32_t n_items;                // heads.n * n_qtiles (work item = (list entry, query tile))
    HeadList heads;                 // the heads this launch computes, in schedule order
    int32_t items_per_xcd;          // ceil(n_items / 8)
    int32_t n_blocks;               // balanced schedule: workgroups (multiple of 8); 0 = one per item
    float *part;                    // balanced schedule: 2 * n_blocks partial-result slots
    uint32_t *item_counters;        // balanced schedule, bf16: arrivals per item (kItemCounterStride apart),
                                    // zero between calls
    int32_t mass_F;                 // attention mass: keys per bin (frame tokens)
    int32_t mass_bins;              // attention mass: bins per head
    int32_t mass_acc;               // attention mass: 1 = add to mass_out, 0 = overwrite
    float *mass_out;                // attention mass: [n_heads][mass_bins]
    const float *fp8_scales;        // FP8 path: per-head scale block (see k_fp8.hip)
    int64_t fp8_rows;               // FP8 path: key rows per head of the packed K / V^T
    float scale;                    // softmax scale
    float scale_log2;               // scale * log2(e)
    // Paged heads (fkv_chunk_attention_static, fkv_chunk_attention_paged): the
    // retained history is read straight from the cache K_hist / V_hist
    // [n_heads][cap][F][d] as a sequence of kept pieces of pg_P tokens (one
    // piece length for the launch; pg_ppf = F / pg_P pieces per frame).  A
    // static entry (st_kept[li] >= 0) keeps frames: kept frame y is logical
    // frame y (y < st_first[li]) or y + st_gap[li], in slot slots.slot[t], and
    // its history length is st_kept[li] * F (kv_len is not read).  A dynamic
    // entry (st_kept[li] < 0) keeps the segments listed in kept_seg[h] (as
    // fkv_select writes them) and its history length is kv_len[h].
    int32_t paged;
    const void *K_hist, *V_hist;
    int32_t F, cap;
    int32_t pg_P, pg_ppf;           // piece tokens, pieces per frame
    uint32_t pg_magic_hi, pg_magic_lo;  // floor(2^64 / pg_P) + 1: j0 / pg_P by multiplication
    int32_t pg_L, pg_nseg;          // segment length and segments per head (dynamic entries)
    const int32_t *kept_seg;        // [n_heads][pg_nseg] (dynamic entries)
    int32_t st_first[FKV_MAX_HEADS], st_gap[FKV_MAX_HEADS], st_kept[FKV_MAX_HEADS];
    SlotTable slots;
};

// ------------------------------------------------------------ FP8 packing
struct Fp8PackArgs {
    const uint16_t *Q, *Kc, *Vc, *K_cur, *V_cur;  // bf16 inputs
    const int32_t *kv_len;
    int64_t slab;
    int32_t n_heads, Lq, d;
    int64_t rows;                   // packed key rows per head (multiple of 64)
    uint8_t *Q8, *K8, *V8T;
    float *scales;                  // [n_heads][fp8_scale_floats(d)]
    double *ws;                     // statistics partials
    int32_t n_kchunks, n_qchunks, chunk_rows;
    // Read in place (fkv_fp8_pack_paged): the history rows of head h are its
    // kept frames (static, st_kept[h] >= 0: kept frame y is logical frame y
    // (y < st_first[h]) or y + st_gap[h]) or its kept segments (dynamic: the
    // ids in kept_seg[h], kv_len[h] tokens), read from K_hist / V_hist
    // [n_heads][cap][F][d] through the slot map; the static heads' lengths
    // are written to kv_out.
    int32_t paged;
    const uint16_t *K_hist, *V_hist;
    int32_t F, L, H, cap, n_seg;
    uint32_t mf_hi, mf_lo, ml_hi, ml_lo;   // floor(2^64 / F) + 1 and floor(2^64 / L) + 1
    const int32_t *kept_seg;        // [n_heads][n_seg]
    int32_t *kv_out;                // [n_heads]: static heads' kv_len
    int32_t st_first[FKV_MAX_HEADS], st_gap[FKV_MAX_HEADS], st_kept[FKV_MAX_HEADS];
    SlotTable slots;
};

constexpr int kScoreThreads = 256;
constexpr int kAttnRowsBf16 = 256;  // query rows per attention workgroup (bf16 MFMA kernel)
constexpr int kAttnKeysPerTile = 64; // keys per tile of the bf16 MFMA kernel
constexpr int kAttnRowsF32 = 32;    // query rows per attention workgroup (fp32 kernel)
constexpr int kScoreWaves = kScoreThreads / 64;

// Scoring workspace: counters, partials and per-head sums for n_list heads.
size_t score_workspace_bytes(int n_list, int H, int units, int n_cg);
int score_column_groups(int64_t unit_vecs);  // workgroups per unit

hipError_t launch_static_copy(const StaticCopyArgs &a, int max_kept, hipStream_t s);
hipError_t launch_dyn_copy(const DynCopyArgs &a, int max_pieces, hipStream_t s);
hipError_t launch_append(const AppendArgs &a, int n_heads, hipStream_t s);
hipError_t launch_select(const SelectArgs &a, hipStream_t s);
hipError_t launch_select_copy(const SelectCopyArgs &a, int max_pieces, hipStream_t s);
// one scoring launch in a.mode (full pass, history statistics, or cached scores)
hipError_t launch_score(const ScoreArgs &a, bool f32, hipStream_t s);
void score_workspace_layout(ScoreArgs &a, void *ws, int n_list, int H, int units, int n_cg);
hipError_t launch_attention_bf16(const AttnArgs &a, int head_dim, hipStream_t s);
size_t attention_part_bytes(int head_dim);  // bytes of one partial-result slot (bf16 kernel)
// Arrival counters of the bf16 balanced schedule: one 256-byte line per item,
// after the 2 * n_blocks partial-result slots of the workspace.
constexpr int kItemCounterStride = 64;   // uint32 per counter
inline size_t attention_counter_bytes(int64_t n_items) { return (size_t)n_items * kItemCounterStride * 4; }

// attention mass per key block (head profiling), k_attn.hip; the workspace holds
// n_heads * n_qtiles * 8 waves * mass_bins floats
hipError_t launch_attention_mass(const AttnArgs &a, int head_dim, hipStream_t s);

// FP8 path (k_fp8.hip)
constexpr int kFp8ChunkRows = 512;          // rows per statistics workgroup
__host__ __device__ inline int fp8_scale_floats(int d) { return 4 + 3 * d; }
inline size_t fp8_stats_doubles(int n_heads, int n_chunks, int d) { return (size_t)n_heads * n_chunks * d * 4; }
hipError_t launch_fp8_pack(const Fp8PackArgs &a, hipStream_t s);
hipError_t launch_attention_fp8(const AttnArgs &a, int head_dim, hipStream_t s);
hipError_t launch_attention_f32(const AttnArgs &a, int head_dim, hipStream_t s);

}  // namespace fkv
