/* fkv.h -- C ABI of the Forcing-KV hot path on AMD MI355X (gfx950).
 *
 * Forcing-KV (arXiv 2605.09681) compresses the KV cache of streaming
 * autoregressive video-diffusion attention head by head:
 *   - static heads keep the sink frame(s) and the transition anchor frame(s)
 *     -- the most recent history frames -- (Sec. 4.2, Eq. 2);
 *   - dynamic heads split every history frame into segments, score each
 *     segment by the cosine similarity of its keys with the same segment of
 *     the next frame, keep the least similar ones (BottomK) and gather them
 *     (Sec. 4.3, Eq. 3 and the union defining the compressed cache);
 *   - the current chunk's queries then attend, without a mask, over
 *     [retained history; current chunk] (Eq. 2, Eq. 4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tensors are DEVICE pointers to row-major, contiguous memory, head_dim
 * innermost, element type `shape->dtype` (bf16 or fp32), 16-byte aligned:
 *   K_hist, V_hist : [n_heads][cap_frames][F][d]   history cache, physical slots
 *   K_cur, V_cur, Q: [n_heads][C*F][d]             current chunk (Lq = C*F tokens)
 *   Kc, Vc         : [n_heads][slab][d]            compressed history per head
 *   O              : [n_heads][C*F][d]             attention output
 *   scores         : float [n_heads][n_seg]        segment similarity (dynamic rows)
 *   kept_seg       : int32 [n_heads][n_seg]        kept segment ids, ascending, -1 padded
 *   kv_len         : int32 [n_heads]               retained history tokens per head
 * `frame_slot` is a HOST array of int32[hist_frames]: logical history frame t
 * (0 = oldest, the sink first) lives in physical slot frame_slot[t] of the
 * cache; this expresses a ring-buffer cache with pinned sink frames.
 * `heads` is a HOST array of fkv_head[n_heads]; `shape` a HOST struct.
 * Logical history tokens are numbered x = t*F + p (frame t, position p);
 * segment g covers tokens [g*L, min(g*L + L, H*F)), n_seg = ceil(H*F / L).
 *
 * Streams and ownership: every call validates its arguments on the host,
 * then enqueues kernels on `stream` (a hipStream_t, NULL = default stream)
 * and returns without synchronising; outputs are valid once the stream has
 * run them.  The caller owns every buffer, workspaces included; the library
 * allocates no device memory and keeps no pointer after a call returns.  K_hist and V_hist are
 * only read: dynamic heads keep their whole history for later similarity
 * scoring (Sec. 5.2), so compaction never modifies the cache.
 *
 * A slab of 0 tokens (nothing retained) may come with NULL Kc / Vc.
 *
 * Errors: a non-OK status is returned before anything is enqueued, so a
 * failed call writes nothing.  FKV_ERR_ARG: null pointer, bad enum, negative
 * budget, non-positive scale, slot out of range.  FKV_ERR_SHAPE: unsupported
 * shape (see fkv_shape; also a frame, the chunk or one head's cache of 2^31
 * bytes or more, which the kernels' 32-bit buffer ranges cannot address).
 * FKV_ERR_CAPACITY: `slab` or the workspace is too
 * small.  FKV_ERR_DEVICE: the HIP runtime reported a launch error.
 * fkv_last_error() returns a message for the last non-OK status of the calling
 * thread.  Calls on distinct streams are independent; calls that share an
 * output buffer must be ordered by the caller.
 */
#ifndef FKV_H
#define FKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FKV_MAX_HEADS 64     /* n_heads limit */
#define FKV_MAX_FRAMES 256   /* cap_frames limit */
#define FKV_MAX_SEGMENTS 4096 /* n_seg limit */

typedef enum {
    FKV_OK = 0,
    FKV_ERR_ARG = 1,
    FKV_ERR_SHAPE = 2,
    FKV_ERR_CAPACITY = 3,
    FKV_ERR_DEVICE = 4
} fkv_status;

typedef enum { FKV_BF16 = 0, FKV_F32 = 1 } fkv_dtype;
typedef enum { FKV_STATIC = 0, FKV_DYNAMIC = 1 } fkv_head_type;
/* Selection group of dynamic heads: FKV_SCOPE_FRAME keeps k segments in every
 * frame (the paper's per-frame BottomK, needs L < F); FKV_SCOPE_GLOBAL keeps k
 * segments among all candidate segments of the history. */
typedef enum { FKV_SCOPE_FRAME = 0, FKV_SCOPE_GLOBAL = 1 } fkv_scope;

typedef struct {
    int32_t n_heads;      /* 1..FKV_MAX_HEADS */
    int32_t head_dim;     /* d: 64 or 128 */
    int32_t frame_tokens; /* F >= 1: tokens per latent frame */
    int32_t hist_frames;  /* H: logical history frames, 0..cap_frames (0: nothing cached) */
    int32_t cap_frames;   /* physical slots in K_hist/V_hist, 1..FKV_MAX_FRAMES */
    int32_t chunk_frames; /* C >= 1: frames of the current chunk */
    int32_t seg_tokens;   /* L >= 1, with F % L == 0 or L % F == 0 */
    int32_t dtype;        /* fkv_dtype */
} fkv_shape;

typedef struct {
    int32_t type;          /* fkv_head_type */
    int32_t sink_frames;   /* >= 0: leading logical frames always kept */
    int32_t recent_frames; /* >= 0: trailing logical frames always kept (the
                              transition anchor frame is recent_frames = 1) */
    int32_t keep_k;        /* >= 0: dynamic heads keep min(keep_k, |group|)
                              segments per selection group */
    int32_t scope;         /* fkv_scope (dynamic heads) */
} fkv_head;

/* Number of segments n_seg = ceil(H*F / L) of `shape` (0 on a bad shape). */
int32_t fkv_num_segments(const fkv_shape *shape);

/* Largest kv_len head `head` can produce under its budget: for a static head
 * the exact |kept frames|*F, for a dynamic head the maximum over all score
 * outcomes (only a partial last segment makes it data dependent).  A `slab`
 * of at least the maximum over the heads of one call is accepted. */
fkv_status fkv_kept_tokens_max(const fkv_shape *shape, const fkv_head *heads,
                               int32_t head, int64_t *tokens);

/* Static structural pruning (Sec. 4.2, Eq. 2).  For every head of type
 * FKV_STATIC: the kept logical frames are [0, min(sink,H)) U [max(H-recent,0),
 * H), ascending, each once; their K and V rows are copied from physical slot
 * frame_slot[t] to Kc[h] / Vc[h] in that order, and kv_len[h] = |kept|*F.
 * Rows of dynamic heads are not touched.  FKV_ERR_CAPACITY if `slab` is below
 * the kept token count of a static head. */
fkv_status fkv_compress_static(const fkv_shape *shape, const fkv_head *heads,
                               const void *K_hist, const void *V_hist,
                               const int32_t *frame_slot, void *Kc, void *Vc,
                               int32_t slab, int32_t *kv_len, void *stream);

/* Device workspace fkv_score_segments needs for `shape` and the dynamic heads
 * of `heads` (a multiple of 256 bytes; 0 when no head is dynamic or H = 0).
 * Every scoring workspace (this one, fkv_score_pooled_workspace_size's) starts
 * with the arrival counters of the one-launch reduction: it must be
 * zero-filled once before its first use (e.g. hipMemset to 0), and every
 * scoring call leaves the counters at zero again when it completes, so
 * consecutive calls need nothing more.  Calls that share a workspace must be
 * ordered (one stream). */
fkv_status fkv_score_workspace_size(const fkv_shape *shape, const fkv_head *heads,
                                    size_t *bytes);

/* Segment-wise similarity (Sec. 4.3, Eq. 3).  For every head of type
 * FKV_DYNAMIC and every segment g: a = the keys of tokens [g*L, min(g*L+L,
 * H*F)), b = the keys of the same tokens shifted by one frame (x + F; tokens
 * at or past H*F are rows x + F - H*F of K_cur, i.e. the first frame of the
 * current chunk follows the last history frame).  Every product is exact in
 * fp64 and summed in fp64: dot = sum a*b, na = sum a*a, nb = sum b*b; then
 * scores[h][g] = (float)(dot / sqrt(na*nb)) rounded to nearest even, or 0 when
 * na*nb == 0.  The cosine is taken over the flattened segment (tokens x d).
 * `workspace` holds the arrival counters and fp64 partial sums (device memory
 * of at least fkv_score_workspace_size bytes, zero-filled before its first
 * use, see above).  Sums are in a fixed order, so the result is the same on
 * every run.  Rows of static heads are not touched.  H = 0 enqueues nothing. */
fkv_status fkv_score_segments(const fkv_shape *shape, const fkv_head *heads,
                              const void *K_hist, const int32_t *frame_slot,
                              const void *K_cur, float *scores, void *workspace,
                              size_t workspace_bytes, void *stream);

/* BottomK selection and compaction (Sec. 4.3, Eq. 3 and the union defining
 * the compressed cache).  For every head of type FKV_DYNAMIC: a segment is
 * forced (kept) when it touches one of the first sink_frames frames or the
 * last recent_frames frames; the other segments are candidates, grouped per
 * frame (FKV_SCOPE_FRAME) or all together (FKV_SCOPE_GLOBAL), and each group
 * keeps the min(keep_k, |group|) candidates of smallest key (isNaN(s), s, g):
 * the least similar segments, NaN scores evicted first, equal scores (-0 ==
 * +0) resolved by the lower index.  kept_seg[h] lists the kept segments in
 * ascending order, padded with -1; their K and V rows are copied to Kc[h] /
 * Vc[h] in that order; kv_len[h] = the number of tokens copied.  Reads
 * `scores` as fkv_score_segments leaves them (any fp32 values are accepted).
 * Rows of static heads are not touched.  FKV_ERR_CAPACITY if `slab` is below
 * fkv_kept_tokens_max of a dynamic head. */
fkv_status fkv_select_compact(const fkv_shape *shape, const fkv_head *heads,
                              const float *scores, const void *K_hist,
                              const void *V_hist, const int32_t *frame_slot,
                              int32_t *kept_seg, void *Kc, void *Vc, int32_t slab,
                              int32_t *kv_len, void *stream);

/* Rolling cache write (the cache keeps a fixed window of past frames, the
 * sink frame(s) pinned; Sec. 4): frame f of K_new / V_new, laid out
 * [n_heads][n_frames*F][d] (a finished chunk's K_cur / V_cur with n_frames =
 * C), is copied into physical slot dst_slot[f] of K_hist / V_hist for every
 * head, overwriting that slot.  dst_slot is a HOST array of n_frames distinct
 * slots in [0, cap_frames); 0 <= n_frames <= cap_frames.  The caller then
 * describes the new logical order with frame_slot on the next calls (the
 * write pointer advances; no cached frame moves). */
fkv_status fkv_append_frames(const fkv_shape *shape, const void *K_new,
                             const void *V_new, int32_t n_frames,
                             const int32_t *dst_slot, void *K_hist, void *V_hist,
                             void *stream);

/* Device workspace fkv_score_pooled needs for `shape` (a multiple of 256
 * bytes; 0 when H = 0). */
fkv_status fkv_score_pooled_workspace_size(const fkv_shape *shape, size_t *bytes);

/* The first-block proxy of Sec. 4.3: one similarity per segment from the key
 * states of ALL n_heads heads together, computed once (from the first
 * transformer block's keys) and reused by every layer.  For segment g, with
 * the per-head quantities of fkv_score_segments summed over the heads,
 *   scores[g] = (float)(sum_h dot_h / sqrt(sum_h na_h * sum_h nb_h)),
 * i.e. the cosine over heads x tokens x head_dim elements (0 when the
 * product of the sums is 0).  Same exact fp64 products, fp64 sums and single
 * rounding as fkv_score_segments.  scores: float [n_seg] (device).  The
 * workspace is zero-filled before its first use, as for fkv_score_segments.
 * H = 0 enqueues nothing. */
fkv_status fkv_score_pooled(const fkv_shape *shape, const void *K_hist,
                            const int32_t *frame_slot, const void *K_cur,
                            float *scores, void *workspace, size_t workspace_bytes,
                            void *stream);

/* Incremental rescoring (the per-step cost of Sec. 4.3's scoring).  Across the
 * AR steps of one chunk the history does not change, only K_cur does, and of
 * all Eq. 3 terms only the pair (frame H-1, first frame of K_cur) depends on
 * it.  fkv_score_history streams the history once and stores, per listed head,
 * unit u (a segment, or a frame when segments span frames) and frame t < H,
 * the fp64 sums SQ(t) = sum K_t^2 and DOT(t) = sum K_t * K_{t+1} (t < H-1) in
 * `stats`, a caller-owned device buffer of fkv_score_stats_size bytes.
 * fkv_score_segments_cached then streams frames H-1 and H only and writes the
 * same scores fkv_score_segments (pooled = 0) or fkv_score_pooled (pooled = 1)
 * would, bit for bit: per listed head [n_heads][n_seg] (rows of static heads
 * untouched), or one row [n_seg].  Both reduce every per-frame sum with the
 * same fixed-order tree, and fkv_score_segments sums a segment's per-frame
 * terms in the same frame order as this call.
 * pooled = 0 lists the dynamic heads of `heads`; pooled = 1 lists every head
 * and `heads` may be NULL.  stats stays valid until the history (K_hist
 * contents or frame_slot) changes; the caller runs fkv_score_history again
 * then (once per chunk).  `workspace` is the scoring workspace
 * (fkv_score_workspace_size, or fkv_score_pooled_workspace_size when pooled).
 * Nothing is enqueued when there is no listed head or H = 0.  Errors as in
 * fkv_score_segments; FKV_ERR_CAPACITY also for a short stats buffer. */
fkv_status fkv_score_stats_size(const fkv_shape *shape, const fkv_head *heads, int32_t pooled,
                                size_t *bytes);
fkv_status fkv_score_history(const fkv_shape *shape, const fkv_head *heads, int32_t pooled,
                             const void *K_hist, const int32_t *frame_slot, double *stats,
                             size_t stats_bytes, void *workspace, size_t workspace_bytes,
                             void *stream);
fkv_status fkv_score_segments_cached(const fkv_shape *shape, const fkv_head *heads,
                                     int32_t pooled, const void *K_hist,
                                     const int32_t *frame_slot, const void *K_cur,
                                     const double *stats, size_t stats_bytes, float *scores,
                                     void *workspace, size_t workspace_bytes, void *stream);

/* fkv_select_compact with one score row shared by every dynamic head: scores
 * is float [n_seg] (as fkv_score_pooled writes it) instead of
 * [n_heads][n_seg].  Everything else, outputs and errors included, is as in
 * fkv_select_compact. */
fkv_status fkv_select_compact_pooled(const fkv_shape *shape, const fkv_head *heads,
                                     const float *scores, const void *K_hist,
                                     const void *V_hist, const int32_t *frame_slot,
                                     int32_t *kept_seg, void *Kc, void *Vc,
                                     int32_t slab, int32_t *kv_len, void *stream);

/* BottomK selection alone (Sec. 4.3, Eq. 3): the kept_seg and kv_len that
 * fkv_select_compact writes for every FKV_DYNAMIC head, without copying any
 * K/V row -- for attention that reads the kept segments in place
 * (fkv_chunk_attention_paged).  scores is float [n_heads][n_seg], or, with
 * shared_row = 1, one row [n_seg] shared by every dynamic head (the pooled
 * first-block proxy).  Rows of static heads are not touched; with H = 0 every
 * dynamic head gets kv_len 0. */
fkv_status fkv_select(const fkv_shape *shape, const fkv_head *heads, const float *scores,
                      int32_t shared_row, int32_t *kept_seg, int32_t *kv_len, void *stream);

/* Bytes of device scratch the library holds per GPU for
 * fkv_score_select_noalloc (8 MiB: a 480P layer's 6 dynamic heads need
 * 0.4 MiB, a 1080P layer's 2.2 MiB). */
#define FKV_NOALLOC_SCRATCH_BYTES (8u << 20)

/* fkv_score_segments followed by fkv_select in ONE kernel launch: the
 * workgroup that completes a dynamic head's scores also selects its kept
 * segments.  scores, kept_seg and kv_len are written exactly as the two calls
 * write them.  Workspace as in fkv_score_segments (same size; zero-filled
 * before its first use).  With H = 0 the dynamic heads get kv_len 0. */
fkv_status fkv_score_select(const fkv_shape *shape, const fkv_head *heads,
                            const void *K_hist, const int32_t *frame_slot,
                            const void *K_cur, float *scores, int32_t *kept_seg,
                            int32_t *kv_len, void *workspace, size_t workspace_bytes,
                            void *stream);

/* Device workspace fkv_chunk_attention takes for its balanced schedule on the
 * CURRENT device (hipGetDevice): 2 x the device's compute units, rounded down
 * to a multiple of 8, partial-result slots of 256 rows x (2*head_dim + 8)
 * bytes (about 34 MB for head_dim 128 on a 256-CU device), then one 256-byte
 * arrival counter per (head, 256-row query tile).  0 for FKV_F32, which has no
 * balanced schedule.  FKV_ERR_DEVICE if the device cannot be queried. */
fkv_status fkv_attention_workspace_size(const fkv_shape *shape, size_t *bytes);

/* Chunk attention over the compressed cache (Eq. 2 for static heads, Eq. 4
 * for dynamic heads).  For every head h and query row r < C*F, with keys
 * [Kc[h][0:n]; K_cur[h]] and values [Vc[h][0:n]; V_cur[h]], n = kv_len[h]
 * (read on the device, clamped to [0, slab]):
 *   O[h][r] = softmax(scale * Q[h][r] . keys^T) . values   (no mask)
 * bf16: bf16 inputs, MFMA products accumulated in fp32, fp32 online softmax,
 * probabilities rounded to bf16 for the value product, output normalised and
 * rounded to bf16.  fp32: all fp32.  scale must be positive and finite
 * (1/sqrt(d) is the usual choice).
 * lse (nullable, float [n_heads][C*F]) receives the natural-log normaliser of
 * the weights that multiply V.  fp32: log(sum_j exp(z_j)), z_j = scale*q.k_j.
 * bf16: m*ln2 + log(sum_j p_j) with p_j = bf16(2^(z_j*log2(e) - m)), the
 * bf16-rounded probabilities the value product uses, and m a per-row reference
 * (the running maximum in log2 units); since every p_j lies within a relative
 * 2^-9 of its exact value, this differs from log(sum_j exp(z_j)) by at most
 * -log(1 - 2^-9) = 1.96e-3 beyond the rounding of the bf16 score products.
 *
 * Work schedule (bf16): with workspace == NULL every (head, 256-row query
 * tile) is one workgroup; heads with longer caches then finish last.  With a
 * device workspace of at least fkv_attention_workspace_size bytes, zero-filled
 * by the caller before its first use (every bf16 call leaves its counters at
 * zero again), the key tiles of all heads and query tiles are split evenly
 * over one workgroup per compute unit, and the parts of a tile cut by a split
 * are combined by the workgroup that completes the last of them
 * (FKV_ERR_CAPACITY if the workspace is smaller).  Both schedules compute the
 * same function; a split tile's parts are normalised and rounded to bf16
 * before they are combined, so its output may differ from the one-workgroup
 * result by about one bf16 step.
 * fp32 ignores the workspace.  Two calls that share a workspace must be
 * ordered by the caller. */
fkv_status fkv_chunk_attention(const fkv_shape *shape, const void *Q,
                               const void *Kc, const void *Vc, int32_t slab,
                               const int32_t *kv_len, const void *K_cur,
                               const void *V_cur, float scale, void *O,
                               float *lse, void *workspace, size_t workspace_bytes,
                               void *stream);

/* fkv_chunk_attention restricted to the heads head_list[0..n_list) (host
 * int32 array; distinct indices in [0, n_heads)): only those heads' rows of O
 * and lse are written, every other byte is left as it was.  Arguments,
 * layouts, schedule and workspace are as in fkv_chunk_attention; the balanced
 * schedule spreads the listed heads' work over all compute units.  This lets a
 * caller attend the heads whose compressed cache is ready (the static heads
 * after fkv_compress_static) while other heads are still being compressed on
 * another stream -- each concurrent call needs its own workspace.  n_list = 0
 * enqueues nothing.  FKV_ERR_ARG for a bad list (out of range, repeated,
 * NULL with n_list > 0). */
fkv_status fkv_chunk_attention_heads(const fkv_shape *shape, const int32_t *head_list,
                                     int32_t n_list, const void *Q, const void *Kc,
                                     const void *Vc, int32_t slab, const int32_t *kv_len,
                                     const void *K_cur, const void *V_cur, float scale,
                                     void *O, float *lse, void *workspace,
                                     size_t workspace_bytes, void *stream);

/* Chunk attention of the static heads (Eq. 2) read in place from the cache:
 * for every head with heads[h].type == FKV_STATIC, the keys are the tokens of
 * its kept history frames -- logical frames [0, min(sink, H)) U
 * [max(H - recent, 0), H) in ascending order, logical frame t in slot
 * frame_slot[t] of K_hist [n_heads][cap_frames][F][d] -- followed by
 * K_cur[h], and likewise for the values.  This is exactly what
 * fkv_compress_static followed by fkv_chunk_attention_heads over the static
 * heads computes (same kernel, same rounding, the same result bit for bit),
 * without the compressed copy: no Kc, Vc or kv_len.  Only the static heads'
 * rows of O and lse are written.  Workspace and schedule as in
 * fkv_chunk_attention.  bf16 only and frame_tokens >= 64 (a key tile then
 * spans at most two cached frames): FKV_ERR_SHAPE otherwise.  frame_slot is
 * a HOST int32 array of hist_frames entries in [0, cap_frames). */
fkv_status fkv_chunk_attention_static(const fkv_shape *shape, const fkv_head *heads,
                                      const void *K_hist, const void *V_hist,
                                      const int32_t *frame_slot, const void *Q,
                                      const void *K_cur, const void *V_cur, float scale,
                                      void *O, float *lse, void *workspace,
                                      size_t workspace_bytes, void *stream);

/* fkv_score_select for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same scores, kept_seg and kv_len, but the scoring workspace
 * is the library's own device array of FKV_NOALLOC_SCRATCH_BYTES on the
 * current device (no workspace argument; the call allocates nothing --
 * no hipMalloc, hipFree or allocating library routine).  Every call on a GPU
 * shares that GPU's array: calls that may overlap on one GPU (other streams,
 * other host threads) race and must be ordered by the caller; each call
 * leaves the array's counters at zero for the next one.  FKV_ERR_CAPACITY
 * when the shape's scoring workspace (fkv_score_workspace_size) exceeds the
 * array; FKV_ERR_DEVICE if the array's address cannot be obtained.  Other
 * arguments and errors as in fkv_score_select. */
fkv_status fkv_score_select_noalloc(const fkv_shape *shape, const fkv_head *heads,
                                    const void *K_hist, const int32_t *frame_slot,
                                    const void *K_cur, float *scores, int32_t *kept_seg,
                                    int32_t *kv_len, void *stream);

/* Chunk attention with every listed head's kept history read in place from
 * the cache (Eq. 2 for static heads, Eq. 4 for dynamic heads), without a
 * compressed copy.  The keys of head h are its kept history tokens in
 * ascending logical order, then K_cur[h]; likewise the values:
 *   FKV_STATIC:  the frames [0, min(sink, H)) U [max(H - recent, 0), H), as
 *                in fkv_chunk_attention_static;
 *   FKV_DYNAMIC: the segments kept_seg[h][0..] covering kv_len[h] tokens, as
 *                fkv_select (or fkv_score_select) writes them (kv_len is read
 *                on the device and clamped to H*F).
 * The result is bit for bit what fkv_compress_static / fkv_select_compact
 * followed by fkv_chunk_attention_heads computes for the same heads.
 * head_list (HOST int32, n_list distinct heads) selects the heads; NULL means
 * every head.  Only the listed heads' rows of O and lse are written.
 * Workspace and schedule as in fkv_chunk_attention.  bf16 only, frame_tokens
 * >= 64; when a dynamic head is listed, also min(seg_tokens, frame_tokens)
 * >= 64 and cap_frames * (frame_tokens / min(seg_tokens, frame_tokens)) <=
 * 256 (the page table holds one byte per piece): FKV_ERR_SHAPE otherwise.
 * kept_seg [n_heads][n_seg] and kv_len [n_heads] are device arrays (needed
 * when a dynamic head is listed and H > 0). */
fkv_status fkv_chunk_attention_paged(const fkv_shape *shape, const fkv_head *heads,
                                     const int32_t *head_list, int32_t n_list,
                                     const void *K_hist, const void *V_hist,
                                     const int32_t *frame_slot, const int32_t *kept_seg,
                                     const int32_t *kv_len, const void *Q, const void *K_cur,
                                     const void *V_cur, float scale, void *O, float *lse,
                                     void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Offline head profiling (Sec. 4.1, Eq. 1).  A profiling pass runs the layer
 * on the uncompressed cache (every head static with recent_frames = H, so Kc
 * holds the whole history in logical order), calls fkv_chunk_attention for
 * the log-normaliser, then fkv_attention_mass, and finally classifies.
 *
 * fkv_attention_mass: for every head h and key block b (keys [bF, bF + F) of
 * [Kc[h][0:kv_len]; K_cur[h]], F = frame_tokens -- with the full history,
 * block t < H is logical frame t and blocks H .. H+C-1 are the chunk's frames):
 *   mass[h][b] (=, or += when accumulate = 1) sum over every query row r of
 *                exp(scale * Q[h][r] . k - lse[h][r])
 * with the same bf16 score product as the attention kernel; fp32 sums in a
 * fixed order (deterministic).  mass: float [n_heads][n_bins] (device),
 * n_bins >= ceil((slab + C*F) / F) (FKV_ERR_CAPACITY otherwise).  bf16 only.
 * The workspace needs no initialisation. */
fkv_status fkv_attention_mass_workspace_size(const fkv_shape *shape, int32_t n_bins,
                                             size_t *bytes);

fkv_status fkv_attention_mass(const fkv_shape *shape, const void *Q, const void *Kc,
                              int32_t slab, const int32_t *kv_len, const void *K_cur,
                              const float *lse, float scale, int32_t n_bins,
                              float *mass, int32_t accumulate, void *workspace,
                              size_t workspace_bytes, void *stream);

/* Eq. 1 on HOST data: mass float [n_heads][n_bins] with bins 0 .. H-1 the
 * history frames (oldest first) and bins H .. n_bins-1 the generated chunk.
 * With A_Total = all bins, A_Generate = bins >= H, A_Transition = the last
 * transition_frames history frames (the paper's transition anchor frame is
 * 1), A_Sink = the first sink_frames history frames, all summed in fp64:
 *   head_type[h] = FKV_STATIC if (A_Generate + A_Transition) /
 *                  (A_Total - A_Sink) > alpha, else FKV_DYNAMIC
 * (FKV_STATIC when the denominator is 0).  head_type: HOST int32 [n_heads]. */
fkv_status fkv_classify_heads(const float *mass, int32_t n_heads, int32_t n_bins,
                              int32_t hist_frames, int32_t sink_frames,
                              int32_t transition_frames, float alpha,
                              int32_t *head_type);

/* ---------------------------------------------------------------------------
 * FP8 variant of the chunk attention (App. F: the method combined with FP8
 * attention), for the FP8 matrix cores of gfx950.  Two steps:
 *
 * fkv_fp8_pack quantises one layer's attention inputs per head to OCP FP8
 * E4M3 (round to nearest even): keys [Kc[0:kv_len]; K_cur] after subtracting
 * their per-channel mean mu (fp64 sum, one rounding to fp32; softmax is
 * unchanged by it), scaled by inv_k = 448 / amax|K - mu|; queries by
 * inv_q = 448 / amax|Q|; values per channel by inv_v[c] = 448 / amax_c|V|
 * (correctly rounded fp32; 0 for an all-zero tensor or channel).
 *   Q8     uint8 [n_heads][C*F][d]
 *   K8     uint8 [n_heads][rows][d], rows = round_up(slab + C*F, 64): row j of
 *          head h is key j of [Kc[h][0:kv_len]; K_cur[h]], rows past it zero
 *   V8T    uint8 [n_heads][rows/64][d][64]: each 64-key tile transposed, its
 *          keys in the order the attention kernel consumes them
 *   scales float [n_heads][4 + 3d]: s_q, s_k, inv_q, inv_k, s_v[d], inv_v[d],
 *          mu[d], with s = amax / 448
 * Inputs are bf16 (FKV_ERR_SHAPE for FKV_F32).  kv_len is read on the device.
 * The workspace (fkv_fp8_sizes) holds statistics and needs no initialisation.
 *
 * fkv_chunk_attention_fp8 computes, from those buffers,
 *   O[h][r] = softmax(scale * (s_q s_k) q8 . k8^T) . (v8 * s_v)
 * with FP8 products accumulated in fp32, fp32 online softmax, and the
 * probabilities themselves rounded to E4M3 (relative error <= 2^-4) before
 * the value product; the normaliser sums the same rounded probabilities.
 * O is bf16 [n_heads][C*F][d]; lse as in fkv_chunk_attention.  The workspace
 * selects the balanced schedule exactly as in fkv_chunk_attention (same size
 * query, fkv_attention_workspace_size; zero-filled before its first use, its
 * counters left at zero by every call; cut items are combined by the
 * workgroup whose part completes last). */
fkv_status fkv_fp8_sizes(const fkv_shape *shape, int32_t slab, size_t *q_bytes,
                         size_t *kv_bytes, size_t *scale_bytes,
                         size_t *workspace_bytes);

fkv_status fkv_fp8_pack(const fkv_shape *shape, const void *Q, const void *Kc,
                        const void *Vc, int32_t slab, const int32_t *kv_len,
                        const void *K_cur, const void *V_cur, void *Q8, void *K8,
                        void *V8T, float *scales, void *workspace,
                        size_t workspace_bytes, void *stream);

/* fkv_fp8_pack_paged: fkv_fp8_pack with every head's retained history read
 * in place from the slot-permuted cache (App. F with Eq. 2 / Eq. 3): the
 * history rows of head h are, in order, the kept frames of a static head
 * (from its budget, as fkv_compress_static gathers them) or the kept
 * segments of a dynamic head (kept_seg[h] and kv_len[h] as fkv_select or
 * fkv_score_select write them, as fkv_select_compact gathers them).  The
 * packed buffers, scales and workspace are byte for byte those of
 * fkv_compress_static + fkv_select_compact + fkv_fp8_pack over the same
 * inputs, with no compressed copy made.
 *   heads      host array [n_heads] (budgets), as for fkv_compress_static
 *   K_hist, V_hist, frame_slot   the cache and its slot map (frame_slot is host
 *              data), as for fkv_chunk_attention_paged
 *   kept_seg   device int32 [n_heads][n_seg], read for dynamic heads
 *   kv_len     device int32 [n_heads]: read for dynamic heads; the static
 *              heads' retained lengths are written to it, so that
 *              fkv_chunk_attention_fp8 can follow (with the same slab)
 *   slab       packed key rows per head before the chunk (as for
 *              fkv_fp8_sizes); FKV_ERR_CAPACITY if any head can retain more
 *              tokens (fkv_kept_tokens_max)
 * Other arguments, the workspace and errors as for fkv_fp8_pack; bf16 only. */
fkv_status fkv_fp8_pack_paged(const fkv_shape *shape, const fkv_head *heads,
                              const void *K_hist, const void *V_hist,
                              const int32_t *frame_slot, const int32_t *kept_seg,
                              int32_t *kv_len, const void *Q, const void *K_cur,
                              const void *V_cur, int32_t slab, void *Q8, void *K8,
                              void *V8T, float *scales, void *workspace,
                              size_t workspace_bytes, void *stream);

fkv_status fkv_chunk_attention_fp8(const fkv_shape *shape, const void *Q8,
                                   const void *K8, const void *V8T, int32_t slab,
                                   const int32_t *kv_len, const float *scales,
                                   float scale, void *O, float *lse,
                                   void *workspace, size_t workspace_bytes,
                                   void *stream);

/* Message describing the calling thread's last non-OK status ("" if none). */
const char *fkv_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FKV_H */
