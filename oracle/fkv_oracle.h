/* fkv_oracle.h -- plain CPU oracle of the Forcing-KV hot path.
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may call this.  It shares no code, header or
 * constant with the HIP library.
 *
 * Every routine works on one attention head, in fp64, in the order the paper
 * states the method:
 *   Eq. 2  (Sec. 4.2)  static structural pruning: sink frames, the transition
 *                      anchor frame(s) and the current chunk;
 *   Eq. 3  (Sec. 4.3)  segment-wise cosine similarity of adjacent frames and
 *                      BottomK selection of the least similar segments;
 *   Sec. 4.3 (the union defining the compressed K/V)  compaction;
 *   Eq. 4 / Eq. 2      attention of the current chunk's queries over
 *                      [compressed history; current chunk].
 *
 * Element storage: FKVO_BF16 = uint16 bf16 bit patterns, FKVO_F32 = float,
 * FKVO_F64 = double (attention inputs only).
 * All tensors are row-major with head_dim innermost.
 */
#ifndef FKV_ORACLE_H
#define FKV_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FKVO_BF16 0
#define FKVO_F32 1
#define FKVO_F64 2  /* attention inputs only (dequantized FP8 values) */

/* Kept logical frames of a static head: [0, sink) U [H - recent, H), ascending,
 * each frame once.  Writes at most H entries; returns the count. */
int fkvo_static_frames(int H, int sink, int recent, int32_t *frames_out);

/* Copies whole logical frames (frame t lives in physical slot frame_slot[t])
 * into a contiguous token list.  hist: [cap][F][d]; out: [n*F][d].
 * Returns the number of tokens written. */
long fkvo_gather_frames(int esize, int F, int d, const void *hist,
                        const int32_t *frame_slot, const int32_t *frames, int n,
                        void *out);

/* Number of segments ceil(H*F / L) of the history token range. */
int fkvo_n_segments(int H, int F, int L);

/* Eq. 3 similarity: for every segment g (logical tokens [gL, min(gL+L, HF))),
 * the cosine between the segment's keys and the keys of the same token range
 * one frame later (tokens at or past H*F come from the current chunk).
 * Exact fp64 products, fp64 sums, one rounding to fp32.
 * hist: [cap][F][d]; cur: [C*F][d]; s32/s64: [n_seg]. */
void fkvo_score_head(int dtype, int d, int F, int H, int L, const void *hist,
                     const int32_t *frame_slot, const void *cur, float *s32,
                     double *s64);

/* Rolling cache: writes frame f of new_frames ([n_frames][F][d]) into
 * physical slot dst_slot[f] of hist ([cap][F][d]). */
void fkvo_append_frames(int esize, int F, int d, int n_frames,
                        const void *new_frames, const int32_t *dst_slot,
                        void *hist);

/* The first-block proxy of Sec. 4.3: one similarity per segment from the keys
 * of all heads together (the cosine over heads x tokens x head_dim elements).
 * hist: [n_heads][cap][F][d]; cur: [n_heads][lq][d]; s32/s64: [n_seg]. */
void fkvo_score_pooled(int dtype, int n_heads, int d, int F, int H, int L,
                       int cap, long lq, const void *hist,
                       const int32_t *frame_slot, const void *cur, float *s32,
                       double *s64);

/* Eq. 3 BottomK: keeps the forced segments (those touching the sink frames or
 * the last `recent` frames) plus, in every selection group, the min(k, |group|)
 * candidates of smallest key (isNaN(s), s, g).  scope 0: one group per frame;
 * scope 1: one group of all candidates.  kept: [n_seg], ascending, -1 padded.
 * Returns the kept count. */
int fkvo_select_head(int H, int F, int L, int sink, int recent, int k, int scope,
                     const float *scores, int32_t *kept);

/* Compaction: concatenation of the kept segments' token rows, ascending.
 * Returns kv_len (tokens written). */
long fkvo_compact_head(int esize, int d, int F, int H, int L,
                       const int32_t *kept, int n_kept, const void *hist,
                       const int32_t *frame_slot, void *out);

/* Eq. 4 / Eq. 2 attention for the listed query rows:
 * O[r] = softmax(scale * q_r . [Kc[0:kv_len]; Kcur]^T) [Vc[0:kv_len]; Vcur].
 * out: [n_rows][d] fp64; lse (nullable): natural-log normaliser per row. */
void fkvo_attention_rows(int dtype, int d, long kv_len, long Lq, const void *Q,
                         const void *Kc, const void *Vc, const void *Kcur,
                         const void *Vcur, double scale, const int32_t *rows,
                         int n_rows, double *out, double *lse);

/* Offline head profiling (Sec. 4.1, Eq. 1): attention mass of every block of
 * F keys of [Kc[0:kv_len]; Kcur], summed over all Lq query rows (exact fp64
 * softmax per row).  mass: [ceil((kv_len + Lq) / F)]. */
void fkvo_attention_mass(int dtype, int d, long kv_len, long Lq, int F, const void *Q,
                         const void *Kc, const void *Kcur, double scale, double *mass);

/* Number of OpenMP threads a parallel region would use. */
int fkvo_max_threads(void);
/* Threads of the following parallel regions (timing only; results do not
 * depend on it). */
void fkvo_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
