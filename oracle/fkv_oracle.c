/* fkv_oracle.c -- plain, slow, obviously correct CPU oracle of the Forcing-KV
 * hot path (arXiv 2605.09681).
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The product path (the
 * HIP library) never calls it, and the two share no code.
 *
 * Arithmetic: fp64 throughout.  Inputs are bf16 or fp32, so every product of
 * two inputs is exact in fp64; sums are plain left-to-right fp64 sums.  Built
 * without -ffast-math and with -ffp-contract=off.
 */
#include "fkv_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Widen one stored element to double (bf16 bits are the top half of an fp32). */
static double load_elem(const void *base, int dtype, size_t i) {
    if (dtype == FKVO_BF16) {
        uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    if (dtype == FKVO_F64) return ((const double *)base)[i];
    return (double)((const float *)base)[i];
}

void fkvo_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int fkvo_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---------------------------------------------------------------------------
 * Eq. 2 (Sec. 4.2): a static head attends to the sink frames and the
 * transition anchor frame(s) -- the most recent history frames -- plus the
 * current chunk.  Logical frame t is kept when it is one of the first `sink`
 * frames or one of the last `recent` frames of the H-frame history.
 * ------------------------------------------------------------------------- */
int fkvo_static_frames(int H, int sink, int recent, int32_t *frames_out) {
    int n = 0;
    for (int t = 0; t < H; ++t)
        if (t < sink || t >= H - recent) frames_out[n++] = t;
    return n;
}

long fkvo_gather_frames(int esize, int F, int d, const void *hist,
                        const int32_t *frame_slot, const int32_t *frames, int n,
                        void *out) {
    const size_t frame_bytes = (size_t)F * d * esize;
    for (int i = 0; i < n; ++i) {
        const char *src = (const char *)hist + (size_t)frame_slot[frames[i]] * frame_bytes;
        memcpy((char *)out + (size_t)i * frame_bytes, src, frame_bytes);
    }
    return (long)n * F;
}

int fkvo_n_segments(int H, int F, int L) {
    long tokens = (long)H * F;
    return (int)((tokens + L - 1) / L);
}

/* Address of logical history token x: frame x / F lives in slot frame_slot[x / F]. */
static size_t hist_row(long x, int F, int d, const int32_t *frame_slot) {
    long t = x / F, p = x % F;
    return ((size_t)frame_slot[t] * F + (size_t)p) * d;
}

/* ---------------------------------------------------------------------------
 * Eq. 3 (Sec. 4.3): s_t^(j) = Cosine(K_{t,j}, K_{t+1,j}).  Each history frame is
 * split into contiguous segments; a segment is compared with the same token
 * range one frame later.  The segment is a matrix of tokens x head_dim; its
 * cosine is taken over all of its elements (flattened).  For the last history
 * frame the "next frame" is the first frame of the current chunk.
 * ------------------------------------------------------------------------- */
void fkvo_score_head(int dtype, int d, int F, int H, int L, const void *hist,
                     const int32_t *frame_slot, const void *cur, float *s32,
                     double *s64) {
    const long HF = (long)H * F;
    const int n_seg = fkvo_n_segments(H, F, L);
#pragma omp parallel for schedule(dynamic, 1)
    for (int g = 0; g < n_seg; ++g) {
        long x0 = (long)g * L;
        long x1 = x0 + L < HF ? x0 + L : HF;
        double dot = 0.0, na = 0.0, nb = 0.0;
        for (long x = x0; x < x1; ++x) {
            size_t ra = hist_row(x, F, d, frame_slot);
            long y = x + F; /* same position, next frame */
            const void *bbase;
            size_t rb;
            if (y < HF) {
                bbase = hist;
                rb = hist_row(y, F, d, frame_slot);
            } else {
                bbase = cur;
                rb = (size_t)(y - HF) * d;
            }
            for (int c = 0; c < d; ++c) {
                double a = load_elem(hist, dtype, ra + c);
                double b = load_elem(bbase, dtype, rb + c);
                dot += a * b;
                na += a * a;
                nb += b * b;
            }
        }
        double cosv = (na * nb == 0.0) ? 0.0 : dot / sqrt(na * nb);
        s64[g] = cosv;
        s32[g] = (float)cosv;
    }
}

/* ---------------------------------------------------------------------------
 * Rolling cache (Sec. 4, the cache keeps a fixed window of past frames with
 * the sink frames pinned): the frames of a finished chunk are written into
 * the physical slots given for them, overwriting what those slots held.
 * new_frames: [n_frames][F][d]; hist: [cap][F][d].
 * ------------------------------------------------------------------------- */
void fkvo_append_frames(int esize, int F, int d, int n_frames,
                        const void *new_frames, const int32_t *dst_slot,
                        void *hist) {
    const size_t frame_bytes = (size_t)F * d * esize;
    for (int f = 0; f < n_frames; ++f)
        memcpy((char *)hist + (size_t)dst_slot[f] * frame_bytes,
               (const char *)new_frames + (size_t)f * frame_bytes, frame_bytes);
}

/* ---------------------------------------------------------------------------
 * The first-block proxy of Sec. 4.3: the similarity is computed from the key
 * states of all attention heads together, i.e. the segment is the matrix
 * heads x tokens x head_dim and its cosine is taken over all of those
 * elements.  Same products, sums and rounding as fkvo_score_head.
 * hist: [n_heads][cap][F][d]; cur: [n_heads][lq][d]; s32/s64: [n_seg].
 * ------------------------------------------------------------------------- */
void fkvo_score_pooled(int dtype, int n_heads, int d, int F, int H, int L,
                       int cap, long lq, const void *hist,
                       const int32_t *frame_slot, const void *cur, float *s32,
                       double *s64) {
    const long HF = (long)H * F;
    const int n_seg = fkvo_n_segments(H, F, L);
    const size_t hist_head = (size_t)cap * F * d, cur_head = (size_t)lq * d;
#pragma omp parallel for schedule(dynamic, 1)
    for (int g = 0; g < n_seg; ++g) {
        long x0 = (long)g * L;
        long x1 = x0 + L < HF ? x0 + L : HF;
        double dot = 0.0, na = 0.0, nb = 0.0;
        for (int h = 0; h < n_heads; ++h) {
            for (long x = x0; x < x1; ++x) {
                size_t ra = h * hist_head + hist_row(x, F, d, frame_slot);
                long y = x + F;
                const void *bbase;
                size_t rb;
                if (y < HF) {
                    bbase = hist;
                    rb = h * hist_head + hist_row(y, F, d, frame_slot);
                } else {
                    bbase = cur;
                    rb = h * cur_head + (size_t)(y - HF) * d;
                }
                for (int c = 0; c < d; ++c) {
                    double a = load_elem(hist, dtype, ra + c);
                    double b = load_elem(bbase, dtype, rb + c);
                    dot += a * b;
                    na += a * a;
                    nb += b * b;
                }
            }
        }
        double cosv = (na * nb == 0.0) ? 0.0 : dot / sqrt(na * nb);
        s64[g] = cosv;
        s32[g] = (float)cosv;
    }
}

/* ---------------------------------------------------------------------------
 * Eq. 3 BottomK.  A segment is forced (always kept) when it touches one of the
 * sink frames or one of the `recent` most recent frames.  The other segments
 * are candidates; within each selection group the min(k, |group|) candidates
 * with the LOWEST similarity are kept (the most similar ones are redundant and
 * evicted).  Order key (isNaN(s), s, g): a NaN score is evicted first, equal
 * scores (with -0 == +0) are resolved by the lower segment index.
 * ------------------------------------------------------------------------- */
typedef struct {
    float s;
    int32_t g;
} cand_t;

static int cand_cmp(const void *pa, const void *pb) {
    const cand_t *a = (const cand_t *)pa, *b = (const cand_t *)pb;
    int na = isnan(a->s) ? 1 : 0, nb = isnan(b->s) ? 1 : 0;
    if (na != nb) return na - nb;
    if (!na) {
        if (a->s < b->s) return -1;
        if (a->s > b->s) return 1;
    }
    return (a->g > b->g) - (a->g < b->g);
}

int fkvo_select_head(int H, int F, int L, int sink, int recent, int k, int scope,
                     const float *scores, int32_t *kept) {
    const long HF = (long)H * F;
    const int n_seg = fkvo_n_segments(H, F, L);
    char *keep = (char *)calloc((size_t)n_seg + 1, 1);
    int *group = (int *)malloc(sizeof(int) * ((size_t)n_seg + 1));
    cand_t *cands = (cand_t *)malloc(sizeof(cand_t) * ((size_t)n_seg + 1));
    int n_groups = 0;

    for (int g = 0; g < n_seg; ++g) {
        long x0 = (long)g * L;
        long x1 = x0 + L < HF ? x0 + L : HF;
        long first = x0 / F, last = (x1 - 1) / F;
        int forced = first < sink || last >= (long)H - recent;
        if (forced) {
            keep[g] = 1;
            group[g] = -1;
        } else {
            group[g] = scope == 0 ? (int)first : 0;
            if (group[g] + 1 > n_groups) n_groups = group[g] + 1;
        }
    }
    for (int grp = 0; grp < n_groups; ++grp) {
        int m = 0;
        for (int g = 0; g < n_seg; ++g)
            if (group[g] == grp) {
                cands[m].s = scores[g];
                cands[m].g = g;
                ++m;
            }
        qsort(cands, (size_t)m, sizeof(cand_t), cand_cmp);
        int kk = k < m ? k : m;
        for (int i = 0; i < kk; ++i) keep[cands[i].g] = 1;
    }
    int n = 0;
    for (int g = 0; g < n_seg; ++g)
        if (keep[g]) kept[n++] = g;
    for (int i = n; i < n_seg; ++i) kept[i] = -1;
    free(keep);
    free(group);
    free(cands);
    return n;
}

/* ---------------------------------------------------------------------------
 * Compaction (Sec. 4.3): the compressed cache is the union over history frames
 * of the kept segments, laid out in ascending segment order (temporal order,
 * sink first).
 * ------------------------------------------------------------------------- */
long fkvo_compact_head(int esize, int d, int F, int H, int L,
                       const int32_t *kept, int n_kept, const void *hist,
                       const int32_t *frame_slot, void *out) {
    const long HF = (long)H * F;
    const size_t row_bytes = (size_t)d * esize;
    long n = 0;
    for (int i = 0; i < n_kept; ++i) {
        long x0 = (long)kept[i] * L;
        long x1 = x0 + L < HF ? x0 + L : HF;
        for (long x = x0; x < x1; ++x, ++n)
            memcpy((char *)out + (size_t)n * row_bytes,
                   (const char *)hist + hist_row(x, F, d, frame_slot) * esize, row_bytes);
    }
    return n;
}

/* ---------------------------------------------------------------------------
 * Eq. 4 / Eq. 2: the current chunk's queries attend, without a mask, to the
 * retained history followed by the chunk's own keys/values.  Softmax written
 * out: z_j = scale <q, k_j>, m = max_j z_j, o = sum_j e^{z_j - m} v_j / sum_j
 * e^{z_j - m}.
 * ------------------------------------------------------------------------- */
void fkvo_attention_rows(int dtype, int d, long kv_len, long Lq, const void *Q,
                         const void *Kc, const void *Vc, const void *Kcur,
                         const void *Vcur, double scale, const int32_t *rows,
                         int n_rows, double *out, double *lse) {
    const long Lk = kv_len + Lq;
#pragma omp parallel
    {
        double *z = (double *)malloc(sizeof(double) * (size_t)(Lk > 0 ? Lk : 1));
        double *q = (double *)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 1)
        for (int i = 0; i < n_rows; ++i) {
            const long r = rows[i];
            for (int c = 0; c < d; ++c) q[c] = load_elem(Q, dtype, (size_t)r * d + c);
            double m = -INFINITY;
            for (long j = 0; j < Lk; ++j) {
                const void *kb = j < kv_len ? Kc : Kcur;
                size_t kr = (size_t)(j < kv_len ? j : j - kv_len) * d;
                double acc = 0.0;
                for (int c = 0; c < d; ++c) acc += q[c] * load_elem(kb, dtype, kr + c);
                z[j] = scale * acc;
                if (z[j] > m) m = z[j];
            }
            double den = 0.0;
            double *o = out + (size_t)i * d;
            for (int c = 0; c < d; ++c) o[c] = 0.0;
            for (long j = 0; j < Lk; ++j) {
                double w = exp(z[j] - m);
                den += w;
                const void *vb = j < kv_len ? Vc : Vcur;
                size_t vr = (size_t)(j < kv_len ? j : j - kv_len) * d;
                for (int c = 0; c < d; ++c) o[c] += w * load_elem(vb, dtype, vr + c);
            }
            for (int c = 0; c < d; ++c) o[c] /= den;
            if (lse) lse[i] = m + log(den);
        }
        free(z);
        free(q);
    }
}

/* ---------------------------------------------------------------------------
 * Offline head profiling, Sec. 4.1 (Eq. 1 uses the attention mass a head puts
 * on the generated chunk, the transition frame, the sink frames and the whole
 * window).  Attention mass of key block b (keys [bF, bF + F) of the key
 * sequence [Kc[0:kv_len]; Kcur]): the sum over every query row of the softmax
 * probabilities of the block's keys.  Exact fp64 softmax per row.
 * mass: [ceil((kv_len + Lq) / F)] fp64, overwritten.
 * ------------------------------------------------------------------------- */
void fkvo_attention_mass(int dtype, int d, long kv_len, long Lq, int F, const void *Q,
                         const void *Kc, const void *Kcur, double scale, double *mass) {
    const long Lk = kv_len + Lq;
    const long n_bins = (Lk + F - 1) / F;
    for (long b = 0; b < n_bins; ++b) mass[b] = 0.0;
#pragma omp parallel
    {
        double *z = (double *)malloc(sizeof(double) * (size_t)(Lk > 0 ? Lk : 1));
        double *q = (double *)malloc(sizeof(double) * (size_t)d);
        double *acc = (double *)calloc((size_t)n_bins, sizeof(double));
#pragma omp for schedule(dynamic, 4)
        for (long r = 0; r < Lq; ++r) {
            for (int c = 0; c < d; ++c) q[c] = load_elem(Q, dtype, (size_t)r * d + c);
            double m = -INFINITY;
            for (long j = 0; j < Lk; ++j) {
                const void *kb = j < kv_len ? Kc : Kcur;
                size_t kr = (size_t)(j < kv_len ? j : j - kv_len) * d;
                double dot = 0.0;
                for (int c = 0; c < d; ++c) dot += q[c] * load_elem(kb, dtype, kr + c);
                z[j] = scale * dot;
                if (z[j] > m) m = z[j];
            }
            double den = 0.0;
            for (long j = 0; j < Lk; ++j) den += exp(z[j] - m);
            for (long j = 0; j < Lk; ++j) acc[j / F] += exp(z[j] - m) / den;
        }
#pragma omp critical
        for (long b = 0; b < n_bins; ++b) mass[b] += acc[b];
        free(acc);
        free(z);
        free(q);
    }
}
