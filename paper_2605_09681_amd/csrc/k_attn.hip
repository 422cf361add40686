// k_attn.hip -- chunk attention over each head's compressed cache (Eq. 2 for
// static heads, Eq. 4 for dynamic heads), bf16 inputs, gfx950 MFMA.
//
// For head h the key sequence is [Kc[h][0:kv_len[h]]; K_cur[h]] (the retained
// history, then the current chunk) and likewise for values; every query row of
// the chunk attends to all of it with no mask.  The per-head key count is
// ragged (it comes from the device-side kv_len), and one key tile may straddle
// the history/chunk boundary.  The PAGED instantiation attends heads in place:
// their retained history -- the kept frames of Eq. 2 for static heads, the
// kept segments of Eq. 3 for dynamic heads -- is read straight from the
// slot-permuted cache through a per-head page table (load_tile_paged), with no
// compressed copy.
//
// Workgroup = 8 waves = 256 query rows of one head (32 per wave), in two
// groups of four waves; one workgroup fills a CU.  Keys are processed in tiles
// of 64.  Per wave and tile, with v_mfma_f32_32x32x16_bf16:
//   S^T = K . Q^T   (A = K rows from LDS, B = the wave's Q rows, held in VGPRs),
//                   2 x (d/16) MFMAs;
//   online softmax in fp32 (exp2 with the scale folded into log2 units; the
//                   row sum adds the bf16-rounded probabilities with v_dot2);
//   O^T += V^T . P^T (A = rows of a V^T tile in LDS, B = P taken straight from
//                    the S^T accumulators, rounded to bf16), 4 x (d/32) MFMAs.
// Computing S transposed makes each lane own one query column, so P needs no
// data movement between the two products: in the 32x32 accumulator layout a
// lane holds 16 keys of its query, which are exactly the 8-element k-slices the
// B operand of the value product takes (any consistent permutation of the
// contraction index is allowed; the V^T tile is stored with the same
// permutation).  Row maxima need one cross-lane exchange (lanes l and l^32
// share a query).  Both operands are read from LDS with 16-byte reads; V is
// transposed on its way into LDS (measured faster than the LDS transpose
// reads).
//
// The two wave groups run the same loop one phase apart (see attn_segment), so
// on every SIMD one wave's softmax overlaps the other wave's MFMA block -- VALU
// and MFMA work of two waves overlap well, that of one wave much less.  The
// running max only moves when a tile's max exceeds it by more than 8 (log2
// units): probabilities stay below 2^8 and the accumulator rescale is skipped
// for most tiles; the final normalisation is exact either way.
//
// Global K/V rows come in through buffer loads whose per-lane offsets are loop
// invariant; rows past the end of a source fall outside the buffer's range and
// read as zero (the straddling tile merges both sources that way).
//
// Schedules: a work item is (entry of the launch's head list, query tile);
// one workgroup per item, or the balanced schedule (attn_common.h) that splits
// the key tiles of all items evenly over one workgroup per CU; the parts of a
// split item are merged by the workgroup that completes the last of them
// (merge_rows).  Heads with longer caches make the per-item
// schedule uneven (at 480P a dynamic head has 342 key tiles per query tile, a
// static head 245, on 228 items for 256 CUs).
#include "attn_common.h"
#include "attn_merge.h"
#include "handover.h"

namespace fkv {
namespace {

using namespace attn;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;      // 8 waves: two groups of 4
constexpr int kGroupThreads = 256; // one group stages a whole K or V tile
constexpr float kRescaleSlack = 8.f;  // log2 units the running max may lag behind
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw 32-bit buffer, range checked
constexpr bf16x2_t kOnes2 = {(__bf16)1.f, (__bf16)1.f};

template <int D>
struct Cfg {
    static constexpr int RSE = D + 8;           // K row stride in LDS (16-byte pad), elements
    static constexpr int TRSE = BN + 8;         // V^T row stride in LDS (16-byte pad), elements
    static constexpr int CPR = D / 8;           // 16-byte chunks per row
    static constexpr int RPP = kGroupThreads / CPR;  // rows one pass of a 256-thread group covers
    static constexpr int NV = BN / RPP;              // 16-byte vectors per thread per staged tile
    static constexpr int KS = D / 16;           // k-steps of S^T = K Q^T
    static constexpr int MB = D / 32;           // 32-row blocks of O^T
    static constexpr int TILE = BN * RSE;       // elements per K tile
    static constexpr int VTILE = D * TRSE;      // elements per V^T tile
    static constexpr int VUNITS = (BN / 4) * CPR;  // (4 keys x 8 dims) units of a V tile
    static_assert(NV >= 1 && BN % RPP == 0, "tile shape");
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// Rows of the key tile starting at j0 of [hist (kvl rows); chunk (Lq rows)] into
// registers, zeros past Lk = kvl + Lq: N 16-byte vectors at byte offsets
// off0 + i*step within the tile.  Rows past the end of a source fall outside
// its buffer range and read as zero; the tile straddling the history/chunk
// boundary merges both sources that way.
template <int D, int N>
__device__ __forceinline__ void load_tile(const uint16_t *hist, const uint16_t *chunk, int j0, int kvl,
                                          int Lk, int Lq, u32x4 *dst, uint32_t off0, uint32_t step) {
    if (j0 + BN <= kvl) {
        const auto r = rsrc(hist + (size_t)j0 * D, BN * D * 2);
#pragma unroll
        for (int i = 0; i < N; ++i) dst[i] = bload(r, off0 + i * step);
    } else if (j0 >= kvl) {
        const auto r = rsrc(chunk + (size_t)(j0 - kvl) * D, (uint32_t)(Lk - j0) * D * 2);
#pragma unroll
        for (int i = 0; i < N; ++i) dst[i] = bload(r, off0 + i * step);
    } else {
        const int nh = kvl - j0;
        const int nc = min(BN - nh, Lq);
        const auto rh = rsrc(hist + (size_t)j0 * D, (uint32_t)nh * D * 2);
        const auto rc = rsrc(chunk, (uint32_t)nc * D * 2);
        const uint32_t shift = (uint32_t)nh * D * 2;  // chunk rows start at tile row nh
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const uint32_t o = off0 + i * step;
            // below tile row nh, o - shift wraps to a huge offset: out of range, reads 0
            dst[i] = bload(rh, o) | bload(rc, o - shift);
        }
    }
}

// Page table of a head read in place: the cache position of each kept piece
// (pg_P tokens), one byte per piece -- piece y's entry sits in byte y >> 6 of
// lane y & 63, up to 256 pieces in one VGPR, looked up with v_readlane, so the
// tile loop never waits on a scalar load (whose counter it shares with the LDS
// reads).  Piece y starts at cache row entry(y) * pg_P of the head, entry =
// slot * pg_ppf + (piece within its frame).
//   static entry: the pieces of kept frame y / pg_ppf, which is logical frame
//                 y' (y' < st_first) or y' + st_gap;
//   dynamic entry: the pieces of the segments in kept_seg[h] (ascending, as
//                 the selection wrote them).
// The host has checked that every entry fits in a byte.
__device__ __forceinline__ uint32_t kept_piece_table(const AttnArgs &a, int li, int kvl, int lane) {
    uint32_t tab = 0;
    const int ppf = a.pg_ppf;
    const int n = a.st_kept[li];
    if (n >= 0) {
        const int first = a.st_first[li], gap = a.st_gap[li];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int y = lane + 64 * k;
            if (y < n * ppf) {
                const int fy = y / ppf, u = y - fy * ppf;
                tab |= (uint32_t)(a.slots.slot[fy < first ? fy : fy + gap] * ppf + u) << (8 * k);
            }
        }
        return tab;
    }
    const int m = a.pg_L > a.F ? a.pg_L / a.F : 1;           // pieces per segment
    const int n_pieces = kvl / a.pg_P;
    const int32_t *ks = a.kept_seg + (size_t)a.heads.head[li] * a.pg_nseg;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int y = lane + 64 * k;
        if (y < n_pieces) {
            // a kept_seg row and kv_len that disagree must not address outside
            // the head's cache: clamp the segment id
            const int q = y / m, g = min(max(ks[q], 0), a.pg_nseg - 1);
            int t, u;
            if (a.pg_L <= a.F) {
                t = g / ppf;
                u = g - t * ppf;
            } else {
                t = min(g * m + (y - q * m), (int)(a.slab / a.F) - 1);   // a short last segment ends at H
                u = 0;
            }
            tab |= (uint32_t)(a.slots.slot[t] * ppf + u) << (8 * k);
        }
    }
    return tab;
}
__device__ __forceinline__ int kept_piece(uint32_t tab, int y) {
    return (int)((uint32_t)__builtin_amdgcn_readlane((int)tab, y & 63) >> (8 * (y >> 6))) & 255;
}

// The same for a head read in place from the cache (paged): history row p is
// row p mod P of kept piece y = p / P, at cache row kept_piece(tab, y) * P.
// With P >= 64 a tile touches at most two kept pieces and the chunk; each part
// has its own range-checked buffer and the three loads are OR-ed, every row
// outside a part reading as zero.
// j0 / P for 0 <= j0 < 2^31 with the launch's 64-bit reciprocal M = floor(2^64 / P) + 1
// (= magic_hi * 2^32 + magic_lo): floor(j0 * M / 2^64) exactly, since j0 * M / 2^64
// exceeds j0 / P by less than 2^-33 < 1 / P.  A few scalar multiplies instead of
// the generic division sequence in every tile load.
__device__ __forceinline__ int div_piece(const AttnArgs &a, int j0) {
    const uint64_t p = (uint64_t)(uint32_t)j0 * a.pg_magic_hi + __umulhi((uint32_t)j0, a.pg_magic_lo);
    return (int)(p >> 32);
}

template <int D, int N>
__device__ __forceinline__ void load_tile_paged(const AttnArgs &a, const uint16_t *hist, uint32_t tab, int P,
                                                const uint16_t *chunk, int j0, int kvl, int Lk, int Lq,
                                                u32x4 *dst, uint32_t off0, uint32_t step) {
    if (j0 >= kvl) {
        const auto r = rsrc(chunk + (size_t)(j0 - kvl) * D, (uint32_t)(Lk - j0) * D * 2);
#pragma unroll
        for (int i = 0; i < N; ++i) dst[i] = bload(r, off0 + i * step);
        return;
    }
    auto piece = [&](int y) { return hist + (size_t)kept_piece(tab, y) * P * D; };
    const int y0 = div_piece(a, j0), r0 = j0 - y0 * P;
    const int na = min(min(P - r0, kvl - j0), BN);            // rows of kept piece y0
    const auto ra = rsrc(piece(y0) + (size_t)r0 * D, (uint32_t)na * D * 2);
    if (na == BN) {
#pragma unroll
        for (int i = 0; i < N; ++i) dst[i] = bload(ra, off0 + i * step);
        return;
    }
    // the rest of the tile: the next kept piece while history lasts, then the chunk
    const int nb = j0 + na < kvl ? min(BN - na, kvl - (j0 + na)) : 0;
    const int nc = j0 + na + nb >= kvl ? min(BN - na - nb, Lq) : 0;
    const auto rb = rsrc(nb > 0 ? piece(y0 + 1) : hist, (uint32_t)nb * D * 2);
    const auto rc = rsrc(chunk, (uint32_t)nc * D * 2);
    const uint32_t sb = (uint32_t)na * D * 2, sc = (uint32_t)(na + nb) * D * 2;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const uint32_t o = off0 + i * step;
        // rows before a part's start wrap to huge offsets: out of range, read 0
        dst[i] = bload(ra, o) | bload(rb, o - sb) | bload(rc, o - sc);
    }
}

// Position of a key tile of a head read in place: its first key j0 and, while
// j0 is in the history, the kept piece y it starts in, the row r within that
// piece (j0 = y * P + r) and that row's offset in the cache.  The tile loop
// advances it by one tile per iteration with a few scalar adds; the page
// table is read again only where a piece ends (reading it for every tile
// measured 0.9% slower: each wave's scalar instructions take issue cycles
// from its own stream).
struct PageCursor {
    int j0, y, r;
    uint32_t off;  // element offset of history row j0 in the head's cache (j0 < kvl)
};

// The tile at `c` (as load_tile_paged).  The history length kvl is a whole
// number of pieces, so a tile starting in piece y holds min(P - r, BN) rows of
// it, then the next piece's rows while history lasts, then the chunk's.
template <int D, int N>
__device__ __forceinline__ void load_tile_cursor(const uint16_t *hist, uint32_t tab, int P, const PageCursor &c,
                                                 const uint16_t *chunk, int kvl, int Lk, int Lq, u32x4 *dst,
                                                 uint32_t off0, uint32_t step) {
    if (c.j0 >= kvl) {
        const auto r = rsrc(chunk + (size_t)(c.j0 - kvl) * D, (uint32_t)(Lk - c.j0) * D * 2);
#pragma unroll
        for (int i = 0; i < N; ++i) dst[i] = bload(r, off0 + i * step);
        return;
    }
    const int na = min(P - c.r, BN);
    const auto ra = rsrc(hist + c.off, (uint32_t)na * D * 2);
    if (na == BN) {
#pragma unroll
        for (int i = 0; i < N; ++i) dst[i] = bload(ra, off0 + i * step);
        return;
    }
    const bool more = c.j0 + na < kvl;  // another kept piece follows, else the chunk
    const auto rb = rsrc(more ? hist + (size_t)kept_piece(tab, c.y + 1) * P * D : chunk,
                         (uint32_t)(more ? BN - na : min(BN - na, Lq)) * D * 2);
    const uint32_t sb = (uint32_t)na * D * 2;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const uint32_t o = off0 + i * step;
        // rows before the second part's start wrap to huge offsets: out of range, read 0
        dst[i] = bload(ra, o) | bload(rb, o - sb);
    }
}

// One MFMA block of a wave: optionally O^T += V^T P^T for one key tile (4 x MB
// products, accumulators o[mb] cycled so consecutive products are independent),
// then optionally S^T = K Q^T for the next tile (KS x 2 products, the two
// accumulators interleaved).  The A operand of every product comes from LDS;
// its reads are issued kPrefetch products ahead so their latency overlaps the
// preceding products.
constexpr int kPrefetch = 4;

template <int D, bool PV, bool QK>
__device__ __forceinline__ void mfma_block(const uint16_t *vs, const uint16_t *ks, int vbase, int kbase,
                                           const bf16x8_t (&pb)[4], const bf16x8_t (&qf)[D / 16],
                                           f32x16_t (&o)[D / 32], f32x16_t (&s)[2]) {
    using C = Cfg<D>;
    constexpr int NPV = PV ? 4 * C::MB : 0;
    constexpr int NQK = QK ? 2 * C::KS : 0;
    constexpr int NSTEP = NPV + NQK;
    // Step order: the value products (accumulators o[mb] cycled) then the score
    // products (accumulators s[0], s[1] alternating).
    auto is_pv = [&](int st) { return st < NPV; };
    auto index = [&](int st) { return st < NPV ? st : st - NPV; };
    auto read_a = [&](int st) -> bf16x8_t {
        const int i = index(st);
        if (is_pv(st)) {
            const int t = i / C::MB, mb = i % C::MB;
            return __builtin_bit_cast(bf16x8_t, *(const u32x4 *)(vs + vbase + (32 * mb) * C::TRSE + 16 * t));
        }
        const int kk = i >> 1, kb = i & 1;
        return __builtin_bit_cast(bf16x8_t, *(const u32x4 *)(ks + kbase + kb * 32 * C::RSE + kk * 16));
    };
    if (QK) {
        s[0] = f32x16_t{};
        s[1] = f32x16_t{};
    }
    bf16x8_t fr[kPrefetch];
#pragma unroll
    for (int i = 0; i < kPrefetch; ++i)
        if (i < NSTEP) fr[i] = read_a(i);
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
        const bf16x8_t a = fr[st % kPrefetch];
        if (st + kPrefetch < NSTEP) fr[st % kPrefetch] = read_a(st + kPrefetch);
        const int i = index(st);
        if (is_pv(st)) {
            const int t = i / C::MB, mb = i % C::MB;
            o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[t], o[mb], 0, 0, 0);
        } else {
            const int kk = i >> 1, kb = i & 1;
            s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s[kb], 0, 0, 0);
        }
    }
    // Keep the operand reads kPrefetch products ahead: kPrefetch LDS reads,
    // then alternate one MFMA and one LDS read.
#pragma unroll
    for (int i = 0; i < kPrefetch && i < NSTEP; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
    for (int st = 0; st < NSTEP; ++st) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (st + kPrefetch < NSTEP) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
}

// One segment: positions [t0, t1) of item (h, qt), where position j is key
// tile (j + rot) mod T of the item's T tiles (the order of key tiles does not
// change the result beyond rounding).  slot == nullptr means the segment is the
// whole item and the normalised output (and lse) is written; otherwise the
// partial result goes to the slot.  Uses every thread of the workgroup and
// leaves no LDS read pending.
template <int D, bool PAGED>
__device__ __forceinline__ void attn_segment(const AttnArgs &a, uint16_t (&Ks)[2][Cfg<D>::TILE],
                                             uint16_t (&Vs)[2][Cfg<D>::VTILE], int li, int qt, int t0,
                                             int t1, int rot, float *slot) {
    using C = Cfg<D>;
    const int h = a.heads.head[li];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = wave >> 2;  // 0: leads by half a tile, 1: trails
    const int l32 = lane & 31, hl = lane >> 5;
    const int Lq = a.Lq;
    const int n = t1 - t0;       // >= 1

    // The wave's 32 query rows, in the B-operand layout: lane holds row l32,
    // dims [16*kk + 8*hl, +8).
    const int qrow = qt * BM + wave * 32 + l32;
    const bool qok = qrow < Lq;
    const uint16_t *Qh = (const uint16_t *)a.Q + (size_t)h * Lq * D;
    bf16x8_t qf[C::KS];
#pragma unroll
    for (int kk = 0; kk < C::KS; ++kk) {
        const u32x4 v = qok ? *(const u32x4 *)(Qh + (size_t)qrow * D + kk * 16 + hl * 8) : u32x4{0, 0, 0, 0};
        qf[kk] = __builtin_bit_cast(bf16x8_t, v);
    }

    const int kvl = entry_kvl<PAGED>(a, li);
    const int Lk = kvl + Lq;
    const uint16_t *Kc = PAGED ? (const uint16_t *)a.K_hist + (size_t)h * a.cap * a.F * D
                               : (const uint16_t *)a.Kc + (size_t)h * a.slab * D;
    const uint16_t *Vc = PAGED ? (const uint16_t *)a.V_hist + (size_t)h * a.cap * a.F * D
                               : (const uint16_t *)a.Vc + (size_t)h * a.slab * D;
    const uint16_t *Kq = (const uint16_t *)a.K_cur + (size_t)h * Lq * D;
    const uint16_t *Vq = (const uint16_t *)a.V_cur + (size_t)h * Lq * D;
    const uint32_t ktab = PAGED ? kept_piece_table(a, li, kvl, lane) : 0u;

    // Loop-invariant per-thread load geometry within the thread's group of 256:
    // rows r0 + RPP*i, chunk c (group 0 stages K tiles, group 1 V tiles).
    const int gtid = tid & 255;
    const int c = gtid % C::CPR, r0 = gtid / C::CPR;
    const uint32_t voff = (uint32_t)(r0 * D + c * 8) * 2u;    // + i*RPP*D*2 bytes
    const int wofs = r0 * C::RSE + c * 8;                      // + i*RPP*RSE elements
    // V staging unit of this thread: keys 4*vq .. 4*vq+3 of the tile, dims 8*vc .. 8*vc+7.
    const int vq = gtid % (BN / 4), vc = gtid / (BN / 4);
    const uint32_t voffv = (uint32_t)(4 * vq * D + vc * 8) * 2u;  // + r*D*2 bytes

    // first key of the segment's tile j
    const int T = (Lk + BN - 1) / BN;
    const int kt0 = (t0 + rot) % T;
    auto tile0 = [&](int j) {
        const int k = kt0 + j;
        return (k >= T ? k - T : k) * BN;
    };
    auto load_k = [&](int j0, u32x4 (&dst)[4]) {
        if (PAGED)
            load_tile_paged<D, C::NV>(a, Kc, ktab, a.pg_P, Kq, j0, kvl, Lk, Lq, dst, voff, C::RPP * D * 2);
        else
            load_tile<D, C::NV>(Kc, Kq, j0, kvl, Lk, Lq, dst, voff, C::RPP * D * 2);
    };
    auto load_v = [&](int j0, u32x4 (&dst)[4]) {
        if (gtid < C::VUNITS) {
            if (PAGED)
                load_tile_paged<D, 4>(a, Vc, ktab, a.pg_P, Vq, j0, kvl, Lk, Lq, dst, voffv, D * 2);
            else
                load_tile<D, 4>(Vc, Vq, j0, kvl, Lk, Lq, dst, voffv, D * 2);
        }
    };
    // In the tile loop each group loads tiles of consecutive positions (group 0
    // V(it + 1), group 1 K(it + 3)); read in place, it follows them with a
    // cursor instead of dividing every tile's first key by the piece length.
    const int P = PAGED ? a.pg_P : 0;
    auto piece_off = [&](int y, int r) { return (uint32_t)(kept_piece(ktab, y) * P + r) * (uint32_t)D; };
    auto cursor_at = [&](int j) {
        const int j0 = tile0(j);
        const int y = j0 < kvl ? div_piece(a, j0) : 0;
        return PageCursor{j0, y, j0 - y * P, j0 < kvl ? piece_off(y, j0 - y * P) : 0u};
    };
    // next tile of the rotated order: inside a piece the offset moves on by a
    // tile; the page table is read again only where a piece ends
    auto advance = [&](PageCursor &cu) {
        cu.j0 += BN;
        if (cu.j0 >= T * BN) {          // the rotated order wraps to the first tile
            cu = PageCursor{0, 0, 0, kvl > 0 ? piece_off(0, 0) : 0u};
        } else {
            cu.r += BN;
            cu.off += BN * D;
            if (cu.r >= P) {
                cu.r -= P;
                ++cu.y;
                if (cu.j0 < kvl) cu.off = piece_off(cu.y, cu.r);
            }
        }
    };
    auto store_k = [&](uint16_t *tile, const u32x4 (&src)[4]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) *(u32x4 *)(tile + wofs + i * C::RPP * C::RSE) = src[i];
    };
    // V^T tile: row d holds the tile's 64 keys; within each 16-key group the key
    // quads are stored in the order 0, 2, 1, 3 so that the 8 keys a lane feeds to
    // the value product (16t + 4hl + 0..3 and 16t + 8 + 4hl + 0..3) are contiguous.
    auto store_vt = [&](uint16_t *vt, const u32x4 (&src)[4]) {
        if (gtid < C::VUNITS) {
            const int qi = vq & 3;
            const int col = 16 * (vq >> 2) + 4 * (((qi & 1) << 1) | (qi >> 1));
            uint16_t *dst = vt + (8 * vc) * C::TRSE + col;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // dims 8vc+2e (low halves) and 8vc+2e+1 (high halves) of the 4 keys
                const uint2 lo = make_uint2((src[0][e] & 0xffffu) | (src[1][e] << 16),
                                            (src[2][e] & 0xffffu) | (src[3][e] << 16));
                const uint2 hi = make_uint2((src[0][e] >> 16) | (src[1][e] & 0xffff0000u),
                                            (src[2][e] >> 16) | (src[3][e] & 0xffff0000u));
                *(uint2 *)(dst + (2 * e) * C::TRSE) = lo;
                *(uint2 *)(dst + (2 * e + 1) * C::TRSE) = hi;
            }
        }
    };

    // LDS read bases of the MFMA operands.
    // K (A of S^T): lane reads row 32*kb + l32, dims 16*kk + 8*hl.
    const int kbase = l32 * C::RSE + hl * 8;
    // V^T (A of O^T): lane reads row 32*mb + l32, keys 16t + 8hl .. +8 of the
    // permuted V^T tile.
    const int vbase = l32 * C::TRSE + 8 * hl;

    f32x16_t o[C::MB];
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) o[mb] = f32x16_t{};
    f32x16_t s[2];
    bf16x8_t pb[4];
    float m_run = -__builtin_inff();  // running max of scale*log2(e)*s (may lag by <= 8)
    float l_run = 0.f;                // this lane's share of the running sum
    const float c2 = a.scale_log2;

    // The row sum adds the bf16-rounded probabilities -- exactly the P the
    // value product consumes -- two at a time (v_dot2 against (1, 1)), in two
    // chains: half the VALU instructions of fp32 adds.  Read in place
    // (PAGED), it runs at the end of the MFMA phase that consumes P, where the
    // wave's VALU is otherwise idle (pinned: the P registers are redefined
    // after the barrier): 3% faster for that instantiation, while the one over
    // a compact copy measured 2.5% slower that way and keeps it in the
    // softmax.
    auto row_sum = [&](bool pin_p) {
        if (pin_p) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                i16x4_t *w = (i16x4_t *)&pb[t];
                __asm__ volatile("" : "+v"(w[0]), "+v"(w[1]));
            }
        }
        float l2 = 0.f;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bf16x2_t pr = {pb[t][2 * j], pb[t][2 * j + 1]};
                if (t & 1) l2 = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, l2, false);
                else l_run = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, l_run, false);
            }
        l_run += l2;
    };

    auto softmax = [&](int j0) {
        if (j0 + BN > Lk) {
            // keys past Lk score -inf.  The in-place kernel does it with a sign
            // mask per entry: compares would hold 32 lane masks (SGPR pairs) at
            // once and push its SGPRs into spills (55 -> 2 spilled, its 480P
            // launch 1.1% faster); for the other kernel the compares measured
            // 1.3% faster.
            if constexpr (PAGED) {
                const int room = Lk - 1 - (j0 + 4 * hl);
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const uint32_t past = (uint32_t)((room - (kb * 32 + 8 * (i >> 2) + (i & 3))) >> 31);
                        s[kb][i] = __uint_as_float((past & 0xff800000u) | (~past & __float_as_uint(s[kb][i])));
                    }
            } else {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int key = j0 + kb * 32 + 8 * (i >> 2) + 4 * hl + (i & 3);
                        if (key >= Lk) s[kb][i] = -__builtin_inff();
                    }
            }
        }
        float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
        for (int i = 2; i < 16; ++i) mx = fmaxf(mx, s[0][i]);
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[1][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * c2;
        if (__ballot(mx > m_run + kRescaleSlack)) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb) o[mb] *= alpha;
        }
        // P^T as the B operand: k-step t covers keys 16t + {4hl..4hl+3, 8+4hl..8+4hl+3},
        // i.e. accumulator entries s[t/2][8*(t%2) + j].
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                pb[t][j] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[t >> 1][8 * (t & 1) + j], c2, -m_run));
        if constexpr (!PAGED) row_sum(false);
    };

    // Prologue: group 0 copies K(0) and K(1) into LDS, group 1 copies V(0);
    // then group 1 fetches K(2) and group 0 fetches V(1) into registers, and
    // group 0 computes S(0).
    u32x4 stage[4];
    if (grp == 0) {
        load_k(tile0(0), stage);
        store_k(Ks[0], stage);
        if (n > 1) {
            load_k(tile0(1), stage);
            store_k(Ks[1], stage);
        }
        if (n > 1) load_v(tile0(1), stage);
    } else {
        load_v(tile0(0), stage);
        store_vt(Vs[0], stage);
        if (n > 2) load_k(tile0(2), stage);
    }
    __syncthreads();
    if (grp == 0) mfma_block<D, false, true>(nullptr, Ks[0], vbase, kbase, pb, qf, o, s);

    // Both groups run the same loop body -- softmax of tile j, barrier, MFMA
    // block (P(j)V(j), then S(j+1) = K(j+1)Q^T), barrier -- with group 1 one
    // phase behind group 0, so on every SIMD one wave's softmax overlaps the
    // other wave's MFMA block.  In global phase terms:
    //   phase 2j:   group 0 softmax(j)     | group 1 MFMA block of tile j-1
    //   phase 2j+1: group 0 MFMA block j   | group 1 softmax(j)
    // K(j) is read in phases 2j-1 and 2j from Ks[j%2]; V(j) in phases 2j+1 and
    // 2j+2 from Vs[j%2].  Group 0 stores V(j) during its softmax(j) and fetches
    // V(j+1); group 1 stores K(j+2) during its softmax(j) and fetches K(j+3).
    // Every store lands in a buffer whose previous tile was last read before the
    // preceding barrier and is first read after the next one.  The MFMA block of
    // the last tile also runs the score product on a stale K buffer; its result
    // is never used.  Both groups meet 2*n + 1 barriers, the last one after
    // every LDS read of the segment.
    if (grp == 1) {
        mfma_block<D, false, true>(nullptr, Ks[0], vbase, kbase, pb, qf, o, s);
        __syncthreads();
    }
    // Let every outstanding load (the Q fragments included) land once here, so
    // the loop's score products carry no wait on the staging loads in flight.
    __builtin_amdgcn_s_waitcnt(0);
    // paged: group 0's next V tile is position 2, group 1's next K tile
    // position 3; both cursors are kept (uniform, scalar) and advanced together
    PageCursor cur_v = PAGED && n > 2 ? cursor_at(2) : PageCursor{0, 0, 0, 0u};
    PageCursor cur_k = PAGED && n > 3 ? cursor_at(3) : PageCursor{0, 0, 0, 0u};
    for (int it = 0; it < n; ++it) {
        const int j0 = tile0(it);
        softmax(j0);
        if (grp == 0) {
            if (it >= 1) store_vt(Vs[it & 1], stage);
            if (it >= 1 && it + 1 < n) {
                if constexpr (PAGED) {
                    if (gtid < C::VUNITS)
                        load_tile_cursor<D, 4>(Vc, ktab, P, cur_v, Vq, kvl, Lk, Lq, stage, voffv, D * 2);
                } else {
                    load_v(tile0(it + 1), stage);
                }
            }
        } else {
            if (it + 2 < n) store_k(Ks[it & 1], stage);
            if (it + 3 < n) {
                if constexpr (PAGED) {
                    load_tile_cursor<D, C::NV>(Kc, ktab, P, cur_k, Kq, kvl, Lk, Lq, stage, voff, C::RPP * D * 2);
                } else {
                    load_k(tile0(it + 3), stage);
                }
            }
        }
        if constexpr (PAGED) {
            if (it >= 1) advance(cur_v);
            advance(cur_k);
        }
        __syncthreads();
        // (no wave-priority raise around the block: measured 1% slower with it)
        mfma_block<D, true, true>(Vs[it & 1], Ks[(it + 1) & 1], vbase, kbase, pb, qf, o, s);
        if constexpr (PAGED) row_sum(true);
        __syncthreads();
    }
    if (grp == 0) __syncthreads();

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (slot) {
        // device-scope stores: the workgroup that merges the item may run on
        // another XCD, within this launch
        unsigned long long *op = (unsigned long long *)slot;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint2 v = pack_bf16x4(o[mb][4 * g] * inv, o[mb][4 * g + 1] * inv, o[mb][4 * g + 2] * inv,
                                            o[mb][4 * g + 3] * inv);
                put_shared(op + ((wave * C::MB + mb) * 4 + g) * 64 + lane, v);
            }
        if (hl == 0) {
            put_shared(slot + BM * D / 2 + wave * 32 + l32, m_run);
            put_shared(slot + BM * D / 2 + BM + wave * 32 + l32, l_tot);
        }
        return;
    }
    if (qok) {
        uint16_t *Oh = (uint16_t *)a.O + ((size_t)h * Lq + qrow) * D;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int g = 0; g < 4; ++g)  // O^T rows d = 32mb + 8g + 4hl + {0..3}
                *(uint2 *)(Oh + mb * 32 + 8 * g + 4 * hl) =
                    pack_bf16x4(o[mb][4 * g] * inv, o[mb][4 * g + 1] * inv, o[mb][4 * g + 2] * inv,
                                o[mb][4 * g + 3] * inv);
        if (a.lse && hl == 0)
            a.lse[(size_t)h * Lq + qrow] = fmaf(m_run, 0.69314718055994530942f, logf(l_tot));
    }
}

// BAL = false: one workgroup per work item (head, query tile), dealt so that
// each XCD (blocks go to the 8 XCDs round-robin) receives a contiguous range
// of items: the query tiles of a head then share that XCD's L2.
// BAL = true: the balanced schedule above, with the same XCD-contiguous
// assignment of ranges (n_blocks is a multiple of 8).
template <int D, bool BAL, bool PAGED>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(AttnArgs a) {
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][C::TILE];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[2][C::VTILE];
    __shared__ uint32_t flag;

    if (!BAL) {
        const int item = (blockIdx.x & 7) * a.items_per_xcd + (blockIdx.x >> 3);
        if (item >= a.n_items) return;
        const int li = item / a.n_qtiles;
        attn_segment<D, PAGED>(a, Ks, Vs, li, item - li * a.n_qtiles, 0, entry_tiles<PAGED>(a, li), 0, nullptr);
        return;
    }
    const WorkList wl = work_list<PAGED>(a);
    const Schedule sc = make_schedule(a, wl);
    const int r = (blockIdx.x & 7) * (a.n_blocks >> 3) + (blockIdx.x >> 3);
    if (r >= sc.G) return;
    const int64_t end = sc.start(r + 1);
    int64_t cur = sc.start(r);
    bool first = true;
    while (cur < end) {
        // locate the item holding tile `cur`
        const ItemPos ip = locate(wl, cur);
        const int qt = ip.qt, T = ip.T;
        const int64_t ibase = ip.ibase;
        const int t0 = (int)(cur - ibase);
        const int t1 = (int)((end < ibase + T ? end : ibase + T) - ibase);
        float *slot = (t0 == 0 && t1 == T)
                          ? nullptr
                          : a.part + (size_t)(2 * r + (first ? 0 : 1)) * slot_floats<D>();
        // Rotate the item's key tiles so that its first part, started at time
        // tau0 = ibase - start(owner(ibase)) of its workgroup, reads key tile
        // tau mod T at time tau: the first parts of all items of a head then
        // sweep its K/V in step (later parts in step among themselves, shifted
        // by a range length), so the XCD's L2 serves the re-reads.
        const int rot = (int)((ibase - sc.start(sc.owner(ibase))) % T);
        attn_segment<D, PAGED>(a, Ks, Vs, ip.li, qt, t0, t1, rot, slot);
        if (slot) {
            // the last of the item's parts to arrive combines them (no wait:
            // every other part is complete when its workgroup arrives)
            const int n_parts = sc.owner(ibase + T - 1) - sc.owner(ibase) + 1;
            uint32_t *cnt = a.item_counters + (size_t)(ip.li * a.n_qtiles + qt) * kItemCounterStride;
            if (arrive_last(cnt, (uint32_t)n_parts, &flag))
                merge_rows<D, 64>(a, sc, ip.li, qt, ibase, T, threadIdx.x >> 6, threadIdx.x & 63);
        }
        cur = ibase + t1;
        first = false;
    }
}

// ------------------------------------------------------------ attention mass
// Offline head profiling (Sec. 4.1, Eq. 1) needs, per head, the attention mass
// each block of F keys of [Kc[0:kv_len]; K_cur] receives: the sum over all
// query rows of the softmax probabilities exp(scale*q.k - lse_row), with lse
// from fkv_chunk_attention over the same keys.  Workgroup = (256-row query
// tile, head), 8 waves x 32 rows.  Per 64-key tile the waves compute S^T with
// the attention kernel's score product (same MFMA sequence, so the same fp32
// scores), form the probabilities, and for every key block the tile touches
// reduce their sum across the wave with a fixed butterfly; lane 0 adds it to
// the wave's own bin array in the workspace, so the result is deterministic.
__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

template <int D>
__global__ __launch_bounds__(kThreads) void attn_mass_kernel(AttnArgs a) {
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[C::TILE];
    const int qt = blockIdx.x, h = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hl = lane >> 5;
    const int Lq = a.Lq;
    float *bins = a.part + (((size_t)h * a.n_qtiles + qt) * 8 + wave) * a.mass_bins;
    for (int b = lane; b < a.mass_bins; b += 64) bins[b] = 0.f;

    const int qrow = qt * BM + wave * 32 + l32;
    const bool qok = qrow < Lq;
    const uint16_t *Qh = (const uint16_t *)a.Q + (size_t)h * Lq * D;
    bf16x8_t qf[C::KS];
#pragma unroll
    for (int kk = 0; kk < C::KS; ++kk) {
        const u32x4 v = qok ? *(const u32x4 *)(Qh + (size_t)qrow * D + kk * 16 + hl * 8) : u32x4{0, 0, 0, 0};
        qf[kk] = __builtin_bit_cast(bf16x8_t, v);
    }
    // rows past Lq contribute nothing: their bias is -inf
    const float bias = qok ? -a.lse[(size_t)h * Lq + qrow] * 1.4426950408889634f : -__builtin_inff();
    const float c2 = a.scale_log2;

    const int kvl = head_kvl(a, h);
    const int Lk = kvl + Lq;
    const uint16_t *Kc = (const uint16_t *)a.Kc + (size_t)h * a.slab * D;
    const uint16_t *Kq = (const uint16_t *)a.K_cur + (size_t)h * Lq * D;
    // staging geometry: all 512 threads, rows r0 + RPP2*i
    constexpr int RPP2 = kThreads / C::CPR;
    constexpr int NV2 = BN / RPP2;
    const int c = tid % C::CPR, r0 = tid / C::CPR;
    const uint32_t voff = (uint32_t)(r0 * D + c * 8) * 2u;
    const int wofs = r0 * C::RSE + c * 8;
    const int kbase = l32 * C::RSE + hl * 8;
    const int vbase = 0;

    f32x16_t o[C::MB];
    f32x16_t s[2];
    bf16x8_t pb[4];
    const int T = (Lk + BN - 1) / BN;
    for (int t = 0; t < T; ++t) {
        const int j0 = t * BN;
        u32x4 stage[4];
        load_tile<D, NV2>(Kc, Kq, j0, kvl, Lk, Lq, stage, voff, RPP2 * D * 2);
        __syncthreads();  // the previous tile's reads are done
#pragma unroll
        for (int i = 0; i < NV2; ++i) *(u32x4 *)(Ks + wofs + i * RPP2 * C::RSE) = stage[i];
        __syncthreads();
        mfma_block<D, false, true>(nullptr, Ks, vbase, kbase, pb, qf, o, s);
        // keys of this lane: j0 + 32kb + 8(i/4) + 4hl + i%4
        const int b_first = j0 / a.mass_F, b_last = (min(j0 + BN, Lk) - 1) / a.mass_F;
        for (int b = b_first; b <= b_last; ++b) {
            const int lo = b * a.mass_F, hi = min(lo + a.mass_F, Lk);
            float v = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = j0 + kb * 32 + 8 * (i >> 2) + 4 * hl + (i & 3);
                    if (key >= lo && key < hi) v += __builtin_amdgcn_exp2f(fmaf(s[kb][i], c2, bias));
                }
            v = wave_sum_f(v);
            if (lane == 0) bins[b] += v;
        }
    }
}

template <int D>
__global__ __launch_bounds__(256) void attn_mass_finalize_kernel(AttnArgs a) {
    const int h = blockIdx.x;
    for (int b = threadIdx.x; b < a.mass_bins; b += 256) {
        float v = 0.f;
        for (int k = 0; k < a.n_qtiles * 8; ++k) v += a.part[((size_t)h * a.n_qtiles * 8 + k) * a.mass_bins + b];
        float *out = a.mass_out + (size_t)h * a.mass_bins + b;
        *out = a.mass_acc ? *out + v : v;
    }
}

}  // namespace

template <bool PAGED>
hipError_t launch_bf16(const AttnArgs &a, int head_dim, hipStream_t s) {
    if (a.n_blocks > 0) {
        if (head_dim == 128)
            hipLaunchKernelGGL((attn_bf16_kernel<128, true, PAGED>), dim3(a.n_blocks), dim3(kThreads), 0, s, a);
        else
            hipLaunchKernelGGL((attn_bf16_kernel<64, true, PAGED>), dim3(a.n_blocks), dim3(kThreads), 0, s, a);
        return hipGetLastError();
    }
    const unsigned blocks = (unsigned)a.items_per_xcd * 8u;
    if (head_dim == 128)
        hipLaunchKernelGGL((attn_bf16_kernel<128, false, PAGED>), dim3(blocks), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL((attn_bf16_kernel<64, false, PAGED>), dim3(blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_attention_bf16(const AttnArgs &a, int head_dim, hipStream_t s) {
    return a.paged ? launch_bf16<true>(a, head_dim, s) : launch_bf16<false>(a, head_dim, s);
}

hipError_t launch_attention_mass(const AttnArgs &a, int head_dim, hipStream_t s) {
    const dim3 grid((unsigned)a.n_qtiles, (unsigned)a.n_heads);
    if (head_dim == 128) {
        hipLaunchKernelGGL(attn_mass_kernel<128>, grid, dim3(kThreads), 0, s, a);
        hipLaunchKernelGGL(attn_mass_finalize_kernel<128>, dim3(a.n_heads), dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL(attn_mass_kernel<64>, grid, dim3(kThreads), 0, s, a);
        hipLaunchKernelGGL(attn_mass_finalize_kernel<64>, dim3(a.n_heads), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

size_t attention_part_bytes(int head_dim) { return (size_t)kAttnRowsBf16 * (head_dim / 2 + 2) * 4; }

}  // namespace fkv
