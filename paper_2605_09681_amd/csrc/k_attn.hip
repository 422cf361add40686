// k_attn.hip -- chunk attention over each head's compressed cache (Eq. 2 for
// static heads, Eq. 4 for dynamic heads), bf16 inputs, gfx950 MFMA.
//
// For head h the key sequence is [Kc[h][0:kv_len[h]]; K_cur[h]] (the retained
// history, then the current chunk) and likewise for values; every query row of
// the chunk attends to all of it with no mask.  The per-head key count is
// ragged (it comes from the device-side kv_len), and one key tile may straddle
// the history/chunk boundary.
//
// Workgroup = 4 waves = 128 query rows of one head (32 per wave); two
// workgroups share a CU.  Keys are processed in tiles of 64.  Per wave and
// tile, with v_mfma_f32_32x32x16_bf16:
//   S^T = K . Q^T   (A = K rows from LDS, B = the wave's Q rows, held in VGPRs
//                    for the whole kernel), 2 x (d/16) MFMAs;
//   online softmax in fp32 (exp2 with the scale folded into log2 units);
//   O^T += V^T . P^T (A = V^T read from the row-major V tile with the gfx950
//                    LDS transpose read, B = P taken straight from the S^T
//                    accumulators, rounded to bf16), 4 x (d/32) MFMAs.
// Computing S transposed makes each lane own one query column, so P needs no
// data movement between the two products: in the 32x32 accumulator layout a
// lane holds 16 keys of its query, which are exactly the 8-element k-slices the
// B operand of the value product takes (any consistent permutation of the
// contraction index is allowed; V^T is read with the same permutation).  Row
// maxima need one cross-lane exchange (lanes l and l^32 share a query).
//
// Pipeline (one barrier per tile): iteration j runs the softmax of tile j on
// the VALU, stores K of tile j+1 and V of tile j (fetched one iteration
// earlier) into LDS, meets the barrier, issues the global loads of K(j+2) and
// V(j+1), then runs one contiguous MFMA block at raised wave priority: the
// value product of tile j followed by the score product of tile j+1.  The two
// workgroups on a CU are not synchronised with each other, so one's softmax
// overlaps the other's MFMA block.  K and V are double-buffered separately.
//
// The running max is only moved when a tile's max exceeds it by more than 8
// (log2 units): probabilities then stay below 2^8 and the accumulator rescale
// is skipped for most tiles; the final normalisation is exact either way.
//
// Global K/V rows come in through buffer loads whose per-lane offsets are loop
// invariant; rows past the end of a source fall outside the buffer's range and
// read as zero (the straddling tile merges both sources that way).  LDS rows
// are padded (K by 16 bytes, V by 64 bytes, measured best for the 16-byte K
// operand reads and the transpose reads of V) so the operand reads spread over
// the banks and every LDS access uses an immediate offset.
//
// Work items (head, 128-row query tile) are dealt so that each XCD (blocks go
// to the 8 XCDs round-robin) receives a contiguous range: the query tiles of a
// head then share that XCD's L2 while they sweep the same K/V.
#include "fkv_internal.h"

namespace fkv {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int BM = kAttnRowsBf16;  // query rows per workgroup
constexpr int BN = 64;             // keys per tile
constexpr float kRescaleSlack = 8.f;  // log2 units the running max may lag behind
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw 32-bit buffer, range checked

template <int D>
struct Cfg {
    static constexpr int RSE = D + 8;           // K row stride in LDS (16-byte pad), elements
    static constexpr int VRSE = D + 32;         // V row stride in LDS (64-byte pad), elements
    static constexpr int CPR = D / 8;           // 16-byte chunks per row
    static constexpr int RPP = kThreads / CPR;  // rows covered by one pass of the workgroup
    static constexpr int NV = BN / RPP;         // 16-byte vectors per thread per tile and tensor
    static constexpr int KS = D / 16;           // k-steps of S^T = K Q^T
    static constexpr int MB = D / 32;           // 32-row blocks of O^T
    static constexpr int TILE = BN * RSE;       // elements per K tile
    static constexpr int VTILE = BN * VRSE;     // elements per V tile
    static_assert(NV >= 1 && BN % RPP == 0, "tile shape");
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(AttnArgs a) {
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][C::TILE];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[2][C::VTILE];

    const int item = (blockIdx.x & 7) * a.items_per_xcd + (blockIdx.x >> 3);
    if (item >= a.n_items) return;
    const int h = item / a.n_qtiles;
    const int qt = item - h * a.n_qtiles;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hl = lane >> 5;
    const int Lq = a.Lq;

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

    int kvl = a.kv_len[h];
    kvl = kvl < 0 ? 0 : (kvl > a.slab ? (int)a.slab : kvl);
    const int Lk = kvl + Lq;
    const int ntiles = (Lk + BN - 1) / BN;
    const uint16_t *Kc = (const uint16_t *)a.Kc + (size_t)h * a.slab * D;
    const uint16_t *Vc = (const uint16_t *)a.Vc + (size_t)h * a.slab * D;
    const uint16_t *Kq = (const uint16_t *)a.K_cur + (size_t)h * Lq * D;
    const uint16_t *Vq = (const uint16_t *)a.V_cur + (size_t)h * Lq * D;

    // Loop-invariant per-thread load geometry: rows r0 + RPP*i, chunk c.
    const int c = tid % C::CPR, r0 = tid / C::CPR;
    const uint32_t voff = (uint32_t)(r0 * D + c * 8) * 2u;   // + i*RPP*D*2 bytes
    const int wofs = r0 * C::RSE + c * 8;                      // + i*RPP*RSE elements
    const int vwofs = r0 * C::VRSE + c * 8;                    // + i*RPP*VRSE elements

    // Rows j0 .. j0+BN-1 of [hist; chunk] into registers, zeros past Lk.
    auto load_rows = [&](const uint16_t *hist, const uint16_t *chunk, int j0, u32x4 (&dst)[C::NV]) {
        if (j0 + BN <= kvl) {
            const auto r = rsrc(hist + (size_t)j0 * D, BN * D * 2);
#pragma unroll
            for (int i = 0; i < C::NV; ++i) dst[i] = bload(r, voff + i * C::RPP * D * 2);
        } else if (j0 >= kvl) {
            const auto r = rsrc(chunk + (size_t)(j0 - kvl) * D, (uint32_t)(Lk - j0) * D * 2);
#pragma unroll
            for (int i = 0; i < C::NV; ++i) dst[i] = bload(r, voff + i * C::RPP * D * 2);
        } else {  // straddles the history/chunk boundary
            const int nh = kvl - j0;
            const int nc = min(BN - nh, Lq);
            const auto rh = rsrc(hist + (size_t)j0 * D, (uint32_t)nh * D * 2);
            const auto rc = rsrc(chunk, (uint32_t)nc * D * 2);
            const uint32_t shift = (uint32_t)nh * D * 2;  // chunk rows start at tile row nh
#pragma unroll
            for (int i = 0; i < C::NV; ++i) {
                const uint32_t o = voff + i * C::RPP * D * 2;
                // below tile row nh, o - shift wraps to a huge offset: out of range, reads 0
                dst[i] = bload(rh, o) | bload(rc, o - shift);
            }
        }
    };
    auto store_rows = [&](uint16_t *tile, const u32x4 (&src)[C::NV]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) *(u32x4 *)(tile + wofs + i * C::RPP * C::RSE) = src[i];
    };
    auto store_vrows = [&](uint16_t *tile, const u32x4 (&src)[C::NV]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) *(u32x4 *)(tile + vwofs + i * C::RPP * C::VRSE) = src[i];
    };

    // LDS read bases of the MFMA operands.
    // K (A of S^T): lane reads row 32*kb + l32, dims 16*kk + 8*hl.
    const int kbase = l32 * C::RSE + hl * 8;
    // V^T (A of O^T) via the transpose read: within each 16-lane group, lane k
    // points at V[4*hl + k/4 (+16t +8half)][16*(group&1) + 4*(k%4) (+32mb)] and
    // receives V[keys 16t + 8half + 4hl + 0..3][dim 32mb + l32].
    const int g16 = lane >> 4, k16 = lane & 15;
    const int vbase = (4 * hl + (k16 >> 2)) * C::VRSE + 16 * (g16 & 1) + 4 * (k16 & 3);

    auto qk = [&](const uint16_t *ks, f32x16_t (&s)[2]) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = f32x16_t{};
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) {
                const u32x4 kv = *(const u32x4 *)(ks + kbase + kb * 32 * C::RSE + kk * 16);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kv),
                                                               qf[kk], s[kb], 0, 0, 0);
            }
        }
    };

    f32x16_t o[C::MB];
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) o[mb] = f32x16_t{};
    float m_run = -__builtin_inff();  // running max of scale*log2(e)*s (may lag by <= 8)
    float l_run = 0.f;                // this lane's share of the running sum
    const float c2 = a.scale_log2;

    u32x4 kreg[C::NV], vreg[C::NV];
    f32x16_t s[2];

    // Prologue: K(0) into LDS and S(0); V(0) and K(1) in flight.
    load_rows(Kc, Kq, 0, kreg);
    store_rows(Ks[0], kreg);
    load_rows(Vc, Vq, 0, vreg);
    if (ntiles > 1) load_rows(Kc, Kq, BN, kreg);
    __syncthreads();
    qk(Ks[0], s);

    for (int it = 0; it < ntiles; ++it) {
        const int j0 = it * BN;
        // ---- softmax of tile it (VALU) ------------------------------------
        if (j0 + BN > Lk) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = j0 + kb * 32 + 8 * (i >> 2) + 4 * hl + (i & 3);
                    if (key >= Lk) s[kb][i] = -__builtin_inff();
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
        bf16x8_t pb[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float p = __builtin_amdgcn_exp2f(fmaf(s[t >> 1][8 * (t & 1) + j], c2, -m_run));
                l_run += p;
                pb[t][j] = (__bf16)p;
            }

        // ---- LDS stores: K(it+1) and V(it) -----------------------------------
        if (it + 1 < ntiles) store_rows(Ks[(it + 1) & 1], kreg);
        store_vrows(Vs[it & 1], vreg);
        __syncthreads();
        if (it + 2 < ntiles) load_rows(Kc, Kq, j0 + 2 * BN, kreg);
        if (it + 1 < ntiles) load_rows(Vc, Vq, j0 + BN, vreg);

        // ---- MFMA block: O += P V(it); S = K(it+1) Q^T ------------------------
        __builtin_amdgcn_s_setprio(1);
        const uint16_t *vs = Vs[it & 1];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb) {
                const uint16_t *p0 = vs + vbase + (16 * t) * C::VRSE + 32 * mb;
                const i16x4_t v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) i16x4_t *)(p0));
                const i16x4_t v2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) i16x4_t *)(p0 + 8 * C::VRSE));
                const bf16x8_t av = __builtin_bit_cast(
                    bf16x8_t, __builtin_shufflevector(v1, v2, 0, 1, 2, 3, 4, 5, 6, 7));
                o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[t], o[mb], 0, 0, 0);
            }
        if (it + 1 < ntiles) qk(Ks[(it + 1) & 1], s);
        __builtin_amdgcn_s_setprio(0);
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (qok) {
        uint16_t *Oh = (uint16_t *)a.O + ((size_t)h * Lq + qrow) * D;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                // O^T rows d = 32mb + 8g + 4hl + {0..3}
                const __bf16 b0 = (__bf16)(o[mb][4 * g + 0] * inv);
                const __bf16 b1 = (__bf16)(o[mb][4 * g + 1] * inv);
                const __bf16 b2 = (__bf16)(o[mb][4 * g + 2] * inv);
                const __bf16 b3 = (__bf16)(o[mb][4 * g + 3] * inv);
                const uint2 pk = make_uint2(
                    (uint32_t)__builtin_bit_cast(uint16_t, b0) | ((uint32_t)__builtin_bit_cast(uint16_t, b1) << 16),
                    (uint32_t)__builtin_bit_cast(uint16_t, b2) | ((uint32_t)__builtin_bit_cast(uint16_t, b3) << 16));
                *(uint2 *)(Oh + mb * 32 + 8 * g + 4 * hl) = pk;
            }
        if (a.lse && hl == 0)
            a.lse[(size_t)h * Lq + qrow] = m_run * 0.69314718055994530942f + logf(l_tot);
    }
}

}  // namespace

hipError_t launch_attention_bf16(const AttnArgs &a, int head_dim, hipStream_t s) {
    const unsigned blocks = (unsigned)a.items_per_xcd * 8u;
    if (head_dim == 128)
        hipLaunchKernelGGL(attn_bf16_kernel<128>, dim3(blocks), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(attn_bf16_kernel<64>, dim3(blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
