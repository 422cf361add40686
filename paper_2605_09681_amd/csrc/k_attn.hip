// k_attn.hip -- chunk attention over each head's compressed cache (Eq. 2 for
// static heads, Eq. 4 for dynamic heads), bf16 inputs, gfx950 MFMA.
//
// For head h the key sequence is [Kc[h][0:kv_len[h]]; K_cur[h]] (the retained
// history, then the current chunk) and likewise for values; every query row of
// the chunk attends to all of it with no mask.  The per-head key count is
// ragged (it comes from the device-side kv_len), and a key tile may straddle
// the history/chunk boundary: rows are fetched from whichever source holds them.
//
// Workgroup = 4 waves = 128 query rows of one head (32 per wave).  Keys are
// processed in tiles of 64, staged through LDS with double buffering (the next
// tile's global loads are in flight while the current tile is computed).  Per
// wave and tile, with v_mfma_f32_32x32x16_bf16:
//   S^T = K . Q^T   (A = K rows from LDS, B = the wave's Q rows held in VGPRs
//                    for the whole kernel), 2 x (d/16) MFMAs;
//   online softmax in fp32 (exp2 with the scale folded into log2 units);
//   O^T += V^T . P^T (A = V^T from a transposed LDS copy, B = P taken straight
//                    from the S^T accumulators, rounded to bf16), 4 x (d/32).
// Computing S transposed makes each lane own one query column, so P needs no
// data movement between the two products: in the 32x32 accumulator layout a
// lane holds 16 keys of its query, which are exactly the 8-element k-slices the
// B operand of the value product wants (any consistent permutation of the
// contraction index is allowed, and V^T is read with the same permutation).
// Row maxima need one cross-lane exchange (lanes l and l^32 share a query).
//
// LDS layouts are XOR-swizzled so both the 16-byte K reads and the 8-byte V^T
// reads of the MFMA operand pattern, and the tile stores, are free of bank
// conflicts beyond the minimum.
//
// Work items (head, 128-row query tile) are assigned so that each XCD (blocks
// are dealt to the 8 XCDs round-robin) receives a contiguous range: the query
// tiles of a head then share that XCD's L2 while they sweep the same K/V.
#include "fkv_internal.h"

namespace fkv {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int BM = kAttnRowsBf16;  // query rows per workgroup
constexpr int BN = 64;   // keys per tile

template <int D>
struct Cfg {
    static constexpr int CPR = D / 8;               // 16-byte chunks per K/V row
    static constexpr int KVEC = BN * CPR / kThreads; // K vectors per thread per tile
    static constexpr int VUNITS = (BN / 4) * CPR;    // (4 keys x 8 dims) V units per tile
    static constexpr int KS = D / 16;                // k-steps of S^T = K Q^T
    static constexpr int MB = D / 32;                // 32-row blocks of O^T
    static_assert(KVEC >= 1 && VUNITS <= kThreads, "tile shape");
};

__device__ __forceinline__ uint4 ld16(const uint16_t *p) { return *(const uint4 *)p; }

// K tile: key row r, 16-byte chunk c stored at chunk c ^ (r % CPR).
template <int D>
__device__ __forceinline__ int k_off(int r, int c) {
    return r * D + ((c ^ (r % Cfg<D>::CPR)) << 3);
}

// V^T tile: dim row d (BN keys = 16 chunks of 4 keys), chunk q stored at q ^ f(d).
__device__ __forceinline__ int vt_off(int d, int q) {
    const int f = ((d & 7) << 1) ^ ((d >> 3) & 15);
    return d * BN + ((q ^ f) << 2);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(AttnArgs a) {
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][BN * D];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[2][D * BN];

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
        const uint4 v = qok ? ld16(Qh + (size_t)qrow * D + kk * 16 + hl * 8) : make_uint4(0, 0, 0, 0);
        qf[kk] = __builtin_bit_cast(bf16x8_t, v);
    }

    int kvl = a.kv_len[h];
    kvl = kvl < 0 ? 0 : (kvl > a.slab ? (int)a.slab : kvl);
    const int Lk = kvl + Lq;
    const uint16_t *Kc = (const uint16_t *)a.Kc + (size_t)h * a.slab * D;
    const uint16_t *Vc = (const uint16_t *)a.Vc + (size_t)h * a.slab * D;
    const uint16_t *Kq = (const uint16_t *)a.K_cur + (size_t)h * Lq * D;
    const uint16_t *Vq = (const uint16_t *)a.V_cur + (size_t)h * Lq * D;

    uint4 kreg[C::KVEC];
    uint4 vreg[4];
    const uint4 zero = make_uint4(0, 0, 0, 0);

    // Row j of the concatenated key (value) sequence: history row j < kvl, else
    // chunk row j - kvl.  Rows past the end read chunk row 0 and are zeroed.
    auto row_ptr = [&](const uint16_t *hist, const uint16_t *chunk, int j) -> const uint16_t * {
        const uint16_t *p = j < kvl ? hist + (size_t)j * D : chunk + (size_t)(j - kvl) * D;
        return j < Lk ? p : chunk;
    };
    auto load_tile = [&](int j0) {
#pragma unroll
        for (int i = 0; i < C::KVEC; ++i) {
            const int vi = tid + i * kThreads;
            const int r = vi / C::CPR, c = vi % C::CPR;
            const int j = j0 + r;
            const uint4 v = ld16(row_ptr(Kc, Kq, j) + c * 8);
            kreg[i] = j < Lk ? v : zero;
        }
        if (tid < C::VUNITS) {
            const int kq = tid / C::CPR, c = tid % C::CPR;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int j = j0 + 4 * kq + r;
                const uint4 v = ld16(row_ptr(Vc, Vq, j) + c * 8);
                vreg[r] = j < Lk ? v : zero;
            }
        }
    };

    auto store_tile = [&](int buf) {
        uint16_t *ks = Ks[buf];
#pragma unroll
        for (int i = 0; i < C::KVEC; ++i) {
            const int vi = tid + i * kThreads;
            const int r = vi / C::CPR, c = vi % C::CPR;
            *(uint4 *)(ks + k_off<D>(r, c)) = kreg[i];
        }
        if (tid < C::VUNITS) {
            const int kq = tid / C::CPR, c = tid % C::CPR;
            uint16_t *vt = Vt[buf];
            const uint32_t w0[4] = {vreg[0].x, vreg[0].y, vreg[0].z, vreg[0].w};
            const uint32_t w1[4] = {vreg[1].x, vreg[1].y, vreg[1].z, vreg[1].w};
            const uint32_t w2[4] = {vreg[2].x, vreg[2].y, vreg[2].z, vreg[2].w};
            const uint32_t w3[4] = {vreg[3].x, vreg[3].y, vreg[3].z, vreg[3].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // dims 8c+2e (low halves) and 8c+2e+1 (high halves) of keys 4kq..4kq+3
                const uint2 lo = make_uint2((w0[e] & 0xffffu) | (w1[e] << 16),
                                            (w2[e] & 0xffffu) | (w3[e] << 16));
                const uint2 hi = make_uint2((w0[e] >> 16) | (w1[e] & 0xffff0000u),
                                            (w2[e] >> 16) | (w3[e] & 0xffff0000u));
                const int d0 = 8 * c + 2 * e;
                *(uint2 *)(vt + vt_off(d0, kq)) = lo;
                *(uint2 *)(vt + vt_off(d0 + 1, kq)) = hi;
            }
        }
    };

    f32x16_t o[C::MB];
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) o[mb] = f32x16_t{};
    float m_run = -__builtin_inff();  // running max of scale*log2(e)*s
    float l_run = 0.f;                // this lane's share of the running sum
    const float c2 = a.scale_log2;
    const int ntiles = (Lk + BN - 1) / BN;

    load_tile(0);
    store_tile(0);
    __syncthreads();

    for (int it = 0; it < ntiles; ++it) {
        const int buf = it & 1;
        const int j0 = it * BN;

        // S^T[key][query] for keys j0 + 32*kb + (8*(i/4) + 4*hl + i%4), query l32.
        const uint16_t *ks = Ks[buf];
        f32x16_t s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = f32x16_t{};
            const int r = kb * 32 + l32;
#pragma unroll
            for (int kk = 0; kk < C::KS; ++kk) {
                const uint4 kv = *(const uint4 *)(ks + k_off<D>(r, 2 * kk + hl));
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kv),
                                                               qf[kk], s[kb], 0, 0, 0);
            }
        }
        if (j0 + BN > Lk) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = j0 + kb * 32 + 8 * (i >> 2) + 4 * hl + (i & 3);
                    if (key >= Lk) s[kb][i] = -__builtin_inff();
                }
        }

        // Next tile's global loads are issued here, after the QK^T phase, so
        // their staging registers are not live at the same time as the K
        // operand fragments; they land in LDS after the value product.
        if (it + 1 < ntiles) load_tile(j0 + BN);

        float mx = s[0][0];
#pragma unroll
        for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s[0][i]);
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[1][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx * c2);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb) o[mb] *= alpha;

        // P^T as the B operand: k-step t covers keys 16t + {4hl..4hl+3, 8+4hl..8+4hl+3},
        // i.e. accumulator entries s[t/2][8*(t%2) + j].
        bf16x8_t pb[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float p = __builtin_amdgcn_exp2f(fmaf(s[t >> 1][8 * (t & 1) + j], c2, -m_new));
                l_run += p;
                pb[t][j] = (__bf16)p;
            }

        const uint16_t *vt = Vt[buf];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb) {
                const int d = mb * 32 + l32;
                const uint2 v1 = *(const uint2 *)(vt + vt_off(d, 4 * t + hl));
                const uint2 v2 = *(const uint2 *)(vt + vt_off(d, 4 * t + 2 + hl));
                const uint4 av = make_uint4(v1.x, v1.y, v2.x, v2.y);
                o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                               pb[t], o[mb], 0, 0, 0);
            }

        if (it + 1 < ntiles) store_tile(buf ^ 1);
        __syncthreads();
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
                __bf16 b0 = (__bf16)(o[mb][4 * g + 0] * inv);
                __bf16 b1 = (__bf16)(o[mb][4 * g + 1] * inv);
                __bf16 b2 = (__bf16)(o[mb][4 * g + 2] * inv);
                __bf16 b3 = (__bf16)(o[mb][4 * g + 3] * inv);
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
