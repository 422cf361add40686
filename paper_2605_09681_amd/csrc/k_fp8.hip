// k_fp8.hip -- FP8 (OCP E4M3) variant of the chunk attention (App. F combines
// the method with FP8 attention), for gfx950's v_mfma_f32_32x32x64_f8f6f4,
// which runs at twice the bf16 MFMA rate.
//
// Packing (three kernels, per head):
//   statistics   per-channel fp64 sum, max and min of the keys [Kc[0:kv_len];
//                K_cur], per-channel max |V| of the values, max |Q|;
//   finalize     key mean mu (fp64 sum / n, one rounding to fp32), amax of
//                K - mu (rounding is monotonic, so it comes from the channel
//                max and min), and for Q, K - mu and every value channel the
//                pair inv = 448 / amax, s = amax / 448 (correctly rounded fp32;
//                0 for an all-zero tensor);
//   pack         E4M3 codes (round to nearest even) of Q * inv_q,
//                (K - mu) * inv_k and V * inv_v[c], each one fp32 operation
//                (two for keys) before the conversion.  Keys become one
//                row-major array [history; chunk] per head; values become
//                V^T per 64-key tile with the key order the value product
//                expects (below); rows past the head's keys are zero.
// Subtracting mu shifts every logit of a query row by the same q . mu, so the
// softmax is unchanged while the keys keep their variation in 3 mantissa bits.
// The history rows come from the compressed copy [Kc[0:kv_len]], or
// (fkv_fp8_pack_paged) straight from the slot-permuted cache: each history row
// is looked up in its head's kept frames or kept segments, in the order the
// compressed copy would hold them, so both give the same bytes.
//
// Attention: the bf16 kernel's structure (two ping-ponging 4-wave groups, 32
// query rows per wave, 64-key tiles, balanced schedule, cut items combined by
// the workgroup whose part arrives last) with
//   S^T = K Q^T    2 x (d/64) MFMAs 32x32x64 per tile (A = K tile from LDS,
//                  lane l reads 32 bytes of key row l%32 at dims 64ks + 32(l/32));
//   P' = 2^(x - m + 6) rounded to E4M3 (x = logit in log2 units, m the running
//                  max, allowed to lag by 2, so P' <= 2^8 < 448 and small
//                  probabilities stay in the normal range);
//   O^T += V^T P'^T  d/32 MFMAs (A = V^T rows from LDS, B = P' straight from
//                  the S^T accumulators: byte j = 16kb + i of lane l is key
//                  32kb + 8(i/4) + 4(l/32) + i%4, the accumulator's own order;
//                  the packed V^T tile stores keys in that order);
//   l += 1^T P'^T  one more MFMA with an all-ones A, so the normaliser sums
//                  exactly the rounded probabilities the value product used
//                  (A in E2M1, whose 1.0 is exact too: 4 VGPRs instead of 8,
//                  which the compiler then keeps live instead of re-creating
//                  every tile; 4% faster at 480P).
// The two operands of an MFMA pair their bytes symmetrically (byte j of lane
// half h of A with byte j of lane half h of B), so any consistent assignment of
// the contraction index to bytes is valid; this was checked on the hardware.
// Output: O = O^T * s_v[d] / l (bf16), lse = ln2 * (m - 6) + ln l.
#include "attn_common.h"
#include "attn_merge.h"

namespace fkv {
namespace {

using namespace attn;

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;
constexpr int kGroupThreads = 256;
constexpr float kSlack = 2.f;   // log2 units the running max may lag behind
constexpr float kPBias = 6.f;   // P' = 2^(x - m + kPBias) <= 2^(kSlack + kPBias)
constexpr float kE4M3Max = 448.f;

// Scale block of head h (fp8_scale_floats(d) floats):
//   [0] s_q  [1] s_k  [2] inv_q  [3] inv_k  [4, 4+d) s_v  [4+d, 4+2d) inv_v  [4+2d, 4+3d) mu_k
enum { SC_SQ = 0, SC_SK = 1, SC_IQ = 2, SC_IK = 3, SC_SV = 4 };

// Position of key k (0..63) of a tile inside the packed V^T row: the byte the
// value product's B operand (the P' accumulator order) assigns to that key.
__device__ __forceinline__ int vt_pos(int k) {
    const int kb = k >> 5, r = k & 31;
    const int hl = (r >> 2) & 1, i = 4 * (r >> 3) + (r & 3);
    return 32 * hl + 16 * kb + i;
}

template <bool HI>
__device__ __forceinline__ int pk_fp8(float a, float b, int old) {
    return __builtin_amdgcn_cvt_pk_fp8_f32(a, b, old, HI);
}

// ------------------------------------------------------------------ statistics
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// j / P for 0 <= j < 2^31 with M = floor(2^64 / P) + 1 = hi * 2^32 + lo:
// floor(j * M / 2^64) exactly (j * M / 2^64 exceeds j / P by less than 2^-33).
// P = 1 (M does not fit in 64 bits) is passed as hi = lo = 0.
__device__ __forceinline__ int div_magic(int j, uint32_t hi, uint32_t lo) {
    if (hi == 0 && lo == 0) return j;
    return (int)(((uint64_t)(uint32_t)j * hi + __umulhi((uint32_t)j, lo)) >> 32);
}

// History length of head h: kv_len clamped to the packed rows, or, read in
// place, the static head's kept frames times F.
__device__ __forceinline__ int pack_kvl(const Fp8PackArgs &a, int h) {
    if (a.paged && a.st_kept[h] >= 0) return a.st_kept[h] * a.F;
    int kvl = a.kv_len[h];
    const int64_t cap = a.paged ? (a.slab < (int64_t)a.H * a.F ? a.slab : (int64_t)a.H * a.F) : a.slab;
    return kvl < 0 ? 0 : (kvl > cap ? (int)cap : kvl);
}

// Read in place, the history of head h is a sequence of kept pieces of P
// rows, each contiguous in the cache: kept frames (static, P = F), kept
// segments (dynamic, L <= F, P = L) or the frames of kept segments (dynamic,
// L > F, P = F).  History row r is row r mod P of piece r / P.
struct Pieces {
    int P;
    uint32_t hi, lo;  // div_magic constants of P
};
// (The choice is made with masks on loaded values: a select between two
// fields of the argument block compiles to a select of their addresses, which
// makes the compiler copy the whole block to scratch memory in every thread.)
__device__ __forceinline__ Pieces pieces_of(const Fp8PackArgs &a, int h) {
    const uint32_t m = (a.st_kept[h] >= 0 || a.L > a.F) ? ~0u : 0u;  // P = F, else P = L
    const uint32_t F = (uint32_t)a.F, L = (uint32_t)a.L;
    return Pieces{(int)((F & m) | (L & ~m)), (a.mf_hi & m) | (a.ml_hi & ~m), (a.mf_lo & m) | (a.ml_lo & ~m)};
}

// Cache row (slot * F + row within the frame) of the first row of kept piece
// p of head h.  A kept_seg entry out of range is clamped, so a row that
// disagrees with kv_len cannot address outside the head's cache.
__device__ __forceinline__ int piece_row(const Fp8PackArgs &a, int h, int p, const int *slots) {
    int t, off = 0;
    if (a.st_kept[h] >= 0) {
        t = p < a.st_first[h] ? p : p + a.st_gap[h];
    } else if (a.L <= a.F) {
        const int g = min(max(a.kept_seg[(size_t)h * a.n_seg + p], 0), a.n_seg - 1);
        const int spf = a.F / a.L;
        t = g / spf;
        off = (g - t * spf) * a.L;
    } else {
        const int m = a.L / a.F;
        const int q = p / m;
        const int g = min(max(a.kept_seg[(size_t)h * a.n_seg + q], 0), a.n_seg - 1);
        t = min(g * m + (p - q * m), a.H - 1);
    }
    return slots[t] * a.F + off;
}

// The workgroup's table of piece start rows for its history rows [r0, r1):
// the slot map is copied to LDS, then entry i (piece p0 + i) is built by all
// threads at once (one round of kept_seg loads per workgroup instead of one
// per row).  At most (r1 - r0) / P + 1 <= cap entries.  Every thread calls it
// (two barriers).
struct PieceTable {
    Pieces pc;
    int p0;
};
__device__ __forceinline__ PieceTable build_pieces(const Fp8PackArgs &a, int h, int r0, int r1, int *slots,
                                                   int *tab, int cap) {
    for (int t = threadIdx.x; t < a.H; t += blockDim.x) slots[t] = a.slots.slot[t];
    __syncthreads();
    PieceTable pt{pieces_of(a, h), 0};
    if (r0 < r1) {
        pt.p0 = div_magic(r0, pt.pc.hi, pt.pc.lo);
        const int np = min(div_magic(r1 - 1, pt.pc.hi, pt.pc.lo) - pt.p0 + 1, cap);
        for (int i = threadIdx.x; i < np; i += blockDim.x) tab[i] = piece_row(a, h, pt.p0 + i, slots);
    }
    __syncthreads();
    return pt;
}

// Element offset of key/value row r of head h (r < kvl: history, else the
// chunk's row r - kvl) and whether it is a history row; read in place, history
// rows go through the workgroup's piece table.
template <int D>
__device__ __forceinline__ size_t pack_row(const Fp8PackArgs &a, int h, int r, int kvl, const PieceTable &pt,
                                           const int *tab, bool *hist) {
    *hist = r < kvl;
    if (!*hist) return ((size_t)h * a.Lq + (r - kvl)) * D;
    if (!a.paged) return ((size_t)h * a.slab + r) * D;
    const int p = div_magic(r, pt.pc.hi, pt.pc.lo);
    return ((size_t)h * a.cap * a.F + tab[p - pt.p0] + (r - p * pt.pc.P)) * D;
}

// grid (n_kchunks + n_qchunks, n_heads); thread = (row group, 8-channel group),
// four rows in flight per thread.  Partials ws[((h * chunks + x) * d + c) * 4 +
// {sum K, max K, min K, max |V|}]; Q chunks store max |Q| in slot 3.
template <int D>
__global__ __launch_bounds__(256) void fp8_stats_kernel(Fp8PackArgs a) {
    constexpr int CG = D / 8;          // channel groups (16-byte bf16 vectors) per row
    constexpr int RG = 256 / CG;       // row groups
    constexpr int U = 4;               // rows in flight per thread
    __shared__ double red_s[RG][D];
    __shared__ float red_mx[RG][D], red_mn[RG][D], red_v[RG][D];
    __shared__ int slots[FKV_MAX_FRAMES], tab[kFp8ChunkRows + 1];  // read in place
    const int x = blockIdx.x, h = blockIdx.y;
    const int tid = threadIdx.x, cg = tid % CG, rg = tid / CG;
    const int chunks = a.n_kchunks + a.n_qchunks;
    const int kvl = pack_kvl(a, h);
    if (a.paged && x == 0 && tid == 0 && a.st_kept[h] >= 0) a.kv_out[h] = kvl;
    double sum[8];
    float mx[8], mn[8], vm[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        sum[e] = 0.0;
        mx[e] = -__builtin_inff();
        mn[e] = __builtin_inff();
        vm[e] = 0.f;
    }
    const bool keys = x < a.n_kchunks;
    const int r0 = (keys ? x : x - a.n_kchunks) * a.chunk_rows;
    const int r1 = min(r0 + a.chunk_rows, keys ? kvl + a.Lq : a.Lq);
    // (chunk_rows is kFp8ChunkRows: at most kFp8ChunkRows + 1 pieces)
    const PieceTable pt = a.paged && keys ? build_pieces(a, h, r0, min(r1, kvl), slots, tab, kFp8ChunkRows + 1)
                                          : PieceTable{};
    for (int rb = r0 + rg; rb < r1; rb += U * RG) {
        u32x4 kv[U], vv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u * RG;
            kv[u] = u32x4{0, 0, 0, 0};
            vv[u] = u32x4{0, 0, 0, 0};
            if (r < r1) {
                if (keys) {
                    bool hist;
                    const size_t off = pack_row<D>(a, h, r, kvl, pt, tab, &hist);
                    kv[u] = *(const u32x4 *)((hist ? (a.paged ? a.K_hist : a.Kc) : a.K_cur) + off + 8 * cg);
                    vv[u] = *(const u32x4 *)((hist ? (a.paged ? a.V_hist : a.Vc) : a.V_cur) + off + 8 * cg);
                } else {
                    vv[u] = *(const u32x4 *)(a.Q + ((size_t)h * a.Lq + r) * D + 8 * cg);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (rb + u * RG >= r1) break;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float fv = (e & 1) ? bf_hi(vv[u][e >> 1]) : bf_lo(vv[u][e >> 1]);
                vm[e] = fmaxf(vm[e], fabsf(fv));
                if (keys) {
                    const float fk = (e & 1) ? bf_hi(kv[u][e >> 1]) : bf_lo(kv[u][e >> 1]);
                    sum[e] += (double)fk;
                    mx[e] = fmaxf(mx[e], fk);
                    mn[e] = fminf(mn[e], fk);
                }
            }
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        red_s[rg][8 * cg + e] = sum[e];
        red_mx[rg][8 * cg + e] = mx[e];
        red_mn[rg][8 * cg + e] = mn[e];
        red_v[rg][8 * cg + e] = vm[e];
    }
    __syncthreads();
    for (int c = tid; c < D; c += 256) {
        double s = 0.0;
        float M = -__builtin_inff(), m = __builtin_inff(), v = 0.f;
        for (int g = 0; g < RG; ++g) {
            s += red_s[g][c];
            M = fmaxf(M, red_mx[g][c]);
            m = fminf(m, red_mn[g][c]);
            v = fmaxf(v, red_v[g][c]);
        }
        double *o = a.ws + (((size_t)h * chunks + x) * D + c) * 4;
        o[0] = s;
        o[1] = M;
        o[2] = m;
        o[3] = v;
    }
}

__device__ __forceinline__ void scale_pair(float amax, float *inv, float *s) {
    *inv = amax > 0.f ? __fdiv_rn(kE4M3Max, amax) : 0.f;
    *s = amax > 0.f ? __fdiv_rn(amax, kE4M3Max) : 0.f;
}

// grid (n_heads), 1024 threads: S = 1024 / D slices of the chunks per channel,
// four chunks in flight per thread, combined in a fixed order.
template <int D>
__global__ __launch_bounds__(1024) void fp8_finalize_kernel(Fp8PackArgs a) {
    constexpr int S = 1024 / D;
    __shared__ double red_s[S][D];
    __shared__ float red_mx[S][D], red_mn[S][D], red_v[S][D], red_q[S][D];
    __shared__ float red_k[D], red_qq[D];
    const int h = blockIdx.x, c = threadIdx.x % D, sl = threadIdx.x / D;
    const int chunks = a.n_kchunks + a.n_qchunks;
    const int kvl = pack_kvl(a, h);
    const double *p = a.ws + ((size_t)h * chunks * D + c) * 4;
    double s = 0.0;
    float M = -__builtin_inff(), m = __builtin_inff(), v = 0.f, q = 0.f;
    for (int x0 = sl; x0 < chunks; x0 += 4 * S) {
        double o[4][4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int x = x0 + u * S;
            if (x < chunks) {
                const double *src = p + (size_t)x * D * 4;
                o[u][0] = src[0];
                o[u][1] = src[1];
                o[u][2] = src[2];
                o[u][3] = src[3];
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int x = x0 + u * S;
            if (x >= chunks) break;
            if (x < a.n_kchunks) {
                s += o[u][0];
                M = fmaxf(M, (float)o[u][1]);
                m = fminf(m, (float)o[u][2]);
                v = fmaxf(v, (float)o[u][3]);
            } else {
                q = fmaxf(q, (float)o[u][3]);
            }
        }
    }
    red_s[sl][c] = s;
    red_mx[sl][c] = M;
    red_mn[sl][c] = m;
    red_v[sl][c] = v;
    red_q[sl][c] = q;
    __syncthreads();
    if (sl == 0) {
        for (int i = 1; i < S; ++i) {
            s += red_s[i][c];
            M = fmaxf(M, red_mx[i][c]);
            m = fminf(m, red_mn[i][c]);
            v = fmaxf(v, red_v[i][c]);
            q = fmaxf(q, red_q[i][c]);
        }
        const float mu = (float)(s / (double)(kvl + a.Lq));
        red_k[c] = fmaxf(fabsf(__fsub_rn(M, mu)), fabsf(__fsub_rn(m, mu)));
        red_qq[c] = q;
        float *sc = a.scales + (size_t)h * fp8_scale_floats(D);
        float inv, sv;
        scale_pair(v, &inv, &sv);
        sc[SC_SV + c] = sv;
        sc[SC_SV + D + c] = inv;
        sc[SC_SV + 2 * D + c] = mu;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float ak = 0.f, aq = 0.f;
        for (int i = 0; i < D; ++i) {
            ak = fmaxf(ak, red_k[i]);
            aq = fmaxf(aq, red_qq[i]);
        }
        float *sc = a.scales + (size_t)h * fp8_scale_floats(D);
        float iq, sq, ik, sk;
        scale_pair(aq, &iq, &sq);
        scale_pair(ak, &ik, &sk);
        sc[SC_SQ] = sq;
        sc[SC_SK] = sk;
        sc[SC_IQ] = iq;
        sc[SC_IK] = ik;
    }
}

// E4M3 codes of 8 bf16 values (one 16-byte vector) times per-element factors.
template <bool SUB>
__device__ __forceinline__ uint2 quant8(const u32x4 &w, const float *mu, const float *inv, bool per_channel,
                                        float inv0) {
    float f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        float x = (e & 1) ? bf_hi(w[e >> 1]) : bf_lo(w[e >> 1]);
        if (SUB) x = __fsub_rn(x, mu[e]);
        f[e] = __fmul_rn(x, per_channel ? inv[e] : inv0);
    }
    int lo = 0, hi = 0;
    lo = pk_fp8<false>(f[0], f[1], lo);
    lo = pk_fp8<true>(f[2], f[3], lo);
    hi = pk_fp8<false>(f[4], f[5], hi);
    hi = pk_fp8<true>(f[6], f[7], hi);
    return make_uint2((uint32_t)lo, (uint32_t)hi);
}

// Transpose of a 4 x 4 byte block: dword i of the result holds byte i of a0..a3.
__device__ __forceinline__ void transpose4(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3, uint32_t (&o)[4]) {
    const uint32_t t0 = __builtin_amdgcn_perm(a1, a0, 0x05010400u);  // a0.b0 a1.b0 a0.b1 a1.b1
    const uint32_t t1 = __builtin_amdgcn_perm(a1, a0, 0x07030602u);  // a0.b2 a1.b2 a0.b3 a1.b3
    const uint32_t t2 = __builtin_amdgcn_perm(a3, a2, 0x05010400u);
    const uint32_t t3 = __builtin_amdgcn_perm(a3, a2, 0x07030602u);
    o[0] = __builtin_amdgcn_perm(t2, t0, 0x05040100u);
    o[1] = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
    o[2] = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
    o[3] = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

// grid (tiles, n_heads), 256 threads.  Tile t < n_ktiles packs keys and values
// [64t, 64t + 64): thread = (key quad kq, 8-channel group cg); the four keys
// 4kq .. 4kq+3 occupy four consecutive bytes of every V^T row, so each of the
// thread's 8 channels is one 4-byte store.  Tiles t >= n_ktiles pack 64 query
// rows, four 8-channel vectors per thread.
template <int D>
__global__ __launch_bounds__(256) void fp8_pack_kernel(Fp8PackArgs a, int n_ktiles) {
    constexpr int CG = D / 8;
    const int t = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const float *sc = a.scales + (size_t)h * fp8_scale_floats(D);
    if (t >= n_ktiles) {  // queries
        constexpr int UPT = BN * CG / 256;
        const float inv = sc[SC_IQ];
        u32x4 w[UPT];
#pragma unroll
        for (int i = 0; i < UPT; ++i) {
            const int u = tid + 256 * i, r = (t - n_ktiles) * BN + u / CG;
            w[i] = r < a.Lq ? *(const u32x4 *)(a.Q + ((size_t)h * a.Lq + r) * D + 8 * (u % CG)) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int i = 0; i < UPT; ++i) {
            const int u = tid + 256 * i, r = (t - n_ktiles) * BN + u / CG;
            if (r < a.Lq)
                *(uint2 *)(a.Q8 + ((size_t)h * a.Lq + r) * D + 8 * (u % CG)) = quant8<false>(w[i], nullptr, nullptr, false, inv);
        }
        return;
    }
    __shared__ int slots[FKV_MAX_FRAMES], tab[BN + 1];  // read in place
    const int kvl = pack_kvl(a, h);
    const int Lk = kvl + a.Lq;
    if (t * BN >= Lk) return;  // never read by the attention kernel
    const PieceTable pt = a.paged ? build_pieces(a, h, t * BN, min(t * BN + BN, kvl), slots, tab, BN + 1) : PieceTable{};
    if (tid >= (BN / 4) * CG) return;
    const int kq = tid % (BN / 4), cg = tid / (BN / 4);
    const float *mu = sc + SC_SV + 2 * D + 8 * cg;
    const float *iv = sc + SC_SV + D + 8 * cg;
    const float ik = sc[SC_IK];
    u32x4 kw[4], vw[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int r = t * BN + 4 * kq + e;
        kw[e] = u32x4{0, 0, 0, 0};
        vw[e] = u32x4{0, 0, 0, 0};
        if (r < Lk) {
            bool hist;
            const size_t off = pack_row<D>(a, h, r, kvl, pt, tab, &hist);
            kw[e] = *(const u32x4 *)((hist ? (a.paged ? a.K_hist : a.Kc) : a.K_cur) + off + 8 * cg);
            vw[e] = *(const u32x4 *)((hist ? (a.paged ? a.V_hist : a.Vc) : a.V_cur) + off + 8 * cg);
        }
    }
    uint2 vq[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int r = t * BN + 4 * kq + e;
        // rows past the head's keys pack as zeros (0 - mu would not be 0)
        const uint2 kc = r < Lk ? quant8<true>(kw[e], mu, nullptr, false, ik) : make_uint2(0u, 0u);
        *(uint2 *)(a.K8 + ((size_t)h * a.rows + r) * D + 8 * cg) = kc;
        vq[e] = quant8<false>(vw[e], nullptr, iv, true, 0.f);
    }
    uint32_t lo[4], hi[4];
    transpose4(vq[0].x, vq[1].x, vq[2].x, vq[3].x, lo);
    transpose4(vq[0].y, vq[1].y, vq[2].y, vq[3].y, hi);
    uint8_t *dst = a.V8T + ((size_t)h * a.rows + (size_t)t * BN) * D + vt_pos(4 * kq);  // tile t: [D][BN] bytes
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        *(uint32_t *)(dst + (8 * cg + j) * BN) = lo[j];
        *(uint32_t *)(dst + (8 * cg + 4 + j) * BN) = hi[j];
    }
}

// ------------------------------------------------------------------ attention
template <int D>
struct Fp8Cfg {
    static constexpr int KROW = D + 16;             // K tile row stride in LDS (bytes)
    static constexpr int VROW = BN + 16;            // V^T tile row stride in LDS (bytes)
    static constexpr int KS = D / 64;               // k-steps of S^T = K Q^T
    static constexpr int MB = D / 32;               // 32-row blocks of O^T
    static constexpr int KTILE = BN * KROW;
    static constexpr int VTILE = D * VROW;
    static constexpr int KCH = D / 16;              // 16-byte chunks per K row
    static constexpr int VCH = BN / 16;             // 16-byte chunks per V^T row
    static constexpr int NV = BN * D / 16 / kGroupThreads;  // staging vectors per thread
    static_assert(NV >= 1 && NV <= 4, "tile shape");
};

__device__ __forceinline__ i32x8 load32(const uint8_t *p) {
    const u32x4 a = *(const u32x4 *)p, b = *(const u32x4 *)(p + 16);
    return i32x8{(int)a[0], (int)a[1], (int)a[2], (int)a[3], (int)b[0], (int)b[1], (int)b[2], (int)b[3]};
}

__device__ __forceinline__ f32x16_t mfma8(const i32x8 &a, const i32x8 &b, const f32x16_t &c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// The same product with A in E2M1 (format code 4; only the first four words
// of a are read) and B in E4M3.
__device__ __forceinline__ f32x16_t mfma4x8(const i32x8 &a, const i32x8 &b, const f32x16_t &c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 4, 0, 0, 0, 0, 0);
}

// One MFMA block of a wave: S^T = K Q^T for the next tile (its K operands kq
// were read from LDS during the previous phase), then, if PV, O^T += V^T P'^T
// and l += 1 P'^T for the current tile.  The V^T operands are read at the start
// of the block and arrive while the score products run.
template <int D, bool PV>
__device__ __forceinline__ void mfma_block8(const uint8_t *vs, int vbase, const i32x8 &pb, const i32x8 &ones,
                                            const i32x8 (&qf)[D / 64], const i32x8 (&kq)[D / 32],
                                            f32x16_t (&o)[D / 32], f32x16_t &lacc, f32x16_t (&s)[2]) {
    using C = Fp8Cfg<D>;
    constexpr int NQ = 2 * C::KS;
    constexpr int NEARLY = NQ < C::MB ? NQ : C::MB;   // V operands read before the score products
    i32x8 va[C::MB];
    if (PV) {
#pragma unroll
        for (int mb = 0; mb < NEARLY / 2; ++mb) va[mb] = load32(vs + vbase + mb * 32 * C::VROW);
    }
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
        const int kk = i >> 1, kb = i & 1;
        s[kb] = mfma8(kq[i], qf[kk], kk == 0 ? f32x16_t{} : s[kb]);
        // the rest of the V operands, issued as the K operands retire
        const int mb = NEARLY / 2 + i;
        if (PV && mb < C::MB) va[mb] = load32(vs + vbase + mb * 32 * C::VROW);
    }
    if (PV) {
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb) o[mb] = mfma8(va[mb], pb, o[mb]);
        lacc = mfma4x8(ones, pb, lacc);
    }
    if (PV) {
#pragma unroll
        for (int mb = 0; mb < NEARLY / 2; ++mb) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (NEARLY / 2 + i < C::MB) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, C::MB + 1, 0);
    } else {
        __builtin_amdgcn_sched_group_barrier(0x008, NQ, 0);
    }
}

// K operands of the score product for one tile: key rows 32kb + l32, dims
// 64kk + 32hl .. +32 (index 2kk + kb).
template <int D>
__device__ __forceinline__ void read_kq(const uint8_t *ks, int kbase, i32x8 (&kq)[D / 32]) {
    using C = Fp8Cfg<D>;
#pragma unroll
    for (int i = 0; i < 2 * C::KS; ++i) kq[i] = load32(ks + kbase + (i & 1) * 32 * C::KROW + 64 * (i >> 1));
}

template <int D>
__device__ __forceinline__ void fp8_segment(const AttnArgs &a, uint8_t (&Ks)[2][Fp8Cfg<D>::KTILE],
                                            uint8_t (&Vs)[2][Fp8Cfg<D>::VTILE], int h, int qt, int t0, int t1,
                                            int rot, float *slot) {
    using C = Fp8Cfg<D>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = wave >> 2;
    const int l32 = lane & 31, hl = lane >> 5;
    const int Lq = a.Lq;
    const int n = t1 - t0;

    const float *sc = a.fp8_scales + (size_t)h * fp8_scale_floats(D);
    float c2 = a.scale_log2 * sc[SC_SQ] * sc[SC_SK];
    c2 = c2 > 0.f ? c2 : 1.f;  // a zero Q or K packs to zeros: every logit is 0 either way

    const int qrow = qt * BM + wave * 32 + l32;
    const bool qok = qrow < Lq;
    const uint8_t *Qh = (const uint8_t *)a.Q + (size_t)h * Lq * D;
    i32x8 qf[C::KS];
#pragma unroll
    for (int kk = 0; kk < C::KS; ++kk)
        qf[kk] = qok ? load32(Qh + (size_t)qrow * D + 64 * kk + 32 * hl) : i32x8{};

    const int Lk = head_kvl(a, h) + Lq;
    const int T = (Lk + BN - 1) / BN;
    const uint8_t *K8 = (const uint8_t *)a.Kc + (size_t)h * a.fp8_rows * D;
    const uint8_t *V8 = (const uint8_t *)a.Vc + (size_t)h * a.fp8_rows * D;

    const int gtid = tid & 255;
    const int kt0 = (t0 + rot) % T;
    auto tile = [&](int j) {
        const int k = kt0 + j;
        return k >= T ? k - T : k;
    };
    auto load_k = [&](int kt, u32x4 (&dst)[4]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) {
            const int v = gtid + i * kGroupThreads;
            dst[i] = __builtin_nontemporal_load((const u32x4 *)(K8 + ((size_t)kt * BN + v / C::KCH) * D + 16 * (v % C::KCH)));
        }
    };
    auto load_v = [&](int kt, u32x4 (&dst)[4]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) {
            const int v = gtid + i * kGroupThreads;
            dst[i] = __builtin_nontemporal_load((const u32x4 *)(V8 + (size_t)kt * BN * D + 16 * v));
        }
    };
    auto store_k = [&](uint8_t *t, const u32x4 (&src)[4]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) {
            const int v = gtid + i * kGroupThreads;
            *(u32x4 *)(t + (v / C::KCH) * C::KROW + 16 * (v % C::KCH)) = src[i];
        }
    };
    auto store_v = [&](uint8_t *t, const u32x4 (&src)[4]) {
#pragma unroll
        for (int i = 0; i < C::NV; ++i) {
            const int v = gtid + i * kGroupThreads;
            *(u32x4 *)(t + (v / C::VCH) * C::VROW + 16 * (v % C::VCH)) = src[i];
        }
    };

    // K (A of S^T): lane reads key row 32kb + l32, dims 64kk + 32hl .. +32.
    const int kbase = l32 * C::KROW + 32 * hl;
    // V^T (A of O^T): lane reads dim row 32mb + l32, packed key bytes 32hl .. +32.
    const int vbase = l32 * C::VROW + 32 * hl;

    f32x16_t o[C::MB];
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) o[mb] = f32x16_t{};
    f32x16_t lacc = f32x16_t{};
    f32x16_t s[2];
    i32x8 pb = i32x8{};
    const i32x8 ones = {0x22222222, 0x22222222, 0x22222222, 0x22222222, 0, 0, 0, 0};  // E2M1 1.0
    float m_run = -__builtin_inff();

    // Row maximum of the current scores (keys past Lk masked), and the lazy
    // update of the running max with the rescale of the accumulators.
    auto row_max = [&](int j0) {
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
        if (__ballot(mx > m_run + kSlack)) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            lacc *= alpha;
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb) o[mb] *= alpha;
        }
    };
    // The rounded probabilities P' of the current scores.
    auto exps = [&]() {
        const float bias = kPBias - m_run;
#pragma unroll
        for (int w = 0; w < 8; ++w) {
            // bytes 4w .. 4w+3 of the B operand: accumulator entries s[w/4][4(w%4) .. +3]
            const int kb = w >> 2, i0 = 4 * (w & 3);
            int r = pb[w];  // both halves are overwritten: no zeroing move
            r = pk_fp8<false>(__builtin_amdgcn_exp2f(fmaf(s[kb][i0], c2, bias)),
                       __builtin_amdgcn_exp2f(fmaf(s[kb][i0 + 1], c2, bias)), r);
            r = pk_fp8<true>(__builtin_amdgcn_exp2f(fmaf(s[kb][i0 + 2], c2, bias)),
                       __builtin_amdgcn_exp2f(fmaf(s[kb][i0 + 3], c2, bias)), r);
            pb[w] = r;
        }
    };

    u32x4 stage[4];
    if (grp == 0) {
        load_k(tile(0), stage);
        store_k(Ks[0], stage);
        if (n > 1) {
            load_k(tile(1), stage);
            store_k(Ks[1], stage);
            load_v(tile(1), stage);
        }
    } else {
        load_v(tile(0), stage);
        store_v(Vs[0], stage);
        if (n > 2) load_k(tile(2), stage);
    }
    __syncthreads();
    i32x8 kq[2 * C::KS];
    read_kq<D>(Ks[0], kbase, kq);
    if (grp == 0) mfma_block8<D, false>(nullptr, vbase, pb, ones, qf, kq, o, lacc, s);
    // Same phase structure and barrier count as the bf16 kernel: group 1 runs
    // one phase behind group 0; 2n + 2 barriers per group, the last one after
    // every LDS read of the segment.  The K operands of the next score product
    // are read at the top of each iteration: that tile was stored two phases
    // before the barrier just passed and is overwritten only after the MFMA
    // block of this iteration.
    if (grp == 1) {
        mfma_block8<D, false>(nullptr, vbase, pb, ones, qf, kq, o, lacc, s);
        __syncthreads();
    }
    __builtin_amdgcn_s_waitcnt(0);
    // The row maximum of tile it + 1 is taken in the MFMA phase of tile it,
    // right after its products are issued (its VALU work overlaps them; 6%
    // faster than at the start of the softmax phase); the softmax phase then
    // only forms the probabilities.
    for (int it = 0; it < n; ++it) {
        read_kq<D>(Ks[(it + 1) & 1], kbase, kq);
        if (it == 0) row_max(tile(0) * BN);
        exps();
        if (grp == 0) {
            if (it >= 1) store_v(Vs[it & 1], stage);
            if (it >= 1 && it + 1 < n) load_v(tile(it + 1), stage);
        } else {
            if (it + 2 < n) store_k(Ks[it & 1], stage);
            if (it + 3 < n) load_k(tile(it + 3), stage);
        }
        __syncthreads();
        // (the priority raise is worth 15% here: the products issue ahead of
        // the other wave's softmax)
        __builtin_amdgcn_s_setprio(1);
        mfma_block8<D, true>(Vs[it & 1], vbase, pb, ones, qf, kq, o, lacc, s);
        __builtin_amdgcn_s_setprio(0);
        if (it + 1 < n) row_max(tile(it + 1) * BN);
        __syncthreads();
    }
    if (grp == 0) __syncthreads();

    const float l_tot = lacc[0];  // every row of the ones product holds this query's sum
    const float inv = 1.f / l_tot;
    const float *sv = sc + SC_SV;
    if (slot) {
        // device-scope stores: the workgroup that combines the item's parts may
        // run on another XCD, within this launch.  The part's maximum is
        // m - kPBias, so that l_tot = sum 2^(x - (m - kPBias)) as for bf16 parts.
        unsigned long long *op = (unsigned long long *)slot;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 w = *(const float4 *)(sv + 32 * mb + 8 * g + 4 * hl);
                put_shared(op + ((wave * C::MB + mb) * 4 + g) * 64 + lane,
                           pack_bf16x4(o[mb][4 * g] * w.x * inv, o[mb][4 * g + 1] * w.y * inv,
                                       o[mb][4 * g + 2] * w.z * inv, o[mb][4 * g + 3] * w.w * inv));
            }
        if (hl == 0) {
            put_shared(slot + BM * D / 2 + wave * 32 + l32, m_run - kPBias);
            put_shared(slot + BM * D / 2 + BM + wave * 32 + l32, l_tot);
        }
        return;
    }
    if (qok) {
        uint16_t *Oh = (uint16_t *)a.O + ((size_t)h * Lq + qrow) * D;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 w = *(const float4 *)(sv + 32 * mb + 8 * g + 4 * hl);
                *(uint2 *)(Oh + mb * 32 + 8 * g + 4 * hl) =
                    pack_bf16x4(o[mb][4 * g] * w.x * inv, o[mb][4 * g + 1] * w.y * inv,
                                o[mb][4 * g + 2] * w.z * inv, o[mb][4 * g + 3] * w.w * inv);
            }
        if (a.lse && hl == 0)
            a.lse[(size_t)h * Lq + qrow] = fmaf(m_run - kPBias, 0.69314718055994530942f, logf(l_tot));
    }
}

template <int D, bool BAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fp8_kernel(AttnArgs a) {
    using C = Fp8Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint8_t Ks[2][C::KTILE];
    __shared__ __attribute__((aligned(16))) uint8_t Vs[2][C::VTILE];
    __shared__ uint32_t flag;
    if (!BAL) {
        const int item = (blockIdx.x & 7) * a.items_per_xcd + (blockIdx.x >> 3);
        if (item >= a.n_items) return;
        const int li = item / a.n_qtiles;
        const int h = a.heads.head[li];
        fp8_segment<D>(a, Ks, Vs, h, item - li * a.n_qtiles, 0, head_tiles(a, h), 0, nullptr);
        return;
    }
    // The schedule walks the head list entry by entry (dependent scalar loads)
    // rather than building the wave-parallel work list of attn_common.h: at
    // 252 VGPRs this kernel has none to spare, and the work list cost it a
    // private segment for no measured gain.
    auto tiles = [&](int l) { return head_tiles(a, a.heads.head[l]); };
    Schedule sc;
    {
        int64_t total = 0;
        for (int l = 0; l < a.heads.n; ++l) total += (int64_t)a.n_qtiles * tiles(l);
        sc.total = total;
        sc.G = (int)(total < a.n_blocks ? total : a.n_blocks);
    }
    const int r = (blockIdx.x & 7) * (a.n_blocks >> 3) + (blockIdx.x >> 3);
    if (r >= sc.G) return;
    const int64_t end = sc.start(r + 1);
    int64_t cur = sc.start(r);
    bool first = true;
    while (cur < end) {
        ItemPos ip;  // the item holding tile `cur`
        {
            int li = 0, T = tiles(0);
            int64_t base = 0;
            while (cur >= base + (int64_t)a.n_qtiles * T) {
                base += (int64_t)a.n_qtiles * T;
                T = tiles(++li);
            }
            const int qt = (int)((cur - base) / T);
            ip = ItemPos{li, qt, T, base + (int64_t)qt * T};
        }
        const int h = a.heads.head[ip.li], qt = ip.qt, T = ip.T;
        const int64_t ibase = ip.ibase;
        const int t0 = (int)(cur - ibase);
        const int t1 = (int)((end < ibase + T ? end : ibase + T) - ibase);
        float *slot = (t0 == 0 && t1 == T) ? nullptr
                                            : a.part + (size_t)(2 * r + (first ? 0 : 1)) * slot_floats<D>();
        const int rot = (int)((ibase - sc.start(sc.owner(ibase))) % T);
        fp8_segment<D>(a, Ks, Vs, h, qt, t0, t1, rot, slot);
        if (slot) {
            // the last of the item's parts to arrive combines them
            const int n_parts = sc.owner(ibase + T - 1) - sc.owner(ibase) + 1;
            uint32_t *cnt = a.item_counters + (size_t)(ip.li * a.n_qtiles + qt) * kItemCounterStride;
            if (arrive_last(cnt, (uint32_t)n_parts, &flag))
                merge_rows<D, 64>(a, sc, ip.li, qt, ibase, T, threadIdx.x >> 6, threadIdx.x & 63);
        }
        cur = ibase + t1;
        first = false;
    }
}

}  // namespace

hipError_t launch_fp8_pack(const Fp8PackArgs &a, hipStream_t s) {
    const dim3 sgrid((unsigned)(a.n_kchunks + a.n_qchunks), (unsigned)a.n_heads);
    const int n_ktiles = (int)(a.rows / BN);
    const int n_qtiles = (a.Lq + BN - 1) / BN;
    const dim3 pgrid((unsigned)(n_ktiles + n_qtiles), (unsigned)a.n_heads);
    if (a.d == 128) {
        hipLaunchKernelGGL(fp8_stats_kernel<128>, sgrid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(fp8_finalize_kernel<128>, dim3(a.n_heads), dim3(1024), 0, s, a);
        hipLaunchKernelGGL(fp8_pack_kernel<128>, pgrid, dim3(256), 0, s, a, n_ktiles);
    } else {
        hipLaunchKernelGGL(fp8_stats_kernel<64>, sgrid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(fp8_finalize_kernel<64>, dim3(a.n_heads), dim3(1024), 0, s, a);
        hipLaunchKernelGGL(fp8_pack_kernel<64>, pgrid, dim3(256), 0, s, a, n_ktiles);
    }
    return hipGetLastError();
}

hipError_t launch_attention_fp8(const AttnArgs &a, int head_dim, hipStream_t s) {
    if (a.n_blocks > 0) {
        if (head_dim == 128)
            hipLaunchKernelGGL((attn_fp8_kernel<128, true>), dim3(a.n_blocks), dim3(kThreads), 0, s, a);
        else
            hipLaunchKernelGGL((attn_fp8_kernel<64, true>), dim3(a.n_blocks), dim3(kThreads), 0, s, a);
        return hipGetLastError();
    }
    const unsigned blocks = (unsigned)a.items_per_xcd * 8u;
    if (head_dim == 128)
        hipLaunchKernelGGL((attn_fp8_kernel<128, false>), dim3(blocks), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL((attn_fp8_kernel<64, false>), dim3(blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
