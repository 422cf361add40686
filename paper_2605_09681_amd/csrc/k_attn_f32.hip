// k_attn_f32.hip -- chunk attention over the compressed cache (Eq. 2 / Eq. 4)
// for fp32 tensors: plain fp32 vector arithmetic, no matrix cores.  This path
// serves small fp32 workloads; the bf16 MFMA kernel is the fast path.
//
// Workgroup = 32 query rows of one head; 8 threads per row.  Keys are staged in
// LDS 32 at a time; each thread scores 4 keys of its row, the row's 8 threads
// combine maxima with shuffles and run an fp32 online softmax; each thread then
// accumulates a d/8-wide slice of the row's output.
#include "fkv_internal.h"

namespace fkv {
namespace {

constexpr int kThreads = 256;
constexpr int RM = kAttnRowsF32;  // query rows per workgroup
constexpr int TN = 32;            // keys per tile
constexpr int TPR = kThreads / RM;  // threads per row (8)

template <int D>
__global__ __launch_bounds__(kThreads) void attn_f32_kernel(AttnArgs a) {
    __shared__ float Qs[RM][D + 1];
    __shared__ float Ks[TN][D + 1];
    __shared__ float Vs[TN][D];
    __shared__ float Ps[RM][TN + 1];

    const int item = blockIdx.x;
    if (item >= a.n_items) return;
    const int li = item / a.n_qtiles;
    const int h = a.heads.head[li];
    const int qt = item - li * a.n_qtiles;
    const int tid = threadIdx.x;
    const int r = tid / TPR, sub = tid % TPR;
    const int Lq = a.Lq;
    const int q0 = qt * RM;

    const float *Qh = (const float *)a.Q + (size_t)h * Lq * D;
    for (int i = tid; i < RM * D; i += kThreads) {
        const int rr = i / D, c = i % D;
        Qs[rr][c] = (q0 + rr < Lq) ? Qh[(size_t)(q0 + rr) * D + c] : 0.f;
    }

    int kvl = a.kv_len[h];
    kvl = kvl < 0 ? 0 : (kvl > a.slab ? (int)a.slab : kvl);
    const int Lk = kvl + Lq;
    const float *Kc = (const float *)a.Kc + (size_t)h * a.slab * D;
    const float *Vc = (const float *)a.Vc + (size_t)h * a.slab * D;
    const float *Kq = (const float *)a.K_cur + (size_t)h * Lq * D;
    const float *Vq = (const float *)a.V_cur + (size_t)h * Lq * D;

    constexpr int SL = D / TPR;  // output slice per thread
    float o[SL];
#pragma unroll
    for (int e = 0; e < SL; ++e) o[e] = 0.f;
    float m_run = -__builtin_inff(), l_run = 0.f;

    for (int j0 = 0; j0 < Lk; j0 += TN) {
        __syncthreads();
        for (int i = tid; i < TN * D; i += kThreads) {
            const int jj = i / D, c = i % D;
            const int j = j0 + jj;
            float kv = 0.f, vv = 0.f;
            if (j < kvl) {
                kv = Kc[(size_t)j * D + c];
                vv = Vc[(size_t)j * D + c];
            } else if (j < Lk) {
                kv = Kq[(size_t)(j - kvl) * D + c];
                vv = Vq[(size_t)(j - kvl) * D + c];
            }
            Ks[jj][c] = kv;
            Vs[jj][c] = vv;
        }
        __syncthreads();

        float sv[TN / TPR];
        float mx = -__builtin_inff();
#pragma unroll
        for (int u = 0; u < TN / TPR; ++u) {
            const int jj = sub + TPR * u;
            float acc = 0.f;
            for (int c = 0; c < D; ++c) acc = fmaf(Qs[r][c], Ks[jj][c], acc);
            sv[u] = (j0 + jj < Lk) ? acc * a.scale : -__builtin_inff();
            mx = fmaxf(mx, sv[u]);
        }
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        const float m_new = fmaxf(m_run, mx);
        const float alpha = expf(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int u = 0; u < TN / TPR; ++u) {
            const float p = expf(sv[u] - m_new);
            l_run += p;
            Ps[r][sub + TPR * u] = p;
        }
#pragma unroll
        for (int e = 0; e < SL; ++e) o[e] *= alpha;
        __syncthreads();
        for (int jj = 0; jj < TN; ++jj) {
            const float p = Ps[r][jj];
#pragma unroll
            for (int e = 0; e < SL; ++e) o[e] = fmaf(p, Vs[jj][sub * SL + e], o[e]);
        }
    }

    float l_tot = l_run;
#pragma unroll
    for (int off = 1; off < TPR; off <<= 1) l_tot += __shfl_xor(l_tot, off);
    const int row = q0 + r;
    if (row < Lq) {
        float *Oh = (float *)a.O + ((size_t)h * Lq + row) * D;
        const float inv = 1.f / l_tot;
#pragma unroll
        for (int e = 0; e < SL; ++e) Oh[sub * SL + e] = o[e] * inv;
        if (a.lse && sub == 0) a.lse[(size_t)h * Lq + row] = m_run + logf(l_tot);
    }
}

}  // namespace

hipError_t launch_attention_f32(const AttnArgs &a, int head_dim, hipStream_t s) {
    if (head_dim == 128)
        hipLaunchKernelGGL(attn_f32_kernel<128>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(attn_f32_kernel<64>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace fkv
