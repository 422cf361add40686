// attn_common.h -- pieces shared by the bf16 and FP8 chunk-attention kernels:
// tile sizes, the balanced work schedule and the partial-result slot format
// in which the parts of a split item are combined.
#pragma once

#include "fkv_internal.h"

namespace fkv {
namespace attn {

constexpr int BM = kAttnRowsBf16;  // query rows per workgroup (8 waves x 32)
constexpr int BN = kAttnKeysPerTile;  // keys per tile

// Number of key tiles of head h: [Kc[h][0:kv_len]; K_cur[h]] in tiles of BN.
__device__ __forceinline__ int head_kvl(const AttnArgs &a, int h) {
    const int kvl = a.kv_len[h];
    return kvl < 0 ? 0 : (kvl > a.slab ? (int)a.slab : kvl);
}
__device__ __forceinline__ int head_tiles(const AttnArgs &a, int h) {
    return (head_kvl(a, h) + a.Lq + BN - 1) / BN;
}
// The same for entry li of the launch's head list.  PAGED (a compile-time
// switch): heads read in place; a static entry's history length follows from
// its budget (stored per list entry), a dynamic entry's is kv_len.
template <bool PAGED = false>
__device__ __forceinline__ int entry_kvl(const AttnArgs &a, int li) {
    if constexpr (PAGED) {
        const int kept = a.st_kept[li];
        if (kept >= 0) return kept * a.F;
    }
    return head_kvl(a, a.heads.head[li]);
}
template <bool PAGED = false>
__device__ __forceinline__ int entry_tiles(const AttnArgs &a, int li) {
    return (entry_kvl<PAGED>(a, li) + a.Lq + BN - 1) / BN;
}

// Work items are (entry li of the launch's head list, query tile qt),
// li-major; the head is h = heads.head[li].
//
// Balanced schedule.  Work item i = (head h, query tile qt), h-major, has
// T_h key tiles; concatenating all items gives one sequence of `total` tiles,
// which G = min(n_blocks, total) workgroups split into equal contiguous ranges:
// workgroup r takes tiles [r*total/G, (r+1)*total/G).  An item cut by a range
// boundary is computed in parts whose results are combined by the workgroup
// completing the last of them (attn_merge.h).  Every kernel derives the same
// schedule from kv_len.
struct Schedule {
    int64_t total;
    int G;
    __device__ __forceinline__ int64_t start(int r) const { return (int64_t)r * total / G; }
    // workgroup whose range holds tile x: the largest r with start(r) <= x
    __device__ __forceinline__ int owner(int64_t x) const { return (int)(((x + 1) * G - 1) / total); }
};

// The launch's work list as one wave sees it: lane l < heads.n holds the key
// tile count T of list entry l and the inclusive prefix sum of n_qtiles * T
// over entries 0..l; lanes past the list repeat the total.  One vector load of
// the entries' lengths and a wave scan, instead of a chain of dependent scalar
// loads (one per entry, each a full memory latency) at the start of every
// workgroup.
struct WorkList {
    int T;
    int64_t incl;
};

__device__ __forceinline__ int64_t readlane64(int64_t v, int l) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <bool PAGED = false>
__device__ __forceinline__ WorkList work_list(const AttnArgs &a) {
    const int lane = threadIdx.x & 63;
    // entry l's head (and, read in place, its kept-frame count) into lane l,
    // with uniform indices into the launch arguments (a per-lane index would
    // copy them to private memory)
    int e = 0, kept = -1;
    for (int l = 0; l < a.heads.n; ++l)
        if (lane == l) {
            e = a.heads.head[l];
            if (PAGED) kept = a.st_kept[l];
        }
    int T = 0;
    if (lane < a.heads.n) {
        const int kvl = kept >= 0 ? kept * a.F : head_kvl(a, e);
        T = (kvl + a.Lq + BN - 1) / BN;
    }
    long long v = (long long)a.n_qtiles * T;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const long long u = __shfl_up(v, d, 64);
        if (lane >= d) v += u;
    }
    return WorkList{T, (int64_t)v};
}

// Tiles of all items before entry li.
__device__ __forceinline__ int64_t entry_base(const WorkList &wl, int li) {
    return li > 0 ? readlane64(wl.incl, li - 1) : 0;
}

// The item holding tile x (0 <= x < total) of the concatenated sequence: list
// entry li, its query tile qt, the item's first tile ibase and its tile count T.
struct ItemPos {
    int li, qt, T;
    int64_t ibase;
};
__device__ __forceinline__ ItemPos locate(const WorkList &wl, int64_t x) {
    const int li = (int)__builtin_ctzll(__ballot(wl.incl > x));   // first entry ending past x
    const int64_t base = entry_base(wl, li);
    const int T = __builtin_amdgcn_readlane(wl.T, li);
    const int qt = (int)((x - base) / T);
    return ItemPos{li, qt, T, base + (int64_t)qt * T};
}

__device__ __forceinline__ Schedule make_schedule(const AttnArgs &a, const WorkList &wl) {
    const int64_t total = readlane64(wl.incl, 63);
    Schedule sc;
    sc.total = total;
    sc.G = (int)(total < a.n_blocks ? total : a.n_blocks);
    return sc;
}

// Partial result of one part of an item, in a slot of BM*(D/2 + 2) floats:
// the part's own normalised output o/l rounded to bf16, in the accumulator
// layout of the waves (4 values per lane and uint2 index
// ((wave*MB + mb)*4 + g)*64 + lane), then the running max m (log2 units) of
// the BM rows, then their probability sums l.
template <int D>
__device__ __forceinline__ size_t slot_floats() { return (size_t)BM * (D / 2 + 2); }

__device__ __forceinline__ uint2 pack_bf16x4(float x0, float x1, float x2, float x3) {
    const uint32_t b0 = __builtin_bit_cast(uint16_t, (__bf16)x0), b1 = __builtin_bit_cast(uint16_t, (__bf16)x1);
    const uint32_t b2 = __builtin_bit_cast(uint16_t, (__bf16)x2), b3 = __builtin_bit_cast(uint16_t, (__bf16)x3);
    return make_uint2(b0 | (b1 << 16), b2 | (b3 << 16));
}

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

}  // namespace attn
}  // namespace fkv
