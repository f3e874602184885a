// Device helpers shared by the cache kernels and the attention kernels:
// bf16 unpacking, 16-lane row sums, block scans, the per-head segment view and
// the append of a step's token.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "layout.h"

namespace headkv {
namespace dev {

template <int NW>
struct alignas(NW * 4) Words {
    uint32_t w[NW];
};

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ __forceinline__ double bf_f64(uint16_t b) {
    return (double)__uint_as_float((uint32_t)b << 16);
}

// Sum over groups of N = 8 or 16 lanes (half or whole DPP rows): quad swaps,
// then the half-row mirror and, for 16, the row mirror; every lane of the
// group ends with the group's sum.
template <int N>
__device__ __forceinline__ float lanes_sum(float v) {
    static_assert(N == 8 || N == 16, "8 or 16 lanes");
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
    if (N == 16)
        v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
    return v;
}

// Inclusive prefix sum over the 64 lanes of a wavefront (all active): within
// each row of 16 lanes by DPP row shifts (lanes whose source lies outside
// the row add 0), then the totals of the rows before, read from lanes 15, 31
// and 47 (no exchange through LDS)
__device__ __forceinline__ int wave_inclusive_scan(int x) {
    int v = x;
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
    const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
              r2 = __builtin_amdgcn_readlane(v, 47);
    const int row = (threadIdx.x & 63) >> 4;
    return v + (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
}

// Exclusive prefix sum over a block of NT threads (256 by default);
// *total receives the sum.  Every thread of the block must call it.
template <int NT = kBlock>
__device__ inline int block_exclusive_scan(int x, int* total) {
    __shared__ int wsum[NT / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int inc = wave_inclusive_scan(x);
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
        off += w < wave ? wsum[w] : 0;
        tot += wsum[w];
    }
    __syncthreads();
    *total = tot;
    return off + inc - x;
}

struct SegPtrs {
    uint16_t* K;
    uint16_t* V;
    int32_t* pos;
};

__device__ __forceinline__ SegPtrs seg_ptrs(char* seg, int C, int cap, int d) {
    SegPtrs p;
    p.K = reinterpret_cast<uint16_t*>(seg);
    p.V = p.K + (size_t)(C + cap) * d;
    p.pos = reinterpret_cast<int32_t*>(p.V + (size_t)(C + cap) * d);
    return p;
}

// ------------------------------------------------------------------- append
// K <- [K, k_t], V <- [V, v_t] for head h by the threads tid < d of a block:
// row C+n, pos[n] = step, and q_t into the head's ring of the last P queries
// (the window an update scores against, Eq. 6).  Split in a load half and a
// store half so that a caller can put other loads between them.  The length
// itself is not stored: the host counts the appended tokens (LayerDev::dn),
// and only prefill and the periodic update write n.  The load half only
// issues loads (no loaded value is used before the store half), so that a
// caller's loads are not held behind their latency.
struct AppendVals {
    uint16_t k = 0, v = 0, qbits = 0;
};

__device__ __forceinline__ uint16_t* ring_slot(const LayerDev& L, int d, int h, int step) {
    return L.qring + ((size_t)h * L.ring_len + step % L.ring_len) * d;
}

__device__ __forceinline__ AppendVals append_load(int d, int h, const AppendArgs& a, int tid) {
    AppendVals r;
    if (tid < d) {
        r.qbits = a.q[(size_t)h * d + tid];
        r.k = a.k[(size_t)h * d + tid];
        r.v = a.v[(size_t)h * d + tid];
    }
    return r;
}

__device__ __forceinline__ void append_store(const LayerDev& L, int C, int d, int h, int n,
                                             const AppendArgs& a, const AppendVals& r, int tid) {
    if (tid >= d) return;
    SegPtrs s = seg_ptrs(L.kv + L.seg_off[h], C, L.cap[h], d);
    const size_t row = (size_t)(C + n) * d;
    s.K[row + tid] = r.k;
    s.V[row + tid] = r.v;
    ring_slot(L, d, h, a.step)[tid] = r.qbits;
    if (tid == 0) s.pos[n] = a.step;
}

__device__ __forceinline__ void append_token(const LayerDev& L, int C, int d, int h, int n,
                                             const AppendArgs& a, int tid) {
    append_store(L, C, d, h, n, a, append_load(d, h, a, tid), tid);
}

// Current length of head h: n as the last kernel that set it wrote it, plus
// the tokens appended since (one per step, for every head alike).
__device__ __forceinline__ int head_len(const LayerDev& L, int h) { return L.n[h] + L.dn; }

// Step 1 for head h of the dense layout, by the nthreads threads of a block:
// layer state reset (segment, capacity, length 0, labels, the dense chunk
// table) and, for prefix rows [r0, r1), the copy of the
// conditional keys and values into the head's first rows.
__device__ inline void prefill_head(const LayerDev& L, int h, int nheads, int C, int d,
                                    const uint16_t* kc, const uint16_t* vc, int64_t seg_bytes,
                                    int dense_cap, int dense_chunks, int r0, int r1,
                                    bool reset, int tid, int nthreads) {
    if (reset) {
        for (int c = tid; c < dense_chunks; c += nthreads)
            L.items[(size_t)h * dense_chunks + c] = ((uint32_t)h << 8) | (uint32_t)c;
        if (tid == 0) {
            L.item_start[h] = h * dense_chunks;
            if (h == nheads - 1) L.item_start[h + 1] = (h + 1) * dense_chunks;
            L.seg_off[h] = (int64_t)h * seg_bytes;
            L.cap[h] = dense_cap;
            L.n[h] = 0;
            L.budget[h] = 0;
            L.nstar[h] = 0;
            L.label[h] = 0;
            L.order[h] = h;
        }
    }
    if (r1 <= r0) return;
    SegPtrs s = seg_ptrs(L.kv + (int64_t)h * seg_bytes, C, dense_cap, d);
    const int w = d / 8;  // 16-byte pieces per row
    const uint4* ks = reinterpret_cast<const uint4*>(kc + (size_t)h * C * d);
    const uint4* vs = reinterpret_cast<const uint4*>(vc + (size_t)h * C * d);
    uint4* kd = reinterpret_cast<uint4*>(s.K);
    uint4* vd = reinterpret_cast<uint4*>(s.V);
    for (int i = r0 * w + tid; i < r1 * w; i += nthreads) {
        kd[i] = ks[i];
        vd[i] = vs[i];
    }
}

}  // namespace dev
}  // namespace headkv
