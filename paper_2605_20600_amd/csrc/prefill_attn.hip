// Causal self-attention over the conditional (prefix) tokens, the dense part
// of Step 1 (cache prefilling, Sec. 4): o_i = softmax(q_i K^T / sqrt(d), keys
// j <= i) V for the C prefix tokens of every (b, h), on the MFMA units of
// gfx950.
//
// A block of 4 wavefronts takes 128 queries of one head, one wavefront per 32
// of them.  The keys arrive in blocks of 128: the block's threads load one
// into LDS together (K and V rows, padded by 16 bytes against bank conflicts)
// with every load issued at once, so the head's keys cost one memory round
// trip per 128 rather than one per 32-key tile and wavefront.  For each tile
// of 32 keys at or before its queries, a wavefront computes
//   S^T = K_tile Q^T   32x32x16 bf16 MFMAs over d (A = key rows from LDS,
//                      B = the wavefront's query rows, held in registers), so
//                      that a lane holds 16 of the 32 scores of one query and
//                      the other 16 sit in lane l ^ 32;
//   online softmax     per query in fp32 (exp2 of pre-scaled scores), the
//                      running max shared by the lane pair;
//   O^T += V^T P^T     32x32x8 bf16 MFMAs: the score accumulators, rounded to
//                      bf16, are exactly the B operand of this shape; each
//                      lane reads its 4 keys of one dim from the LDS V rows.
// The normaliser sums the bf16-rounded weights that multiply V.  The same
// launch stores the prefix keys and values into the cache (headkv_prefill):
// the block of query tile t writes key block t from the registers it loaded
// it into.  Prefixes shorter than 128 tokens, where most of a key block would
// be clamped rows, take k_prefill_attn_tiles instead: each wavefront loads its
// own 32-key tiles (the same MFMA steps).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/headkv.h"
#include "device_common.h"
#include "layout.h"

namespace headkv {
namespace {

using namespace dev;

typedef short bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// fp32 -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint16_t bf16_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ bf16x8_t load8(const uint16_t* p) {
    const uint4 w = *reinterpret_cast<const uint4*>(p);
    return __builtin_bit_cast(bf16x8_t, w);
}

// grid: ceil(C / 128) x B*H blocks, the query tiles of a head adjacent;
// block: 256 threads = 4 wavefronts of 32 queries
// Each block also does Step 1's cache work for its head: the block of the
// first query tile resets the head's layer state, and every block stores the
// keys and values of its own 128 prefix rows into the cache.
template <int D>
__global__ __launch_bounds__(256) void k_prefill_attn_keys(LayerDev L, int nheads,
                                                      const uint16_t* __restrict__ qc,
                                                      const uint16_t* __restrict__ kc,
                                                      const uint16_t* __restrict__ vc,
                                                      float* __restrict__ out, int C,
                                                      float qscale, int64_t seg_bytes,
                                                      int dense_cap, int dense_chunks) {
    constexpr int KS = D / 16;            // 32x32x16 steps over d
    constexpr int MB = D / 32;            // 32-dim blocks of the output
    constexpr int CH = D / 8;             // 16-byte pieces of a row
    constexpr int PER = 128 * CH / 256;   // pieces of a 128-key block per thread (K or V)
    constexpr int PITCH = D + 8;          // LDS row pitch in bf16
    __shared__ __align__(16) uint16_t ks[128 * PITCH];
    __shared__ __align__(16) uint16_t vs[128 * PITCH];
    const int tiles = (C + 127) / 128;
    const int bh = blockIdx.x / tiles;
    const int tile = blockIdx.x - bh * tiles;
    prefill_head(L, bh, nheads, C, D, kc, vc, seg_bytes, dense_cap, dense_chunks, 0, 0, tile == 0,
                 threadIdx.x, 256);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int q0 = tile * 128 + wave * 32;
    const bool active = q0 < C;  // a wavefront past C still loads and meets the barriers
    const int half = lane >> 5, j = lane & 31;  // j: this lane's query (and key row of a tile)
    const size_t base = (size_t)bh * C * D;
    const uint16_t* Q = qc + base;
    const uint4* K4 = reinterpret_cast<const uint4*>(kc + base);
    const uint4* V4 = reinterpret_cast<const uint4*>(vc + base);
    const int qrow = min(q0 + j, C - 1);
    bf16x8_t qb[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qb[s] = load8(Q + (size_t)qrow * D + 16 * s + 8 * half);

    f32x16_t acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mb][r] = 0.f;
    float m = -INFINITY, lsum = 0.f;
    const int q = q0 + j;  // this lane's query
    const SegPtrs cache = seg_ptrs(L.kv + (int64_t)bh * seg_bytes, C, dense_cap, D);
    uint4* cK = reinterpret_cast<uint4*>(cache.K);
    uint4* cV = reinterpret_cast<uint4*>(cache.V);
    for (int kb = 0; kb <= tile; ++kb) {
        // keys kb*128 .. kb*128 + 127 (rows past C clamped to C - 1: finite,
        // and masked by the causal mask since every query is below C).  The
        // barrier comes first, and every row is loaded and written: otherwise
        // the compiler keeps the loaded rows in scratch memory, or sinks each
        // load into the branch that uses it and waits for them one at a time.
        if (kb > 0) __syncthreads();  // every wavefront is done with the previous block
        uint4 kr[PER], vr[PER];
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int c = tid + 256 * i, row = c / CH, col = c % CH;
            const size_t key = (size_t)min(kb * 128 + row, C - 1);
            kr[i] = K4[key * CH + col];
            vr[i] = V4[key * CH + col];
        }
        // every load out before the first write: the empty asm makes the
        // loaded values opaque, so that the register allocator cannot reload
        // them one at a time next to their writes
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            asm volatile("" : "+v"(kr[i].x), "+v"(kr[i].y), "+v"(kr[i].z), "+v"(kr[i].w));
            asm volatile("" : "+v"(vr[i].x), "+v"(vr[i].y), "+v"(vr[i].z), "+v"(vr[i].w));
        }
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int c = tid + 256 * i, row = c / CH, col = c % CH;
            *reinterpret_cast<uint4*>(ks + row * PITCH + col * 8) = kr[i];
            *reinterpret_cast<uint4*>(vs + row * PITCH + col * 8) = vr[i];
        }
        if (kb == tile) {  // this block's own prefix rows into the cache
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int c = tid + 256 * i, row = c / CH, col = c % CH;
                const int key = kb * 128 + row;
                if (key < C) {
                    cK[(size_t)key * CH + col] = kr[i];
                    cV[(size_t)key * CH + col] = vr[i];
                }
            }
        }
        __syncthreads();
        if (!active) continue;
        for (int t = 0; t < 4; ++t) {
            const int k0 = kb * 128 + 32 * t;
            if (k0 > q0 + 31 || k0 >= C) break;  // causal: tiles at or before the queries
            const uint16_t* kt = ks + (32 * t) * PITCH;
            const uint16_t* vt = vs + (32 * t) * PITCH;
            // S^T[key i][query j] for keys k0 .. k0 + 31
            f32x16_t st;
#pragma unroll
            for (int r = 0; r < 16; ++r) st[r] = 0.f;
#pragma unroll
            for (int s = 0; s < KS; ++s)
                st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    *reinterpret_cast<const bf16x8_t*>(kt + j * PITCH + 16 * s + 8 * half), qb[s],
                    st, 0, 0, 0);
            // keys of accumulator r: k0 + 8 (r / 4) + 4 half + r % 4; causal mask
            float mx = m;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = k0 + 8 * (r / 4) + 4 * half + (r & 3);
                st[r] = key <= q ? st[r] * qscale : -INFINITY;
                mx = fmaxf(mx, st[r]);
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float f = __builtin_amdgcn_exp2f(m - mx);  // m = -inf gives 0
            m = mx;
            lsum *= f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mb][r] *= f;
            // weights, rounded to bf16: B operands of the four 32x32x8 steps
            bf16x4_t pb[4];
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint16_t w = bf16_rne(__builtin_amdgcn_exp2f(st[4 * g + e] - mx));
                    lsum += __uint_as_float((uint32_t)w << 16);
                    pb[g][e] = (short)w;
                }
            // O^T[dim][query] += V^T[dim][key] P^T[key][query]
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    bf16x4_t va;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        va[e] = (short)vt[(8 * g + 4 * half + e) * PITCH + 32 * mb + j];
                    acc[mb] = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(va, pb[g], acc[mb], 0, 0, 0);
                }
        }
    }
    if (!active) return;
    lsum += __shfl_xor(lsum, 32);
    if (q >= C) return;
    const float inv = 1.f / lsum;
    float* o = out + base + (size_t)q * D;
    // accumulator r of block mb: dim 32 mb + 8 (r / 4) + 4 half + r % 4
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            float4 v;
            v.x = acc[mb][4 * g] * inv;
            v.y = acc[mb][4 * g + 1] * inv;
            v.z = acc[mb][4 * g + 2] * inv;
            v.w = acc[mb][4 * g + 3] * inv;
            *reinterpret_cast<float4*>(o + 32 * mb + 8 * g + 4 * half) = v;
        }
}

// A tile of 32 keys: the A operands of S^T (key row j, 16 dims per step, this
// half's 8 of them) and 16-byte pieces of the V rows.
template <int D>
struct KeyTile {
    bf16x8_t k[D / 16];
    uint4 v[32 / (64 / (D / 8))];
};

template <int D>
__device__ __forceinline__ KeyTile<D> load_tile(const uint16_t* K, const uint16_t* V, int t0, int j,
                                                int half, int lane, int C) {
    constexpr int LPR = D / 8, RPL = 64 / LPR;
    KeyTile<D> t;
    const int krow = min(t0 + j, C - 1);
#pragma unroll
    for (int s = 0; s < D / 16; ++s) t.k[s] = load8(K + (size_t)krow * D + 16 * s + 8 * half);
#pragma unroll
    for (int i = 0; i < 32 / RPL; ++i) {
        const int key = min(t0 + i * RPL + lane / LPR, C - 1);
        t.v[i] = *reinterpret_cast<const uint4*>(V + (size_t)key * D + (lane % LPR) * 8);
    }
    return t;
}

// Prefixes shorter than 128 tokens (one query tile per head; most of a key
// block would be clamped rows): each wavefront loads its own key tiles, one
// at a time, the V tile through its own LDS rows.  Grid and block as for
// k_prefill_attn_keys; the block copies its head's prefix rows into the cache.
template <int D>
__global__ __launch_bounds__(256) void k_prefill_attn_tiles(LayerDev L, int nheads,
                                                      const uint16_t* __restrict__ qc,
                                                      const uint16_t* __restrict__ kc,
                                                      const uint16_t* __restrict__ vc,
                                                      float* __restrict__ out, int C,
                                                      float qscale, int64_t seg_bytes,
                                                      int dense_cap, int dense_chunks) {
    constexpr int KS = D / 16;  // 32x32x16 steps over d
    constexpr int MB = D / 32;  // 32-dim blocks of the output
    const int tiles = (C + 127) / 128;
    const int bh = blockIdx.x / tiles;
    const int tile = blockIdx.x - bh * tiles;
    prefill_head(L, bh, nheads, C, D, kc, vc, seg_bytes, dense_cap, dense_chunks, tile * 128,
                 min(C, tile * 128 + 128), tile == 0, threadIdx.x, 256);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q0 = tile * 128 + wave * 32;
    if (q0 >= C) return;
    const int half = lane >> 5, j = lane & 31;  // j: this lane's query (and key row)
    const size_t base = (size_t)bh * C * D;
    const uint16_t* Q = qc + base;
    const uint16_t* K = kc + base;
    const uint16_t* V = vc + base;
    const int qrow = min(q0 + j, C - 1);
    bf16x8_t qb[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qb[s] = load8(Q + (size_t)qrow * D + 16 * s + 8 * half);

    f32x16_t acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mb][r] = 0.f;
    float m = -INFINITY, lsum = 0.f;
    const int q = q0 + j;                              // this lane's query
    const int k_last = min(q0 + 31, C - 1);            // last key any query here sees
    constexpr int LPR = D / 8;                         // lanes per V row (16 bytes each)
    constexpr int RPL = 64 / LPR;                      // V rows per wavefront load
    __shared__ __align__(16) uint16_t sv_all[4][32 * D];
    uint16_t* sv = sv_all[wave];                       // this wavefront's V tile [key][dim]
    for (int k0 = 0; k0 <= k_last; k0 += 32) {
        const KeyTile<D> cur = load_tile<D>(K, V, k0, j, half, lane, C);
        const bf16x8_t* kb = cur.k;
        const uint4* vrow = cur.v;
        // S^T[key i][query j] for keys k0 .. k0 + 31
        f32x16_t st;
#pragma unroll
        for (int r = 0; r < 16; ++r) st[r] = 0.f;
#pragma unroll
        for (int s = 0; s < KS; ++s)
            st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[s], qb[s], st, 0, 0, 0);
        // keys of accumulator r: k0 + 8 (r / 4) + 4 half + r % 4; causal mask
        float mx = m;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = k0 + 8 * (r / 4) + 4 * half + (r & 3);
            st[r] = key <= q ? st[r] * qscale : -INFINITY;
            mx = fmaxf(mx, st[r]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float f = __builtin_amdgcn_exp2f(m - mx);  // m = -inf gives 0
        m = mx;
        lsum *= f;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[mb][r] *= f;
        // weights, rounded to bf16: B operands of the four 32x32x8 steps
        bf16x4_t pb[4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint16_t w = bf16_rne(__builtin_amdgcn_exp2f(st[4 * g + e] - mx));
                lsum += __uint_as_float((uint32_t)w << 16);
                pb[g][e] = (short)w;
            }
        // O^T[dim][query] += V^T[dim][key] P^T[key][query]; the wavefront's
        // own LDS rows, so program order is the only ordering needed
#pragma unroll
        for (int i = 0; i < 32 / RPL; ++i)
            *reinterpret_cast<uint4*>(sv + (i * RPL + lane / LPR) * D + (lane % LPR) * 8) = vrow[i];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                bf16x4_t va;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    va[e] = (short)sv[(8 * g + 4 * half + e) * D + 32 * mb + j];
                acc[mb] = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(va, pb[g], acc[mb], 0, 0, 0);
            }
    }
    lsum += __shfl_xor(lsum, 32);
    if (q >= C) return;
    const float inv = 1.f / lsum;
    float* o = out + base + (size_t)q * D;
    // accumulator r of block mb: dim 32 mb + 8 (r / 4) + 4 half + r % 4
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            float4 v;
            v.x = acc[mb][4 * g] * inv;
            v.y = acc[mb][4 * g + 1] * inv;
            v.z = acc[mb][4 * g + 2] * inv;
            v.w = acc[mb][4 * g + 3] * inv;
            *reinterpret_cast<float4*>(o + 32 * mb + 8 * g + 4 * half) = v;
        }
}

inline int last_error() { return (int)hipGetLastError(); }

}  // namespace

int launch_prefill_attn(const LayerDev& L, const Shape& s, const uint16_t* qc, const uint16_t* kc,
                        const uint16_t* vc, float* out, int64_t dense_seg_bytes, int dense_cap,
                        int dense_chunks, void* stream, void* ev_start, void* ev_stop) {
    const dim3 grid((unsigned)((s.C + 127) / 128) * (unsigned)s.BH), block(256);
    const float qscale = (float)(1.4426950408889634 / std::sqrt((double)s.d));
    hipStream_t st = (hipStream_t)stream;
    hipEvent_t e0 = static_cast<hipEvent_t>(ev_start), e1 = static_cast<hipEvent_t>(ev_stop);
#define HEADKV_PREFILL_LAUNCH(KERNEL)                                                        \
    hipExtLaunchKernelGGL(KERNEL, grid, block, 0, st, e0, e1, 0, L, s.BH, qc, kc, vc, out, s.C, \
                          qscale, dense_seg_bytes, dense_cap, dense_chunks)
    if (s.C >= 128) {
        if (s.d == 128) HEADKV_PREFILL_LAUNCH(k_prefill_attn_keys<128>);
        else HEADKV_PREFILL_LAUNCH(k_prefill_attn_keys<64>);
    } else {
        if (s.d == 128) HEADKV_PREFILL_LAUNCH(k_prefill_attn_tiles<128>);
        else HEADKV_PREFILL_LAUNCH(k_prefill_attn_tiles<64>);
    }
#undef HEADKV_PREFILL_LAUNCH
    return last_error();
}

}  // namespace headkv
