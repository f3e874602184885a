// The decode-attention block of Eq. (1) over one head of the compressed cache,
// shared by the attention kernels and the fused update + attention kernel.
//
// A block of T threads is rows of d/8 lanes (16 at d = 128, 8 at d = 64); each
// row holds one token at a time, 8 elements per lane (one 16-byte load), so the
// rows of a wavefront read consecutive K or V rows of the segment (1 KB).  A
// pass covers T/(d/8) x TPR tokens: every load of the pass is issued before
// the first one is used (row indices past the end are clamped to the last
// token and their logits masked, so no load sits behind a branch), the K rows
// before the V rows.  K/V are read once per step, so the loads are
// non-temporal.  The softmax is online, with one running max per wavefront:
// the rows of a wavefront are summed with lane exchanges, and the wavefronts
// merged through LDS.  With an append, the step's token is attended from the
// input by wavefront 0 of the block whose range holds it (as the first token
// of its online softmax), which also writes it into the cache.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "device_common.h"
#include "layout.h"

namespace headkv {
namespace dev {

template <int D>
struct AttnRegs {
    static constexpr int LPR = D / 8;   // lanes per token row
    static constexpr int VPL = 8;       // bf16 elements per lane
    static constexpr int NW = VPL / 2;  // 32-bit words per lane
    using Vec = Words<NW>;
};

template <int NW>
__device__ __forceinline__ Words<NW> nt_load(const uint16_t* p) {
    typedef unsigned int vec_t __attribute__((ext_vector_type(NW)));
    const vec_t t = __builtin_nontemporal_load(reinterpret_cast<const vec_t*>(p));
    Words<NW> w;
#pragma unroll
    for (int e = 0; e < NW; ++e) w.w[e] = t[e];
    return w;
}

// Merge of the chunks of a head, column by column: lane tid < D of a chunk
// holds its column's normalised output o = sum_j p_j v_j / sum_j p_j and the
// chunk's log2-sum-exp s = m + log2(l).  Chunks are the leaves of a binary
// tree over chunk indices; at every inner node the two subtrees' (o, s) meet
// through one 64-bit atomic exchange on the node's word (the first to arrive
// leaves its pair there and is done; the second receives it, clears the word,
// merges left with right and goes up), and the chunk that completes the root
// writes the head's output.  The partner's data comes back in the atomic's
// own return value, so nothing waits for another chunk's stores, and the
// fixed left-right order makes the result independent of arrival order.  The
// node whose right subtree starts at chunk c owns the words of slot i0 + c
// (one per column; c = 1 .. nch - 1 name the nch - 1 inner nodes); a word is
// zero between launches, and a pair never packs to zero: its high half is
// bits(s) XOR kPartKey, a signalling-NaN pattern that no arithmetic result
// carries.
constexpr uint32_t kPartKey = 0x7fbadbadu;

__device__ __forceinline__ uint64_t pair_pack(float o, float s) {
    return ((uint64_t)(__float_as_uint(s) ^ kPartKey) << 32) | (uint64_t)__float_as_uint(o);
}
// (o, s) <- (o, s) merged with (ob, sb), in that order
__device__ __forceinline__ void pair_merge(float& o, float& s, float ob, float sb) {
    const float mx = fmaxf(s, sb);
    const float wa = __builtin_amdgcn_exp2f(s - mx);
    const float wb = __builtin_amdgcn_exp2f(sb - mx);
    const float w = wa + wb;
    o = (o * wa + ob * wb) / w;
    s = mx + __builtin_amdgcn_logf(w);
}

// Chunk c of the nch chunks of head h, column tid < D with (o, s): climbs the
// tree while it is the second to reach a node.  i0: the head's first slot
// (item_start[h]); part: D words per slot.
template <int D>
__device__ __forceinline__ void chunk_merge(int h, int nch, int c, int i0, float o, float s,
                                            float* __restrict__ out,
                                            uint64_t* __restrict__ part, int tid) {
    int c0 = c;  // first chunk of the subtree that (o, s) covers
    for (int lvl = 0;; ++lvl) {
        const int size = 1 << lvl;
        if (c0 == 0 && size >= nch) {
            out[(size_t)h * D + tid] = o;
            return;
        }
        const bool left = ((c0 >> lvl) & 1) == 0;
        const int right = left ? c0 + size : c0;  // first chunk of the right subtree
        if (right >= nch) continue;               // no right subtree: up a level
        uint64_t* w = part + (size_t)(i0 + right) * D + tid;
        const uint64_t other =
            __hip_atomic_exchange(w, pair_pack(o, s), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (other == 0) return;  // the other subtree's chunk goes on
        __hip_atomic_store(w, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        float ob = __uint_as_float((uint32_t)other);
        float sb = __uint_as_float((uint32_t)(other >> 32) ^ kPartKey);
        if (left) {
            pair_merge(o, s, ob, sb);
        } else {
            pair_merge(ob, sb, o, s);
            o = ob;
            s = sb;
            c0 -= size;
        }
    }
}

// Partial logit of one lane: its NW words of q and of a K row, bf16 pairs,
// multiplied and summed in fp32 (the products of bf16 values are exact in fp32)
template <int NW>
__device__ __forceinline__ float lane_dot(const uint32_t* qw, const Words<NW>& k) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    float dp = 0.f;
#pragma unroll
    for (int e = 0; e < NW; ++e)
        dp = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, qw[e]),
                                             __builtin_bit_cast(bf16x2_t, k.w[e]), dp, false);
    return dp;
}

// Row padding (floats) of the end-of-block merge buffer: lane g of a column
// reads row g * wpg + k, so rows wpg apart must start 64 / g_lanes banks
// apart (64 banks of 4 bytes) for the g_lanes lanes of a column to read
// without conflicts
constexpr int merge_pad(int wpg, int d, int g_lanes) {
    if (g_lanes == 1) return 0;
    for (int pad = 0; pad < 64; ++pad)
        if ((wpg * (d + pad)) % 64 == 64 / g_lanes) return pad;
    return -1;
}

// Online-softmax update of one row's state with NT tokens t0 + j * ROWS + row
// (those at or past t_end masked); k/v hold the lane's 8 elements of each row.
// The running max is the wavefront's (the same in all its rows), taken over
// the logits before the V rows are used, so that the rows of a wavefront
// merge at the end by plain sums.  In two halves: the logits and the new
// running max from the K rows, then the weights and their V rows.
template <int D, int NT, int ROWS>
__device__ __forceinline__ float attn_logits(const typename AttnRegs<D>::Vec (&kk)[NT], int t0,
                                             int row, int t_end, const uint32_t* qw, float qscale,
                                             float m, float (&s)[NT]) {
    constexpr int NW = AttnRegs<D>::NW;
    float mx = m;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const float dp = lanes_sum<AttnRegs<D>::LPR>(lane_dot<NW>(qw, kk[j])) * qscale;
        s[j] = (t0 + j * ROWS + row < t_end) ? dp : -INFINITY;
        mx = fmaxf(mx, s[j]);
    }
    // the wavefront's max: the row sums leave the same value in every lane of
    // a row (each of their steps adds a symmetric pair of lanes), so one lane
    // per row is read directly instead of exchanging through LDS
    constexpr int LPR = AttnRegs<D>::LPR;
    float wm = mx;
#pragma unroll
    for (int r = 0; r < 64 / LPR; ++r)
        wm = fmaxf(wm, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mx), r * LPR)));
    return wm;
}

template <int D, int NT>
__device__ __forceinline__ void attn_weigh(const typename AttnRegs<D>::Vec (&vv)[NT],
                                           const float (&s)[NT], float mx, float& m, float& l,
                                           float* acc) {
    constexpr int NW = AttnRegs<D>::NW;
    constexpr int VPL = AttnRegs<D>::VPL;
    if (mx != -INFINITY) {
        const float f = __builtin_amdgcn_exp2f(m - mx);  // m = -inf gives 0
        l *= f;
#pragma unroll
        for (int e = 0; e < VPL; ++e) acc[e] *= f;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const float p = __builtin_amdgcn_exp2f(s[j] - mx);
            l += p;
#pragma unroll
            for (int e = 0; e < NW; ++e) {
                acc[2 * e] += p * bf_lo(vv[j].w[e]);
                acc[2 * e + 1] += p * bf_hi(vv[j].w[e]);
            }
        }
        m = mx;
    }
}

template <int D, int NT, int ROWS>
__device__ __forceinline__ void attn_accumulate(const typename AttnRegs<D>::Vec (&kk)[NT],
                                                const typename AttnRegs<D>::Vec (&vv)[NT],
                                                int t0, int row, int t_end,
                                                const uint32_t* qw, float qscale,
                                                float& m, float& l, float* acc) {
    float s[NT];
    const float mx = attn_logits<D, NT, ROWS>(kk, t0, row, t_end, qw, qscale, m, s);
    attn_weigh<D, NT>(vv, s, mx, m, l, acc);
}

// The work of one attention block; `item` is its index among the blocks of
// the layer.  TPR tokens per row and pass: 8, or 4 (6) when every head fits
// in half (three quarters of) a pass, or 9 when that gives one pass where 8
// would need two.
template <int D, bool APPEND, int T, bool CHUNKED, int TPR>
__device__ __forceinline__ void attn_block(const LayerDev& L, int C, const AppendArgs& a,
                                           const uint16_t* __restrict__ q,
                                           float* __restrict__ out, uint64_t* __restrict__ part,
                                           int use_order, int order_base, int pad_len,
                                           float qscale, int item, int n_given = -1) {
    using Vec = typename AttnRegs<D>::Vec;
    constexpr int VPL = AttnRegs<D>::VPL;
    constexpr int NW = AttnRegs<D>::NW;
    constexpr int LPR = AttnRegs<D>::LPR;
    constexpr int ROWS = T / LPR;
    constexpr int TP = ROWS * TPR;  // tokens per pass
    constexpr int WAVES = T / 64;
    int h, chunk = 0;
    if (CHUNKED) {
        const uint32_t it = L.items[item];
        h = (int)(it >> 8);
        chunk = (int)(it & 255u);
    } else {
        // through a vector load: a scalar one would leave its wait at the
        // join of the two paths, where it also waits for the kernel arguments
        // still in flight, and the block's first metadata loads would follow
        // them on the path without the order as well
        h = item;
        if (use_order) {
            int lane0 = 0;
            asm("" : "+v"(lane0));
            h = __builtin_amdgcn_readfirstlane(L.order[order_base + item + lane0]);
        }
    }
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = tid / LPR, col = tid % LPR;
    // the head's segment, capacity and length, read together up front
    const int64_t seg = L.seg_off[h];
    const int cap = L.cap[h];
    // n_given: the length as the caller already knows it (a kernel that has
    // just changed it), else the one in memory
    const int n = n_given >= 0 ? n_given : head_len(L, h);
    const int i0 = CHUNKED ? L.item_start[h] : 0;  // the head's first chunk slot
    // Everything the first K/V load waits for comes in one round of scalar
    // loads when the kernel preloads its leading arguments (the metadata, with
    // the rest of the arguments), else two (the arguments first).  Left to
    // itself, the compiler fetches arguments late, each behind the previous
    // wait (up to four rounds); an empty asm statement that takes these values
    // pins them before any load that follows.  (Placed before the metadata
    // loads, it would make them vector loads.)
    asm volatile("" ::"s"(q), "s"(seg), "s"(cap), "s"(n), "s"(C), "s"(pad_len), "s"(qscale));
    if (CHUNKED) asm volatile("" ::"s"(i0), "s"(part));
    if (APPEND) asm volatile("" ::"s"(a.k), "s"(a.v), "s"(L.qring), "s"(L.ring_len));
    const Vec qraw = *reinterpret_cast<const Vec*>(q + (size_t)h * D + col * VPL);
    // the cache holds len_c tokens; with the append, the step's token is
    // attended as token len_c, from the input
    const int len_c = C + n;
    const int len = len_c + (APPEND ? 1 : 0);
    // chunked: the fewest chunks of at most one pass that hold the head's
    // tokens take part, with equal shares of them (the later table entries of
    // the head have nothing to do), and the only chunk of a head that fits in
    // one writes the output itself, without partials
    const int nch = len > TP ? (len + TP - 1) / TP : 1;
    const int per = (len + nch - 1) / nch;  // at most TP
    if (CHUNKED && chunk >= nch) return;
    const int t_begin = CHUNKED ? chunk * per : 0;
    const int t_end = CHUNKED ? min(len, t_begin + per) : len;
    // cache rows this block streams: [t_begin, s_end); the padding strategy
    // reads the rows of the layer's longest head (pad_len attended tokens, the
    // appended one included, which comes from the input), those past s_end
    // masked
    const int s_end = min(t_end, len_c);
    const int s_stop = CHUNKED ? s_end : max(s_end, pad_len - (APPEND ? 1 : 0));
    // the block whose range holds the new token (always the one block of a head
    // that is not chunked) performs the append; its wavefront 0 attends the
    // token and moves its K/V row.  The head's length is not stored: the host
    // counts the appended tokens
    const bool owner = APPEND && (!CHUNKED || (t_begin <= len_c && len_c < t_end));
    const bool newtok = owner && wave == 0;
    uint16_t* K = reinterpret_cast<uint16_t*>(L.kv + seg);
    uint16_t* V = K + (size_t)(C + cap) * D;

    // the append's loads (the new token's K/V row, by wavefront 0) go out
    // before the K/V stream and its stores right after it
    Vec kn, vn;
    if (newtok) {
        kn = *reinterpret_cast<const Vec*>(a.k + (size_t)h * D + col * VPL);
        vn = *reinterpret_cast<const Vec*>(a.v + (size_t)h * D + col * VPL);
    }
    float m = -INFINITY, l = 0.f;
    float acc[VPL];
#pragma unroll
    for (int e = 0; e < VPL; ++e) acc[e] = 0.f;
    uint32_t qw[NW];
    // q's bf16 pairs (the logits are scaled after the dot products); then the
    // append's stores, and the new token as the first token of the softmax:
    // every row of wavefront 0 holds its K/V row, so each computes its logit
    // and takes it as the starting max; row 0 counts it and writes its K/V
    // row, its position and q's row of the query ring
    auto begin = [&]() {
        // an opaque copy of q, so that its use (common to both branches
        // below) is not hoisted in front of the K/V loads, where it would
        // wait for q
        Vec qv = qraw;
        static_assert(NW == 4, "four words per lane");
        asm volatile("" : "+v"(qv.w[0]), "+v"(qv.w[1]), "+v"(qv.w[2]), "+v"(qv.w[3]));
#pragma unroll
        for (int e = 0; e < NW; ++e) qw[e] = qv.w[e];
        if (newtok) {
            m = lanes_sum<LPR>(lane_dot<NW>(qw, kn)) * qscale;
            if (row == 0) {
                *reinterpret_cast<Vec*>(K + (size_t)len_c * D + col * VPL) = kn;
                *reinterpret_cast<Vec*>(V + (size_t)len_c * D + col * VPL) = vn;
                *reinterpret_cast<Vec*>(ring_slot(L, D, h, a.step) + col * VPL) = qraw;
                if (col == 0) reinterpret_cast<int32_t*>(V + (size_t)(C + cap) * D)[n] = a.step;
                l = 1.f;
#pragma unroll
                for (int e = 0; e < NW; ++e) {
                    acc[2 * e] = bf_lo(vn.w[e]);
                    acc[2 * e + 1] = bf_hi(vn.w[e]);
                }
            }
        }
    };
    // first pass, straight-line code from its loads to its use (a join in
    // between would make the compiler wait for every load at it): all K rows,
    // then all V rows, so that the logits and their max are computed while the
    // V rows are still arriving.  A chunk past the head's cached length reads
    // nothing.
    Vec kk[TPR], vv[TPR];
    auto load_k = [&](int t0) {
#pragma unroll
        for (int j = 0; j < TPR; ++j)
            kk[j] = nt_load<NW>(K + (size_t)min(t0 + j * ROWS + row, s_stop - 1) * D + col * VPL);
    };
    auto load_v = [&](int t0) {
#pragma unroll
        for (int j = 0; j < TPR; ++j)
            vv[j] = nt_load<NW>(V + (size_t)min(t0 + j * ROWS + row, s_stop - 1) * D + col * VPL);
    };
    // a head longer than one pass (only at 8 or 6 tokens per row: the other
    // widths are picked when every head fits in one pass, and a chunk holds
    // at most one) requests the next pass's K rows as soon as
    // this pass's logits are taken, and its V rows once this pass's are
    // accumulated, so that the stream runs on across passes; every request
    // is unconditional, so that no join makes the compiler wait for all
    constexpr bool kPipe = (TPR == kAttnTpr || TPR == kAttnTprShort) && !CHUNKED;
    int t0 = t_begin;
    if (t_begin < s_stop) {
        load_k(t_begin);
        load_v(t_begin);
        // keep every load of the pass ahead of its first use
        __builtin_amdgcn_sched_barrier(0);
        begin();
        if constexpr (kPipe) {
            for (; t0 + TP < s_stop; t0 += TP) {
                float s[TPR];
                const float mx = attn_logits<D, TPR, ROWS>(kk, t0, row, s_end, qw, qscale, m, s);
                load_k(t0 + TP);
                __builtin_amdgcn_sched_barrier(0);
                attn_weigh<D, TPR>(vv, s, mx, m, l, acc);
                load_v(t0 + TP);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        attn_accumulate<D, TPR, ROWS>(kk, vv, t0, row, s_end, qw, qscale, m, l, acc);
    } else {
        begin();
    }
    if constexpr (!kPipe) {
        for (t0 += TP; t0 < s_stop; t0 += TP) {
            load_k(t0);
            load_v(t0);
            __builtin_amdgcn_sched_barrier(0);
            attn_accumulate<D, TPR, ROWS>(kk, vv, t0, row, s_end, qw, qscale, m, l, acc);
        }
    }
    // merge the rows of each wavefront: they share its max, so by sums; every
    // exchange of a step is issued before the first is used
#pragma unroll
    for (int off = LPR; off <= 32; off <<= 1) {
        const float lo = __shfl_xor(l, off);
        float ao[VPL];
#pragma unroll
        for (int e = 0; e < VPL; ++e) ao[e] = __shfl_xor(acc[e], off);
        __builtin_amdgcn_sched_barrier(0);
        l += lo;
#pragma unroll
        for (int e = 0; e < VPL; ++e) acc[e] += ao[e];
    }
    // G adjacent lanes per output column merge the wavefronts' partials
    // below: 4 in a 1024-thread block that owns its CU, where the tail of the
    // merge is the launch's; 1 elsewhere (in 512-thread blocks, two to a CU,
    // and with the chunk merge's atomics after it, spreading it measured
    // slower).  The rows of sacc are padded so that the G lanes of a column,
    // which read different rows, fall in different LDS banks.
    constexpr int G = (!CHUNKED && T == 1024 && T / D >= 4) ? 4 : 1;
    constexpr int WPG = WAVES / G;
    static_assert(WAVES % G == 0 && G * D <= T, "merge groups");
    constexpr int PAD = merge_pad(WPG, D, G);
    static_assert(PAD >= 0, "no conflict-free padding");
    __shared__ float sm[WAVES], sl[WAVES];
    __shared__ float sacc[WAVES][D + PAD];
    if (lane < LPR) {
#pragma unroll
        for (int e = 0; e < VPL; ++e) sacc[wave][col * VPL + e] = acc[e];
        if (lane == 0) {
            sm[wave] = m;
            sl[wave] = l;
        }
    }
    __syncthreads();
    // each of a column's G lanes merges WAVES / G of the wavefronts'
    // partials, then the G lanes are combined with DPP steps: the merge at
    // the very end of the block, where every serial step adds to the launch,
    // is spread over G times the lanes.  All LDS reads are issued first.
    if (tid < G * D) {
        const int c = tid / G, g = tid % G;
        float mw[WPG], lw[WPG], xw[WPG];
#pragma unroll
        for (int k = 0; k < WPG; ++k) {
            mw[k] = sm[g * WPG + k];
            lw[k] = sl[g * WPG + k];
            xw[k] = sacc[g * WPG + k][c];
        }
        __builtin_amdgcn_sched_barrier(0);
        float mx = -INFINITY;
#pragma unroll
        for (int k = 0; k < WPG; ++k) mx = fmaxf(mx, mw[k]);
        // the column's max over its G lanes (symmetric pairs: the same value
        // in all of them)
        if (G >= 2)
            mx = fmaxf(mx, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(mx), 0xB1, 0xF, 0xF, false)));
        if (G >= 4)
            mx = fmaxf(mx, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(mx), 0x4E, 0xF, 0xF, false)));
        float o = 0.f, z = 0.f;
#pragma unroll
        for (int k = 0; k < WPG; ++k) {
            const float f = (mw[k] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw[k] - mx);
            o += f * xw[k];
            z += f * lw[k];
        }
        if (G >= 2) {
            o += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(o), 0xB1, 0xF, 0xF, false));
            z += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(z), 0xB1, 0xF, 0xF, false));
        }
        if (G >= 4) {
            o += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(o), 0x4E, 0xF, 0xF, false));
            z += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(z), 0x4E, 0xF, 0xF, false));
        }
        if (g == 0) {
            if (!CHUNKED || nch == 1)
                out[(size_t)h * D + c] = o / z;
            else
                chunk_merge<D>(h, nch, chunk, i0, o / z, mx + __builtin_amdgcn_logf(z),
                               out, part, c);
        }
    }
}

}  // namespace dev
}  // namespace headkv
