// Decode attention over the ragged compressed cache, Eq. (1), written for
// gfx950 (CDNA4: 64-lane wavefronts, 16 wavefronts of 128 VGPRs per CU).
//
//   k_attn   one block per work item.  A work item is either a whole head
//            (every pass over its tokens) or one chunk of a head of at most
//            one pass, taken from the layer's chunk table; optionally fused
//            with the step's append.  Whole heads may come from a range of the
//            dispatch order (one head group per launch) and may read up to a
//            padded length with the rows past their own length masked (the
//            other two strategies of Sec. 5.1 for heads of unequal length).
//   k_merge  merge of the chunks of every head of a chunked launch, and the
//            commit of the fused append's length.
//
// A block of T threads is rows of d/8 lanes (16 at d = 128, 8 at d = 64); each
// row holds one token at a time, 8 elements per lane (one 16-byte load), so the
// rows of a wavefront read consecutive K or V rows of the segment (1 KB).  A
// pass covers T/(d/8) x kAttnTpr tokens (512 at T = 1024 and d = 128, 1024 at
// d = 64): every load of the pass is issued
// before the first one is used (row indices past the end are clamped to the
// last token and their logits masked, so no load sits behind a branch).  K/V
// are read once per step, so the loads are non-temporal.  The softmax is
// online per row; rows are merged with cross-lane swaps and the wavefronts
// through LDS.  With an append, the step's token is attended from the input
// and written into the cache by the block whose range holds it.
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

// Online-softmax update of one row's state with NT tokens t0 + j * ROWS + row
// (those at or past t_end masked); k/v hold their d/16 elements of the lane.
template <int D, int NT, int ROWS>
__device__ __forceinline__ void attn_accumulate(const typename AttnRegs<D>::Vec (&kk)[NT],
                                                const typename AttnRegs<D>::Vec (&vv)[NT],
                                                int t0, int row, int t_end, const float* qf,
                                                float& m, float& l, float* acc) {
    constexpr int NW = AttnRegs<D>::NW;
    constexpr int VPL = AttnRegs<D>::VPL;
    float s[NT];
    float mx = m;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        float dp = 0.f;
#pragma unroll
        for (int e = 0; e < NW; ++e) {
            dp += qf[2 * e] * bf_lo(kk[j].w[e]);
            dp += qf[2 * e + 1] * bf_hi(kk[j].w[e]);
        }
        dp = lanes_sum<AttnRegs<D>::LPR>(dp);
        s[j] = (t0 + j * ROWS + row < t_end) ? dp : -INFINITY;
        mx = fmaxf(mx, s[j]);
    }
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

// The work of one attention block; `item` is its index among the blocks of
// the layer.  TPR tokens per row and pass: 8, or 4 when every head fits in
// half a pass, or 9 when that gives one pass where 8 would need two.
template <int D, bool APPEND, int T, bool CHUNKED, int TPR>
__device__ __forceinline__ void attn_block(const LayerDev& L, int C, const AppendArgs& a,
                                           const uint16_t* __restrict__ q,
                                           float* __restrict__ out, float* __restrict__ part,
                                           int use_order, int order_base, int pad_len,
                                           float qscale, int item) {
    using Vec = typename AttnRegs<D>::Vec;
    constexpr int VPL = AttnRegs<D>::VPL;
    constexpr int NW = AttnRegs<D>::NW;
    constexpr int LPR = AttnRegs<D>::LPR;
    constexpr int ROWS = T / LPR;
    constexpr int TP = ROWS * TPR;  // tokens per pass
    constexpr int WAVES = T / 64;
    int h, t_begin;
    if (CHUNKED) {
        const uint32_t it = L.items[item];
        h = (int)(it >> 8);
        t_begin = (int)(it & 255u) * TP;
    } else {
        h = use_order ? L.order[order_base + item] : item;
        t_begin = 0;
    }
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = tid / LPR, col = tid % LPR;
    const Vec qraw = *reinterpret_cast<const Vec*>(q + (size_t)h * D + col * VPL);
    const int n = L.n[h];
    const int len = C + n + (APPEND ? 1 : 0);
    const int t_end = CHUNKED ? min(len, t_begin + TP) : len;
    // padding strategy: rows up to pad_len are read, those past len masked
    const int t_stop = CHUNKED ? t_end : max(len, pad_len);
    // the block whose range holds the new token (always the one block of a head
    // that is not chunked) performs the append
    const bool owner = APPEND && (!CHUNKED || (t_begin <= len - 1 && len - 1 < t_end));
    const uint16_t* K = reinterpret_cast<const uint16_t*>(L.kv + L.seg_off[h]);
    const uint16_t* V = K + (size_t)(C + L.cap[h]) * D;
    // K (or V) row of token `tok`: the step's new token comes from the input
    auto krow = [&](int tok) {
        return (APPEND && tok == len - 1) ? a.k + (size_t)h * D : K + (size_t)tok * D;
    };
    auto vrow = [&](int tok) {
        return (APPEND && tok == len - 1) ? a.v + (size_t)h * D : V + (size_t)tok * D;
    };

    // the append's loads go out before the K/V stream and its stores right
    // after (the attention reads the new token from the input, never from row
    // C+n); n itself changes once no block reads it
    AppendVals av;
    if (owner) av = append_load(L, D, h, a, tid);
    float m = -INFINITY, l = 0.f;
    float acc[VPL];
#pragma unroll
    for (int e = 0; e < VPL; ++e) acc[e] = 0.f;
    float qf[VPL];
    // first pass: the append's store and q's conversion go between its loads
    // and their first use
    if (t_begin < t_stop) {  // a chunk past the head's length reads nothing
        Vec kk[TPR], vv[TPR];
        // all K rows of the pass, then all V rows: the logits and their max
        // are computed while the V rows are still arriving
#pragma unroll
        for (int j = 0; j < TPR; ++j)
            kk[j] = nt_load<NW>(krow(min(t_begin + j * ROWS + row, t_stop - 1)) + col * VPL);
#pragma unroll
        for (int j = 0; j < TPR; ++j)
            vv[j] = nt_load<NW>(vrow(min(t_begin + j * ROWS + row, t_stop - 1)) + col * VPL);
        // keep every load of the pass ahead of its first use
        __builtin_amdgcn_sched_barrier(0);
        if (owner) append_store(L, C, D, h, n, a, av, tid);
#pragma unroll
        for (int e = 0; e < NW; ++e) {
            qf[2 * e] = bf_lo(qraw.w[e]) * qscale;
            qf[2 * e + 1] = bf_hi(qraw.w[e]) * qscale;
        }
        attn_accumulate<D, TPR, ROWS>(kk, vv, t_begin, row, t_end, qf, m, l, acc);
    }
    // further passes of a head longer than one pass
    for (int t0 = t_begin + TP; t0 < t_stop; t0 += TP) {
        Vec kk[TPR], vv[TPR];
#pragma unroll
        for (int j = 0; j < TPR; ++j)
            kk[j] = nt_load<NW>(krow(min(t0 + j * ROWS + row, t_stop - 1)) + col * VPL);
#pragma unroll
        for (int j = 0; j < TPR; ++j)
            vv[j] = nt_load<NW>(vrow(min(t0 + j * ROWS + row, t_stop - 1)) + col * VPL);
        __builtin_amdgcn_sched_barrier(0);
        attn_accumulate<D, TPR, ROWS>(kk, vv, t0, row, t_end, qf, m, l, acc);
    }
    // merge the rows of each wavefront
#pragma unroll
    for (int off = LPR; off <= 32; off <<= 1) {
        const float mo = __shfl_xor(m, off);
        const float lo = __shfl_xor(l, off);
        const float mn = fmaxf(m, mo);
        const float fa = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m - mn);
        const float fb = (mo == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mo - mn);
        l = l * fa + lo * fb;
#pragma unroll
        for (int e = 0; e < VPL; ++e) {
            const float ao = __shfl_xor(acc[e], off);
            acc[e] = acc[e] * fa + ao * fb;
        }
        m = mn;
    }
    __shared__ float sm[WAVES], sl[WAVES];
    __shared__ float sacc[WAVES][D];
    if (lane < LPR) {
#pragma unroll
        for (int e = 0; e < VPL; ++e) sacc[wave][col * VPL + e] = acc[e];
        if (lane == 0) {
            sm[wave] = m;
            sl[wave] = l;
        }
    }
    __syncthreads();  // every wavefront has read n before the append changes it
    if (owner && !CHUNKED) append_commit(L, h, n, tid);
    if (tid < D) {
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) mx = fmaxf(mx, sm[w]);
        float o = 0.f, z = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            const float f = (sm[w] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(sm[w] - mx);
            o += f * sacc[w][tid];
            z += f * sl[w];
        }
        if (!CHUNKED) {
            out[(size_t)h * D + tid] = o / z;
        } else {
            float* pp = part + (size_t)item * (D + 2);
            pp[tid] = o;
            if (tid == 0) {
                pp[D] = mx;
                pp[D + 1] = z;
            }
        }
    }
}

// 4 wavefronts per SIMD (16 per CU) at every block size: at most 128 VGPRs.
template <int D, bool APPEND, int T, bool CHUNKED, int TPR>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(4))) void k_attn(
    LayerDev L, int C, AppendArgs a, const uint16_t* __restrict__ q, float* __restrict__ out,
    float* __restrict__ part, int use_order, int order_base, int pad_len, float qscale) {
    attn_block<D, APPEND, T, CHUNKED, TPR>(L, C, a, q, out, part, use_order, order_base, pad_len,
                                           qscale, (int)blockIdx.x);
}

// Several layers in one launch: layer blockIdx.x / BH, head blockIdx.x % BH.
template <int D, int T, int TPR>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(4))) void k_attn_layers(
    LayersArg args, MetaLayout ml, int BH, int C, float qscale) {
    const int layer = (int)blockIdx.x / BH;
    const LayerDev L = make_layer_dev(args.kv[layer], args.meta[layer], ml);
    const AppendArgs none{};
    attn_block<D, false, T, false, TPR>(L, C, none, args.q[layer], args.out[layer], nullptr, 0, 0,
                                        0, qscale, (int)blockIdx.x - layer * BH);
}

// Merge of the chunks of every head: a kernel of its own, since plain device
// memory is only coherent across the XCDs' L2 caches at kernel boundaries.
// With `commit`, the length grows by the token the attention appended.
template <int D>
__global__ __launch_bounds__(D) void k_merge(LayerDev L, float* __restrict__ out,
                                             const float* __restrict__ part, int commit) {
    constexpr int PS = D + 2;
    const int h = blockIdx.x, tid = threadIdx.x;
    const int i0 = L.item_start[h], i1 = L.item_start[h + 1];
    float mx = -INFINITY;
    for (int i = i0; i < i1; ++i) mx = fmaxf(mx, part[(size_t)i * PS + D]);
    float num = 0.f, den = 0.f;
    for (int i = i0; i < i1; ++i) {
        const float mi = part[(size_t)i * PS + D];
        if (mi != -INFINITY) {
            const float f = __builtin_amdgcn_exp2f(mi - mx);
            num += f * part[(size_t)i * PS + tid];
            den += f * part[(size_t)i * PS + D + 1];
        }
    }
    out[(size_t)h * D + tid] = num / den;
    if (commit && tid == 0) L.n[h] = L.n[h] + 1;
}

inline int last_error() { return (int)hipGetLastError(); }

template <int D, int T, bool CHUNKED, int TPR>
void attn_launch(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                 float* out, float* partials, const AttnPlan& p, hipStream_t st, hipEvent_t ev0,
                 hipEvent_t ev1) {
    const float qscale = (float)(1.4426950408889634 / std::sqrt((double)D));
    const dim3 grid(CHUNKED ? p.items : p.heads), block(T);
    // with events, they take the kernel's own start and end timestamps
    if (a.k != nullptr)
        hipExtLaunchKernelGGL((k_attn<D, true, T, CHUNKED, TPR>), grid, block, 0, st, ev0, ev1, 0, L,
                              s.C, a, q, out, partials, p.use_order, p.order_base, p.pad_len,
                              qscale);
    else
        hipExtLaunchKernelGGL((k_attn<D, false, T, CHUNKED, TPR>), grid, block, 0, st, ev0, ev1, 0, L,
                              s.C, a, q, out, partials, p.use_order, p.order_base, p.pad_len,
                              qscale);
    if (CHUNKED)
        hipLaunchKernelGGL(k_merge<D>, dim3(s.BH), dim3(D), 0, st, L, out, partials,
                           a.k != nullptr ? 1 : 0);
}

template <int D, int T>
void attn_dispatch_t(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                     float* out, float* partials, const AttnPlan& p, hipStream_t st,
                     hipEvent_t ev0, hipEvent_t ev1) {
    if (p.chunked)
        attn_launch<D, T, true, kAttnTpr>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else if (p.tpr == kAttnTpr)
        attn_launch<D, T, false, kAttnTpr>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else if (p.tpr == kAttnTprWide)
        attn_launch<D, T, false, kAttnTprWide>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else
        attn_launch<D, T, false, kAttnTpr / 2>(L, s, a, q, out, partials, p, st, ev0, ev1);
}

template <int D>
void attn_dispatch(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                   float* out, float* partials, const AttnPlan& p, hipStream_t st,
                   hipEvent_t ev0, hipEvent_t ev1) {
    if (p.threads == 1024)
        attn_dispatch_t<D, 1024>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else if (p.threads == 512)
        attn_dispatch_t<D, 512>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else
        attn_dispatch_t<D, 256>(L, s, a, q, out, partials, p, st, ev0, ev1);
}

}  // namespace

template <int D, int T>
void layers_launch(const LayersArg& a, int layers, const MetaLayout& ml, const Shape& s, int tpr,
                   hipStream_t st) {
    const float qscale = (float)(1.4426950408889634 / std::sqrt((double)D));
    const dim3 grid((unsigned)layers * (unsigned)s.BH), block(T);
    if (tpr == kAttnTpr)
        hipLaunchKernelGGL((k_attn_layers<D, T, kAttnTpr>), grid, block, 0, st, a, ml, s.BH, s.C,
                           qscale);
    else if (tpr == kAttnTprWide)
        hipLaunchKernelGGL((k_attn_layers<D, T, kAttnTprWide>), grid, block, 0, st, a, ml, s.BH,
                           s.C, qscale);
    else
        hipLaunchKernelGGL((k_attn_layers<D, T, kAttnTpr / 2>), grid, block, 0, st, a, ml, s.BH,
                           s.C, qscale);
}

template <int D>
void layers_dispatch(const LayersArg& a, int layers, const MetaLayout& ml, const Shape& s,
                     int threads, int tpr, hipStream_t st) {
    if (threads == 1024)
        layers_launch<D, 1024>(a, layers, ml, s, tpr, st);
    else if (threads == 512)
        layers_launch<D, 512>(a, layers, ml, s, tpr, st);
    else
        layers_launch<D, 256>(a, layers, ml, s, tpr, st);
}

int launch_attn(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                float* out, float* partials, const AttnPlan& p, void* stream, void* ev_start,
                void* ev_stop) {
    hipEvent_t e0 = static_cast<hipEvent_t>(ev_start), e1 = static_cast<hipEvent_t>(ev_stop);
    if (s.d == 128)
        attn_dispatch<128>(L, s, a, q, out, partials, p, (hipStream_t)stream, e0, e1);
    else
        attn_dispatch<64>(L, s, a, q, out, partials, p, (hipStream_t)stream, e0, e1);
    return last_error();
}

int launch_attn_layers(const LayersArg& a, int layers, const MetaLayout& ml, const Shape& s,
                       int threads, int tpr, void* stream) {
    if (s.d == 128)
        layers_dispatch<128>(a, layers, ml, s, threads, tpr, (hipStream_t)stream);
    else
        layers_dispatch<64>(a, layers, ml, s, threads, tpr, (hipStream_t)stream);
    return last_error();
}

}  // namespace headkv
