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
//            In a chunked launch the chunks of a head merge their results
//            through a tree of atomic exchanges, in the same kernel.
//
// The block itself (rows of d/8 lanes, all loads of a pass issued before
// use, online softmax, merge through LDS) is attn_block in attn_block.h.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "../../include/headkv.h"
#include "attn_block.h"
#include "device_common.h"
#include "layout.h"

namespace headkv {
namespace {

using namespace dev;

// 4 wavefronts per SIMD (16 per CU) at every block size: at most 128 VGPRs.
// The arguments that the block's first loads need lead the list, as plain
// pointers and an integer, so that they are preloaded into scalar registers
// at wave launch: the first metadata loads then go out without waiting for
// the kernel-argument fetch.  `sel` is the chunk table (chunked launches),
// else the dispatch order from the launch's first head, or null for block i =
// head i.  The same fields of L are not read.
template <int D, bool APPEND, int T, bool CHUNKED, int TPR>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(4))) void k_attn(
    char* kv, int64_t* seg_off, int32_t* len_n, int32_t* cap, const uint16_t* q, int32_t* sel,
    int dn, LayerDev L, int C, AppendArgs a, float* __restrict__ out,
    uint64_t* __restrict__ part, int pad_len, float qscale) {
    LayerDev M = L;
    M.kv = kv;
    M.seg_off = seg_off;
    M.n = len_n;
    M.cap = cap;
    M.dn = dn;
    if (CHUNKED)
        M.items = reinterpret_cast<uint32_t*>(sel);
    else
        M.order = sel;
    attn_block<D, APPEND, T, CHUNKED, TPR>(M, C, a, q, out, part, sel != nullptr, 0, pad_len,
                                           qscale, (int)blockIdx.x);
}

// Several layers in one launch: layer blockIdx.x / BH, head blockIdx.x % BH.
template <int D, int T, int TPR>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(4))) void k_attn_layers(
    LayersArg args, MetaLayout ml, int BH, int C, float qscale) {
    const int layer = (int)blockIdx.x / BH;
    LayerDev L = make_layer_dev(args.kv[layer], args.meta[layer], ml);
    L.dn = args.dn[layer];
    const AppendArgs none{};
    attn_block<D, false, T, false, TPR>(L, C, none, args.q[layer], args.out[layer], nullptr, 0, 0,
                                        0, qscale, (int)blockIdx.x - layer * BH);
}

// Sets n words to zero: a partial buffer before its first chunked launch.
__global__ __launch_bounds__(256) void k_zero(uint64_t* __restrict__ p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
        p[i] = 0u;
}

inline int last_error() { return (int)hipGetLastError(); }

template <int D, int T, bool CHUNKED, int TPR>
void attn_launch(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                 float* out, uint64_t* partials, const AttnPlan& p, hipStream_t st, hipEvent_t ev0,
                 hipEvent_t ev1) {
    const float qscale = (float)(1.4426950408889634 / std::sqrt((double)D));
    const dim3 grid(CHUNKED ? p.items : p.heads), block(T);
    int32_t* sel = CHUNKED ? reinterpret_cast<int32_t*>(L.items)
                           : (p.use_order ? L.order + p.order_base : nullptr);
    // with events, they take the kernel's own start and end timestamps
    if (a.k != nullptr)
        hipExtLaunchKernelGGL((k_attn<D, true, T, CHUNKED, TPR>), grid, block, 0, st, ev0, ev1, 0,
                              L.kv, L.seg_off, L.n, L.cap, q, sel, L.dn, L, s.C, a, out, partials,
                              p.pad_len, qscale);
    else
        hipExtLaunchKernelGGL((k_attn<D, false, T, CHUNKED, TPR>), grid, block, 0, st, ev0, ev1, 0,
                              L.kv, L.seg_off, L.n, L.cap, q, sel, L.dn, L, s.C, a, out, partials,
                              p.pad_len, qscale);
}

template <int D, int T>
void attn_dispatch_t(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                     float* out, uint64_t* partials, const AttnPlan& p, hipStream_t st,
                     hipEvent_t ev0, hipEvent_t ev1) {
    if (p.chunked)
        attn_launch<D, T, true, kAttnTpr>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else if (p.tpr == kAttnTpr)
        attn_launch<D, T, false, kAttnTpr>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else if (p.tpr == kAttnTprWide)
        attn_launch<D, T, false, kAttnTprWide>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else if (p.tpr == kAttnTprShort)
        attn_launch<D, T, false, kAttnTprShort>(L, s, a, q, out, partials, p, st, ev0, ev1);
    else
        attn_launch<D, T, false, kAttnTpr / 2>(L, s, a, q, out, partials, p, st, ev0, ev1);
}

template <int D>
void attn_dispatch(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                   float* out, uint64_t* partials, const AttnPlan& p, hipStream_t st,
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
    else if (tpr == kAttnTprShort)
        hipLaunchKernelGGL((k_attn_layers<D, T, kAttnTprShort>), grid, block, 0, st, a, ml, s.BH,
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

int launch_zero_words(uint64_t* p, size_t n, void* stream) {
    if (n == 0) return 0;
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 1024);
    hipLaunchKernelGGL(k_zero, dim3(blocks), dim3(256), 0, (hipStream_t)stream, p, n);
    return last_error();
}

int launch_attn(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                float* out, uint64_t* partials, const AttnPlan& p, void* stream, void* ev_start,
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
