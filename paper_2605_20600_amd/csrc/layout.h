// Shared host/device description of the per-layer cache layout.
//
// Cache of one head ("segment", 256-byte aligned, inside the layer's KV
// buffer):
//   K rows   [C + cap][d] bf16   rows 0..C-1: conditional prefix (Eq. 2, k_c),
//                                rows C+s: visual slot s (any order of positions)
//   V rows   [C + cap][d] bf16   same rows as K
//   pos      [cap] int32         visual position held by slot s
// Slots 0..n-1 of a head are occupied; an update compacts them again.
//
// Per-layer metadata buffer: one array per field, each 256-byte aligned.
#pragma once

#include <cstddef>
#include <cstdint>

namespace headkv {

constexpr int kChunk = 64;          // tokens per decode work item
constexpr int kBlock = 256;         // threads per block of the cache kernels
constexpr int kXcds = 8;            // MI355X: 8 accelerator complex dies

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline size_t segment_bytes(int C, int cap, int d) {
    return align_up(2 * (size_t)(C + cap) * d * sizeof(uint16_t) + (size_t)cap * sizeof(int32_t), 256);
}

struct MetaLayout {
    size_t seg_off, cap, n, budget, nstar, label, counter, chunk_base, qsum, work, total;
    int max_items;

    void compute(int BH, int d, int max_items_) {
        max_items = max_items_;
        size_t o = 0;
        auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
        seg_off = take(sizeof(int64_t) * BH);
        cap = take(sizeof(int32_t) * BH);
        n = take(sizeof(int32_t) * BH);
        budget = take(sizeof(int32_t) * BH);
        nstar = take(sizeof(int32_t) * BH);
        label = take(sizeof(int32_t) * BH);
        counter = take(sizeof(uint32_t) * BH);
        chunk_base = take(sizeof(int32_t) * BH);
        qsum = take(sizeof(double) * (size_t)BH * d);
        work = take(sizeof(int32_t) * 2 * (size_t)max_items);
        total = o;
    }
};

// Device view of one layer, passed to kernels by value.
struct LayerDev {
    char* kv;             // base of the layer's current KV buffer
    int64_t* seg_off;     // byte offset of each head's segment in kv
    int32_t* cap;         // visual slots of each head
    int32_t* n;           // occupied visual slots
    int32_t* budget;      // visual-token budget (after grouping)
    int32_t* nstar;       // n* from grouping
    int32_t* label;       // 1 = local head
    uint32_t* counter;    // split-K arrival counters, zero between launches
    int32_t* chunk_base;  // first partial slot of each head
    double* qsum;         // [BH][d] running sum of the queries of this window
    int32_t* work;        // [max_items][2] (head, chunk) work items, head < 0 = idle
};

inline LayerDev make_layer_dev(void* kv, void* meta, const MetaLayout& m) {
    char* b = static_cast<char*>(meta);
    LayerDev L;
    L.kv = static_cast<char*>(kv);
    L.seg_off = reinterpret_cast<int64_t*>(b + m.seg_off);
    L.cap = reinterpret_cast<int32_t*>(b + m.cap);
    L.n = reinterpret_cast<int32_t*>(b + m.n);
    L.budget = reinterpret_cast<int32_t*>(b + m.budget);
    L.nstar = reinterpret_cast<int32_t*>(b + m.nstar);
    L.label = reinterpret_cast<int32_t*>(b + m.label);
    L.counter = reinterpret_cast<uint32_t*>(b + m.counter);
    L.chunk_base = reinterpret_cast<int32_t*>(b + m.chunk_base);
    L.qsum = reinterpret_cast<double*>(b + m.qsum);
    L.work = reinterpret_cast<int32_t*>(b + m.work);
    return L;
}

// Launchers (kernels.hip).  All return hipGetLastError() as an int.
struct Shape {
    int BH, B, H, d, C, N;
};

int launch_prefill(const LayerDev& L, const Shape& s, const uint16_t* kc, const uint16_t* vc,
                   int64_t dense_seg_bytes, int dense_cap, int dense_cph, void* stream);
int launch_append(const LayerDev& L, const Shape& s, const uint16_t* q, const uint16_t* k,
                  const uint16_t* v, int step, int accumulate, int reset, void* stream);
int launch_score(const LayerDev& L, const Shape& s, const uint16_t* q, int32_t* n_star,
                 uint8_t* is_local, int len, double sqrt_d, double tau, int local_window,
                 void* stream);
int launch_budgets(const LayerDev& L, const Shape& s, const uint8_t* is_local,
                   const int32_t* override_b, int32_t* budgets, int mode, int row_len,
                   int recent_len, int rho_num, int rho_den, void* stream);
int launch_update(const LayerDev& L, const Shape& s, const char* src_kv, int relayout,
                  int64_t dense_seg_bytes, int dense_cap, int recent_len, int rs_num,
                  int rs_den, int u, void* stream);
int launch_decode(const LayerDev& L, const Shape& s, const uint16_t* q, float* out,
                  float* partials, int uniform_active, int n_items, void* stream);
int launch_export(const LayerDev& L, const Shape& s, uint8_t* mask, int32_t* count,
                  void* stream);

}  // namespace headkv
