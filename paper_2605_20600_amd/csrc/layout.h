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

constexpr int kBlock = 256;  // threads per block of the cache kernels
constexpr int kAttnTpr = 8;  // tokens per 16-lane row per attention pass
// A wider pass (9 tokens per row, still under 128 VGPRs) for launches whose
// longest head just misses one pass of 8: one pass instead of two.
constexpr int kAttnTprWide = 9;
// Three quarters of a pass, for launches whose longest head fits it: fewer
// clamped duplicate loads than a pass of 8.
constexpr int kAttnTprShort = 6;
constexpr int kCus = 256;    // MI355X compute units
// Attention blocks have 1024, 512 or 256 threads; 1024 threads of at most 128
// VGPRs fill a CU, so a CU holds 1024 / threads blocks at once.  A token row
// of d bf16 is read by d/8 lanes, 16 bytes each.
constexpr int kAttnMinThreads = 256;
constexpr int kAttnMaxThreads = 1024;
inline constexpr int attn_tokens_per_pass(int threads, int d, int tpr = kAttnTpr) {
    return threads / (d / 8) * tpr;
}
inline constexpr int attn_resident_blocks(int threads) { return kCus * (kAttnMaxThreads / threads); }
// Chunks per head in a chunk table: bounded so that the chunk index fits in
// the 8 low bits of a table entry.
constexpr int kMaxChunksPerHead = 255;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline size_t segment_bytes(int C, int cap, int d) {
    return align_up(2 * (size_t)(C + cap) * d * sizeof(uint16_t) + (size_t)cap * sizeof(int32_t), 256);
}

struct MetaLayout {
    size_t seg_off, cap, n, budget, nstar, label, order, items, item_start, qring, total;
    int max_items, ring_len, attn_scores;

    // max_items: largest chunk table of a layer (every head at its largest
    // capacity, in chunks of the smallest attention pass); ring_len: queries
    // kept per head, the update period (the window of Eq. 6); attn_scores: 1
    // when global heads are scored by the window's attention weights.
    void compute(int BH, int d, int max_items_, int ring_len_, int attn_scores_ = 0) {
        max_items = max_items_;
        ring_len = ring_len_;
        attn_scores = attn_scores_;
        size_t o = 0;
        auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
        seg_off = take(sizeof(int64_t) * BH);
        cap = take(sizeof(int32_t) * BH);
        n = take(sizeof(int32_t) * BH);
        budget = take(sizeof(int32_t) * BH);
        nstar = take(sizeof(int32_t) * BH);
        label = take(sizeof(int32_t) * BH);
        order = take(sizeof(int32_t) * BH);
        items = take(sizeof(uint32_t) * (size_t)max_items);
        item_start = take(sizeof(int32_t) * ((size_t)BH + 1));
        qring = take(sizeof(uint16_t) * (size_t)BH * ring_len * d);
        total = o;
    }
};

// Device view of one layer, passed to kernels by value.
struct LayerDev {
    char* kv;             // base of the layer's current KV buffer
    int64_t* seg_off;     // byte offset of each head's segment in kv
    int32_t* cap;         // visual slots of each head
    int32_t* n;           // occupied visual slots as of the last kernel that set them
                          // (prefill, an update): the length is n[h] + dn
    int32_t* budget;      // visual-token budget (after grouping)
    int32_t* nstar;       // n* from grouping
    int32_t* label;       // 1 = local head
    int32_t* order;       // attention dispatch order of the heads (longest first)
    // chunk table: entry = head << 8 | chunk, the chunks of a head contiguous;
    // head h owns entries item_start[h] .. item_start[h+1]-1
    uint32_t* items;
    int32_t* item_start;  // [BH + 1]
    // the queries of the last ring_len steps, [BH][ring_len][d] bf16, step t
    // in slot t % ring_len: the window that an update scores against
    uint16_t* qring;
    int ring_len;
    int attn_scores;      // 1: attention-sum scores instead of Eq. 6
    int dn;               // tokens every head appended since n was written
};

#if defined(__HIPCC__)
__host__ __device__
#endif
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
    L.order = reinterpret_cast<int32_t*>(b + m.order);
    L.items = reinterpret_cast<uint32_t*>(b + m.items);
    L.item_start = reinterpret_cast<int32_t*>(b + m.item_start);
    L.qring = reinterpret_cast<uint16_t*>(b + m.qring);
    L.ring_len = m.ring_len;
    L.attn_scores = m.attn_scores;
    L.dn = 0;
    return L;
}

// Launchers (cache_kernels.hip, attn_kernels.hip).  All return
// hipGetLastError() as an int.
struct Shape {
    int BH, B, H, d, C, N;
};

// The token appended by a step (fused into the kernel that consumes it).
struct AppendArgs {
    const uint16_t* q;   // [BH][d] bf16
    const uint16_t* k;
    const uint16_t* v;
    int step;            // visual position of the token
};

// Also writes the dense layout's chunk table: dense_chunks chunks per head.
int launch_prefill(const LayerDev& L, const Shape& s, const uint16_t* kc, const uint16_t* vc,
                   int64_t dense_seg_bytes, int dense_cap, int dense_chunks, void* stream);
int launch_append(const LayerDev& L, const Shape& s, const AppendArgs& a, void* stream);
// Causal attention over the C >= 1 prefix tokens of every head, fused with
// launch_prefill's work (prefill_attn.hip).
int launch_prefill_attn(const LayerDev& L, const Shape& s, const uint16_t* qc, const uint16_t* kc,
                        const uint16_t* vc, float* out, int64_t dense_seg_bytes, int dense_cap,
                        int dense_chunks, void* stream, void* ev_start = nullptr,
                        void* ev_stop = nullptr);
int launch_score(const LayerDev& L, const Shape& s, const uint16_t* q, int32_t* n_star,
                 uint8_t* is_local, int len, double sqrt_d, double tau, int local_window,
                 void* stream);
// Writes budgets and the labels the updates use (L.label) for every head.
int launch_budgets(const LayerDev& L, const Shape& s, const uint8_t* is_local,
                   const int32_t* override_b, int32_t* budgets, int mode, int row_len,
                   int recent_len, int rho_num, int rho_den, int cfg_pairs, void* stream);
// a.k == nullptr: no append.  step: the visual step of the update.
// lds_cap: largest visual capacity among the launch's source segments.
// With L.attn_scores, global heads are scored by the window's attention weights.
int launch_update(const LayerDev& L, const Shape& s, const AppendArgs& a, const char* src_kv,
                  int relayout, int64_t dense_seg_bytes, int dense_cap, int recent_len,
                  int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                  void* stream, void* ev_start, void* ev_stop);
// Append + update (Eq. 6 scores) + attention of one layer step in one launch,
// for attention plans of one block per head; use_order, pad_len, threads and
// tpr as in that plan; q, out as in launch_attn.
int launch_update_attn(const LayerDev& L, const Shape& s, const AppendArgs& a, int recent_len,
                       int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                       const uint16_t* q, float* out, int use_order, int pad_len, int threads,
                       int tpr, void* stream, void* ev_start, void* ev_stop);
// Dynamic LDS of one update block (C: prefix rows, with attention-sum scores).
size_t update_lds_bytes(int N, int cap, int d, int C, bool attn_scores, int period);
// Dynamic LDS an update block may take: the CU's 160 KB less a margin for the
// kernel's static LDS (block scans, radix histogram, reductions).
constexpr size_t kUpdateLdsBudget = 156 * 1024;
// How one attention launch covers a layer (or a group of its heads).
struct AttnPlan {
    int threads;     // 1024, 512 or 256
    int chunked;     // 0: one block per head, every pass; 1: one block per entry
                     //    of the chunk table (chunks of one pass), merged in
                     //    the kernel
    int items;       // entries of the chunk table (chunked)
    int heads;       // blocks of a launch with one block per head
    int use_order;   // one block per head: head = order[order_base + block]
    int order_base;
    int pad_len;     // one block per head: read rows up to this length, those
                     // past the head's own length masked (0: none)
    int tpr;         // tokens per row and pass: kAttnTpr, or 3/4 or half of it
                     // (one block per head, every head within that pass), or
                     // kAttnTprWide
};
// Per-layer pointers of a multi-layer attention launch (up to kMaxLayersPerLaunch).
constexpr int kMaxLayersPerLaunch = 64;
struct LayersArg {
    void* kv[kMaxLayersPerLaunch];
    void* meta[kMaxLayersPerLaunch];
    int dn[kMaxLayersPerLaunch];
    const uint16_t* q[kMaxLayersPerLaunch];
    float* out[kMaxLayersPerLaunch];
};
// Attention of `layers` layers (no append, one block per head, every head
// resident): heads of layer i are blocks i*BH .. i*BH + BH - 1.
int launch_attn_layers(const LayersArg& a, int layers, const MetaLayout& ml, const Shape& s,
                       int threads, int tpr, void* stream);
// a.k == nullptr: no append.  partials: d 64-bit words per table entry, zero
// between launches (every word a chunked launch writes, it also clears).
// ev_start / ev_stop (hipEvent_t or nullptr) receive the attention kernel's
// own start and end timestamps.
int launch_attn(const LayerDev& L, const Shape& s, const AppendArgs& a, const uint16_t* q,
                float* out, uint64_t* partials, const AttnPlan& p, void* stream,
                void* ev_start = nullptr, void* ev_stop = nullptr);
// Sets n 64-bit words at p to zero (a partial buffer before its first use).
int launch_zero_words(uint64_t* p, size_t n, void* stream);
int launch_export(const LayerDev& L, const Shape& s, uint8_t* mask, int32_t* count,
                  void* stream);

}  // namespace headkv
