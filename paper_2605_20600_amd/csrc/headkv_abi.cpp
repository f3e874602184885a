// Host runtime and C ABI of the head-aware compressed-KV decode path.
//
// The handle mirrors, per layer, what the device state must be (step, phase,
// every head's length, budget and capacity) so that every call is validated
// before anything is launched, grids are sized without reading the device
// back, and the only device-to-host wait is the one in assign_budgets, where
// the budgets decide the layout of the per-head segments.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/headkv.h"
#include "layout.h"
#include "scratch.h"

using namespace headkv;

namespace {

thread_local std::string g_err;

headkv_status fail(headkv_status code, const std::string& msg) {
    g_err = msg;
    return code;
}

headkv_status ok() { return HEADKV_OK; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Layer {
    void* dense = nullptr;
    void* meta = nullptr;
    void* ragged = nullptr;
    bool prefilled = false;
    bool grouped = false;
    int last_step = -1;
    std::vector<int> n, budget, cap;
    // tokens every head appended since the device lengths were last written
    // (by prefill or an update); kernels take the length as n[h] + dn
    int dn = 0;
    std::vector<uint8_t> label_local;  // labels used by the updates (host copy)
    int chunk_threads = kAttnMaxThreads;  // block size the chunk table is cut for
    int items = 0;                        // entries of the chunk table
    int n_global = 0;                     // global heads (first in the dispatch
                                          // order with HEADKV_ATTN_GROUPED)
};

}  // namespace

struct headkv_ctx {
    headkv_config cfg;
    Shape shape;
    MetaLayout ml;
    int t_g = 0;
    int dense_cap = 0;             // visual slots per head before grouping
    int64_t dense_seg = 0;         // bytes per head segment before grouping
    size_t ws_bytes = 0;
    void* ws = nullptr;
    bool ws_clear = false;         // the workspace has been zeroed (the chunked
                                   // attention keeps it zero between launches)
    std::vector<Layer> layers;
    // timing of sampled launches: event pairs, kind and algorithmic bytes
    std::vector<hipEvent_t> events;
    std::vector<double> timed_bytes;
    std::vector<int> timed_kind;
    size_t timed = 0;
    int64_t timing_dropped = 0;
    ~headkv_ctx() {
        for (hipEvent_t e : events) (void)hipEventDestroy(e);
    }
};

namespace {

headkv_status validate_config(const headkv_config* c) {
    if (!c) return fail(HEADKV_ERR_INVALID_ARG, "config is NULL");
    if (c->batch < 1 || c->num_layers < 1 || c->num_heads < 1)
        return fail(HEADKV_ERR_INVALID_ARG, "batch, num_layers and num_heads must be >= 1");
    if (c->num_heads > 1024) return fail(HEADKV_ERR_UNSUPPORTED, "num_heads > 1024");
    if ((long long)c->batch * c->num_heads > (1 << 24))
        return fail(HEADKV_ERR_UNSUPPORTED, "batch * num_heads > 2^24");
    if (c->head_dim != 64 && c->head_dim != 128)
        return fail(HEADKV_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (c->prefix_len < 0 || c->prefix_len > HEADKV_MAX_PREFIX)
        return fail(HEADKV_ERR_INVALID_ARG, "prefix_len out of [0, HEADKV_MAX_PREFIX]");
    if (c->num_visual < 1 || c->num_visual > HEADKV_MAX_VISUAL)
        return fail(HEADKV_ERR_INVALID_ARG, "num_visual out of [1, HEADKV_MAX_VISUAL]");
    if (c->row_len < 1 || c->row_len > c->num_visual)
        return fail(HEADKV_ERR_INVALID_ARG, "row_len out of [1, num_visual]");
    if (c->recent_len < 1 || c->local_window < 1 || c->period < 1)
        return fail(HEADKV_ERR_INVALID_ARG, "recent_len, local_window and period must be >= 1");
    if (c->group_threshold < 1 || c->group_threshold > c->num_visual)
        return fail(HEADKV_ERR_INVALID_ARG, "group_threshold out of [1, num_visual]");
    if (c->group_threshold > HEADKV_MAX_CAPACITY)
        return fail(HEADKV_ERR_UNSUPPORTED, "group_threshold > HEADKV_MAX_CAPACITY");
    if (c->budget_mode < HEADKV_BUDGET_PAPER || c->budget_mode > HEADKV_BUDGET_TOTAL)
        return fail(HEADKV_ERR_INVALID_ARG, "unknown budget_mode");
    if (c->rho_num < 1 || c->rho_den < 1 || c->rho_num > c->rho_den)
        return fail(HEADKV_ERR_INVALID_ARG, "rho must be in (0, 1]");
    if (c->rs_num < 0 || c->rs_den < 1 || c->rs_num > c->rs_den)
        return fail(HEADKV_ERR_INVALID_ARG, "r_s must be in [0, 1]");
    if (!(c->tau > 0.0 && c->tau <= 1.0)) return fail(HEADKV_ERR_INVALID_ARG, "tau must be in (0, 1]");
    if (c->attn_strategy < HEADKV_ATTN_VARLEN || c->attn_strategy > HEADKV_ATTN_GROUPED)
        return fail(HEADKV_ERR_INVALID_ARG, "unknown attn_strategy");
    if (c->cfg_pairs != 0 && c->cfg_pairs != 1) return fail(HEADKV_ERR_INVALID_ARG, "cfg_pairs must be 0 or 1");
    if (c->score_mode != HEADKV_SCORE_MEAN_LOGIT && c->score_mode != HEADKV_SCORE_ATTN_SUM)
        return fail(HEADKV_ERR_INVALID_ARG, "unknown score_mode");
    if (c->score_mode == HEADKV_SCORE_ATTN_SUM &&
        update_lds_bytes(c->num_visual, std::min(c->num_visual, HEADKV_MAX_CAPACITY), c->head_dim,
                         c->prefix_len, true, c->period) > kUpdateLdsBudget)
        return fail(HEADKV_ERR_UNSUPPORTED, "attention-sum scores: prefix + capacity too large for LDS");
    if (c->cfg_pairs && c->batch % 2 != 0)
        return fail(HEADKV_ERR_INVALID_ARG, "cfg_pairs needs an even batch");
    // chunk indices must fit the 8 bits of a chunk table entry (always true
    // within the prefix and capacity limits)
    const int max_cap = std::max(c->group_threshold, std::min(c->num_visual, HEADKV_MAX_CAPACITY));
    const int tp = attn_tokens_per_pass(kAttnMinThreads, c->head_dim);
    if ((c->prefix_len + max_cap + 1 + tp - 1) / tp > kMaxChunksPerHead)
        return fail(HEADKV_ERR_UNSUPPORTED, "too many attention chunks per head");
    return ok();
}

struct Plan {
    int BH, dense_cap;
    int64_t dense_seg;
    size_t dense_bytes, ws_bytes;
    MetaLayout ml;
};

// Chunks of one pass of a `threads`-thread block that cover a head of
// capacity `cap` (prefix, slots and the token being appended).
int chunks_of(int C, int cap, int threads, int d) {
    const int tp = attn_tokens_per_pass(threads, d);
    return (C + cap + 1 + tp - 1) / tp;
}

Plan make_plan(const headkv_config& c) {
    Plan p;
    p.BH = c.batch * c.num_heads;
    p.dense_cap = c.group_threshold;
    p.dense_seg = (int64_t)segment_bytes(c.prefix_len, p.dense_cap, c.head_dim);
    p.dense_bytes = (size_t)p.dense_seg * p.BH;
    // the largest capacity any head can have, dense or after grouping
    const int max_cap = std::max(p.dense_cap, std::min(c.num_visual, HEADKV_MAX_CAPACITY));
    const int per_head = chunks_of(c.prefix_len, max_cap, kAttnMinThreads, c.head_dim);
    // ring of the window queries: an update's window never holds more than
    // min(P, N) steps (with P > N the grouping step's update is the only one,
    // and its window starts at step 0 either way)
    p.ml.compute(p.BH, c.head_dim, p.BH * per_head, std::min(c.period, c.num_visual),
                 c.score_mode == HEADKV_SCORE_ATTN_SUM ? 1 : 0);
    // partial (max, sum, weighted V) of every chunk table entry
    p.ws_bytes = align_up((size_t)p.BH * per_head * c.head_dim * sizeof(uint64_t), 256);
    return p;
}

// Block size of a chunk table for the given capacities: the fewest rounds of
// resident blocks, then the largest blocks (fewest partial results).
int pick_chunk_threads(int C, int d, const std::vector<int>& cap) {
    int best = kAttnMaxThreads;
    long long best_rounds = -1;
    for (int t = kAttnMaxThreads; t >= kAttnMinThreads; t /= 2) {
        long long items = 0;
        for (int x : cap) items += chunks_of(C, x, t, d);
        const long long slots = attn_resident_blocks(t);
        const long long rounds = (items + slots - 1) / slots;
        if (best_rounds < 0 || rounds < best_rounds) {
            best = t;
            best_rounds = rounds;
        }
    }
    return best;
}

// Block size of the full-cache chunk table.  Before grouping every head grows
// from the prefix to group_threshold tokens, so the size is chosen for the
// phase's mean length, not the capacity: the largest block whose chunks of a
// head of that length give at least one block per CU (Lumina-1024 full-cache
// phase: 1024 threads, one chunk per head for most steps, 10.43 us per
// launch; 512 threads 9.68 us).
int dense_chunk_threads(int BH, int C, int thr, int d) {
    for (int t = kAttnMaxThreads; t > kAttnMinThreads; t /= 2)
        if ((long long)BH * chunks_of(C, thr / 2, t, d) >= kCus) return t;
    return kAttnMinThreads;
}

headkv_status check_layer(headkv_t h, int32_t layer) {
    if (!h) return fail(HEADKV_ERR_INVALID_ARG, "handle is NULL");
    if (layer < 0 || layer >= h->cfg.num_layers) return fail(HEADKV_ERR_INVALID_ARG, "layer out of range");
    return ok();
}

headkv_status hip_status(int e, const char* what) {
    if (e != 0) return fail(HEADKV_ERR_HIP, std::string(what) + ": " + hipGetErrorString((hipError_t)e));
    return ok();
}

double sqrt_d(headkv_t h) { return std::sqrt((double)h->cfg.head_dim); }

LayerDev dev_of(headkv_t h, const Layer& L) {
    LayerDev D = make_layer_dev(L.grouped ? L.ragged : L.dense, L.meta, h->ml);
    D.dn = L.dn;
    return D;
}

// Event pair for a sampled launch of `kind`, or nullptrs.
void take_events(headkv_t h, bool time_it, int kind, double bytes, void** e0, void** e1) {
    *e0 = *e1 = nullptr;
    if (!time_it) return;
    if (2 * (h->timed + 1) > h->events.size()) {
        ++h->timing_dropped;
        return;
    }
    *e0 = h->events[2 * h->timed];
    *e1 = h->events[2 * h->timed + 1];
    h->timed_bytes[h->timed] = bytes;
    h->timed_kind[h->timed] = kind;
    ++h->timed;
}

}  // namespace

extern "C" {

headkv_status headkv_plan(const headkv_config* cfg, size_t* dense_kv_bytes, size_t* meta_bytes,
                          size_t* workspace_bytes) {
    headkv_status st = validate_config(cfg);
    if (st) return st;
    if (!dense_kv_bytes || !meta_bytes || !workspace_bytes)
        return fail(HEADKV_ERR_INVALID_ARG, "output pointer is NULL");
    Plan p = make_plan(*cfg);
    *dense_kv_bytes = p.dense_bytes;
    *meta_bytes = p.ml.total;
    *workspace_bytes = p.ws_bytes;
    return ok();
}

headkv_status headkv_create(const headkv_config* cfg, void* const* dense_kv, void* const* meta,
                            void* workspace, headkv_t* out) {
    headkv_status st = validate_config(cfg);
    if (st) return st;
    if (!dense_kv || !meta || !out) return fail(HEADKV_ERR_INVALID_ARG, "NULL pointer");
    // a NULL workspace is allowed: chunked attention then needs the
    // allocation-free entry point
    if (workspace && !aligned(workspace, 256))
        return fail(HEADKV_ERR_INVALID_ARG, "workspace not 256-byte aligned");
    for (int l = 0; l < cfg->num_layers; ++l) {
        if (!dense_kv[l] || !meta[l]) return fail(HEADKV_ERR_INVALID_ARG, "NULL layer buffer");
        if (!aligned(dense_kv[l], 256) || !aligned(meta[l], 256))
            return fail(HEADKV_ERR_INVALID_ARG, "layer buffer not 256-byte aligned");
    }
    headkv_ctx* h = new (std::nothrow) headkv_ctx();
    if (!h) return fail(HEADKV_ERR_INVALID_ARG, "out of host memory");
    Plan p = make_plan(*cfg);
    h->cfg = *cfg;
    h->shape = Shape{p.BH, cfg->batch, cfg->num_heads, cfg->head_dim, cfg->prefix_len, cfg->num_visual};
    h->ml = p.ml;
    h->t_g = cfg->group_threshold - 1;
    h->dense_cap = p.dense_cap;
    h->dense_seg = p.dense_seg;
    h->ws_bytes = p.ws_bytes;
    h->ws = workspace;
    h->layers.resize(cfg->num_layers);
    for (int l = 0; l < cfg->num_layers; ++l) {
        h->layers[l].dense = dense_kv[l];
        h->layers[l].meta = meta[l];
    }
    *out = h;
    return ok();
}

void headkv_destroy(headkv_t h) { delete h; }

}  // extern "C"

namespace {

// Step 1 of `layer`: host mirror reset and one launch that resets the device
// state and stores the prefix (with q_c, also the prefix attention).
headkv_status prefill_impl(headkv_t h, int32_t layer, const uint16_t* q_c, const uint16_t* k_c,
                           const uint16_t* v_c, float* out_c, void* stream) {
    headkv_status st = check_layer(h, layer);
    if (st) return st;
    const headkv_config& c = h->cfg;
    if (c.prefix_len > 0 && (!k_c || !v_c)) return fail(HEADKV_ERR_INVALID_ARG, "k_c / v_c is NULL");
    if (c.prefix_len > 0 && (!aligned(k_c, 16) || !aligned(v_c, 16)))
        return fail(HEADKV_ERR_INVALID_ARG, "k_c / v_c not 16-byte aligned");
    if (q_c || out_c) {
        if (c.prefix_len < 1) return fail(HEADKV_ERR_INVALID_ARG, "prefill attention needs prefix_len >= 1");
        if (!q_c || !out_c) return fail(HEADKV_ERR_INVALID_ARG, "q_c / out_c is NULL");
        if (!aligned(q_c, 16) || !aligned(out_c, 16))
            return fail(HEADKV_ERR_INVALID_ARG, "q_c / out_c not 16-byte aligned");
    }
    Layer& L = h->layers[layer];
    L.grouped = false;
    L.prefilled = false;
    L.ragged = nullptr;
    L.last_step = -1;
    L.n.assign(h->shape.BH, 0);
    L.dn = 0;
    L.cap.assign(h->shape.BH, h->dense_cap);
    L.budget.assign(h->shape.BH, 0);
    L.label_local.assign(h->shape.BH, 0);
    L.chunk_threads = dense_chunk_threads(h->shape.BH, c.prefix_len, h->dense_cap, c.head_dim);
    const int dense_chunks = chunks_of(c.prefix_len, h->dense_cap, L.chunk_threads, c.head_dim);
    L.items = h->shape.BH * dense_chunks;
    if (q_c) {
        // timed whenever events are reserved: q, k, v read, k, v stored, fp32 out
        const double Cd = (double)c.prefix_len * c.head_dim;
        void *e0, *e1;
        take_events(h, !h->events.empty(), HEADKV_TIMED_PREFILL,
                    h->shape.BH * (3 * Cd * 2 + 2 * Cd * 2 + Cd * 4), &e0, &e1);
        st = hip_status(launch_prefill_attn(dev_of(h, L), h->shape, q_c, k_c, v_c, out_c,
                                            h->dense_seg, h->dense_cap, dense_chunks, stream,
                                            e0, e1),
                        "prefill attention launch");
    }
    else
        st = hip_status(launch_prefill(dev_of(h, L), h->shape, k_c, v_c, h->dense_seg,
                                       h->dense_cap, dense_chunks, stream),
                        "prefill launch");
    if (st) return st;
    L.prefilled = true;
    return ok();
}

}  // namespace

extern "C" {

headkv_status headkv_prefill(headkv_t h, int32_t layer, const uint16_t* k_c, const uint16_t* v_c,
                             void* stream) {
    return prefill_impl(h, layer, nullptr, k_c, v_c, nullptr, stream);
}

headkv_status headkv_prefill_attn(headkv_t h, int32_t layer, const uint16_t* q_c,
                                  const uint16_t* k_c, const uint16_t* v_c, float* out_c,
                                  void* stream) {
    if (!q_c || !out_c) return fail(HEADKV_ERR_INVALID_ARG, "q_c / out_c is NULL");
    return prefill_impl(h, layer, q_c, k_c, v_c, out_c, stream);
}

}  // extern "C"

namespace {

// Checks shared by every call that appends the token of `step`; fills the
// append arguments and tells whether a periodic update follows the append.
headkv_status prepare_append(headkv_t h, int32_t layer, int32_t step, const uint16_t* q,
                             const uint16_t* k, const uint16_t* v, AppendArgs* a, bool* update,
                             int* u) {
    headkv_status st = check_layer(h, layer);
    if (st) return st;
    if (!q || !k || !v) return fail(HEADKV_ERR_INVALID_ARG, "q / k / v is NULL");
    // the kernels read q, k and v rows with 16-byte vector loads
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16))
        return fail(HEADKV_ERR_INVALID_ARG, "q / k / v not 16-byte aligned");
    Layer& L = h->layers[layer];
    const headkv_config& c = h->cfg;
    if (!L.prefilled) return fail(HEADKV_ERR_STATE, "append before prefill");
    if (step != L.last_step + 1) return fail(HEADKV_ERR_STATE, "steps must be consecutive from 0");
    if (step >= c.num_visual) return fail(HEADKV_ERR_INVALID_ARG, "step >= num_visual");
    if (!L.grouped && step > h->t_g)
        return fail(HEADKV_ERR_STATE, "heads must be grouped at step group_threshold - 1");
    for (int i = 0; i < h->shape.BH; ++i)
        if (L.n[i] >= L.cap[i]) return fail(HEADKV_ERR_CAPACITY, "head capacity exhausted");
    // every append writes q into the head's ring of the last P queries, the
    // window that the next update scores against (Eq. 6)
    const int P = c.period;
    a->q = q;
    a->k = k;
    a->v = v;
    a->step = step;
    *update = L.grouped && step > h->t_g && (step - h->t_g) % P == 0;
    *u = (step - h->t_g) / P;
    return ok();
}

// Host mirror after the append (and update) of `step`.
void commit_append(headkv_t h, Layer& L, int32_t step, bool update) {
    for (int i = 0; i < h->shape.BH; ++i) L.n[i] += 1;
    // the update kernel writes every head's length; an append alone does not
    L.dn = update ? 0 : L.dn + 1;
    if (update)
        for (int i = 0; i < h->shape.BH; ++i) L.n[i] = std::min(L.n[i], L.budget[i]);
    L.last_step = step;
}

int max_cap(const Layer& L) { return *std::max_element(L.cap.begin(), L.cap.end()); }

// Tokens per row of a pass for a launch whose longest head reads `len`
// tokens: half or three quarters of a pass when that suffices (LlamaGen shape,
// heads of up to 168 tokens in 256-token passes: 233,250 -> 242,940 tokens/s
// with 192-token passes), the wide pass when it makes one pass of what would
// otherwise take two, else the normal pass, or three-quarter passes when
// their rows of loads (passes x tokens per row) are fewer: rows past a head's
// end are loaded clamped to its last row, and a mostly empty last pass costs
// (Lumina-768 rho 1/4, heads of up to 765 tokens: two passes of 384 instead
// of 512, 14.07-14.11 -> 13.21 us per launch, whole job +5.7 %; Janus +1.7 %).
int pass_tpr(int len, int threads, int d) {
    if (len <= attn_tokens_per_pass(threads, d, kAttnTpr / 2)) return kAttnTpr / 2;
    if (len <= attn_tokens_per_pass(threads, d, kAttnTprShort)) return kAttnTprShort;
    if (len > attn_tokens_per_pass(threads, d, kAttnTpr) &&
        len <= attn_tokens_per_pass(threads, d, kAttnTprWide))
        return kAttnTprWide;
    const int p8 = (len + attn_tokens_per_pass(threads, d) - 1) / attn_tokens_per_pass(threads, d);
    const int p6 = (len + attn_tokens_per_pass(threads, d, kAttnTprShort) - 1) /
                   attn_tokens_per_pass(threads, d, kAttnTprShort);
    if (p6 * kAttnTprShort < p8 * kAttnTpr) return kAttnTprShort;
    return kAttnTpr;
}

// Largest block size at which `heads` one-block-per-head blocks are all
// resident at once (256 beyond that; 1024 when they do not fill the CUs).
int resident_threads(int heads) {
    for (int t = kAttnMaxThreads; t >= kAttnMinThreads; t /= 2)
        if (heads <= attn_resident_blocks(t)) return t;
    return kAttnMinThreads;
}

// The attention launches of one layer step (appended: the step's token is
// attended from the input).  Returns their number (1 or 2).
//  VARLEN, fewer heads than CUs: the layer's chunk table, chunks of at most
//    one pass (at each launch the fewest that hold a head's length, sharing
//    its tokens evenly), balanced across heads of unequal length, merged in
//    the same kernel (a tree of atomic exchanges over each head's chunks).
//  VARLEN otherwise: one block per head over all its passes (no merge, the
//    append fused), at the largest block size at which every head's block is
//    resident at once (beyond that 256-thread blocks); longest heads first
//    whenever a CU takes more than one block.
//  PADDED: one block per head, every head reading the layer's longest length.
//  GROUPED (after grouping): one launch per non-empty group, global heads
//    first, each like VARLEN's one block per head over its own heads.
int attn_plans(headkv_t h, const Layer& L, bool appended, AttnPlan* out) {
    const int BH = h->shape.BH;
    const int strategy = h->cfg.attn_strategy;
    const int len_max = h->cfg.prefix_len + *std::max_element(L.n.begin(), L.n.end()) +
                        (appended ? 1 : 0);
    const int d = h->cfg.head_dim;
    auto whole = [&](int t, int heads, int use_order, int base, int pad) {
        int tpr = pass_tpr(std::max(len_max, pad), t, d);
        // every head within half a pass: half the threads with full rows read
        // the same tokens per pass, and merge half as many wavefronts at the
        // end (Lumina-768 full-cache steps of 148-248 tokens: 6.3-7.8 ->
        // 5.8-7.4 us per launch without the append, 0.02-0.25 us less with
        // it); every head stays resident, halving the block doubles the blocks
        // a CU holds
        if (tpr == kAttnTpr / 2 && t > kAttnMinThreads) {
            t /= 2;
            tpr = kAttnTpr;
        }
        return AttnPlan{t, 0, 0, heads, use_order, base, pad, tpr};
    };
    if (strategy == HEADKV_ATTN_PADDED) {
        out[0] = whole(resident_threads(BH), BH, 0, 0, len_max);
        return 1;
    }
    if (strategy == HEADKV_ATTN_GROUPED && L.grouped) {
        int k = 0;
        const int sizes[2] = {L.n_global, BH - L.n_global};
        for (int g = 0, base = 0; g < 2; base += sizes[g], ++g)
            if (sizes[g] > 0) out[k++] = whole(resident_threads(sizes[g]), sizes[g], 1, base, 0);
        return k;
    }
    if (BH < kCus) {
        out[0] = AttnPlan{L.chunk_threads, 1, L.items, BH, 0, 0, 0, kAttnTpr};
        return 1;
    }
    // with more than one block per CU, longest heads first (after grouping;
    // before it every head has the same length): the first round of dispatch
    // gives every CU one of the long heads, the second one of the short ones
    // (Janus, 512 heads, 2 blocks per CU: 13.35 -> 12.28 us; stress, 2048
    // heads in two rounds: 20,900 -> 24,200 tokens/s).  With more rounds the
    // dispatcher balances by itself and the order's load sits in front of
    // every round (LlamaGen shape, 5120 heads in five rounds: 31.2 us sorted,
    // 30.0 us in head order)
    const int t = resident_threads(BH);
    const int rounds = (BH + attn_resident_blocks(t) - 1) / attn_resident_blocks(t);
    const bool by_length = L.grouped && BH > kCus && rounds <= 2;
    out[0] = whole(t, BH, by_length ? 1 : 0, 0, 0);
    return 1;
}

// Launches the attention of a layer step with the split-K partials of chunked
// plans in `partials` (the handle's workspace, or the allocation-free entry
// point's scratch); the event pair brackets the first kernel's start and the
// last kernel's end.
headkv_status launch_attention(headkv_t h, const Layer& L, const LayerDev& D, const AppendArgs& a,
                               const uint16_t* q, float* out, uint64_t* partials, void* stream,
                               void* e0, void* e1, const char* what) {
    AttnPlan plans[2];
    const int np = attn_plans(h, L, a.k != nullptr, plans);
    for (int i = 0; i < np; ++i)
        if (plans[i].chunked && partials == nullptr)
            return fail(HEADKV_ERR_STATE,
                        "the handle has no workspace and this layer's attention is split into "
                        "chunks: use headkv_decode_attn_noalloc");
    // the merge words of a chunked launch are zero until written; the static
    // scratch starts zero, the caller's workspace is zeroed once
    if (partials != nullptr && partials == h->ws && !h->ws_clear) {
        for (int i = 0; i < np; ++i) {
            if (!plans[i].chunked) continue;
            const int e = launch_zero_words(partials, h->ws_bytes / sizeof(uint64_t), stream);
            if (e) return hip_status(e, "workspace clear");
            h->ws_clear = true;
            break;
        }
    }
    for (int i = 0; i < np; ++i) {
        const int e = launch_attn(D, h->shape, a, q, out, partials, plans[i], stream,
                                  i == 0 ? e0 : nullptr, i == np - 1 ? e1 : nullptr);
        if (e) return hip_status(e, what);
    }
    return ok();
}

}  // namespace

extern "C" {

headkv_status headkv_append_and_evict(headkv_t h, int32_t layer, int32_t step, const uint16_t* q,
                                      const uint16_t* k, const uint16_t* v, void* stream) {
    AppendArgs a;
    bool update = false;
    int u = 0;
    headkv_status st = prepare_append(h, layer, step, q, k, v, &a, &update, &u);
    if (st) return st;
    Layer& L = h->layers[layer];
    const headkv_config& c = h->cfg;
    LayerDev D = dev_of(h, L);
    if (update)
        st = hip_status(launch_update(D, h->shape, a, nullptr, 0, 0, 0, c.recent_len, c.rs_num,
                                      c.rs_den, u, step, max_cap(L), sqrt_d(h), stream, nullptr,
                                      nullptr),
                        "append + update launch");
    else
        st = hip_status(launch_append(D, h->shape, a, stream), "append launch");
    if (st) return st;
    commit_append(h, L, step, update);
    return ok();
}

}  // extern "C"

namespace {

// Algorithmic HBM bytes of the kernels of a decode step, from the host mirror
// (n before the step's append).
//   fused append + attention: K and V of the prefix, the retained tokens and
//   the new token; q in, the output out; the new K/V row, its position and q's
//   ring row written.
double fused_step_bytes(headkv_t h, const Layer& L) {
    const headkv_config& c = h->cfg;
    const double d = c.head_dim;
    double tokens = 0;
    for (int n : L.n) tokens += c.prefix_len + n + 1;
    const double per_head = d * 2 + d * 4 + 3 * d * 2 + 4;
    return tokens * 2 * d * 2 + h->shape.BH * per_head;
}

//   attention alone (n after the step's update): K, V, q and the output.
double attn_bytes(headkv_t h, const Layer& L) {
    const headkv_config& c = h->cfg;
    const double d = c.head_dim;
    double tokens = 0;
    for (int n : L.n) tokens += c.prefix_len + n;
    return tokens * 2 * d * 2 + h->shape.BH * (d * 2 + d * 4);
}

//   append + periodic update: the append (q, k, v in; K/V row, position and
//   q's ring row written); every head's positions; for a global head that
//   evicts, the keys of its history and the window's queries from the ring;
//   and at most M K/V rows and positions moved by the compaction.
double update_bytes(headkv_t h, const Layer& L) {
    const headkv_config& c = h->cfg;
    const double d = c.head_dim;
    double b = 0;
    for (int i = 0; i < h->shape.BH; ++i) {
        const int n = L.n[i] + 1, B = L.budget[i];
        const int w_eff = std::min(c.recent_len, B);
        const int T = std::max(0, n - w_eff);
        const int M = std::max(0, T - (B - w_eff));
        b += 3 * 2 * d + 3 * 2 * d + 4 + 4.0 * n;
        if (M > 0) {
            if (!L.label_local[i]) b += T * 2 * d + std::min(c.period, L.last_step + 2) * 2 * d;
            b += M * (2 * 2 * 2 * d + 8);
        }
    }
    return b;
}

headkv_status decode_step_impl(headkv_t h, int32_t layer, int32_t step, const uint16_t* q,
                               const uint16_t* k, const uint16_t* v, float* out, void* stream,
                               bool time_it) {
    if (!out) return fail(HEADKV_ERR_INVALID_ARG, "out is NULL");
    if (!aligned(out, 16)) return fail(HEADKV_ERR_INVALID_ARG, "out not 16-byte aligned");
    AppendArgs a;
    bool update = false;
    int u = 0;
    headkv_status st = prepare_append(h, layer, step, q, k, v, &a, &update, &u);
    if (st) return st;
    Layer& L = h->layers[layer];
    const headkv_config& c = h->cfg;
    if (!L.grouped && step == h->t_g)
        return fail(HEADKV_ERR_STATE, "the grouping step needs the separate calls");
    LayerDev D = dev_of(h, L);
    AppendArgs none = a;
    none.k = none.v = none.q = nullptr;
    void *e0, *e1;
    if (update) {
        const double ub = update_bytes(h, L);  // over the lengths before the step
        const int lds_cap = max_cap(L);
        commit_append(h, L, step, update);
        // the attention that follows, over the lengths after the update: with
        // one block per head, the update's block attends too
        AttnPlan plans[2];
        const int np = attn_plans(h, L, false, plans);
        if (c.score_mode == HEADKV_SCORE_MEAN_LOGIT && np == 1 && !plans[0].chunked) {
            take_events(h, time_it, HEADKV_TIMED_UPDATE_ATTN, ub + attn_bytes(h, L), &e0, &e1);
            return hip_status(launch_update_attn(D, h->shape, a, c.recent_len, c.rs_num, c.rs_den,
                                                 u, step, lds_cap, sqrt_d(h), q, out,
                                                 plans[0].use_order, plans[0].pad_len,
                                                 plans[0].threads, plans[0].tpr, stream, e0, e1),
                              "append + update + attention launch");
        }
        take_events(h, time_it, HEADKV_TIMED_UPDATE, ub, &e0, &e1);
        st = hip_status(launch_update(D, h->shape, a, nullptr, 0, 0, 0, c.recent_len, c.rs_num,
                                      c.rs_den, u, step, lds_cap, sqrt_d(h), stream, e0, e1),
                        "append + update launch");
        if (st) return st;
        take_events(h, time_it, HEADKV_TIMED_ATTN, attn_bytes(h, L), &e0, &e1);
        // over the lengths the update wrote (D still counts the step's append)
        return launch_attention(h, L, dev_of(h, L), none, q, out, static_cast<uint64_t*>(h->ws),
                                stream, e0, e1, "attention launch");
    }
    // the append is fused into the attention; the host counts it (dn)
    take_events(h, time_it, L.grouped ? HEADKV_TIMED_ATTN_APPEND : HEADKV_TIMED_ATTN_APPEND_DENSE,
                fused_step_bytes(h, L), &e0, &e1);
    st = launch_attention(h, L, D, a, q, out, static_cast<uint64_t*>(h->ws), stream, e0, e1,
                          "append + attention launch");
    if (st) return st;
    commit_append(h, L, step, update);
    return ok();
}

}  // namespace

extern "C" {

headkv_status headkv_decode_step(headkv_t h, int32_t layer, int32_t step, const uint16_t* q,
                                 const uint16_t* k, const uint16_t* v, float* out, void* stream) {
    return decode_step_impl(h, layer, step, q, k, v, out, stream, false);
}

headkv_status headkv_run_steps(headkv_t h, int32_t step_begin, int32_t step_end,
                               const uint16_t* const* q, const uint16_t* const* k,
                               const uint16_t* const* v, int64_t step_stride, float* const* out,
                               int32_t timing_every, void* stream) {
    if (!h) return fail(HEADKV_ERR_INVALID_ARG, "handle is NULL");
    if (!q || !k || !v || !out) return fail(HEADKV_ERR_INVALID_ARG, "NULL pointer array");
    if (step_begin < 0 || step_end < step_begin || step_stride < 0 || timing_every < 0)
        return fail(HEADKV_ERR_INVALID_ARG, "bad step range, stride or timing interval");
    // every step's rows must keep the 16-byte alignment of the first
    if ((step_stride * (int64_t)sizeof(uint16_t)) % 16 != 0)
        return fail(HEADKV_ERR_INVALID_ARG, "step_stride is not a multiple of 8 elements");
    const int NL = h->cfg.num_layers;
    for (int t = step_begin; t < step_end; ++t) {
        const bool time_it = timing_every > 0 && t % timing_every == 0;
        for (int l = 0; l < NL; ++l) {
            if (!q[l] || !k[l] || !v[l] || !out[l])
                return fail(HEADKV_ERR_INVALID_ARG, "NULL layer pointer");
            const size_t off = (size_t)t * (size_t)step_stride;
            headkv_status st = decode_step_impl(h, l, t, q[l] + off, k[l] + off, v[l] + off,
                                                out[l], stream, time_it);
            if (st) return st;
        }
    }
    return ok();
}

headkv_status headkv_timing_reserve(headkv_t h, int64_t launches) {
    if (!h || launches < 0) return fail(HEADKV_ERR_INVALID_ARG, "bad handle or count");
    while ((int64_t)h->events.size() < 2 * launches) {
        hipEvent_t e;
        headkv_status st = hip_status(hipEventCreate(&e), "event create");
        if (st) return st;
        h->events.push_back(e);
    }
    h->timed_bytes.resize(h->events.size() / 2);
    h->timed_kind.resize(h->events.size() / 2);
    return ok();
}

headkv_status headkv_timing_collect(headkv_t h, double* kernel_ms, int64_t* launches,
                                    double* alg_bytes, int64_t* dropped) {
    if (!h || !kernel_ms || !launches || !alg_bytes || !dropped)
        return fail(HEADKV_ERR_INVALID_ARG, "NULL pointer");
    for (int k = 0; k < HEADKV_TIMED_KINDS; ++k) {
        kernel_ms[k] = 0;
        launches[k] = 0;
        alg_bytes[k] = 0;
    }
    if (h->timed > 0) {
        headkv_status st = hip_status(hipEventSynchronize(h->events[2 * h->timed - 1]), "event wait");
        if (st) return st;
    }
    for (size_t i = 0; i < h->timed; ++i) {
        float e = 0;
        headkv_status st = hip_status(hipEventElapsedTime(&e, h->events[2 * i], h->events[2 * i + 1]),
                                      "event time");
        if (st) return st;
        const int k = h->timed_kind[i];
        kernel_ms[k] += e;
        launches[k] += 1;
        alg_bytes[k] += h->timed_bytes[i];
    }
    *dropped = h->timing_dropped;
    h->timed = 0;
    h->timing_dropped = 0;
    return ok();
}

headkv_status headkv_score_heads(headkv_t h, int32_t layer, const uint16_t* q, int32_t* n_star,
                                 uint8_t* is_local, void* stream) {
    headkv_status st = check_layer(h, layer);
    if (st) return st;
    if (!q || !n_star || !is_local) return fail(HEADKV_ERR_INVALID_ARG, "NULL pointer");
    if (!aligned(q, 16)) return fail(HEADKV_ERR_INVALID_ARG, "q not 16-byte aligned");
    Layer& L = h->layers[layer];
    if (!L.prefilled || L.grouped || L.last_step != h->t_g)
        return fail(HEADKV_ERR_STATE, "score_heads runs once, right after the append of step group_threshold - 1");
    const headkv_config& c = h->cfg;
    const int len = c.prefix_len + h->t_g + 1;
    return hip_status(launch_score(dev_of(h, L), h->shape, q, n_star, is_local, len,
                                   std::sqrt((double)c.head_dim), c.tau, c.local_window, stream),
                      "score launch");
}

headkv_status headkv_assign_budgets(headkv_t h, int32_t layer, const uint8_t* is_local,
                                    const int32_t* budget_override, int32_t* budgets,
                                    void* ragged_kv, size_t ragged_bytes,
                                    size_t* ragged_bytes_needed, void* stream) {
    headkv_status st = check_layer(h, layer);
    if (st) return st;
    if (!is_local || !budgets || !ragged_bytes_needed) return fail(HEADKV_ERR_INVALID_ARG, "NULL pointer");
    const headkv_config& c = h->cfg;
    if (c.budget_mode == HEADKV_BUDGET_OVERRIDE && !budget_override)
        return fail(HEADKV_ERR_INVALID_ARG, "budget_override is NULL in override mode");
    if (ragged_kv && !aligned(ragged_kv, 256)) return fail(HEADKV_ERR_INVALID_ARG, "ragged_kv not 256-byte aligned");
    Layer& L = h->layers[layer];
    if (!L.prefilled || L.grouped || L.last_step != h->t_g)
        return fail(HEADKV_ERR_STATE, "assign_budgets runs once, at step group_threshold - 1");
    const int BH = h->shape.BH;
    hipStream_t s = (hipStream_t)stream;
    LayerDev Dold = dev_of(h, L);
    st = hip_status(launch_budgets(Dold, h->shape, is_local, budget_override, budgets, c.budget_mode,
                                   c.row_len, c.recent_len, c.rho_num, c.rho_den, c.cfg_pairs, stream),
                    "budget launch");
    if (st) return st;
    std::vector<int32_t> bud(BH);
    std::vector<int32_t> lab(BH);  // the labels the budgets used (cfg pairs applied)
    st = hip_status(hipMemcpyAsync(bud.data(), budgets, sizeof(int32_t) * BH, hipMemcpyDeviceToHost, s),
                    "budget read-back");
    if (!st) st = hip_status(hipMemcpyAsync(lab.data(), Dold.label, sizeof(int32_t) * BH,
                                            hipMemcpyDeviceToHost, s),
                             "label read-back");
    if (st) {
        (void)hipStreamSynchronize(s);
        return st;
    }
    st = hip_status(hipStreamSynchronize(s), "stream wait");
    if (st) return st;
    // segments: prefix + min(budget + P, N) slots each, in head order
    std::vector<int64_t> off(BH);
    std::vector<int32_t> cap(BH);
    std::vector<int> cap_i(BH);
    size_t total = 0;
    for (int i = 0; i < BH; ++i) {
        if (bud[i] < 1 || bud[i] > c.num_visual)
            return fail(HEADKV_ERR_INVALID_ARG, "a budget is outside [1, num_visual]");
        cap[i] = std::min(bud[i] + c.period, c.num_visual);
        if (cap[i] > HEADKV_MAX_CAPACITY)
            return fail(HEADKV_ERR_UNSUPPORTED, "budget + period exceeds HEADKV_MAX_CAPACITY");
    }
    if (c.attn_strategy == HEADKV_ATTN_PADDED) {  // every head padded to the largest
        const int32_t cmax = *std::max_element(cap.begin(), cap.end());
        std::fill(cap.begin(), cap.end(), cmax);
    }
    for (int i = 0; i < BH; ++i) {
        cap_i[i] = cap[i];
        off[i] = (int64_t)total;
        total += segment_bytes(c.prefix_len, cap[i], c.head_dim);
    }
    *ragged_bytes_needed = total;
    if (!ragged_kv || ragged_bytes < total)
        return fail(HEADKV_ERR_CAPACITY, "ragged_kv is NULL or smaller than *ragged_bytes_needed");
    // attention dispatch order: longest heads first, so that when a layer
    // needs more than one round of blocks the short heads fill the tail; with
    // HEADKV_ATTN_GROUPED the global heads, then the local heads
    std::vector<int32_t> order(BH);
    for (int i = 0; i < BH; ++i) order[i] = i;
    if (c.attn_strategy == HEADKV_ATTN_GROUPED)
        std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return lab[a] < lab[b]; });
    else
        std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return cap[a] > cap[b]; });
    int n_global = 0;
    for (int i = 0; i < BH; ++i) n_global += lab[i] ? 0 : 1;
    // chunk table of the new layout, the chunks of a head contiguous
    const int chunk_threads = pick_chunk_threads(c.prefix_len, c.head_dim, cap_i);
    std::vector<uint32_t> items;
    std::vector<int32_t> item_start(BH + 1);
    for (int i = 0; i < BH; ++i) {
        item_start[i] = (int32_t)items.size();
        const int nc = chunks_of(c.prefix_len, cap[i], chunk_threads, c.head_dim);
        for (int k = 0; k < nc; ++k) items.push_back(((uint32_t)i << 8) | (uint32_t)k);
    }
    item_start[BH] = (int32_t)items.size();
    // tables of the new layout (the host vectors outlive the copies: the stream
    // is waited for below on every path)
    char* mb = static_cast<char*>(L.meta);
    st = hip_status(hipMemcpyAsync(mb + h->ml.seg_off, off.data(), sizeof(int64_t) * BH, hipMemcpyHostToDevice, s), "table upload");
    if (!st) st = hip_status(hipMemcpyAsync(mb + h->ml.cap, cap.data(), sizeof(int32_t) * BH, hipMemcpyHostToDevice, s), "table upload");
    if (!st) st = hip_status(hipMemcpyAsync(mb + h->ml.order, order.data(), sizeof(int32_t) * BH, hipMemcpyHostToDevice, s), "table upload");
    if (!st) st = hip_status(hipMemcpyAsync(mb + h->ml.items, items.data(), sizeof(uint32_t) * items.size(), hipMemcpyHostToDevice, s), "table upload");
    if (!st) st = hip_status(hipMemcpyAsync(mb + h->ml.item_start, item_start.data(), sizeof(int32_t) * (BH + 1), hipMemcpyHostToDevice, s), "table upload");
    // padded rows are read (and masked) by the attention: keep them finite
    if (!st && c.attn_strategy == HEADKV_ATTN_PADDED)
        st = hip_status(hipMemsetAsync(ragged_kv, 0, total, s), "ragged clear");
    // first update, fused with the move from the dense buffer into the segments
    if (!st) {
        LayerDev Dnew = make_layer_dev(ragged_kv, L.meta, h->ml);
        Dnew.dn = L.dn;  // the lengths it moves: prefill's 0 plus every append since
        AppendArgs none{};
        st = hip_status(launch_update(Dnew, h->shape, none, static_cast<const char*>(L.dense), 1,
                                      h->dense_seg, h->dense_cap, c.recent_len, c.rs_num, c.rs_den,
                                      0, h->t_g, h->dense_cap, sqrt_d(h), stream, nullptr, nullptr),
                        "relayout launch");
    }
    headkv_status st_wait = hip_status(hipStreamSynchronize(s), "stream wait");
    if (st || st_wait) {
        // the metadata may already describe the per-head segments while the
        // move into them did not run: nothing may use this layer until it is
        // prefilled again
        L.prefilled = false;
        return fail(st ? st : st_wait, g_err + " (the layer must be prefilled again)");
    }
    L.ragged = ragged_kv;
    L.grouped = true;
    L.budget.assign(bud.begin(), bud.end());
    L.label_local.assign(lab.begin(), lab.end());
    L.cap.assign(cap.begin(), cap.end());
    L.chunk_threads = chunk_threads;
    L.items = (int)items.size();
    L.n_global = n_global;
    for (int i = 0; i < BH; ++i) L.n[i] = std::min(L.n[i], L.budget[i]);
    L.dn = 0;  // the relayout wrote every head's length
    return ok();
}

}  // extern "C"

namespace {

headkv_status check_decode_attn(headkv_t h, int32_t layer, const uint16_t* q, float* out) {
    headkv_status st = check_layer(h, layer);
    if (st) return st;
    if (!q || !out) return fail(HEADKV_ERR_INVALID_ARG, "q / out is NULL");
    if (!aligned(q, 16) || !aligned(out, 16))
        return fail(HEADKV_ERR_INVALID_ARG, "q / out not 16-byte aligned");
    Layer& L = h->layers[layer];
    if (!L.prefilled || L.last_step < 0) return fail(HEADKV_ERR_STATE, "decode_attn before the first append");
    if (!L.grouped && L.last_step == h->t_g)
        return fail(HEADKV_ERR_STATE, "assign_budgets must run before attention at step group_threshold - 1");
    return ok();
}

}  // namespace

extern "C" {

headkv_status headkv_decode_attn(headkv_t h, int32_t layer, const uint16_t* q, float* out,
                                 void* stream) {
    headkv_status st = check_decode_attn(h, layer, q, out);
    if (st) return st;
    const Layer& L = h->layers[layer];
    AppendArgs none{};
    return launch_attention(h, L, dev_of(h, L), none, q, out, static_cast<uint64_t*>(h->ws), stream,
                            nullptr, nullptr, "attention launch");
}

headkv_status headkv_decode_attn_noalloc(headkv_t h, int32_t layer, const uint16_t* q, float* out,
                                         void* stream) {
    headkv_status st = check_decode_attn(h, layer, q, out);
    if (st) return st;
    const Layer& L = h->layers[layer];
    AttnPlan plans[2];
    const int np = attn_plans(h, L, false, plans);
    bool chunked = false;
    for (int i = 0; i < np; ++i) {
        if (!plans[i].chunked) continue;
        chunked = true;
        const size_t need = (size_t)plans[i].items * h->cfg.head_dim * sizeof(uint64_t);
        if (need > kScratchBytes)
            return fail(HEADKV_ERR_CAPACITY, "the layer's chunked attention needs " +
                                                 std::to_string(need) + " bytes of partials, more "
                                                 "than the " + std::to_string(kScratchBytes) +
                                                 "-byte scratch: use headkv_decode_attn");
    }
    void* scratch = nullptr;
    if (chunked) {
        st = hip_status(scratch_address(&scratch), "scratch address");
        if (st) return st;
    }
    AppendArgs none{};
    return launch_attention(h, L, dev_of(h, L), none, q, out, static_cast<uint64_t*>(scratch), stream,
                            nullptr, nullptr, "attention launch");
}

headkv_status headkv_decode_attn_layers(headkv_t h, int32_t layer_begin, int32_t layer_end,
                                        const uint16_t* const* q, float* const* out,
                                        void* stream) {
    if (!h) return fail(HEADKV_ERR_INVALID_ARG, "handle is NULL");
    if (!q || !out) return fail(HEADKV_ERR_INVALID_ARG, "NULL pointer array");
    const int n = layer_end - layer_begin;
    if (layer_begin < 0 || layer_end > h->cfg.num_layers || n < 1)
        return fail(HEADKV_ERR_INVALID_ARG, "bad layer range");
    if (n > kMaxLayersPerLaunch) return fail(HEADKV_ERR_UNSUPPORTED, "more than 64 layers");
    const int BH = h->shape.BH;
    if (BH < kCus || h->cfg.attn_strategy != HEADKV_ATTN_VARLEN)
        return fail(HEADKV_ERR_UNSUPPORTED, "multi-layer attention needs >= 256 heads and the varlen strategy");
    for (int i = 0; i < n; ++i) {
        if (!q[i] || !out[i]) return fail(HEADKV_ERR_INVALID_ARG, "NULL layer pointer");
        if (!aligned(q[i], 16) || !aligned(out[i], 16))
            return fail(HEADKV_ERR_INVALID_ARG, "q / out not 16-byte aligned");
    }
    LayersArg args{};
    int len_max = 0;
    for (int i = 0; i < n; ++i) {
        Layer& L = h->layers[layer_begin + i];
        if (!L.prefilled || L.last_step < 0)
            return fail(HEADKV_ERR_STATE, "decode_attn before the first append");
        if (!L.grouped && L.last_step == h->t_g)
            return fail(HEADKV_ERR_STATE, "assign_budgets must run before attention at step group_threshold - 1");
        args.kv[i] = L.grouped ? L.ragged : L.dense;
        args.meta[i] = L.meta;
        args.dn[i] = L.dn;
        args.q[i] = q[i];
        args.out[i] = out[i];
        len_max = std::max(len_max, h->cfg.prefix_len + *std::max_element(L.n.begin(), L.n.end()));
    }
    const int t = resident_threads(BH);
    if (BH > attn_resident_blocks(t))
        return fail(HEADKV_ERR_UNSUPPORTED, "multi-layer attention needs every head resident");
    const int tpr = pass_tpr(len_max, t, h->cfg.head_dim);
    return hip_status(launch_attn_layers(args, n, h->ml, h->shape, t, tpr, stream),
                      "multi-layer attention launch");
}

headkv_status headkv_export_retained(headkv_t h, int32_t layer, uint8_t* mask, int32_t* count,
                                     void* stream) {
    headkv_status st = check_layer(h, layer);
    if (st) return st;
    if (!mask || !count) return fail(HEADKV_ERR_INVALID_ARG, "mask / count is NULL");
    Layer& L = h->layers[layer];
    if (!L.prefilled) return fail(HEADKV_ERR_STATE, "export before prefill");
    return hip_status(launch_export(dev_of(h, L), h->shape, mask, count, stream), "export launch");
}

const char* headkv_last_error(void) { return g_err.c_str(); }

}  // extern "C"
