// HIP kernels of the compressed cache, written for gfx950 (CDNA4: 64-lane
// wavefronts, 160 KB LDS per CU, 8 XCDs).
//
//   k_prefill  Step 1 cache prefilling (Sec. 4): conditional keys/values into
//              rows 0..C-1 of every head, layer state reset.
//   k_append   cache append (Sec. 3, KV Cache) + running sum of the queries of
//              the current update window (Eq. 6 is linear in the queries);
//              also fused into k_update and the attention kernels.
//   k_score    head grouping (Sec. 4, Step 2), fp64.
//   k_budgets  per-head budgets (Sec. 5.1, Implementation Details).
//   k_update   periodic update (Eqs. 2-6): sliding window (Eq. 3) or
//              Stratified Token Eviction (Eqs. 4-6), fused with the
//              compaction of the head's slots or, at the grouping step, with
//              the move into the head's own segment.
//   k_export   retained-position masks for parity checks.
//
// Everything that decides an index (grouping mass, eviction scores) is
// computed in fp64 with one fixed summation order, so the decisions do not
// depend on thread scheduling; multiplies and adds stay separate wherever a
// product can round (the attention-sum logits multiply two bf16 values, exact
// in fp64, and use fma).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/headkv.h"
#include "attn_block.h"
#include "device_common.h"
#include "layout.h"

namespace headkv {
namespace {

using namespace dev;

// ------------------------------------------------------------------ prefill
__global__ __launch_bounds__(kBlock) void k_prefill(LayerDev L, int C, int d, const uint16_t* kc,
                                                    const uint16_t* vc, int64_t seg_bytes,
                                                    int dense_cap, int dense_chunks) {
    prefill_head(L, blockIdx.x, gridDim.x, C, d, kc, vc, seg_bytes, dense_cap, dense_chunks, 0, C,
                 true, threadIdx.x, kBlock);
}

__global__ void k_append(LayerDev L, int C, int d, AppendArgs a) {
    const int h = blockIdx.x;
    append_token(L, C, d, h, head_len(L, h), a, threadIdx.x);
}

// ------------------------------------------------------------ head grouping
__global__ __launch_bounds__(kBlock) void k_score(LayerDev L, int d, const uint16_t* q,
                                                  int32_t* n_star, uint8_t* is_local, int len,
                                                  double sqrt_d, double tau, int local_window) {
#pragma clang fp contract(off)
    extern __shared__ double a[];  // [len]
    __shared__ double qd[128];
    __shared__ double red[kBlock / 64];
    __shared__ double zsh;
    const int h = blockIdx.x, tid = threadIdx.x;
    for (int i = tid; i < d; i += kBlock) qd[i] = bf_f64(q[(size_t)h * d + i]);
    __syncthreads();
    const uint16_t* K = reinterpret_cast<const uint16_t*>(L.kv + L.seg_off[h]);
    // logits q.k_j / sqrt(d), dims summed in order
    double m = -INFINITY;
    for (int j = tid; j < len; j += kBlock) {
        const uint16_t* kr = K + (size_t)j * d;
        double acc = 0.0;
        for (int i = 0; i < d; i += 8) {
            const Words<4> u = *reinterpret_cast<const Words<4>*>(kr + i);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc = acc + qd[i + 2 * e] * (double)bf_lo(u.w[e]);
                acc = acc + qd[i + 2 * e + 1] * (double)bf_hi(u.w[e]);
            }
        }
        a[j] = acc / sqrt_d;
        m = fmax(m, a[j]);
    }
    for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
    if ((tid & 63) == 0) red[tid >> 6] = m;
    __syncthreads();
    m = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
    for (int j = tid; j < len; j += kBlock) a[j] = exp(a[j] - m);
    __syncthreads();
    if (tid == 0) {  // normaliser, summed over the cache in order
        double z = 0.0;
        for (int j = 0; j < len; ++j) z += a[j];
        zsh = z;
    }
    __syncthreads();
    const double z = zsh;
    for (int j = tid; j < len; j += kBlock) a[j] = a[j] / z;
    __syncthreads();
    if (tid == 0) {  // mass accumulated backward from the newest token
        double S = 0.0;
        int ns = len;
        for (int nn = 1; nn <= len; ++nn) {
            S += a[len - nn];
            if (S >= tau) {
                ns = nn;
                break;
            }
        }
        const int loc = ns < local_window ? 1 : 0;
        n_star[h] = ns;
        is_local[h] = (uint8_t)loc;
        L.nstar[h] = ns;
        L.label[h] = loc;
    }
}

// ------------------------------------------------------------------ budgets
// With cfg_pairs, batch rows 2i (conditional) and 2i+1 (unconditional) form a
// guidance pair and both take the labels of row 2i.
__global__ void k_budgets(LayerDev L, int H, int N, const uint8_t* is_local,
                          const int32_t* override_b, int32_t* budgets, int mode, int row_len,
                          int recent_len, int rho_num, int rho_den, int cfg_pairs) {
    __shared__ int n_local;
    const int b = blockIdx.x, h = threadIdx.x, idx = b * H + h;
    if (h == 0) n_local = 0;
    __syncthreads();
    const int loc = is_local[cfg_pairs ? (b & ~1) * H + h : idx] ? 1 : 0;
    if (loc) atomicAdd(&n_local, 1);
    __syncthreads();
    const long long rhoN = (long long)N * rho_num / rho_den;
    const int b_local = recent_len < N ? recent_len : N;
    int B;
    if (mode == HEADKV_BUDGET_OVERRIDE) {
        B = override_b[idx];
    } else if (mode == HEADKV_BUDGET_PAPER) {
        B = loc ? b_local : (int)(rhoN < 1 ? 1 : rhoN);
    } else {
        const int n_global = H - n_local;
        const long long rest = rhoN * H - (long long)n_local * b_local;
        const long long per = (n_global > 0 && rest > 0) ? rest / n_global : 0;
        long long bg = per / row_len * row_len;
        if (bg < b_local) bg = b_local;
        if (bg > N) bg = N;
        B = loc ? b_local : (int)bg;
    }
    budgets[idx] = B;
    L.budget[idx] = B;
    L.label[idx] = loc;
}

// ------------------------------------------------------------------- update
// LDS of one update block, sized by the host from the largest source capacity
// of the launch (`cap`) and the number of visual positions (`N`).
// Steps of the query ring staged through LDS at a time when an update sums
// its window (Eq. 6 scores).
constexpr int kRingChunk = 64;

struct UpdateLds {
    static __host__ __device__ int words(int N) { return (N + 31) >> 5; }
    static __host__ __device__ size_t a16(size_t x) { return (x + 15) & ~(size_t)15; }
    // staged ring rows: the window's first chunk, rounded up to whole groups of
    // eight rows (read eight at a time)
    static __host__ __device__ int stage_steps(int P) { return ((P < kRingChunk ? P : kRingChunk) + 7) & ~7; }
    // bitmap | word prefix | order (u16) | evict (u8) | positions (i32) |
    // scores (f64, also two int lists) | query sum (f64 [d]), or with
    // attention-sum scores G queries (f64 [G][d]) | with Eq. 6 scores: ring
    // rows of the window staged for its sum (bf16 [min(P, kRingChunk)][d]);
    // with attention-sum scores: weights of the cache for each query of a
    // group (f64 [G][C + cap])
    static __host__ __device__ size_t off_wpre(int N) { return a16(4 * (size_t)words(N)); }
    static __host__ __device__ size_t off_order(int N) { return off_wpre(N) + a16(4 * (size_t)words(N)); }
    static __host__ __device__ size_t off_evict(int N, int cap) { return off_order(N) + a16(2 * (size_t)cap); }
    static __host__ __device__ size_t off_pos(int N, int cap) { return off_evict(N, cap) + a16((size_t)cap); }
    static __host__ __device__ size_t off_sig(int N, int cap) { return off_pos(N, cap) + a16(4 * (size_t)cap); }
    static __host__ __device__ size_t off_qs(int N, int cap) { return off_sig(N, cap) + a16(8 * (size_t)cap); }
    static __host__ __device__ size_t off_w(int N, int cap, int d, int g) {
        return off_qs(N, cap) + a16(8 * (size_t)d * g);
    }
    static __host__ __device__ size_t bytes(int N, int cap, int d, int C, bool attn, int g, int P) {
        return off_w(N, cap, d, attn ? g : 1) +
               (attn ? a16(8 * (size_t)g * ((size_t)C + cap)) : a16(2 * (size_t)d * stage_steps(P)));
    }
};

// Window queries scored together by the attention-sum variant: up to 8 when
// the period and the LDS allow, else one at a time.
constexpr int kQueryGroup = 8;

// fp64 score -> unsigned key with the same order (-0 and +0 map to one key,
// since they compare equal).
__device__ __forceinline__ uint64_t score_key(double x) {
    if (x == 0.0) x = 0.0;
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Marks for eviction the mq lowest entries of part [lo, hi) by (score, rank):
// a radix select over the keys, 8 bits per pass from the top, that stops as
// soon as the chosen digit's bucket leaves entirely; if the exact threshold key
// is reached, the entries equal to it leave in rank order.
template <int NT>
__device__ void select_lowest(const double* sig, const uint16_t* order, uint8_t* evict, int lo,
                              int hi, int mq, int tid) {
    __shared__ uint32_t hist[256];
    __shared__ int pick[3];  // digit, entries below its bucket, bucket size
    if (mq <= 0) return;
    if (mq >= hi - lo) {
        for (int r = lo + tid; r < hi; r += NT) evict[order[r]] = 1;
        return;
    }
    uint64_t prefix = 0;  // chosen digits so far
    int want = mq;        // entries still to take at or above the prefix
    for (int shift = 56;; shift -= 8) {
        const uint64_t above = shift == 56 ? 0ull : ~0ull << (shift + 8);
        if (tid < 256) hist[tid] = 0u;
        __syncthreads();
        for (int r = lo + tid; r < hi; r += NT) {
            const uint64_t k = score_key(sig[r]);
            if ((k & above) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
        }
        __syncthreads();
        const int c = tid < 256 ? (int)hist[tid] : 0;
        int tot;
        const int ex = block_exclusive_scan<NT>(c, &tot);
        if (ex < want && want <= ex + c) {
            pick[0] = tid;
            pick[1] = ex;
            pick[2] = c;
        }
        __syncthreads();
        prefix |= (uint64_t)pick[0] << shift;
        want -= pick[1];
        const uint64_t upto = ~0ull << shift;
        if (want == pick[2]) {  // the whole bucket leaves with everything below it
            for (int r = lo + tid; r < hi; r += NT)
                if ((score_key(sig[r]) & upto) <= prefix) evict[order[r]] = 1;
            return;
        }
        if (shift == 0) {  // prefix is the exact threshold key
            int taken = 0;
            for (int r0 = lo; r0 < hi && taken < want; r0 += NT) {
                const int r = r0 + tid;
                const uint64_t k = r < hi ? score_key(sig[r]) : ~0ull;
                const int eq = (r < hi && k == prefix) ? 1 : 0;
                int t;
                const int e = block_exclusive_scan<NT>(eq, &t);
                if (eq && taken + e < want) evict[order[r]] = 1;
                taken += t;
            }
            for (int r = lo + tid; r < hi; r += NT)
                if (score_key(sig[r]) < prefix) evict[order[r]] = 1;
            return;
        }
        __syncthreads();  // hist and pick are rewritten next pass
    }
}

// The same two selections as select_lowest on parts [0, n_long) and
// [n_long, T), when T <= NT / Q: Q consecutive lanes (4 or 2) count the
// entries of an entry's part that come before it by (score, rank),
// and the entry leaves if fewer than its part's m do.  One pass over the part
// instead of up to eight radix passes with their barriers; the count grows
// with the part's size, so larger parts keep the radix select.  A part is
// ranked only if it keeps some and loses some entries (the only parts whose
// scores exist).
template <int NT, int Q>
__device__ void select_small(double* sig, const uint16_t* order, uint8_t* evict, int n_long,
                             int T, int m_long, int m_near, int tid) {
    static_assert(Q == 2 || Q == 4, "two or four lanes per entry");
    uint64_t* key = reinterpret_cast<uint64_t*>(sig);  // keys replace the scores in place
    auto part_of = [&](int r, int& lo, int& hi, int& mq) {
        const bool lng = r < n_long;
        lo = lng ? 0 : n_long;
        hi = lng ? n_long : T;
        mq = lng ? m_long : m_near;
    };
    {
        int lo, hi, mq;
        part_of(tid, lo, hi, mq);
        if (tid < T && mq > 0 && mq < hi - lo) key[tid] = score_key(sig[tid]);
    }
    __syncthreads();
    const int r = tid / Q, q = tid % Q;
    int lo, hi, mq;
    part_of(r, lo, hi, mq);
    if (r >= T || mq <= 0) return;
    if (mq >= hi - lo) {
        if (q == 0) evict[order[r]] = 1;
        return;
    }
    // entries before r count when not greater, those after when less
    const uint64_t kr = key[r];
    int c = 0;
#pragma unroll 4
    for (int j = lo + q; j < hi; j += Q) {
        const uint64_t kj = key[j];
        c += (j < r ? kj <= kr : kj < kr) ? 1 : 0;
    }
    // the Q lanes of an entry (an aligned pair or quad) are all here: summed
    // within the quad by DPP
    c += __builtin_amdgcn_update_dpp(0, c, 0xB1, 0xF, 0xF, false);  // lane ^ 1
    if (Q == 4) c += __builtin_amdgcn_update_dpp(0, c, 0x4E, 0xF, 0xF, false);  // lane ^ 2
    if (q == 0 && c < mq) evict[order[r]] = 1;
}

// q . k of a cached row in fp64, the dims summed in order, without FMA.
template <int D>
__device__ __forceinline__ double dot_row(const double* qd, const uint16_t* row) {
#pragma clang fp contract(off)
    const uint4* kr = reinterpret_cast<const uint4*>(row);
    uint4 v[D / 8];
#pragma unroll
    for (int c = 0; c < D / 8; ++c) v[c] = kr[c];
    double acc = 0.0;
#pragma unroll
    for (int c = 0; c < D / 8; ++c) {
        const uint32_t wv[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc = acc + qd[8 * c + 2 * e] * (double)bf_lo(wv[e]);
            acc = acc + qd[8 * c + 2 * e + 1] * (double)bf_hi(wv[e]);
        }
    }
    return acc;
}

// The attention-sum variant of the eviction score (the oracle's
// ORC_SCORE_ATTN_SUM): for each window query p (steps max(0, step-P+1) ..
// step, from the query ring), its softmax over the cache it attended -- the
// prefix rows, then the retained tokens with position <= p in position order
// -- with logits q.k / sqrt(d) in fp64 and exp(l - max) summed in that order;
// sig[r] for the history ranks [r_lo, r_hi) accumulates the weights query by
// query, in step order.
// The window is taken G queries at a time: each thread reads a cached row once
// and runs the G dot products as G independent fp64 chains (dims in order);
// the G normalisers are summed by G threads at once, each over its query's
// cache in order.  qd: LDS [D][G]; w: LDS [G][wst] with wst >= C + n.
template <int D, int G>
__device__ void attention_sum_scores(const LayerDev& L, const SegPtrs& S, int C, int h, int n,
                                     int r_lo, int r_hi, int step,
                                     const uint16_t* order, const int32_t* pos, double* qd,
                                     double* sig, double* w, int wst, double sqrt_d, int tid) {
#pragma clang fp contract(off)
    constexpr int WAVES = kBlock / 64;
    __shared__ double red[WAVES][G];
    __shared__ double msh[G], zsh[G];
    __shared__ int nvs[G];
    const int P = L.ring_len;
    const int p0 = step - P + 1 > 0 ? step - P + 1 : 0;
    const int lane = tid & 63, wave = tid >> 6;
    for (int r = r_lo + tid; r < r_hi; r += kBlock) sig[r] = 0.0;
    for (int pa = p0; pa <= step; pa += G) {
        const int ng = step + 1 - pa < G ? step + 1 - pa : G;  // queries of this group
        // the group's queries in fp64 (rows past ng are zero and unused)
        for (int i = tid; i < G * D; i += kBlock) {
            const int g = i / D, e = i - g * D;
            qd[e * G + g] = g < ng ? bf_f64(L.qring[((size_t)h * P + (pa + g) % P) * D + e]) : 0.0;
        }
        if (tid < ng) {  // visible visual tokens of query pa + tid: ranks with position <= p
            const int p = pa + tid;
            int lo = 0, hi = n;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (pos[order[mid]] <= p) lo = mid + 1; else hi = mid;
            }
            nvs[tid] = lo;
        }
        __syncthreads();
        int vis[G];  // cache length seen by each query (non-decreasing in g)
#pragma unroll
        for (int g = 0; g < G; ++g) vis[g] = C + nvs[g < ng ? g : ng - 1];
        const int rows = vis[G - 1];
        // logits of every visible row for all queries of the group, and maxima
        double m[G];
#pragma unroll
        for (int g = 0; g < G; ++g) m[g] = -INFINITY;
        for (int j = tid; j < rows; j += kBlock) {
            const uint16_t* row =
                j < C ? S.K + (size_t)j * D : S.K + (size_t)(C + order[j - C]) * D;
            const uint4* kr = reinterpret_cast<const uint4*>(row);
            // the queries are read from LDS for every row: an offset of zero
            // the compiler cannot see through keeps it from hoisting all G x D
            // of them out of the loop
            int zo;
            asm volatile("s_mov_b32 %0, 0" : "=s"(zo));
            const double* qz = qd + zo;
            // qz is dim-major ([D][G]): the query values of the next S dims are
            // read while this S dims' products are added (a scheduling barrier
            // keeps the reads a stage ahead).  The product of two bf16 values
            // is exact in fp64, so an fma rounds exactly like the oracle's
            // multiply and add.
            constexpr int S = 4;
            double acc[G], qa[S][G], qb[S][G];
#pragma unroll
            for (int g = 0; g < G; ++g) acc[g] = 0.0;
#pragma unroll
            for (int e = 0; e < S; ++e)
#pragma unroll
                for (int g = 0; g < G; ++g) qa[e][g] = qz[e * G + g];
            constexpr int HR = D / 16;  // half a row in flight at a time
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                uint4 v[HR];
#pragma unroll
                for (int c = 0; c < HR; ++c) v[c] = kr[half * HR + c];
#pragma unroll
                for (int c = 0; c < HR; ++c) {
                    const uint32_t wv[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
#pragma unroll
                    for (int st = 0; st < 8 / S; ++st) {
                        const int i0 = 8 * (half * HR + c) + st * S;  // first dim of the stage
                        if (i0 + S < D) {
#pragma unroll
                            for (int e = 0; e < S; ++e)
#pragma unroll
                                for (int g = 0; g < G; ++g) qb[e][g] = qz[(i0 + S + e) * G + g];
                        }
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int e = 0; e < S; ++e) {
                            const int k = st * S + e;  // dim within the 16-byte chunk
                            const double kv =
                                (double)((k & 1) ? bf_hi(wv[k / 2]) : bf_lo(wv[k / 2]));
#pragma unroll
                            for (int g = 0; g < G; ++g) acc[g] = fma(qa[e][g], kv, acc[g]);
                        }
#pragma unroll
                        for (int e = 0; e < S; ++e)
#pragma unroll
                            for (int g = 0; g < G; ++g) qa[e][g] = qb[e][g];
                    }
                }
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const double l = acc[g] / sqrt_d;
                w[(size_t)g * wst + j] = l;
                if (j < vis[g]) m[g] = fmax(m[g], l);
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            for (int o = 32; o > 0; o >>= 1) m[g] = fmax(m[g], __shfl_xor(m[g], o));
            if (lane == 0) red[wave][g] = m[g];
        }
        __syncthreads();
        if (tid < G) {
            double mx = red[0][tid];
            for (int i = 1; i < WAVES; ++i) mx = fmax(mx, red[i][tid]);
            msh[tid] = mx;
        }
        __syncthreads();
        for (int j = tid; j < rows; j += kBlock)
#pragma unroll
            for (int g = 0; g < G; ++g)
                if (j < vis[g]) w[(size_t)g * wst + j] = exp(w[(size_t)g * wst + j] - msh[g]);
        __syncthreads();
        if (tid < ng) {  // normaliser of query pa + tid, summed over its cache in order
            const double* wg = w + (size_t)tid * wst;
            const int len = C + nvs[tid];
            double z = 0.0;
            int j = 0;
            // the reads go out eight at a time, the additions stay in order
            for (; j + 8 <= len; j += 8) {
                double t[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) t[u] = wg[j + u];
#pragma unroll
                for (int u = 0; u < 8; ++u) z += t[u];
            }
            for (; j < len; ++j) z += wg[j];
            zsh[tid] = z;
        }
        __syncthreads();
        for (int r = r_lo + tid; r < r_hi; r += kBlock) {
            double a = sig[r];
            for (int g = 0; g < ng; ++g)
                if (r < nvs[g]) a = a + w[(size_t)g * wst + C + r] / zsh[g];
            sig[r] = a;
        }
        __syncthreads();  // qd, w, nvs, msh and zsh are rewritten for the next group
    }
}

// One block per head: optional append, then the periodic update of Eqs. 2-6
// (or, with `relayout`, the first update fused with the move into the head's
// new segment).  ATTN_SUM: the attention-sum scores instead of Eq. 6; a
// separate instantiation, since its fp64 exp needs about twice the registers
// (the Eq. 6 kernel stays under 64 VGPRs: eight 256-thread blocks per CU).
// The update of head h by the block's NT threads (body of k_update and of the
// fused update + attention kernel); returns the head's length afterwards.
// FUSED: the block goes on to the attention, so it has the attention's 128
// VGPRs: where no K row was loaded ahead, a whole row is scored per round
// trip instead of half of one.
template <int D, bool ATTN_SUM, int G, int NT = kBlock, bool FUSED = false>
__device__ __forceinline__ int update_block(const LayerDev& L, int C, int N, const AppendArgs& a,
                                            const char* src_kv, int relayout,
                                            int64_t dense_seg_bytes, int dense_cap,
                                            int recent_len, int rs_num, int rs_den, int u,
                                            int step, int lds_cap, double sqrt_d, int h) {
#pragma clang fp contract(off)
    static_assert(!ATTN_SUM || NT == kBlock, "attention-sum scores run in 256-thread blocks");
    static_assert(NT >= 256 && NT % 64 == 0, "the radix select needs at least 256 threads");
    constexpr int kRow16 = D / 8;  // 16-byte chunks per row
    extern __shared__ __align__(16) unsigned char lds[];
    uint32_t* bm = reinterpret_cast<uint32_t*>(lds);
    int32_t* wpre = reinterpret_cast<int32_t*>(lds + UpdateLds::off_wpre(N));
    uint16_t* order = reinterpret_cast<uint16_t*>(lds + UpdateLds::off_order(N));
    uint8_t* evict = lds + UpdateLds::off_evict(N, lds_cap);
    double* sig = reinterpret_cast<double*>(lds + UpdateLds::off_sig(N, lds_cap));
    double* qs = reinterpret_cast<double*>(lds + UpdateLds::off_qs(N, lds_cap));
    int32_t* pos = reinterpret_cast<int32_t*>(lds + UpdateLds::off_pos(N, lds_cap));
    const int tid = threadIdx.x;
    const int n0 = head_len(L, h);
    const int B = L.budget[h];
    const int local = L.label[h];
    // the segment's metadata too, before the append's stores (after them, the
    // compiler can no longer read it through the scalar cache)
    const int cap_h = L.cap[h];
    const int64_t seg_h = L.seg_off[h];
    // the step's append, then the update that follows it; the update takes the
    // new token's position and query from the append's own values rather than
    // reading them back from memory
    const bool app = a.k != nullptr;
    AppendVals av;
    if (app) {
        av = append_load(D, h, a, tid);
        append_store(L, C, D, h, n0, a, av, tid);
    }
    const int n = n0 + (app ? 1 : 0);
    // Eq. (2): history = retained tokens older than the recent window
    const int w_eff = recent_len < B ? recent_len : B;
    const int T = n > w_eff ? n - w_eff : 0;
    const int keep = B - w_eff;
    const int M = T > keep ? T - keep : 0;
    if (!relayout && M == 0) {
        // every head's length is written at an update (the host's count of
        // appended tokens starts again from it)
        if (tid == 0) L.n[h] = n;
        return n;
    }
    // Eq. 6 window of a global head that evicts: steps w0..step of the query
    // ring (the step's own query, when this kernel appends it, from the
    // append's values)
    const int w0 = step - L.ring_len + 1 > 0 ? step - L.ring_len + 1 : 0;
    const int wlast = app ? step - 1 : step;  // last step read from the ring
    const bool window = !ATTN_SUM && !local && M > 0;

    const int src_cap = relayout ? dense_cap : cap_h;
    char* src_seg = relayout ? const_cast<char*>(src_kv) + (int64_t)h * dense_seg_bytes
                             : L.kv + seg_h;
    SegPtrs S = seg_ptrs(src_seg, C, src_cap, D);
    // With at most one slot per thread, thread s loads its slot's position
    // now, and, for a global head that scores (with registers for a whole row:
    // NT >= 512, or d = 64), its K row right after the positions, so that their round
    // trips overlap the ranking and the window sum.  The appended row is still
    // being stored: its position comes from the step, its row is read when it
    // is scored.
    constexpr bool kRowAhead = (NT >= 512 || D <= 64) && !ATTN_SUM;
    const bool one_slot = n <= NT;
    const int n_ahead = app ? n0 : n;
    const bool ahead = kRowAhead && window && one_slot;
    int p_own = 0;
    if (one_slot && tid < n) p_own = (app && tid == n0) ? a.step : S.pos[tid];
    // The window's first kRingChunk ring rows, loaded now so that their round
    // trip overlaps the ranking.  Every thread loads (past the window's rows,
    // and for a head without a window, the window's first piece again), so
    // that no branch holds a load: the wait for the position before them
    // then leaves them in flight.  16-byte pieces as a vector type: copies of
    // the struct type were kept in scratch memory.
    typedef unsigned int piece_t __attribute__((ext_vector_type(4)));
    constexpr int PER = (kRingChunk * kRow16 + NT - 1) / NT;
    piece_t wbuf[PER];
    {
        const int cw = wlast + 1 - w0 < kRingChunk ? wlast + 1 - w0 : kRingChunk;
        const int cn = window ? cw : 0;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int v0 = tid + k * NT;
            const int v = v0 < cn * kRow16 ? v0 : 0;
            wbuf[k] = reinterpret_cast<const piece_t*>(ring_slot(L, D, h, w0 + v / kRow16))[v % kRow16];
        }
    }
    uint4 krow[kRowAhead ? kRow16 : 1];

    // rank every occupied slot by its position: bitmap + prefix popcount
    const int nw = UpdateLds::words(N);
    for (int i = tid; i < nw; i += NT) bm[i] = 0u;
    for (int i = tid; i < n; i += NT) evict[i] = 0;
    __syncthreads();
    if (one_slot) {
        if (tid < n) {
            pos[tid] = p_own;
            atomicOr(&bm[p_own >> 5], 1u << (p_own & 31));
        }
    } else {
        // PB positions per thread in flight at a time (slot 0 stands in for the
        // slots past n, so that no branch holds a load)
        constexpr int PB = 4;
        for (int s0 = 0; s0 < n; s0 += PB * NT) {
            int pv[PB];
#pragma unroll
            for (int k = 0; k < PB; ++k) {
                const int s = s0 + tid + k * NT;
                pv[k] = S.pos[s < n ? s : 0];
            }
#pragma unroll
            for (int k = 0; k < PB; ++k) {
                const int s = s0 + tid + k * NT;
                if (s < n) {
                    const int p = (app && s == n0) ? a.step : pv[k];
                    pos[s] = p;
                    atomicOr(&bm[p >> 5], 1u << (p & 31));
                }
            }
        }
    }
    // the K rows go out once the positions are in (a wait for a position
    // would otherwise also wait for them); the empty asm completes the
    // position's load on every path, so that no later wait counts the rows
    asm volatile("" ::"v"(p_own));
    if (ahead && tid < n_ahead) {
        const uint4* kr = reinterpret_cast<const uint4*>(S.K + (size_t)(C + tid) * D);
#pragma unroll
        for (int c = 0; c < (kRowAhead ? kRow16 : 1); ++c) krow[c] = kr[c];
    }
    __syncthreads();
    {
        const int w0 = 2 * tid;
        const int c0 = w0 < nw ? __popc(bm[w0]) : 0;
        const int c1 = w0 + 1 < nw ? __popc(bm[w0 + 1]) : 0;
        int tot;
        const int ex = block_exclusive_scan<NT>(c0 + c1, &tot);
        if (w0 < nw) wpre[w0] = ex;
        if (w0 + 1 < nw) wpre[w0 + 1] = ex + c0;
    }
    __syncthreads();
    int r_own = -1;  // rank of this thread's slot (one slot per thread)
    for (int s = tid; s < n; s += NT) {
        const int p = pos[s];
        const int r = wpre[p >> 5] + __popc(bm[p >> 5] & ((1u << (p & 31)) - 1u));
        order[r] = (uint16_t)s;
        r_own = r;
    }
    __syncthreads();

    if (M > 0) {
        if (local) {
            // Eq. (3): sliding window, the M oldest leave
            for (int r = tid; r < M; r += NT) evict[order[r]] = 1;
        } else {
            // Eq. (5): long-range part = the oldest floor(T r_s) history tokens
            const int n_long = (int)((long long)T * rs_num / rs_den);
            const int n_near = T - n_long;
            int m_long = (M + (u & 1)) >> 1;
            int m_near = M - m_long;
            if (m_long > n_long) {
                m_near += m_long - n_long;
                m_long = n_long;
            }
            if (m_near > n_near) {
                m_long += m_near - n_near;
                m_near = n_near;
            }
            // a part is scored only if it keeps some and loses some tokens
            const bool sel_long = m_long > 0 && m_long < n_long;
            const bool sel_near = m_near > 0 && m_near < n_near;
            const int r_lo = sel_long ? 0 : n_long;
            const int r_hi = sel_near ? T : n_long;
            if (ATTN_SUM) {
                attention_sum_scores<D, G>(
                    L, S, C, h, n, r_lo, r_hi, step, order, pos, qs, sig,
                    reinterpret_cast<double*>(lds + UpdateLds::off_w(N, lds_cap, D, G)),
                    C + lds_cap, sqrt_d, tid);
            } else {
            // Eq. (6): mean raw logit of the past-P queries; the positive factor
            // 1/(P sqrt(d)) is dropped, the order is that of (sum q) . k, summed
            // over the dims in order in fp64.  Each thread reads half of its row's
            // 16-byte chunks together and then walks them in order.
            // the window's query sum, q_{w0} + ... + q_step in step order in
            // fp64: up to kRingChunk ring rows at a time (the first chunk loaded
            // above) are staged through LDS, then each of D threads adds its
            // dim's column
            {
                uint16_t* stage = reinterpret_cast<uint16_t*>(lds + UpdateLds::off_w(N, lds_cap, D, 1));
                double qacc = 0.0;
                for (int c0 = w0; c0 <= wlast; c0 += kRingChunk) {
                    const int cn = wlast + 1 - c0 < kRingChunk ? wlast + 1 - c0 : kRingChunk;
                    if (c0 != w0) {
#pragma unroll
                        for (int k = 0; k < PER; ++k) {
                            const int v = tid + k * NT;
                            if (v < cn * kRow16)
                                wbuf[k] = reinterpret_cast<const piece_t*>(
                                    ring_slot(L, D, h, c0 + v / kRow16))[v % kRow16];
                        }
                    }
#pragma unroll
                    for (int k = 0; k < PER; ++k) {
                        const int v = tid + k * NT;
                        if (v < cn * kRow16) reinterpret_cast<piece_t*>(stage)[v] = wbuf[k];
                    }
                    __syncthreads();
                    // eight LDS reads in flight ahead of the in-order adds (the
                    // stage holds whole groups of eight rows; rows past cn are
                    // read and not added)
                    if (tid < D)
                        for (int j0 = 0; j0 < cn; j0 += 8) {
                            uint16_t x[8];
#pragma unroll
                            for (int j = 0; j < 8; ++j) x[j] = stage[(j0 + j) * D + tid];
#pragma unroll
                            for (int j = 0; j < 8; ++j)
                                if (j0 + j < cn) qacc = qacc + bf_f64(x[j]);
                        }
                    __syncthreads();
                }
                if (app && tid < D) qacc = qacc + bf_f64(av.qbits);
                if (tid < D) qs[tid] = qacc;
            }
            __syncthreads();
            if (ahead) {
                // thread s scores its own slot from the row it loaded
                if (tid < n && r_own >= r_lo && r_own < r_hi) {
                    if (tid >= n_ahead) {
                        const uint4* kr = reinterpret_cast<const uint4*>(S.K + (size_t)(C + tid) * D);
#pragma unroll
                        for (int c = 0; c < (kRowAhead ? kRow16 : 1); ++c) krow[c] = kr[c];
                    }
                    double acc = 0.0;
#pragma unroll
                    for (int c = 0; c < (kRowAhead ? kRow16 : 1); ++c) {
                        const uint32_t wv[4] = {krow[c].x, krow[c].y, krow[c].z, krow[c].w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            acc = acc + qs[8 * c + 2 * e] * (double)bf_lo(wv[e]);
                            acc = acc + qs[8 * c + 2 * e + 1] * (double)bf_hi(wv[e]);
                        }
                    }
                    sig[r_own] = acc;
                }
            } else {
                for (int r = r_lo + tid; r < r_hi; r += NT) {
                    const uint4* kr = reinterpret_cast<const uint4*>(S.K + (size_t)(C + order[r]) * D);
                    double acc = 0.0;
                    // half a row in flight at a time keeps the update kernel
                    // under 64 VGPRs (eight blocks per CU), which pays more
                    // than one round trip per row; the fused kernel takes the
                    // whole row unless the row loaded ahead holds registers
                    constexpr int NH = (FUSED && !kRowAhead) ? 1 : 2;
                    constexpr int HR = kRow16 / NH;
#pragma unroll
                    for (int half = 0; half < NH; ++half) {
                        uint4 v[HR];
#pragma unroll
                        for (int c = 0; c < HR; ++c) v[c] = kr[half * HR + c];
#pragma unroll
                        for (int c = 0; c < HR; ++c) {
                            const uint32_t wv[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
                            const int i0 = 8 * (half * HR + c);
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                acc = acc + qs[i0 + 2 * e] * (double)bf_lo(wv[e]);
                                acc = acc + qs[i0 + 2 * e + 1] * (double)bf_hi(wv[e]);
                            }
                        }
                    }
                    sig[r] = acc;
                }
            }
            }
            __syncthreads();
            // per part, evict the m lowest by (score, position)
            if (T <= NT / 4) {
                select_small<NT, 4>(sig, order, evict, n_long, T, m_long, m_near, tid);
            } else if (T <= NT / 2) {
                select_small<NT, 2>(sig, order, evict, n_long, T, m_long, m_near, tid);
            } else {
                select_lowest<NT>(sig, order, evict, 0, n_long, m_long, tid);
                select_lowest<NT>(sig, order, evict, n_long, T, m_near, tid);
            }
        }
    }
    __syncthreads();
    const int n_new = n - M;
    int32_t* list_a = reinterpret_cast<int32_t*>(sig);
    int32_t* list_b = list_a + lds_cap;

    if (relayout) {
        // prefix rows, then kept slots in position order, into the new segment
        SegPtrs Dd = seg_ptrs(L.kv + L.seg_off[h], C, L.cap[h], D);
        const uint4* sk = reinterpret_cast<const uint4*>(S.K);
        const uint4* sv = reinterpret_cast<const uint4*>(S.V);
        uint4* dk = reinterpret_cast<uint4*>(Dd.K);
        uint4* dv = reinterpret_cast<uint4*>(Dd.V);
        for (int i = tid; i < C * kRow16; i += NT) {
            dk[i] = sk[i];
            dv[i] = sv[i];
        }
        int base = 0;
        for (int r0 = 0; r0 < n; r0 += NT) {
            const int r = r0 + tid;
            const int kf = (r < n && !evict[order[r]]) ? 1 : 0;
            int tot;
            const int ex = block_exclusive_scan<NT>(kf, &tot);
            if (kf) {
                list_a[base + ex] = order[r];
                Dd.pos[base + ex] = pos[order[r]];
            }
            base += tot;
        }
        __syncthreads();
        for (int i = tid; i < n_new * kRow16; i += NT) {
            const int j = i / kRow16, c = i - j * kRow16;
            const size_t src = (size_t)(C + list_a[j]) * kRow16 + c;
            const size_t dst = (size_t)(C + j) * kRow16 + c;
            dk[dst] = sk[src];
            dv[dst] = sv[src];
        }
    } else {
        // in place: evicted slots below n_new are refilled from kept slots at or
        // above n_new; the two sets are disjoint, so no copy reads a written row
        int nh = 0, nf = 0;
        for (int s0 = 0; s0 < n; s0 += NT) {
            const int s = s0 + tid;
            const int hf = (s < n_new && evict[s]) ? 1 : 0;
            const int ff = (s >= n_new && s < n && !evict[s]) ? 1 : 0;
            int th, tf;
            const int eh = block_exclusive_scan<NT>(hf, &th);
            const int ef = block_exclusive_scan<NT>(ff, &tf);
            if (hf) list_a[nh + eh] = s;
            if (ff) list_b[nf + ef] = s;
            nh += th;
            nf += tf;
        }
        __syncthreads();
        // the two lists have the same length when exactly M slots were
        // selected; the moves never read past either list
        nh = nh < nf ? nh : nf;
        uint4* k4 = reinterpret_cast<uint4*>(S.K);
        uint4* v4 = reinterpret_cast<uint4*>(S.V);
        for (int i = tid; i < nh * kRow16; i += NT) {
            const int j = i / kRow16, c = i - j * kRow16;
            const size_t dst = (size_t)(C + list_a[j]) * kRow16 + c;
            const size_t src = (size_t)(C + list_b[j]) * kRow16 + c;
            k4[dst] = k4[src];
            v4[dst] = v4[src];
        }
        for (int j = tid; j < nh; j += NT) S.pos[list_a[j]] = pos[list_b[j]];
    }
    if (tid == 0) L.n[h] = n_new;
    return n_new;
}

// NT threads per block: 256 with more heads than CUs (eight blocks per CU),
// 1024 when each head has a CU to itself.
template <int D, bool ATTN_SUM, int G, int NT>
__global__ __launch_bounds__(NT) void k_update(LayerDev L, int C, int N, AppendArgs a,
                                               const char* src_kv, int relayout,
                                               int64_t dense_seg_bytes, int dense_cap,
                                               int recent_len, int rs_num, int rs_den, int u,
                                               int step, int lds_cap, double sqrt_d) {
    update_block<D, ATTN_SUM, G, NT>(L, C, N, a, src_kv, relayout, dense_seg_bytes, dense_cap,
                                     recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d,
                                     (int)blockIdx.x);
}

// A step's append, periodic update and attention in one launch, for layers
// whose attention runs one T-thread block per head: the block updates its
// head (Eq. 6 scores) with all its threads, then attends over the updated
// cache with the length it has just computed.  The head comes from the
// dispatch order when `order` is not null.  At most 128 VGPRs, as the
// attention kernels: 1024 / T blocks per CU.  The metadata tables the first
// loads need, the order and the appended count lead the argument list as
// plain pointers and an integer, preloaded into scalar registers at wave
// launch (the same fields of L are not read); the order is read by a vector
// load, whose wait stays on its own path.
template <int D, int T, int TPR>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(4))) void k_update_attn(
    int32_t* len_n, int32_t* budget, int32_t* label, int64_t* seg_off, int32_t* cap,
    const int32_t* order, int dn, LayerDev L, int C, int N, AppendArgs a, int recent_len,
    int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
    const uint16_t* __restrict__ q, float* __restrict__ out, int pad_len, float qscale) {
    LayerDev M = L;
    M.n = len_n;
    M.budget = budget;
    M.label = label;
    M.seg_off = seg_off;
    M.cap = cap;
    M.dn = dn;
    int h = (int)blockIdx.x;
    if (order != nullptr) {
        int lane0 = 0;
        asm("" : "+v"(lane0));
        h = __builtin_amdgcn_readfirstlane(order[(int)blockIdx.x + lane0]);
    }
    const int n = update_block<D, false, 1, T, true>(M, C, N, a, nullptr, 0, 0, 0, recent_len,
                                               rs_num, rs_den, u, step, lds_cap, sqrt_d, h);
    __syncthreads();  // the rows the update moved are read by other threads
    const AppendArgs none{};
    attn_block<D, false, T, false, TPR>(M, C, none, q, out, nullptr, 0, 0, pad_len, qscale, h,
                                        n);
}

// ------------------------------------------------------------------- export
__global__ __launch_bounds__(kBlock) void k_export(LayerDev L, int C, int d, int N, uint8_t* mask,
                                                   int32_t* count) {
    const int h = blockIdx.x, tid = threadIdx.x;
    const int n = head_len(L, h);
    SegPtrs s = seg_ptrs(L.kv + L.seg_off[h], C, L.cap[h], d);
    for (int p = tid; p < N; p += kBlock) mask[(size_t)h * N + p] = 0;
    __syncthreads();
    for (int j = tid; j < n; j += kBlock) mask[(size_t)h * N + s.pos[j]] = 1;
    if (tid == 0) count[h] = n;
}

inline int last_error() { return (int)hipGetLastError(); }

}  // namespace

int launch_prefill(const LayerDev& L, const Shape& s, const uint16_t* kc, const uint16_t* vc,
                   int64_t dense_seg_bytes, int dense_cap, int dense_chunks, void* stream) {
    hipLaunchKernelGGL(k_prefill, dim3(s.BH), dim3(kBlock), 0, (hipStream_t)stream, L, s.C, s.d,
                       kc, vc, dense_seg_bytes, dense_cap, dense_chunks);
    return last_error();
}

int launch_append(const LayerDev& L, const Shape& s, const AppendArgs& a, void* stream) {
    hipLaunchKernelGGL(k_append, dim3(s.BH), dim3(s.d), 0, (hipStream_t)stream, L, s.C, s.d, a);
    return last_error();
}

int launch_score(const LayerDev& L, const Shape& s, const uint16_t* q, int32_t* n_star,
                 uint8_t* is_local, int len, double sqrt_d, double tau, int local_window,
                 void* stream) {
    hipLaunchKernelGGL(k_score, dim3(s.BH), dim3(kBlock), sizeof(double) * (size_t)len,
                       (hipStream_t)stream, L, s.d, q, n_star, is_local, len, sqrt_d, tau,
                       local_window);
    return last_error();
}

int launch_budgets(const LayerDev& L, const Shape& s, const uint8_t* is_local,
                   const int32_t* override_b, int32_t* budgets, int mode, int row_len,
                   int recent_len, int rho_num, int rho_den, int cfg_pairs, void* stream) {
    hipLaunchKernelGGL(k_budgets, dim3(s.B), dim3(s.H), 0, (hipStream_t)stream, L, s.H, s.N,
                       is_local, override_b, budgets, mode, row_len, recent_len, rho_num, rho_den,
                       cfg_pairs);
    return last_error();
}

// Queries per group of the attention-sum scores: kQueryGroup when the period
// has that many and their weights fit in the LDS, else 1.
int update_query_group(int N, int cap, int d, int C, bool attn_scores, int period) {
    if (!attn_scores || period < kQueryGroup) return 1;
    return UpdateLds::bytes(N, cap, d, C, true, kQueryGroup, period) <= kUpdateLdsBudget ? kQueryGroup : 1;
}

int launch_update(const LayerDev& L, const Shape& s, const AppendArgs& a, const char* src_kv,
                  int relayout, int64_t dense_seg_bytes, int dense_cap, int recent_len,
                  int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                  void* stream, void* ev_start, void* ev_stop) {
    hipStream_t st = (hipStream_t)stream;
    hipEvent_t e0 = static_cast<hipEvent_t>(ev_start), e1 = static_cast<hipEvent_t>(ev_stop);
    const bool attn = L.attn_scores != 0;
    const int G = update_query_group(s.N, lds_cap, s.d, s.C, attn, L.ring_len);
    const size_t lds = UpdateLds::bytes(s.N, lds_cap, s.d, s.C, attn, G, L.ring_len);
    // allow the update block more than 64 KB of dynamic LDS (gfx950: 160 KB)
    static const bool lds_ok = [] {
        const int max_lds = 160 * 1024;
        const void* fns[8] = {reinterpret_cast<const void*>(&k_update<128, false, 1, kBlock>),
                              reinterpret_cast<const void*>(&k_update<128, false, 1, 1024>),
                              reinterpret_cast<const void*>(&k_update<128, true, 1, kBlock>),
                              reinterpret_cast<const void*>(&k_update<128, true, kQueryGroup, kBlock>),
                              reinterpret_cast<const void*>(&k_update<64, false, 1, kBlock>),
                              reinterpret_cast<const void*>(&k_update<64, false, 1, 1024>),
                              reinterpret_cast<const void*>(&k_update<64, true, 1, kBlock>),
                              reinterpret_cast<const void*>(&k_update<64, true, kQueryGroup, kBlock>)};
        bool ok = true;
        for (const void* f : fns)
            ok = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, max_lds) ==
                     hipSuccess && ok;
        (void)hipGetLastError();
        return ok;
    }();
    (void)lds_ok;
    // a CU per head: the whole CU's threads on it (the attention-sum variant
    // keeps 256)
    const bool wide = !attn && s.BH <= kCus;
#define HEADKV_UPDATE(D_, A_, G_, NT_)                                                             \
    hipExtLaunchKernelGGL((k_update<D_, A_, G_, NT_>), dim3(s.BH), dim3(NT_), lds, st, e0, e1, 0,  \
                          L, s.C, s.N, a, src_kv, relayout, dense_seg_bytes, dense_cap,           \
                          recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d)
    if (s.d == 128) {
        if (wide) HEADKV_UPDATE(128, false, 1, 1024);
        else if (!attn) HEADKV_UPDATE(128, false, 1, kBlock);
        else if (G == kQueryGroup) HEADKV_UPDATE(128, true, kQueryGroup, kBlock);
        else HEADKV_UPDATE(128, true, 1, kBlock);
    } else {
        if (wide) HEADKV_UPDATE(64, false, 1, 1024);
        else if (!attn) HEADKV_UPDATE(64, false, 1, kBlock);
        else if (G == kQueryGroup) HEADKV_UPDATE(64, true, kQueryGroup, kBlock);
        else HEADKV_UPDATE(64, true, 1, kBlock);
    }
#undef HEADKV_UPDATE
    return last_error();
}

namespace {

template <int D, int T, int TPR>
void update_attn_launch(const LayerDev& L, const Shape& s, const AppendArgs& a, int recent_len,
                        int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                        const uint16_t* q, float* out, int use_order, int pad_len, size_t lds,
                        hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    // allow more than 64 KB of dynamic LDS (gfx950: 160 KB), once per kernel
    static const bool lds_ok = [] {
        const bool ok = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_update_attn<D, T, TPR>),
                                            hipFuncAttributeMaxDynamicSharedMemorySize,
                                            160 * 1024) == hipSuccess;
        (void)hipGetLastError();
        return ok;
    }();
    (void)lds_ok;
    const float qscale = (float)(1.4426950408889634 / sqrt_d);
    hipExtLaunchKernelGGL((k_update_attn<D, T, TPR>), dim3(s.BH), dim3(T), lds, st, e0, e1, 0,
                          L.n, L.budget, L.label, L.seg_off, L.cap,
                          use_order ? L.order : static_cast<int32_t*>(nullptr), L.dn, L, s.C, s.N,
                          a, recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d, q, out,
                          pad_len, qscale);
}

template <int D, int T>
void update_attn_tpr(const LayerDev& L, const Shape& s, const AppendArgs& a, int recent_len,
                     int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                     const uint16_t* q, float* out, int use_order, int pad_len, int tpr,
                     size_t lds, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    if (tpr == kAttnTpr)
        update_attn_launch<D, T, kAttnTpr>(L, s, a, recent_len, rs_num, rs_den, u, step, lds_cap,
                                           sqrt_d, q, out, use_order, pad_len, lds, st, e0, e1);
    else if (tpr == kAttnTprShort)
        update_attn_launch<D, T, kAttnTprShort>(L, s, a, recent_len, rs_num, rs_den, u, step,
                                                lds_cap, sqrt_d, q, out, use_order, pad_len, lds,
                                                st, e0, e1);
    else if (tpr == kAttnTprWide)
        update_attn_launch<D, T, kAttnTprWide>(L, s, a, recent_len, rs_num, rs_den, u, step,
                                               lds_cap, sqrt_d, q, out, use_order, pad_len, lds,
                                               st, e0, e1);
    else
        update_attn_launch<D, T, kAttnTpr / 2>(L, s, a, recent_len, rs_num, rs_den, u, step,
                                               lds_cap, sqrt_d, q, out, use_order, pad_len, lds,
                                               st, e0, e1);
}

template <int D>
void update_attn_threads(const LayerDev& L, const Shape& s, const AppendArgs& a, int recent_len,
                         int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                         const uint16_t* q, float* out, int use_order, int pad_len, int threads,
                         int tpr, size_t lds, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    if (threads == 1024)
        update_attn_tpr<D, 1024>(L, s, a, recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d, q,
                                 out, use_order, pad_len, tpr, lds, st, e0, e1);
    else if (threads == 512)
        update_attn_tpr<D, 512>(L, s, a, recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d, q,
                                out, use_order, pad_len, tpr, lds, st, e0, e1);
    else
        update_attn_tpr<D, 256>(L, s, a, recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d, q,
                                out, use_order, pad_len, tpr, lds, st, e0, e1);
}

}  // namespace

int launch_update_attn(const LayerDev& L, const Shape& s, const AppendArgs& a, int recent_len,
                       int rs_num, int rs_den, int u, int step, int lds_cap, double sqrt_d,
                       const uint16_t* q, float* out, int use_order, int pad_len, int threads,
                       int tpr, void* stream, void* ev_start, void* ev_stop) {
    hipStream_t st = (hipStream_t)stream;
    hipEvent_t e0 = static_cast<hipEvent_t>(ev_start), e1 = static_cast<hipEvent_t>(ev_stop);
    const size_t lds = UpdateLds::bytes(s.N, lds_cap, s.d, s.C, false, 1, L.ring_len);
    if (s.d == 128)
        update_attn_threads<128>(L, s, a, recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d, q,
                                 out, use_order, pad_len, threads, tpr, lds, st, e0, e1);
    else
        update_attn_threads<64>(L, s, a, recent_len, rs_num, rs_den, u, step, lds_cap, sqrt_d, q,
                                out, use_order, pad_len, threads, tpr, lds, st, e0, e1);
    return last_error();
}

size_t update_lds_bytes(int N, int cap, int d, int C, bool attn_scores, int period) {
    return UpdateLds::bytes(N, cap, d, C, attn_scores, 1, period);
}

int launch_export(const LayerDev& L, const Shape& s, uint8_t* mask, int32_t* count,
                  void* stream) {
    hipLaunchKernelGGL(k_export, dim3(s.BH), dim3(kBlock), 0, (hipStream_t)stream, L, s.C, s.d,
                       s.N, mask, count);
    return last_error();
}

}  // namespace headkv
