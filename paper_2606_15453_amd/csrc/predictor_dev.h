// Predictor state and device code (Section 4.2): the Table Update
// (Algorithm 3, with the HT overwrite and the hit count of the verify step)
// and the Expert Predict function (Algorithm 2 with Eq. 1).  Shared by the
// standalone predictor kernels and the decode path's router + predictor
// kernel.  Both bodies run in one 256-thread workgroup on an LDS image of
// the tables.
#pragma once

#include "common.h"

// Per-layer byte tables start on 4-byte boundaries (strides rounded up) so
// the kernels copy them into LDS as whole words.
struct stmoe_predictor {
    int L, E, K, B;
    size_t cct_stride;           // bytes per layer pair: E*K rounded up to 4
    size_t ht_stride;            // bytes per layer: B*K rounded up to 4
    size_t pend_stride;          // bytes per layer: B*E rounded up to 4
    int32_t* co;                 // [L-1][E][E] profiling co-activation counts
    uint8_t* cct_idx;            // [L-1] x cct_stride, each [E][K]
    uint8_t* cct_conf;           // [L-1] x cct_stride, each [E][K]
    uint8_t* ht;                 // [L] x ht_stride, each [B][K], rows sorted ascending
    uint8_t* pend;               // [L] x pend_stride, each [B][E]: last prediction per layer
    unsigned long long* stats;   // [L][3]: hits, |A|, |P|
    int32_t* stage;              // profiling selections staged in chunks of whole tokens
    size_t stage_bytes;
    bool profiled;
};

inline size_t round4(size_t n) { return (n + 3) / 4 * 4; }

namespace stmoe {
namespace pred {

constexpr int kThreads = 256;
constexpr int kConfInit = 2;   // "10", preferred
constexpr int kConfMax = 3;    // "11", strongly preferred
constexpr int kThreshold = 2;  // prefetch when the score reaches "10"
constexpr int kHtScore = 2;    // HT confidences stay at "10"

struct UpdateArgs {
    const int32_t* sel_prev;   // [B][K] or null at layer 0
    const int32_t* sel_cur;    // [B][K], or null when the selection is already in LDS
    uint8_t* cidx;             // CCT_{layer-1} [E][K] or null
    uint8_t* cconf;
    uint8_t* ht;               // HT[layer] [B][K]
    const uint8_t* pend;       // [B][E] prediction for this layer
    unsigned long long* stats; // [3]
    int B, E, K, online;
};

struct PredictArgs {
    const int32_t* sel_cur;    // [B][K], or null when in LDS or unused (cidx null)
    const uint8_t* cidx;       // CCT_layer [E][K] or null (layer -1 or HT-only)
    const uint8_t* cconf;
    const uint8_t* ht_next;    // HT[layer+1] [B][K] or null (CCT-only)
    uint8_t* pend;             // [B][E] kept for the next update's hit count
    uint8_t* score;            // [B][E] or null
    uint8_t* mask;             // [E] or null
    uint8_t* max_score;        // [E] or null: max over rows of the score
    int32_t* ranked;           // [E] or null
    int32_t* n_ranked;         // [1] or null
    int B, E, K;
};

// Scores rank through a 64-bin histogram.  With distinct experts in every
// CCT entry a score is at most K * 3 + 2 = 50; larger ones (repeated experts
// in an imported entry) take an exact O(E) ranking instead.
constexpr int kScoreBins = 64;
static_assert(kMaxK * kConfMax + kHtScore < kScoreBins, "score histogram too small");
static_assert(kMaxE <= kThreads, "one expert per thread in the ranking");

// LDS image of every table one update + predict touches.  The tables are
// small (at most E*K = 4 KB each), so each kernel copies them in with one
// round of independent loads and then works from LDS: the dependent chains
// (selection -> CCT entry -> slot) cost LDS latency instead of HBM latency.
struct TableShared {
    union {
        float z[kMaxB * kMaxE];       // router logits (fused kernel, before top-K)
        int sc[kMaxB * kMaxE];        // prediction scores
    };
    __align__(16) uint8_t uidx[kMaxE * kMaxK];    // CCT_{layer-1} (update)
    __align__(16) uint8_t uconf[kMaxE * kMaxK];
    __align__(16) uint8_t pidx[kMaxE * kMaxK];    // CCT_layer (predict)
    __align__(16) uint8_t pconf[kMaxE * kMaxK];
    __align__(16) uint8_t pend[kMaxB * kMaxE];    // prediction made for this layer
    __align__(16) uint8_t htn[kMaxB * kMaxK];     // HT[layer+1]
    __align__(16) uint8_t htnew[kMaxB * kMaxK];   // HT[layer] after the update
    __align__(16) int32_t prev[kMaxB * kMaxK];
    __align__(16) int32_t sel[kMaxB * kMaxK];
    __align__(16) int32_t Fs[kMaxB * kMaxK];  // every row's actual set, ascending (row stride kMaxK)
    int mx[kMaxE];                    // max score over rows
    int whist[kThreads / 64][kScoreBins];  // per-wave histogram of candidate scores
    int greater[kScoreBins];          // candidates scoring above each value
    unsigned hits, npred;
};

// One contiguous global -> LDS copy of n 4-byte words (null src: nothing).
struct Seg {
    const uint32_t* src;
    uint32_t* dst;
    int n;
};

__device__ __forceinline__ Seg seg(const void* src, void* dst, size_t bytes) {
    Seg g;
    g.src = reinterpret_cast<const uint32_t*>(src);
    g.dst = reinterpret_cast<uint32_t*>(dst);
    g.n = src ? int((bytes + 3) / 4) : 0;
    return g;
}

constexpr int kMaxSegs = 10;
constexpr int kStageRegs = 4;   // words per thread per segment in one pass

// Copy every segment into LDS.  In each pass a thread loads up to
// kStageRegs words of every segment before its first LDS store, so the whole
// copy is one memory round trip at decode sizes.  Ends with a barrier.
__device__ void stage(const Seg* g, int nseg) {
    int most = 0;
#pragma unroll
    for (int j = 0; j < kMaxSegs; ++j)
        if (j < nseg) most = max(most, g[j].n);
    for (int base = 0; base < most; base += kThreads * kStageRegs) {
        uint32_t val[kMaxSegs][kStageRegs];
#pragma unroll
        for (int j = 0; j < kMaxSegs; ++j)
#pragma unroll
            for (int r = 0; r < kStageRegs; ++r) {
                const int i = base + r * kThreads + int(threadIdx.x);
                val[j][r] = j < nseg && i < g[j].n ? g[j].src[i] : 0u;
            }
#pragma unroll
        for (int j = 0; j < kMaxSegs; ++j)
#pragma unroll
            for (int r = 0; r < kStageRegs; ++r) {
                const int i = base + r * kThreads + int(threadIdx.x);
                if (j < nseg && i < g[j].n) g[j].dst[i] = val[j][r];
            }
    }
    __syncthreads();
}

// Segments for an update (always 5 slots, unused ones empty, so that the
// slot positions are compile-time constants); returns the count.
__device__ __forceinline__ int update_segs(const UpdateArgs& a, TableShared& sh, Seg* g) {
    const int EK = a.E * a.K, BK = a.B * a.K;
    const bool cct = a.cidx != nullptr && a.online;
    int n = 0;
    g[n++] = seg(cct ? a.cidx : nullptr, sh.uidx, EK);
    g[n++] = seg(cct ? a.cconf : nullptr, sh.uconf, EK);
    g[n++] = seg(cct ? a.sel_prev : nullptr, sh.prev, BK * sizeof(int32_t));
    g[n++] = seg(a.pend, sh.pend, a.B * a.E);
    g[n++] = seg(a.sel_cur, sh.sel, BK * sizeof(int32_t));
    return n;
}

// Segments for a prediction (always 4 slots); returns the count.
__device__ __forceinline__ int predict_segs(const PredictArgs& a, TableShared& sh, Seg* g) {
    const int EK = a.E * a.K, BK = a.B * a.K;
    int n = 0;
    g[n++] = seg(a.cidx, sh.pidx, EK);
    g[n++] = seg(a.cconf, sh.pconf, EK);
    g[n++] = seg(a.ht_next, sh.htn, BK);
    g[n++] = seg(a.cidx ? a.sel_cur : nullptr, sh.sel, BK * sizeof(int32_t));
    return n;
}

// Algorithm 3 on CCT_{layer-1} for rows b = 0..B-1 in order.  Lane t of a
// group of GS lanes (one wave holds whole groups) owns slot s = t % GS of
// entry g = t / GS, the g-th expert of A_{layer-1}[b]; the entries of one row
// are distinct, so the groups of a row are independent and only the order of
// rows is serial.  Each lane reads its entry's whole snapshot with its own
// slot (one LDS round trip per row: the next row's entry index is loaded a
// row ahead, since the update never writes it), and the group's replaced
// slots and absent experts meet in two ballots.  With GS = 8 (K <= 8) every
// group sits in wave 0 and rows follow each other without a workgroup
// barrier (a wave's LDS accesses complete in order); with GS = 16 groups
// span the four waves and a barrier separates rows.  Loops run to GS with
// reads that stay inside the LDS arrays, so their reads issue together.
template <int GS>
__device__ __forceinline__ void cct_rows(const UpdateArgs& a, TableShared& sh) {
    constexpr bool one_wave = GS * GS <= 64;
    const int t = threadIdx.x, K = a.K, E = a.E;
    const int g = t / GS, s = t % GS, first = (t & 63) - s;
    const bool on = g < K && s < K;
    if (one_wave && t >= 64) return;
    const unsigned gmask = (1u << K) - 1u;
    int e = on ? sh.prev[g] : -1;
    for (int b = 0; b < a.B; ++b) {
        const bool ok = e >= 0 && e < E;      // out-of-range selections are ignored
        const int ec = ok ? e : 0;
        const int32_t* F = sh.Fs + b * kMaxK;
        const uint8_t* entry = sh.uidx + ec * K;   // + j < kMaxE * kMaxK for j < GS
        int Fv[GS], snap[GS];
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            Fv[j] = F[j];
            snap[j] = entry[j];
        }
        const int mine = F[s], f = entry[s];
        int conf = sh.uconf[ec * K + s];
        const int e_next = on && b + 1 < a.B ? sh.prev[(b + 1) * K + g] : -1;
        bool hit = false, held = false;
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            hit |= j < K && Fv[j] == f;
            held |= j < K && snap[j] == mine;
        }
        // slots replaced in this entry, and experts of F absent from it
        const unsigned long long rm = __ballot(ok && !hit && conf == 0);
        const unsigned long long am = __ballot(on && !held);
        if (ok) {
            if (hit) {
                conf = min(conf + 1, kConfMax);
            } else if (conf > 0) {
                conf -= 1;
            } else {
                // the rank-th absent expert of F (ascending), rank = replaced
                // slots before this one
                const int rank = __popc(unsigned(rm >> first) & gmask & ((1u << s) - 1u));
                unsigned abs_ = unsigned(am >> first) & gmask;
#pragma unroll
                for (int q = 0; q < GS; ++q)
                    if (q < rank) abs_ &= abs_ - 1u;
                const int at = __ffs(abs_) - 1;
                int pick = 0;
#pragma unroll
                for (int j = 0; j < GS; ++j) pick = j == at ? Fv[j] : pick;
                if (abs_) sh.uidx[e * K + s] = uint8_t(pick);
                conf = kConfInit;
            }
            sh.uconf[e * K + s] = uint8_t(conf);
        }
        e = e_next;
        // the next row may update the same entries
        if (one_wave)
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        else
            __syncthreads();
    }
}

// The verify step and Algorithm 3 for one layer: hits of the selection
// against the prediction made for this layer, HT[layer][b] <- sorted
// selection, then the CCT_{layer-1} entries of every row (cct_rows).  Works
// on the LDS image (staged by the caller), then writes the touched CCT
// entries, HT and the hit counts back.  Ends with a barrier.
__device__ void update_body(const UpdateArgs& a, TableShared& sh) {
    const int tid = threadIdx.x, K = a.K, E = a.E, BK = a.B * K;
    const bool cct = a.cidx != nullptr && a.online;
    // every row sorted ascending: a lane per selected expert finds its rank
    // (reads past the last row stay inside sel: B, K <= 16)
    for (int i = tid; i < BK; i += kThreads) {
        const int32_t* row = sh.sel + (i / K) * K;
        const int v = sh.sel[i];
        int rank = 0;
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            const int w = row[j];
            rank += j < K && w < v;
        }
        sh.Fs[(i / K) * kMaxK + rank] = v;
    }
    unsigned my_hits = 0, my_pred = 0;
    for (int i = tid; i < BK; i += kThreads) {
        const int v = sh.sel[i];
        if (v >= 0 && v < E) my_hits += sh.pend[(i / K) * E + v] >= kThreshold;
    }
    for (int i = tid; i < a.B * E; i += kThreads) my_pred += sh.pend[i] >= kThreshold;
    if (tid == 0) { sh.hits = 0; sh.npred = 0; }
    __syncthreads();
    for (int i = tid; i < BK; i += kThreads) {
        const uint8_t v = uint8_t(sh.Fs[(i / K) * kMaxK + i % K]);
        sh.htnew[i] = v;
        a.ht[i] = v;
    }
    if (cct) {
        if (K <= 8)
            cct_rows<8>(a, sh);
        else
            cct_rows<16>(a, sh);
    }
    __syncthreads();
    if (cct) {
        // write back every entry slot this layer's rows touched (duplicates
        // carry the same final value)
        for (int i = tid; i < a.B * K * K; i += kThreads) {
            const int e = sh.prev[i / K], s = i % K;
            if (e >= 0 && e < E) {
                a.cidx[e * K + s] = sh.uidx[e * K + s];
                a.cconf[e * K + s] = sh.uconf[e * K + s];
            }
        }
    }
    if (my_hits) atomicAdd(&sh.hits, my_hits);
    if (my_pred) atomicAdd(&sh.npred, my_pred);
    __syncthreads();
    if (tid == 0) {
        atomicAdd(&a.stats[0], (unsigned long long)sh.hits);
        atomicAdd(&a.stats[1], (unsigned long long)(a.B * K));
        atomicAdd(&a.stats[2], (unsigned long long)sh.npred);
    }
}

// Algorithm 2 with Eq. 1: score_b[f] = sum_{e in A[b]} conf of f in CCT[e]
// + 2 [f in HT_next[b]]; PrefetchSet = {f : score >= 2}; the union over rows
// ranked by (max score desc, index asc).  Integer atomics in LDS: exact.
// Reads the LDS image (staged by the caller; htn holds HT[layer+1]).
__device__ void predict_body(const PredictArgs& a, TableShared& sh) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int K = a.K, KK = a.K * a.K, E = a.E;
    for (int i = tid; i < a.B * E; i += kThreads) sh.sc[i] = 0;
    for (int i = tid; i < (kThreads / 64) * kScoreBins; i += kThreads) (&sh.whist[0][0])[i] = 0;
    __syncthreads();
    if (a.cidx) {
        for (int i = tid; i < a.B * KK; i += kThreads) {
            const int b = i / KK, e = sh.sel[b * K + (i % KK) / K], s = i % K;
            const int f = e >= 0 && e < E ? sh.pidx[e * K + s] : E;
            if (f < E) atomicAdd(&sh.sc[b * E + f], int(sh.pconf[e * K + s]));
        }
    }
    if (a.ht_next)
        for (int i = tid; i < a.B * K; i += kThreads)
            if (sh.htn[i] < E) atomicAdd(&sh.sc[(i / K) * E + sh.htn[i]], kHtScore);
    __syncthreads();
    for (int i = tid; i < a.B * E; i += kThreads) {
        a.pend[i] = uint8_t(sh.sc[i]);
        if (a.score) a.score[i] = uint8_t(sh.sc[i]);
    }
    // one expert per thread: max over rows, then its place in the ranking
    const int f = tid;
    int m = 0;
    if (f < E) {
#pragma unroll
        for (int b = 0; b < kMaxB; ++b) {
            const int v = sh.sc[b * E + f];      // inside sc for every b < kMaxB
            m = max(m, b < a.B ? v : 0);
        }
        if (a.mask) a.mask[f] = m >= kThreshold;
        if (a.max_score) a.max_score[f] = uint8_t(m);
    }
    if (!a.ranked && !a.n_ranked) return;
    const bool cand = f < E && m >= kThreshold;
    if (f < E) sh.mx[f] = m;
    if (cand && m < kScoreBins) atomicAdd(&sh.whist[wave][m], 1);
    if (__syncthreads_or(cand && m >= kScoreBins)) {
        // exact fallback for out-of-histogram scores
        int total = 0;
        for (int g = 0; g < E; ++g) total += sh.mx[g] >= kThreshold;
        if (a.ranked && f < E) {
            if (cand) {
                int rank = 0;
                for (int g = 0; g < E; ++g)
                    rank += sh.mx[g] >= kThreshold && (sh.mx[g] > m || (sh.mx[g] == m && g < f));
                a.ranked[rank] = f;
            }
            if (f >= total) a.ranked[f] = -1;
        }
        if (a.n_ranked && tid == 0) *a.n_ranked = total;
        return;
    }
    if (wave == 0) {
        // greater[t] = candidates with score > t: suffix sum of the histogram
        int h = 0;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) h += sh.whist[w][lane];
        int suf = h;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_down(suf, o, 64);
            if (lane + o < 64) suf += y;
        }
        sh.greater[lane] = suf - h;
    }
    __syncthreads();
    // lanes of this wave with the same score and a lower index: equality of
    // all six score bits, one ballot per bit
    unsigned long long same = __ballot(cand);
#pragma unroll
    for (int bit = 0; bit < 6; ++bit) {
        const bool on = (m >> bit) & 1;
        const unsigned long long bm = __ballot(cand && on);
        same &= on ? bm : ~bm;
    }
    const int total = sh.greater[kThreshold - 1];
    if (a.ranked && f < E) {
        if (cand) {
            int rank = sh.greater[m] + __popcll(same & ((1ull << lane) - 1ull));
#pragma unroll
            for (int w = 0; w < kThreads / 64; ++w)
                if (w < wave) rank += sh.whist[w][m];
            a.ranked[rank] = f;
        }
        if (f >= total) a.ranked[f] = -1;
    }
    if (a.n_ranked && tid == 0) *a.n_ranked = total;
}

// Host-side construction of the per-layer argument blocks.
inline UpdateArgs update_args(stmoe_predictor* p, int layer, const int32_t* sel_prev,
                              const int32_t* sel_cur, int online) {
    UpdateArgs a;
    a.sel_prev = sel_prev;
    a.sel_cur = sel_cur;
    a.cidx = layer >= 1 ? p->cct_idx + size_t(layer - 1) * p->cct_stride : nullptr;
    a.cconf = layer >= 1 ? p->cct_conf + size_t(layer - 1) * p->cct_stride : nullptr;
    a.ht = p->ht + size_t(layer) * p->ht_stride;
    a.pend = p->pend + size_t(layer) * p->pend_stride;
    a.stats = p->stats + size_t(layer) * 3;
    a.B = p->B;
    a.E = p->E;
    a.K = p->K;
    a.online = online ? 1 : 0;
    return a;
}

// layer -1 predicts layer 0 from HT[0] alone
inline PredictArgs predict_args(stmoe_predictor* p, int layer, const int32_t* sel_cur, int use,
                                uint8_t* score, uint8_t* mask, uint8_t* max_score, int32_t* ranked,
                                int32_t* n_ranked) {
    const bool cct = (use & STMOE_USE_CCT) && layer >= 0;
    const int tgt = layer + 1;
    PredictArgs a;
    a.sel_cur = sel_cur;
    a.cidx = cct ? p->cct_idx + size_t(layer) * p->cct_stride : nullptr;
    a.cconf = cct ? p->cct_conf + size_t(layer) * p->cct_stride : nullptr;
    a.ht_next = (use & STMOE_USE_HT) ? p->ht + size_t(tgt) * p->ht_stride : nullptr;
    a.pend = p->pend + size_t(tgt) * p->pend_stride;
    a.score = score;
    a.mask = mask;
    a.max_score = max_score;
    a.ranked = ranked;
    a.n_ranked = n_ranked;
    a.B = p->B;
    a.E = p->E;
    a.K = p->K;
    return a;
}

}  // namespace pred
}  // namespace stmoe
