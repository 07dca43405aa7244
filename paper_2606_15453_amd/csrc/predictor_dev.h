// Predictor state and device code (Section 4.2): the Table Update
// (Algorithm 3, with the HT overwrite and the hit count of the verify step)
// and the Expert Predict function (Algorithm 2 with Eq. 1).  Shared by the
// standalone predictor kernels and the fused router + predictor kernel.
// Both bodies run in one 256-thread workgroup.
#pragma once

#include "common.h"

struct stmoe_predictor {
    int L, E, K, B;
    int32_t* co;                 // [L-1][E][E] profiling co-activation counts
    uint8_t* cct_idx;            // [L-1][E][K]
    uint8_t* cct_conf;           // [L-1][E][K]
    uint8_t* ht;                 // [L][B][K], each row sorted ascending
    uint8_t* pend;               // [L][B][E] last prediction scores made for each layer
    unsigned long long* stats;   // [L][3]: hits, |A|, |P|
    bool profiled;
};

namespace stmoe {
namespace pred {

constexpr int kThreads = 256;
constexpr int kConfInit = 2;   // "10", preferred
constexpr int kConfMax = 3;    // "11", strongly preferred
constexpr int kThreshold = 2;  // prefetch when the score reaches "10"
constexpr int kHtScore = 2;    // HT confidences stay at "10"

struct UpdateArgs {
    const int32_t* sel_prev;   // [B][K] or null at layer 0
    const int32_t* sel_cur;    // [B][K] (global or LDS)
    uint8_t* cidx;             // CCT_{layer-1} [E][K] or null
    uint8_t* cconf;
    uint8_t* ht;               // HT[layer] [B][K]
    const uint8_t* pend;       // [B][E] prediction for this layer
    unsigned long long* stats; // [3]
    int B, E, K, online;
};

struct UpdateShared {
    int32_t F[kMaxK];                 // actual set, ascending
    uint8_t snap[kMaxK * kMaxK];      // entries before this row's update
    uint8_t repl[kMaxK * kMaxK];      // slot is replaced
    unsigned hits, npred;
};

// Algorithm 3 on CCT_{layer-1} for the entries selected at layer-1, rows
// b = 0..B-1 in order; HT[layer][b] <- sorted selection; hits against the
// prediction made for this layer.  One lane per (entry, slot).
__device__ void update_body(const UpdateArgs& a, UpdateShared& sh) {
    const int tid = threadIdx.x, K = a.K, KK = a.K * a.K;
    if (tid == 0) { sh.hits = 0; sh.npred = 0; }
    for (int b = 0; b < a.B; ++b) {
        const int32_t* cur = a.sel_cur + b * K;
        if (tid < K) {
            const int v = cur[tid];
            int rank = 0;
            for (int j = 0; j < K; ++j) rank += cur[j] < v;
            sh.F[rank] = v;
        }
        int e = 0, s = 0, conf = 0;
        bool hit = false;
        const bool upd = a.cidx != nullptr && a.online && tid < KK;
        bool upd_ok = upd;
        if (upd) {
            e = a.sel_prev[b * K + tid / K];
            s = tid % K;
            upd_ok = e >= 0 && e < a.E;      // out-of-range selections are ignored
            sh.snap[tid] = upd_ok ? a.cidx[e * K + s] : 0xff;
            conf = upd_ok ? a.cconf[e * K + s] : 1;
        }
        __syncthreads();
        if (upd) {
            const int f = sh.snap[tid];
            for (int j = 0; j < K; ++j) hit |= (sh.F[j] == f);
            sh.repl[tid] = upd_ok && (!hit && conf == 0);
        }
        __syncthreads();
        if (upd_ok) {
            if (hit) {
                conf = min(conf + 1, kConfMax);
            } else if (conf > 0) {
                conf -= 1;
            } else {
                // the rank-th expert of F (ascending) absent from the entry's snapshot
                const int base = tid - s;
                int rank = 0;
                for (int q = 0; q < s; ++q) rank += sh.repl[base + q];
                int pick = -1;
                for (int j = 0; j < K && pick < 0; ++j) {
                    bool held = false;
                    for (int q = 0; q < K; ++q) held |= (sh.snap[base + q] == sh.F[j]);
                    if (!held) {
                        if (rank == 0) pick = sh.F[j];
                        --rank;
                    }
                }
                if (pick >= 0) a.cidx[e * K + s] = uint8_t(pick);
                conf = kConfInit;
            }
            a.cconf[e * K + s] = uint8_t(conf);
        }
        // verification against the prediction made for this layer
        if (tid < K && cur[tid] >= 0 && cur[tid] < a.E && a.pend[b * a.E + cur[tid]] >= kThreshold)
            atomicAdd(&sh.hits, 1u);
        for (int f = tid; f < a.E; f += kThreads)
            if (a.pend[b * a.E + f] >= kThreshold) atomicAdd(&sh.npred, 1u);
        if (tid < K) a.ht[b * K + tid] = uint8_t(sh.F[tid]);
        // the next row may update the same entries: make this row's writes visible
        __threadfence_block();
        __syncthreads();
    }
    if (tid == 0) {
        atomicAdd(&a.stats[0], (unsigned long long)sh.hits);
        atomicAdd(&a.stats[1], (unsigned long long)(a.B * K));
        atomicAdd(&a.stats[2], (unsigned long long)sh.npred);
    }
}

struct PredictArgs {
    const int32_t* sel_cur;    // [B][K] (global or LDS; unused when cidx is null)
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

struct PredictShared {
    int sc[kMaxB * kMaxE];
    int mx[kMaxE];
};

// Algorithm 2 with Eq. 1: score_b[f] = sum_{e in A[b]} conf of f in CCT[e]
// + 2 [f in HT_next[b]]; PrefetchSet = {f : score >= 2}; the union over rows
// ranked by (max score desc, index asc).  Integer atomics in LDS: exact.
__device__ void predict_body(const PredictArgs& a, PredictShared& sh) {
    const int tid = threadIdx.x, K = a.K, E = a.E;
    for (int i = tid; i < a.B * E; i += kThreads) sh.sc[i] = 0;
    __syncthreads();
    for (int b = 0; b < a.B; ++b) {
        if (a.cidx && tid < K * K) {
            const int e = a.sel_cur[b * K + tid / K], s = tid % K;
            if (e >= 0 && e < E) atomicAdd(&sh.sc[b * E + a.cidx[e * K + s]], int(a.cconf[e * K + s]));
        }
        if (a.ht_next && tid < K) atomicAdd(&sh.sc[b * E + a.ht_next[b * K + tid]], kHtScore);
    }
    __syncthreads();
    for (int i = tid; i < a.B * E; i += kThreads) {
        a.pend[i] = uint8_t(sh.sc[i]);
        if (a.score) a.score[i] = uint8_t(sh.sc[i]);
    }
    for (int f = tid; f < E; f += kThreads) {
        int m = 0;
        for (int b = 0; b < a.B; ++b) m = max(m, sh.sc[b * E + f]);
        sh.mx[f] = m;
        if (a.mask) a.mask[f] = m >= kThreshold;
        if (a.max_score) a.max_score[f] = uint8_t(m);
    }
    __syncthreads();
    if (a.ranked || a.n_ranked) {
        if (a.ranked)
            for (int f = tid; f < E; f += kThreads) a.ranked[f] = -1;
        __syncthreads();
        for (int f = tid; f < E; f += kThreads) {
            if (sh.mx[f] < kThreshold) continue;
            int rank = 0;
            for (int g = 0; g < E; ++g)
                rank += sh.mx[g] >= kThreshold && (sh.mx[g] > sh.mx[f] || (sh.mx[g] == sh.mx[f] && g < f));
            if (a.ranked) a.ranked[rank] = f;
        }
        if (a.n_ranked && tid == 0) {
            int count = 0;
            for (int g = 0; g < E; ++g) count += sh.mx[g] >= kThreshold;
            *a.n_ranked = count;
        }
    }
}

// Host-side construction of the per-layer argument blocks.
inline UpdateArgs update_args(stmoe_predictor* p, int layer, const int32_t* sel_prev,
                              const int32_t* sel_cur, int online) {
    UpdateArgs a;
    a.sel_prev = sel_prev;
    a.sel_cur = sel_cur;
    a.cidx = layer >= 1 ? p->cct_idx + size_t(layer - 1) * p->E * p->K : nullptr;
    a.cconf = layer >= 1 ? p->cct_conf + size_t(layer - 1) * p->E * p->K : nullptr;
    a.ht = p->ht + size_t(layer) * p->B * p->K;
    a.pend = p->pend + size_t(layer) * p->B * p->E;
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
    a.cidx = cct ? p->cct_idx + size_t(layer) * p->E * p->K : nullptr;
    a.cconf = cct ? p->cct_conf + size_t(layer) * p->E * p->K : nullptr;
    a.ht_next = (use & STMOE_USE_HT) ? p->ht + size_t(tgt) * p->B * p->K : nullptr;
    a.pend = p->pend + size_t(tgt) * p->B * p->E;
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
