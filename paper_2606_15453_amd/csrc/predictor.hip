// Spatio-temporal expert predictor (Section 4.2): Cross-layer Correlation
// Tables with 2-bit confidences and a per-layer History Table.
//
// Tables live in HBM and are small (for 94 layers x 128 experts x top-8:
// 94 KB of CCT indices and 94 KB of confidences), so the runtime kernels run
// as a single workgroup each: the update of one batch row touches K entries
// x K slots (at most 256 lanes, one lane per slot), and the prediction sums
// K x K contributions into per-row score bins in LDS with integer atomics,
// which is exact and order-free.
#include <vector>

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
namespace {

constexpr int kThreads = 256;
constexpr int kConfInit = 2;   // "10", preferred
constexpr int kConfMax = 3;    // "11", strongly preferred
constexpr int kThreshold = 2;  // prefetch when the score reaches "10"
constexpr int kHtScore = 2;    // HT confidences stay at "10"

// ---------------------------------------------------------------- profiling
// Algorithm 1, counting: one workgroup per (profiling token, layer pair).
__global__ __launch_bounds__(kThreads) void co_count_kernel(const int32_t* sel, int P, int B, int L,
                                                            int E, int K, int32_t* co) {
    const int p = blockIdx.x, i = blockIdx.y;
    const int pairs = B * K * K;
    for (int t = threadIdx.x; t < pairs; t += kThreads) {
        const int b = t / (K * K), r = (t / K) % K, s = t % K;
        const int32_t* row = sel + ((size_t(p) * B + b) * L) * K;
        const int e = row[i * K + r], f = row[(i + 1) * K + s];
        atomicAdd(&co[(size_t(i) * E + e) * E + f], 1);
    }
}

// Algorithm 1, selection: CCT_i[e] = the K largest counts of Co_i[e][*]
// (equal counts -> lower index), all with confidence "10".
__global__ __launch_bounds__(kThreads) void cct_build_kernel(const int32_t* co, int E, int K,
                                                             uint8_t* idx, uint8_t* conf) {
    __shared__ int32_t row[kMaxE];
    const size_t r = blockIdx.x;   // (pair, expert) row
    for (int f = threadIdx.x; f < E; f += kThreads) row[f] = co[r * E + f];
    __syncthreads();
    for (int f = threadIdx.x; f < E; f += kThreads) {
        const int32_t c = row[f];
        int rank = 0;
        for (int g = 0; g < E; ++g) rank += (row[g] > c) || (row[g] == c && g < f);
        if (rank < K) {
            idx[r * K + rank] = uint8_t(f);
            conf[r * K + rank] = uint8_t(kConfInit);
        }
    }
}

// Sort one K-row of distinct expert indices ascending into dst (by ranking).
__device__ __forceinline__ void sorted_row(const int32_t* src, int K, uint8_t* dst) {
    for (int k = threadIdx.x; k < K; k += kThreads) {
        const int v = src[k];
        int rank = 0;
        for (int j = 0; j < K; ++j) rank += src[j] < v;
        dst[rank] = uint8_t(v);
    }
}

__global__ __launch_bounds__(kThreads) void ht_init_kernel(const int32_t* sel_last, int B, int L,
                                                           int K, uint8_t* ht) {
    const int l = blockIdx.x, b = blockIdx.y;
    sorted_row(sel_last + (size_t(b) * L + l) * K, K, ht + (size_t(l) * B + b) * K);
}

// ------------------------------------------------------------------- update
// Algorithm 3 on CCT_{layer-1} for the rows selected at layer-1, then the HT
// overwrite and the hit count against the prediction made for this layer.
struct UpdateArgs {
    const int32_t* sel_prev;   // [B][K] or null at layer 0
    const int32_t* sel_cur;    // [B][K]
    uint8_t* cidx;             // CCT_{layer-1} [E][K] or null
    uint8_t* cconf;
    uint8_t* ht;               // HT[layer] [B][K]
    const uint8_t* pend;       // [B][E] prediction for this layer
    unsigned long long* stats; // [3]
    int B, E, K, online;
};

__global__ __launch_bounds__(kThreads) void update_kernel(UpdateArgs a) {
    __shared__ int32_t F[kMaxK];          // actual set, ascending
    __shared__ uint8_t snap[kMaxK * kMaxK];  // entries before this row's update
    __shared__ uint8_t repl[kMaxK * kMaxK];  // slot is replaced
    __shared__ unsigned hits, npred;
    const int tid = threadIdx.x, K = a.K, KK = a.K * a.K;
    if (tid == 0) { hits = 0; npred = 0; }
    for (int b = 0; b < a.B; ++b) {
        const int32_t* cur = a.sel_cur + b * K;
        if (tid < K) {
            const int v = cur[tid];
            int rank = 0;
            for (int j = 0; j < K; ++j) rank += cur[j] < v;
            F[rank] = v;
        }
        int e = 0, s = 0, conf = 0;
        bool hit = false;
        const bool upd = a.cidx != nullptr && a.online && tid < KK;
        bool upd_ok = upd;
        if (upd) {
            e = a.sel_prev[b * K + tid / K];
            s = tid % K;
            upd_ok = e >= 0 && e < a.E;      // out-of-range selections are ignored
            snap[tid] = upd_ok ? a.cidx[e * K + s] : 0xff;
            conf = upd_ok ? a.cconf[e * K + s] : 1;
        }
        __syncthreads();
        if (upd) {
            const int f = snap[tid];
            for (int j = 0; j < K; ++j) hit |= (F[j] == f);
            repl[tid] = upd_ok && (!hit && conf == 0);
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
                for (int q = 0; q < s; ++q) rank += repl[base + q];
                int pick = -1;
                for (int j = 0; j < K && pick < 0; ++j) {
                    bool held = false;
                    for (int q = 0; q < K; ++q) held |= (snap[base + q] == F[j]);
                    if (!held) {
                        if (rank == 0) pick = F[j];
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
            atomicAdd(&hits, 1u);
        for (int f = tid; f < a.E; f += kThreads)
            if (a.pend[b * a.E + f] >= kThreshold) atomicAdd(&npred, 1u);
        if (tid < K) a.ht[b * K + tid] = uint8_t(F[tid]);
        // next row may update the same entries: make this row's writes visible
        __threadfence_block();
        __syncthreads();
    }
    if (tid == 0) {
        atomicAdd(&a.stats[0], (unsigned long long)hits);
        atomicAdd(&a.stats[1], (unsigned long long)(a.B * K));
        atomicAdd(&a.stats[2], (unsigned long long)npred);
    }
}

// ------------------------------------------------------------------ predict
// Algorithm 2 with Eq. 1: score_b[f] = sum_{e in A[b]} conf of f in CCT[e]
// + 2 [f in HT_next[b]]; PrefetchSet = {f : score >= 2}.
struct PredictArgs {
    const int32_t* sel_cur;    // [B][K] (unused when cidx is null)
    const uint8_t* cidx;       // CCT_layer [E][K] or null (layer -1 or HT-only)
    const uint8_t* cconf;
    const uint8_t* ht_next;    // HT[layer+1] [B][K] or null (CCT-only)
    uint8_t* pend;             // [B][E] kept for the next update's hit count
    uint8_t* score;            // [B][E] or null
    uint8_t* mask;             // [E] or null
    int32_t* ranked;           // [E] or null
    int32_t* n_ranked;         // [1] or null
    int B, E, K;
};

__global__ __launch_bounds__(kThreads) void predict_kernel(PredictArgs a) {
    __shared__ int sc[kMaxB * kMaxE];
    __shared__ int mx[kMaxE];
    const int tid = threadIdx.x, K = a.K, E = a.E;
    for (int i = tid; i < a.B * E; i += kThreads) sc[i] = 0;
    __syncthreads();
    for (int b = 0; b < a.B; ++b) {
        if (a.cidx && tid < K * K) {
            const int e = a.sel_cur[b * K + tid / K], s = tid % K;
            if (e >= 0 && e < E) atomicAdd(&sc[b * E + a.cidx[e * K + s]], int(a.cconf[e * K + s]));
        }
        if (a.ht_next && tid < K) atomicAdd(&sc[b * E + a.ht_next[b * K + tid]], kHtScore);
    }
    __syncthreads();
    for (int i = tid; i < a.B * E; i += kThreads) {
        a.pend[i] = uint8_t(sc[i]);
        if (a.score) a.score[i] = uint8_t(sc[i]);
    }
    for (int f = tid; f < E; f += kThreads) {
        int m = 0;
        for (int b = 0; b < a.B; ++b) m = max(m, sc[b * E + f]);
        mx[f] = m;
        if (a.mask) a.mask[f] = m >= kThreshold;
    }
    __syncthreads();
    if (a.ranked || a.n_ranked) {
        int count = 0;
        for (int f = tid; f < E; f += kThreads) {
            if (a.ranked) a.ranked[f] = -1;
        }
        __syncthreads();
        for (int f = tid; f < E; f += kThreads) {
            if (mx[f] < kThreshold) continue;
            int rank = 0;
            for (int g = 0; g < E; ++g)
                rank += mx[g] >= kThreshold && (mx[g] > mx[f] || (mx[g] == mx[f] && g < f));
            if (a.ranked) a.ranked[rank] = f;
        }
        if (a.n_ranked && tid == 0) {
            for (int g = 0; g < E; ++g) count += mx[g] >= kThreshold;
            *a.n_ranked = count;
        }
    }
}

int check_sel_host(const int32_t* sel, size_t rows, int E, int K) {
    for (size_t r = 0; r < rows; ++r) {
        const int32_t* row = sel + r * K;
        for (int k = 0; k < K; ++k) {
            STMOE_CHECK(row[k] >= 0 && row[k] < E, "selection index out of range");
            for (int j = 0; j < k; ++j) STMOE_CHECK(row[j] != row[k], "selection row has a repeated expert");
        }
    }
    return STMOE_OK;
}

}  // namespace
}  // namespace stmoe

using namespace stmoe;

extern "C" int stmoe_create(int L, int E, int K, int B, stmoe_predictor** out) {
    clear_error();
    STMOE_CHECK(out, "null output");
    STMOE_CHECK(L >= 1 && L <= 4096, "L must be in [1, 4096]");
    STMOE_CHECK(E >= 1 && E <= kMaxE, "E must be in [1, 256]");
    STMOE_CHECK(K >= 1 && K <= E && K <= kMaxK, "K must be in [1, min(E, 16)]");
    STMOE_CHECK(B >= 1 && B <= kMaxB, "B must be in [1, 16]");
    auto* p = new stmoe_predictor();
    p->L = L; p->E = E; p->K = K; p->B = B;
    p->profiled = false;
    const size_t pairs = size_t(L > 1 ? L - 1 : 1);
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = hipMalloc(&p->co, pairs * E * E * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc(&p->cct_idx, pairs * E * K);
    if (e == hipSuccess) e = hipMalloc(&p->cct_conf, pairs * E * K);
    if (e == hipSuccess) e = hipMalloc(&p->ht, size_t(L) * B * K);
    if (e == hipSuccess) e = hipMalloc(&p->pend, size_t(L) * B * E);
    if (e == hipSuccess) e = hipMalloc(&p->stats, size_t(L) * 3 * sizeof(unsigned long long));
    if (e == hipSuccess) e = hipMemset(p->co, 0, pairs * E * E * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(p->cct_idx, 0, pairs * E * K);
    if (e == hipSuccess) e = hipMemset(p->cct_conf, 0, pairs * E * K);
    if (e == hipSuccess) e = hipMemset(p->ht, 0, size_t(L) * B * K);
    if (e == hipSuccess) e = hipMemset(p->pend, 0, size_t(L) * B * E);
    if (e == hipSuccess) e = hipMemset(p->stats, 0, size_t(L) * 3 * sizeof(unsigned long long));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        set_error(std::string("stmoe_create: ") + hipGetErrorString(e));
        stmoe_destroy(p);
        return e == hipErrorOutOfMemory ? STMOE_ENOMEM : STMOE_EHIP;
    }
    *out = p;
    return STMOE_OK;
}

extern "C" int stmoe_destroy(stmoe_predictor* p) {
    if (!p) return STMOE_OK;
    (void)hipFree(p->co);
    (void)hipFree(p->cct_idx);
    (void)hipFree(p->cct_conf);
    (void)hipFree(p->ht);
    (void)hipFree(p->pend);
    (void)hipFree(p->stats);
    delete p;
    return STMOE_OK;
}

extern "C" int stmoe_profile(stmoe_predictor* p, const int32_t* sel, int P) {
    clear_error();
    STMOE_CHECK(p && sel, "null pointer");
    STMOE_CHECK(P >= 1, "P must be >= 1");
    const int L = p->L, E = p->E, K = p->K, B = p->B;
    if (int rc = check_sel_host(sel, size_t(P) * B * L, E, K)) return rc;
    const size_t n = size_t(P) * B * L * K;
    const size_t pairs = size_t(L > 1 ? L - 1 : 1);
    int32_t* dsel = nullptr;
    STMOE_HIP(hipMalloc(&dsel, n * sizeof(int32_t)));
    hipError_t e = hipMemcpy(dsel, sel, n * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(p->co, 0, pairs * E * E * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(p->pend, 0, size_t(L) * B * E);
    if (e == hipSuccess) e = hipMemset(p->stats, 0, size_t(L) * 3 * sizeof(unsigned long long));
    if (e == hipSuccess && L > 1) {
        hipLaunchKernelGGL(co_count_kernel, dim3(P, L - 1), dim3(kThreads), 0, 0, dsel, P, B, L, E,
                           K, p->co);
        e = hipGetLastError();
        if (e == hipSuccess) {
            hipLaunchKernelGGL(cct_build_kernel, dim3(unsigned((L - 1) * E)), dim3(kThreads), 0, 0,
                               p->co, E, K, p->cct_idx, p->cct_conf);
            e = hipGetLastError();
        }
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(ht_init_kernel, dim3(L, B), dim3(kThreads), 0, 0,
                           dsel + size_t(P - 1) * B * L * K, B, L, K, p->ht);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipDeviceSynchronize();
    (void)hipFree(dsel);
    if (e != hipSuccess) {
        set_error(std::string("stmoe_profile: ") + hipGetErrorString(e));
        return STMOE_EHIP;
    }
    p->profiled = true;
    return STMOE_OK;
}

extern "C" int stmoe_update(stmoe_predictor* p, int layer, const int32_t* sel_prev,
                            const int32_t* sel_cur, int online, void* stream) {
    clear_error();
    STMOE_CHECK(p && sel_cur, "null pointer");
    STMOE_CHECK(layer >= 0 && layer < p->L, "layer out of range");
    STMOE_CHECK(layer == 0 || sel_prev, "sel_prev is required for layer >= 1");
    if (!p->profiled) {
        set_error("stmoe_update: predictor has not been profiled");
        return STMOE_ESTATE;
    }
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
    hipLaunchKernelGGL(update_kernel, dim3(1), dim3(kThreads), 0, as_stream(stream), a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

extern "C" int stmoe_predict(stmoe_predictor* p, int layer, const int32_t* sel_cur, int use,
                             uint8_t* score, uint8_t* mask, int32_t* ranked, int32_t* n_ranked,
                             void* stream) {
    clear_error();
    STMOE_CHECK(p, "null predictor");
    STMOE_CHECK(layer >= -1 && layer < p->L - 1, "layer must be in [-1, L-2]");
    STMOE_CHECK((use & ~STMOE_USE_BOTH) == 0, "use must be a STMOE_USE_* bit set");
    const bool cct = (use & STMOE_USE_CCT) && layer >= 0;
    STMOE_CHECK(!cct || sel_cur, "sel_cur is required when the CCT is used");
    if (!p->profiled) {
        set_error("stmoe_predict: predictor has not been profiled");
        return STMOE_ESTATE;
    }
    const int tgt = layer + 1;
    PredictArgs a;
    a.sel_cur = sel_cur;
    a.cidx = cct ? p->cct_idx + size_t(layer) * p->E * p->K : nullptr;
    a.cconf = cct ? p->cct_conf + size_t(layer) * p->E * p->K : nullptr;
    a.ht_next = (use & STMOE_USE_HT) ? p->ht + size_t(tgt) * p->B * p->K : nullptr;
    a.pend = p->pend + size_t(tgt) * p->B * p->E;
    a.score = score;
    a.mask = mask;
    a.ranked = ranked;
    a.n_ranked = n_ranked;
    a.B = p->B;
    a.E = p->E;
    a.K = p->K;
    hipLaunchKernelGGL(predict_kernel, dim3(1), dim3(kThreads), 0, as_stream(stream), a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

extern "C" int stmoe_export(stmoe_predictor* p, int32_t* co, uint8_t* cct_idx, uint8_t* cct_conf,
                            uint8_t* ht) {
    clear_error();
    STMOE_CHECK(p, "null predictor");
    const size_t pairs = size_t(p->L > 1 ? p->L - 1 : 0);
    STMOE_HIP(hipDeviceSynchronize());
    if (co && pairs)
        STMOE_HIP(hipMemcpy(co, p->co, pairs * p->E * p->E * sizeof(int32_t), hipMemcpyDeviceToHost));
    if (cct_idx && pairs)
        STMOE_HIP(hipMemcpy(cct_idx, p->cct_idx, pairs * p->E * p->K, hipMemcpyDeviceToHost));
    if (cct_conf && pairs)
        STMOE_HIP(hipMemcpy(cct_conf, p->cct_conf, pairs * p->E * p->K, hipMemcpyDeviceToHost));
    if (ht) STMOE_HIP(hipMemcpy(ht, p->ht, size_t(p->L) * p->B * p->K, hipMemcpyDeviceToHost));
    return STMOE_OK;
}

extern "C" int stmoe_import(stmoe_predictor* p, const uint8_t* cct_idx, const uint8_t* cct_conf,
                            const uint8_t* ht) {
    clear_error();
    STMOE_CHECK(p && cct_idx && cct_conf && ht, "null pointer");
    const size_t pairs = size_t(p->L > 1 ? p->L - 1 : 0);
    for (size_t i = 0; i < pairs * p->E * p->K; ++i) {
        STMOE_CHECK(cct_idx[i] < p->E, "CCT index out of range");
        STMOE_CHECK(cct_conf[i] <= 3, "CCT confidence out of range");
    }
    for (size_t i = 0; i < size_t(p->L) * p->B * p->K; ++i) STMOE_CHECK(ht[i] < p->E, "HT index out of range");
    STMOE_HIP(hipDeviceSynchronize());
    if (pairs) {
        STMOE_HIP(hipMemcpy(p->cct_idx, cct_idx, pairs * p->E * p->K, hipMemcpyHostToDevice));
        STMOE_HIP(hipMemcpy(p->cct_conf, cct_conf, pairs * p->E * p->K, hipMemcpyHostToDevice));
    }
    STMOE_HIP(hipMemcpy(p->ht, ht, size_t(p->L) * p->B * p->K, hipMemcpyHostToDevice));
    p->profiled = true;
    return STMOE_OK;
}

extern "C" int stmoe_stats(stmoe_predictor* p, int64_t* out) {
    clear_error();
    STMOE_CHECK(p && out, "null pointer");
    STMOE_HIP(hipDeviceSynchronize());
    STMOE_HIP(hipMemcpy(out, p->stats, size_t(p->L) * 3 * sizeof(int64_t), hipMemcpyDeviceToHost));
    return STMOE_OK;
}
