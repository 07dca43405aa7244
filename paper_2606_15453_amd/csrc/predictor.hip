// Spatio-temporal expert predictor (Section 4.2): Cross-layer Correlation
// Tables with 2-bit confidences and a per-layer History Table.
//
// Tables live in HBM and are small (for 94 layers x 128 experts x top-8:
// 94 KB of CCT indices and 94 KB of confidences), so the runtime kernels run
// as a single workgroup each: the update of one batch row touches K entries
// x K slots (at most 256 lanes, one lane per slot), and the prediction sums
// K x K contributions into per-row score bins in LDS with integer atomics,
// which is exact and order-free.
#include <algorithm>
#include <vector>

#include "gating_dev.h"
#include "predictor_dev.h"


namespace stmoe {
namespace {

using namespace pred;

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
                                                             size_t stride, uint8_t* idx, uint8_t* conf) {
    __shared__ int32_t row[kMaxE];
    const size_t r = blockIdx.x;   // (pair, expert) row
    const size_t out = (r / E) * stride + (r % E) * K;
    for (int f = threadIdx.x; f < E; f += kThreads) row[f] = co[r * E + f];
    __syncthreads();
    for (int f = threadIdx.x; f < E; f += kThreads) {
        const int32_t c = row[f];
        int rank = 0;
        for (int g = 0; g < E; ++g) rank += (row[g] > c) || (row[g] == c && g < f);
        if (rank < K) {
            idx[out + rank] = uint8_t(f);
            conf[out + rank] = uint8_t(kConfInit);
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
                                                           int K, size_t stride, uint8_t* ht) {
    const int l = blockIdx.x, b = blockIdx.y;
    sorted_row(sel_last + (size_t(b) * L + l) * K, K, ht + size_t(l) * stride + size_t(b) * K);
}

// ------------------------------------------------------ update and predict
__global__ __launch_bounds__(kThreads) void update_kernel(UpdateArgs a) {
    __shared__ TableShared sh;
    Seg g[kMaxSegs];
    stage(g, update_segs(a, sh, g));
    update_body(a, sh);
}

__global__ __launch_bounds__(kThreads) void predict_kernel(PredictArgs a) {
    __shared__ TableShared sh;
    Seg g[kMaxSegs];
    stage(g, predict_segs(a, sh, g));
    predict_body(a, sh);
}

// The decode path's router tail, verify/update and next-layer prediction in
// one workgroup (after the router's logits launch).  One round of loads
// brings the logits and every table into LDS; softmax/top-K writes the
// selection there, and the update and the prediction run on it.
__global__ __launch_bounds__(kThreads) void route_update_predict_kernel(gating::RouteArgs r, UpdateArgs u,
                                                                        PredictArgs p) {
    __shared__ TableShared sh;
    Seg g[kMaxSegs];
    u.sel_cur = nullptr;     // the selection is produced in LDS
    p.sel_cur = nullptr;
    int n = 0;
    g[n++] = seg(r.zbuf, sh.z, size_t(r.B) * r.E * sizeof(float));
    n += update_segs(u, sh, g + n);
    n += predict_segs(p, sh, g + n);
    stage(g, n);
    gating::softmax_topk_tail(r, sh.z, sh.sel);
    update_body(u, sh);
    // with one layer the prediction reads the HT row the update just wrote
    if (p.ht_next && p.ht_next == u.ht)
        for (int i = threadIdx.x; i < r.B * r.K; i += kThreads) sh.htn[i] = sh.htnew[i];
    __syncthreads();
    predict_body(p, sh);
}

// The decode path's verify/update and next-layer prediction without the
// router (the selection is read from global memory): used where the router
// runs as its own launches and this work overlaps the expert FFN.
__global__ __launch_bounds__(kThreads) void update_predict_kernel(UpdateArgs u, PredictArgs p) {
    __shared__ TableShared sh;
    Seg g[kMaxSegs];
    p.sel_cur = nullptr;     // the update's copy of the selection serves both
    int n = 0;
    n += update_segs(u, sh, g + n);
    n += predict_segs(p, sh, g + n);
    stage(g, n);
    update_body(u, sh);
    // with one layer the prediction reads the HT row the update just wrote
    if (p.ht_next && p.ht_next == u.ht)
        for (int i = threadIdx.x; i < u.B * u.K; i += kThreads) sh.htn[i] = sh.htnew[i];
    __syncthreads();
    predict_body(p, sh);
}

// One layer's arguments of the sequential kernel below.
struct UpdPred {
    UpdateArgs u;
    PredictArgs p;
};

// The verify/update and next-layer prediction of every layer of one token,
// in layer order, in one workgroup: each layer runs the steps of
// update_predict_kernel on the arguments built for it; the barrier between
// layers orders the tables one layer writes before the next layer stages
// them.
// The arguments are built for both prediction sources with the online
// update on; `use` and `online` select the ablation at launch time.
__global__ __launch_bounds__(kThreads) void update_predict_seq_kernel(const UpdPred* args, int n, int use,
                                                                      int online) {
    __shared__ TableShared sh;
    for (int l = 0; l < n; ++l) {
        UpdateArgs u = args[l].u;
        PredictArgs p = args[l].p;
        u.online = online;
        if (!(use & STMOE_USE_CCT)) {
            p.cidx = nullptr;
            p.cconf = nullptr;
        }
        if (!(use & STMOE_USE_HT)) p.ht_next = nullptr;
        Seg g[kMaxSegs];
        p.sel_cur = nullptr;     // the update's copy of the selection serves both
        int k = 0;
        k += update_segs(u, sh, g + k);
        k += predict_segs(p, sh, g + k);
        stage(g, k);
        update_body(u, sh);
        if (p.ht_next && p.ht_next == u.ht)
            for (int i = threadIdx.x; i < u.B * u.K; i += kThreads) sh.htn[i] = sh.htnew[i];
        __syncthreads();
        predict_body(p, sh);
        __syncthreads();
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

namespace {

// Layout of a predictor's device workspace: every table at a 256-byte
// aligned offset, then the staging area of the profiling selections (at
// least one token's [B][L][K], at least 1 MiB).
struct PredLayout {
    size_t co, cct_idx, cct_conf, ht, pend, stats, stage, stage_bytes, total;
};

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

PredLayout pred_layout(int L, int E, int K, int B) {
    PredLayout y{};
    const size_t pairs = size_t(L > 1 ? L - 1 : 1);
    size_t off = 0;
    auto take = [&](size_t n) { const size_t at = off; off = align256(off + n); return at; };
    y.co = take(pairs * E * E * sizeof(int32_t));
    y.cct_idx = take(pairs * round4(size_t(E) * K));
    y.cct_conf = take(pairs * round4(size_t(E) * K));
    y.ht = take(size_t(L) * round4(size_t(B) * K));
    y.pend = take(size_t(L) * round4(size_t(B) * E));
    y.stats = take(size_t(L) * 3 * sizeof(unsigned long long));
    const size_t token = size_t(B) * L * K * sizeof(int32_t);
    y.stage_bytes = std::max(token, size_t(1) << 20) / token * token;
    y.stage = take(y.stage_bytes);
    y.total = off;
    return y;
}

int check_shape(int L, int E, int K, int B) {
    STMOE_CHECK(L >= 1 && L <= 4096, "L must be in [1, 4096]");
    STMOE_CHECK(E >= 1 && E <= kMaxE, "E must be in [1, 256]");
    STMOE_CHECK(K >= 1 && K <= E && K <= kMaxK, "K must be in [1, min(E, 16)]");
    STMOE_CHECK(B >= 1 && B <= kMaxB, "B must be in [1, 16]");
    return STMOE_OK;
}

}  // namespace

extern "C" size_t stmoe_workspace_bytes(int L, int E, int K, int B) {
    if (check_shape(L, E, K, B) != STMOE_OK) return 0;
    return pred_layout(L, E, K, B).total;
}

extern "C" int stmoe_create(int L, int E, int K, int B, void* dev_ws, size_t ws_bytes, stmoe_predictor** out) {
    clear_error();
    STMOE_CHECK(out && dev_ws, "null pointer");
    if (int rc = check_shape(L, E, K, B)) return rc;
    const PredLayout y = pred_layout(L, E, K, B);
    STMOE_CHECK(ws_bytes >= y.total, "workspace smaller than stmoe_workspace_bytes()");
    STMOE_CHECK(reinterpret_cast<uintptr_t>(dev_ws) % 256 == 0, "workspace must be 256-byte aligned");
    char* base = static_cast<char*>(dev_ws);
    auto* p = new stmoe_predictor();
    p->L = L; p->E = E; p->K = K; p->B = B;
    p->profiled = false;
    p->cct_stride = round4(size_t(E) * K);
    p->ht_stride = round4(size_t(B) * K);
    p->pend_stride = round4(size_t(B) * E);
    p->co = reinterpret_cast<int32_t*>(base + y.co);
    p->cct_idx = reinterpret_cast<uint8_t*>(base + y.cct_idx);
    p->cct_conf = reinterpret_cast<uint8_t*>(base + y.cct_conf);
    p->ht = reinterpret_cast<uint8_t*>(base + y.ht);
    p->pend = reinterpret_cast<uint8_t*>(base + y.pend);
    p->stats = reinterpret_cast<unsigned long long*>(base + y.stats);
    p->stage = reinterpret_cast<int32_t*>(base + y.stage);
    p->stage_bytes = y.stage_bytes;
    hipError_t e = hipMemset(dev_ws, 0, y.stage);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        set_error(std::string("stmoe_create: ") + hipGetErrorString(e));
        delete p;
        return STMOE_EHIP;
    }
    *out = p;
    return STMOE_OK;
}

extern "C" int stmoe_destroy(stmoe_predictor* p) {
    delete p;       // the tables live in the caller's workspace
    return STMOE_OK;
}

extern "C" int stmoe_profile(stmoe_predictor* p, const int32_t* sel, int P) {
    clear_error();
    STMOE_CHECK(p && sel, "null pointer");
    STMOE_CHECK(P >= 1, "P must be >= 1");
    const int L = p->L, E = p->E, K = p->K, B = p->B;
    if (int rc = check_sel_host(sel, size_t(P) * B * L, E, K)) return rc;
    const size_t tok = size_t(B) * L * K;                 // int32 per profiling token
    const int chunk = int(p->stage_bytes / (tok * sizeof(int32_t)));
    const size_t pairs = size_t(L > 1 ? L - 1 : 1);
    // the legacy null stream orders the blocking copies and the kernels
    hipError_t e = hipMemset(p->co, 0, pairs * E * E * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(p->pend, 0, size_t(L) * p->pend_stride);
    if (e == hipSuccess) e = hipMemset(p->stats, 0, size_t(L) * 3 * sizeof(unsigned long long));
    int last_at = 0;
    for (int t0 = 0; t0 < P && e == hipSuccess; t0 += chunk) {
        const int n = std::min(chunk, P - t0);
        e = hipMemcpy(p->stage, sel + size_t(t0) * tok, size_t(n) * tok * sizeof(int32_t), hipMemcpyHostToDevice);
        if (e == hipSuccess && L > 1) {
            hipLaunchKernelGGL(co_count_kernel, dim3(n, L - 1), dim3(kThreads), 0, 0, p->stage, n, B, L, E, K,
                               p->co);
            e = hipGetLastError();
        }
        last_at = P - 1 - t0;                             // the last token's row within the final chunk
    }
    if (e == hipSuccess && L > 1) {
        hipLaunchKernelGGL(cct_build_kernel, dim3(unsigned((L - 1) * E)), dim3(kThreads), 0, 0,
                           p->co, E, K, p->cct_stride, p->cct_idx, p->cct_conf);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(ht_init_kernel, dim3(L, B), dim3(kThreads), 0, 0, p->stage + size_t(last_at) * tok,
                           B, L, K, p->ht_stride, p->ht);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipDeviceSynchronize();
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
    const UpdateArgs a = update_args(p, layer, sel_prev, sel_cur, online);
    hipLaunchKernelGGL(update_kernel, dim3(1), dim3(kThreads), 0, as_stream(stream), a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

extern "C" int stmoe_predict(stmoe_predictor* p, int layer, const int32_t* sel_cur, int use,
                             uint8_t* score, uint8_t* mask, uint8_t* max_score, int32_t* ranked,
                             int32_t* n_ranked, void* stream) {
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
    const PredictArgs a = predict_args(p, layer, sel_cur, use, score, mask, max_score, ranked, n_ranked);
    hipLaunchKernelGGL(predict_kernel, dim3(1), dim3(kThreads), 0, as_stream(stream), a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

namespace stmoe {
int launch_route_logits(const gating::RouteArgs& a, hipStream_t s);

// Internal: router + verify/update at `layer` + prediction of the next layer
// (layer 0 of the next token after the last layer) in two launches.  The
// caller has validated the shapes; the routing workspace follows
// moe_route_workspace_bytes.
int fused_route_predict(const void* x, const void* w_gate, int H, int dtype, int renorm, int32_t* idx,
                        float* w, void* route_ws, stmoe_predictor* p, int layer, const int32_t* sel_prev,
                        int use, int online, int32_t* ranked, int32_t* n_ranked, uint8_t* max_score,
                        hipStream_t s) {
    if (!p->profiled) {
        set_error("moe_decode_layer: predictor has not been profiled");
        return STMOE_ESTATE;
    }
    gating::RouteArgs r;
    r.x = x;
    r.wg = w_gate;
    r.B = p->B;
    r.H = H;
    r.E = p->E;
    r.K = p->K;
    r.renorm = renorm ? 1 : 0;
    r.bf16 = dtype == STMOE_BF16;
    r.idx = idx;
    r.w = w;
    r.logits = nullptr;
    r.zbuf = reinterpret_cast<float*>(route_ws);
    const UpdateArgs u = update_args(p, layer, sel_prev, idx, online);
    const PredictArgs q = layer + 1 < p->L
                              ? predict_args(p, layer, idx, use, nullptr, nullptr, max_score, ranked, n_ranked)
                              : predict_args(p, -1, nullptr, use & STMOE_USE_HT, nullptr, nullptr, max_score,
                                             ranked, n_ranked);
    if (int rc = launch_route_logits(r, s)) return rc;
    hipLaunchKernelGGL(route_update_predict_kernel, dim3(1), dim3(kThreads), 0, s, r, u, q);
    STMOE_LAUNCHED();
    return STMOE_OK;
}
}  // namespace stmoe

extern "C" int stmoe_export(stmoe_predictor* p, int32_t* co, uint8_t* cct_idx, uint8_t* cct_conf,
                            int32_t* ht) {
    clear_error();
    STMOE_CHECK(p, "null predictor");
    const size_t pairs = size_t(p->L > 1 ? p->L - 1 : 0);
    STMOE_HIP(hipDeviceSynchronize());
    if (co && pairs)
        STMOE_HIP(hipMemcpy(co, p->co, pairs * p->E * p->E * sizeof(int32_t), hipMemcpyDeviceToHost));
    const size_t ek = size_t(p->E) * p->K, bk = size_t(p->B) * p->K;
    if (cct_idx && pairs)
        STMOE_HIP(hipMemcpy2D(cct_idx, ek, p->cct_idx, p->cct_stride, ek, pairs, hipMemcpyDeviceToHost));
    if (cct_conf && pairs)
        STMOE_HIP(hipMemcpy2D(cct_conf, ek, p->cct_conf, p->cct_stride, ek, pairs, hipMemcpyDeviceToHost));
    if (ht) {
        std::vector<uint8_t> h(size_t(p->L) * bk);
        STMOE_HIP(hipMemcpy2D(h.data(), bk, p->ht, p->ht_stride, bk, p->L, hipMemcpyDeviceToHost));
        for (size_t i = 0; i < h.size(); ++i) ht[i] = h[i];
    }
    return STMOE_OK;
}

extern "C" int stmoe_import(stmoe_predictor* p, const uint8_t* cct_idx, const uint8_t* cct_conf,
                            const int32_t* ht) {
    clear_error();
    STMOE_CHECK(p && cct_idx && cct_conf && ht, "null pointer");
    const int E = p->E, K = p->K;
    const size_t pairs = size_t(p->L > 1 ? p->L - 1 : 0);
    // an entry names K distinct experts (Algorithm 1 builds it so and Algorithm 3
    // keeps it so), which bounds every Eq. 1 score by 3K + 2
    for (size_t r = 0; r < pairs * E; ++r) {
        const uint8_t* row = cct_idx + r * K;
        for (int k = 0; k < K; ++k) {
            STMOE_CHECK(row[k] < E, "CCT index out of range");
            STMOE_CHECK(cct_conf[r * K + k] <= 3, "CCT confidence out of range");
            for (int j = 0; j < k; ++j) STMOE_CHECK(row[j] != row[k], "CCT entry repeats an expert");
        }
    }
    const size_t bk = size_t(p->B) * K;
    std::vector<uint8_t> h(size_t(p->L) * bk);
    for (size_t r = 0; r < size_t(p->L) * p->B; ++r) {
        const int32_t* row = ht + r * K;
        for (int k = 0; k < K; ++k) {
            STMOE_CHECK(row[k] >= 0 && row[k] < E, "HT index out of range");
            for (int j = 0; j < k; ++j) STMOE_CHECK(row[j] != row[k], "HT row repeats an expert");
        }
        // HT rows are kept sorted ascending
        std::vector<int32_t> v(row, row + K);
        std::sort(v.begin(), v.end());
        for (int k = 0; k < K; ++k) h[r * K + k] = uint8_t(v[size_t(k)]);
    }
    STMOE_HIP(hipDeviceSynchronize());
    const size_t ek = size_t(E) * K;
    if (pairs) {
        STMOE_HIP(hipMemcpy2D(p->cct_idx, p->cct_stride, cct_idx, ek, ek, pairs, hipMemcpyHostToDevice));
        STMOE_HIP(hipMemcpy2D(p->cct_conf, p->cct_stride, cct_conf, ek, ek, pairs, hipMemcpyHostToDevice));
    }
    STMOE_HIP(hipMemcpy2D(p->ht, p->ht_stride, h.data(), bk, bk, p->L, hipMemcpyHostToDevice));
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

namespace stmoe {
// Internal: verify/update at `layer` from the selection sel_cur (device
// [B][K]) + prediction of the next layer, one launch on `s`.  The caller has
// validated the shapes.
int update_predict(stmoe_predictor* p, int layer, const int32_t* sel_prev, const int32_t* sel_cur,
                   int use, int online, int32_t* ranked, int32_t* n_ranked, uint8_t* max_score,
                   hipStream_t s) {
    if (!p->profiled) {
        set_error("moe_decode_layer: predictor has not been profiled");
        return STMOE_ESTATE;
    }
    const UpdateArgs u = update_args(p, layer, sel_prev, sel_cur, online);
    const PredictArgs q = layer + 1 < p->L
                              ? predict_args(p, layer, sel_cur, use, nullptr, nullptr, max_score, ranked, n_ranked)
                              : predict_args(p, -1, nullptr, use & STMOE_USE_HT, nullptr, nullptr, max_score,
                                             ranked, n_ranked);
    hipLaunchKernelGGL(update_predict_kernel, dim3(1), dim3(kThreads), 0, s, u, q);
    STMOE_LAUNCHED();
    return STMOE_OK;
}
}  // namespace stmoe

namespace stmoe {
// Internal: device bytes of the per-layer arguments of update_predict_seq.
size_t update_predict_seq_bytes(int L) { return size_t(L) * sizeof(UpdPred); }

// Internal: build the arguments of every layer for the selections idx_all
// (device [L][B][K]) into dev_args (device, update_predict_seq_bytes(L)),
// for both prediction sources with the online update on; synchronous.
int update_predict_seq_args(stmoe_predictor* p, const int32_t* idx_all, void* dev_args) {
    std::vector<UpdPred> v(size_t(p->L));
    const size_t bk = size_t(p->B) * p->K;
    for (int l = 0; l < p->L; ++l) {
        const int32_t* cur = idx_all + size_t(l) * bk;
        const int32_t* prev = l > 0 ? idx_all + size_t(l - 1) * bk : nullptr;
        v[size_t(l)].u = update_args(p, l, prev, cur, 1);
        v[size_t(l)].p = l + 1 < p->L
                             ? predict_args(p, l, cur, STMOE_USE_BOTH, nullptr, nullptr, nullptr, nullptr, nullptr)
                             : predict_args(p, -1, nullptr, STMOE_USE_HT, nullptr, nullptr, nullptr, nullptr,
                                            nullptr);
    }
    STMOE_HIP(hipMemcpy(dev_args, v.data(), v.size() * sizeof(UpdPred), hipMemcpyHostToDevice));
    return STMOE_OK;
}

// Internal: one token's verify/update and predictions for every layer, in
// layer order, one launch on `s` (the arguments from update_predict_seq_args).
int update_predict_seq(stmoe_predictor* p, const void* dev_args, int use, int online, hipStream_t s) {
    if (!p->profiled) {
        set_error("moe_decode_token: predictor has not been profiled");
        return STMOE_ESTATE;
    }
    hipLaunchKernelGGL(update_predict_seq_kernel, dim3(1), dim3(kThreads), 0, s,
                       static_cast<const UpdPred*>(dev_args), p->L, use, online ? 1 : 0);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

// Internal: the shape a predictor was created with (checked by moe_ctx_create).
void stmoe_shape(const stmoe_predictor* p, int* L, int* E, int* K, int* B) {
    *L = p->L;
    *E = p->E;
    *K = p->K;
    *B = p->B;
}
}  // namespace stmoe
