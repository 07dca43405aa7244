// One decode-step MoE layer (Section 4.3.4, pipelined workflow):
//   route (R) -> verify + table update (V) -> predict the next layer (P)
//   -> missed loading of experts the prediction did not stage (ML)
//   -> expert computation (Com.) -> prefetch of the next layer's predicted
//   experts (EP), overlapping the computation.
//
// Without a cache (every routed expert resident in HBM) the layer never
// waits on the host.  Only the router is on the FFN's critical path: the
// verify/update and the next layer's prediction run on an internal side
// stream that waits for the layer's selection and overlaps the FFN.
// With a cache, the host reads one small routing record per layer (the
// selection and the ranked prediction) because hipMemcpyAsync needs
// host-known source addresses; that is the layer's only host wait.
#include <algorithm>
#include <string>
#include <vector>

#include "cache_device.h"
#include "common.h"

namespace stmoe {
int ffn_launch(const void* x, const int32_t* idx, const float* w, int B, int K, int H, int I, int E,
               int dtype, const void* const* eptr, const void* const* sptr, int n_shared,
               float* y, void* ws, hipStream_t s, unsigned long long* n_experts, hipEvent_t ev_mid,
               const float* logits, int renorm, const void* ebase, size_t estride);
int route_logits(const void* x, const void* w_gate, int B, int H, int E, int dtype, float* z, hipStream_t s);
size_t update_predict_seq_bytes(int L);
int update_predict_seq_args(stmoe_predictor* p, const int32_t* idx_all, void* dev_args);
int update_predict_seq(stmoe_predictor* p, const void* dev_args, int use, int online, hipStream_t s);
void expert_cache_shape(const expert_cache* c, int* L, int* E, size_t* blob_bytes);
DeviceCache* expert_cache_device(expert_cache* c);
int expert_cache_after_demand(const expert_cache* c);
uint64_t expert_cache_version(const expert_cache* c);
void stmoe_shape(const stmoe_predictor* p, int* L, int* E, int* K, int* B);
int fused_route_predict(const void* x, const void* w_gate, int H, int dtype, int renorm, int32_t* idx,
                        float* w, void* route_ws, stmoe_predictor* p, int layer, const int32_t* sel_prev,
                        int use, int online, int32_t* ranked, int32_t* n_ranked, uint8_t* max_score,
                        hipStream_t s);
int update_predict(stmoe_predictor* p, int layer, const int32_t* sel_prev, const int32_t* sel_cur,
                   int use, int online, int32_t* ranked, int32_t* n_ranked, uint8_t* max_score,
                   hipStream_t s);

namespace {

struct PtrTable {
    const void* p[kMaxE];
};

// Write one layer's expert pointer table; the pointers travel as kernel
// arguments, so the host may reuse its copy as soon as the launch returns.
__global__ void set_table_kernel(PtrTable t, const void** dst, int E) {
    for (int e = threadIdx.x; e < E; e += blockDim.x) dst[e] = t.p[e];
}

// The device copy of the decode token that the cache's decisions stamp with
// (a replayed graph advances it by one per token).
__global__ void set_token_kernel(int64_t* tok, int64_t v) { *tok = v; }
__global__ void next_token_kernel(int64_t* tok) { *tok += 1; }

}  // namespace
}  // namespace stmoe

using namespace stmoe;

struct moe_ctx {
    int L, E, K, B, H, I, n_shared, dtype, renorm;
    size_t esz;
    std::vector<const void*> router;       // [L]
    // resident blobs at a fixed stride within every layer (one allocation,
    // as the seeded stacks lay them out): the FFN computes expert e's blob
    // as rbase[layer] + e * rstride instead of loading it from the table
    std::vector<const char*> rbase;        // [L], empty if the table has no such layout
    size_t rstride = 0;
    stmoe_predictor* pred = nullptr;
    expert_cache* cache = nullptr;
    hipStream_t s = nullptr;
    // side stream of the predictor (no cache): ev_sel orders it after the
    // layer's router; ev_side marks its queued work, which the compute stream
    // waits for before selections it may still read are overwritten
    hipStream_t side = nullptr;
    hipEvent_t ev_sel = nullptr, ev_side = nullptr;
    bool side_pending = false;
    // per-token predictor work (resident contexts, moe_decode_token): the
    // layers' selections go to the buffer of the token's parity, and one
    // side-stream launch per token runs every layer's update and prediction;
    // ev_tok[par] marks it, and the buffer is rewritten two tokens later
    bool pred_batch = false;
    int cur_par = 0, last_par = 0;
    hipEvent_t ev_tok[2] = {nullptr, nullptr};
    bool tok_pending[2] = {false, false};
    void* seq_args[2] = {nullptr, nullptr};   // device arguments of update_predict_seq per parity
    int32_t* idx = nullptr;                // [2][L][B][K] device (parity 0 unless pred_batch)
    float* w = nullptr;                    // [2][L][B][K] device
    int32_t* ranked = nullptr;             // device: ranked [E], n_ranked [1], max scores [E] (uint8)
    void* route_ws = nullptr;
    size_t route_ws_bytes = 0;
    void* ffn_ws = nullptr;
    size_t ffn_ws_bytes = 0;
    const void** tables = nullptr;         // [L][E] device blob pointers
    const void** shared = nullptr;         // [L][n_shared] device blob pointers
    int32_t* rec = nullptr;                // pinned host: idx [B][K], ranked [E], n_ranked, max scores [E] (uint8)
    int64_t* tok = nullptr;                // device: decode token of the cache's stamps
    int64_t tok_value = -1;                // what *tok holds once the queued work has run
    bool capturing = false;                // a token's layers are being captured into a graph
    int pf_min_score = 2, pf_max = 1 << 30;
    bool want_ranked = false;              // a report asks for the side path's ranked prediction
    int online = 1;                        // Algorithm 3's CCT update on (1) or frozen CCTs (0)
    hipEvent_t rec_ev = nullptr;
    std::vector<const void*> host_table;   // [E] scratch for the cache's answers
    bool started = false;
    int last_token = -1, last_layer = -1;
    // one HIP graph per token (resident contexts): the whole layer sequence,
    // side branch included, replays with one launch on the graph stream;
    // inputs and outputs pass through the staging buffers
    bool graph_on = false;
    int graph_mode = -1;
    uint64_t settings = 0;                 // bumped by the setters whose values a captured graph bakes in
    uint64_t graph_settings = 0;           // ... and their value when the graph was captured,
    uint64_t graph_cache_version = 0;      // with the cache's configuration version then
    hipStream_t gs = nullptr;
    hipEvent_t ev_in = nullptr, ev_out = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t graph_exec = nullptr;
    void* x_stage = nullptr;               // [L][B][H] dtype
    float* y_stage = nullptr;              // [L][B][H] fp32
    // FFN timing: events around the FFN of every `timing_every`-th token (0: off)
    int timing_every = 0;
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;
    // per timed layer: event indices into ev_pool (-1: not recorded)
    struct TimedLayer {
        int route0 = -1, route1 = -1;      // around the routing launches (compute stream)
        int up0 = -1, mid = -1, down1 = -1;  // around the FFN's two kernels
        int pred0 = -1, pred1 = -1;        // around update/predict on the side stream
    };
    std::vector<TimedLayer> timed_layers;
    unsigned long long* n_experts = nullptr;   // device counter
    int64_t n_calls = 0;
};

namespace {

// device/host record of one prediction: ranked [E] int32, n_ranked int32, max scores [E] uint8
size_t ranked_bytes(int E) { return size_t(E + 1) * sizeof(int32_t) + size_t(E); }
uint8_t* max_scores(int32_t* ranked, int E) { return reinterpret_cast<uint8_t*>(ranked + E + 1); }

void free_ctx(moe_ctx* c) {
    if (!c) return;
    if (c->s) (void)hipStreamSynchronize(c->s);
    if (c->side) {
        (void)hipStreamSynchronize(c->side);
        (void)hipStreamDestroy(c->side);
    }
    if (c->ev_sel) (void)hipEventDestroy(c->ev_sel);
    if (c->ev_side) (void)hipEventDestroy(c->ev_side);
    for (int i = 0; i < 2; ++i)
        if (c->ev_tok[i]) (void)hipEventDestroy(c->ev_tok[i]);
    if (c->gs) {
        (void)hipStreamSynchronize(c->gs);
        (void)hipStreamDestroy(c->gs);
    }
    if (c->graph_exec) (void)hipGraphExecDestroy(c->graph_exec);
    if (c->graph) (void)hipGraphDestroy(c->graph);
    if (c->ev_in) (void)hipEventDestroy(c->ev_in);
    if (c->ev_out) (void)hipEventDestroy(c->ev_out);
    if (c->rec) (void)hipHostFree(c->rec);
    if (c->rec_ev) (void)hipEventDestroy(c->rec_ev);
    for (auto e : c->ev_pool) (void)hipEventDestroy(e);
    delete c;       // device buffers live in the caller's workspace
}

// Layout of a context's device workspace (every region 256-byte aligned).
struct CtxLayout {
    size_t idx, w, ranked, route_ws, ffn_ws, tables, shared, n_experts, seq_args, x_stage, y_stage, tok, total;
    size_t route_ws_bytes, ffn_ws_bytes, seq_bytes;
};

CtxLayout ctx_layout(const moe_model_desc* d) {
    CtxLayout y{};
    const size_t LBK = size_t(d->L) * d->B * d->K, LBH = size_t(d->L) * d->B * d->H;
    const size_t esz = d->dtype == STMOE_BF16 ? 2 : 4;
    y.route_ws_bytes = moe_route_workspace_bytes(d->B, d->E);
    y.ffn_ws_bytes = moe_expert_ffn_workspace_bytes(d->B, d->K, d->E, d->H, d->I, d->n_shared, d->dtype);
    y.seq_bytes = update_predict_seq_bytes(d->L);
    size_t off = 0;
    auto take = [&](size_t n) { const size_t at = off; off = (off + n + 255) / 256 * 256; return at; };
    y.idx = take(2 * LBK * sizeof(int32_t));
    y.w = take(2 * LBK * sizeof(float));
    y.ranked = take(ranked_bytes(d->E));
    y.route_ws = take(y.route_ws_bytes);
    y.ffn_ws = take(y.ffn_ws_bytes);
    y.tables = take(size_t(d->L) * d->E * sizeof(void*));
    y.shared = take(size_t(d->L) * d->n_shared * sizeof(void*));
    y.n_experts = take(sizeof(unsigned long long));
    y.seq_args = take(2 * y.seq_bytes);
    y.x_stage = take(LBH * esz);
    y.y_stage = take(LBH * sizeof(float));
    y.tok = take(sizeof(int64_t));
    y.total = off;
    return y;
}

int check_desc(const moe_model_desc* d) {
    STMOE_CHECK(d && d->router_w, "null pointer");
    STMOE_CHECK(d->L >= 1 && d->E >= 1 && d->E <= kMaxE, "bad L/E");
    STMOE_CHECK(d->K >= 1 && d->K <= d->E && d->K <= kMaxK, "bad K");
    STMOE_CHECK(d->B >= 1 && d->B <= kMaxB, "bad B");
    STMOE_CHECK(d->H >= 8 && d->H % 8 == 0 && d->H <= kMaxH, "bad H");
    STMOE_CHECK(d->I >= 8 && d->I % 8 == 0, "bad I");
    STMOE_CHECK(d->n_shared >= 0 && d->n_shared <= 8, "bad n_shared");
    STMOE_CHECK(d->n_shared == 0 || d->shared_w, "shared_w is required when n_shared > 0");
    STMOE_CHECK(d->dtype == STMOE_BF16 || d->dtype == STMOE_F32, "bad dtype");
    return STMOE_OK;
}

int use_bits(int mode) {
    switch (mode) {
        case MOE_MODE_STMOE: return STMOE_USE_BOTH;
        case MOE_MODE_HT_ONLY: return STMOE_USE_HT;
        case MOE_MODE_CCT_ONLY: return STMOE_USE_CCT;
        default: return 0;
    }
}

int set_table(moe_ctx* c, int layer, const std::vector<const void*>& tab) {
    PtrTable t;
    for (int e = 0; e < c->E; ++e) t.p[e] = tab[e];
    hipLaunchKernelGGL(set_table_kernel, dim3(1), dim3(256), 0, c->s, t, c->tables + size_t(layer) * c->E,
                       c->E);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

// Prefetch the ranked prediction held in the host record, subject to the
// admission knobs (minimum score, maximum per layer).
int prefetch_from_record(moe_ctx* c, int target, int64_t stamp) {
    int32_t* ranked = c->rec + c->B * c->K;
    const uint8_t* ms = max_scores(ranked, c->E);
    int n = 0;
    const int total = ranked[c->E];
    while (n < total && n < c->pf_max && ms[ranked[n]] >= c->pf_min_score) ++n;
    if (n <= 0) return STMOE_OK;
    const int rc = expert_cache_prefetch(c->cache, target, ranked, n, stamp);
    return rc < 0 ? rc : STMOE_OK;
}

int fetch_record(moe_ctx* c, const int32_t* idx_dev, bool with_ranked) {
    STMOE_HIP(hipMemcpyAsync(c->rec, idx_dev, size_t(c->B) * c->K * sizeof(int32_t),
                             hipMemcpyDeviceToHost, c->s));
    if (with_ranked)
        STMOE_HIP(hipMemcpyAsync(c->rec + c->B * c->K, c->ranked, ranked_bytes(c->E), hipMemcpyDeviceToHost,
                                 c->s));
    STMOE_HIP(hipEventRecord(c->rec_ev, c->s));
    STMOE_HIP(hipEventSynchronize(c->rec_ev));
    return STMOE_OK;
}

// Timing events are only read after a device-wide sync, so they skip the
// system-scope fence (a cache writeback at every record that would stretch
// the measured intervals).
hipEvent_t next_event(moe_ctx* c) {
    if (c->ev_used == c->ev_pool.size()) {
        hipEvent_t e;
        if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
        c->ev_pool.push_back(e);
    }
    return c->ev_pool[c->ev_used++];
}

}  // namespace

extern "C" size_t moe_ctx_workspace_bytes(const moe_model_desc* d) {
    if (!d || check_desc(d) != STMOE_OK) return 0;
    return ctx_layout(d).total;
}

extern "C" int moe_ctx_create(const moe_model_desc* d, stmoe_predictor* pred, expert_cache* cache,
                              void* compute_stream, void* dev_ws, size_t ws_bytes, moe_ctx** out) {
    clear_error();
    STMOE_CHECK(out && dev_ws, "null pointer");
    if (int rc = check_desc(d)) return rc;
    STMOE_CHECK((cache == nullptr) != (d->resident_w == nullptr),
                "give exactly one of a cache or resident expert pointers");
    for (int l = 0; l < d->L; ++l) STMOE_CHECK(d->router_w[l], "null router pointer");
    const CtxLayout y = ctx_layout(d);
    STMOE_CHECK(ws_bytes >= y.total, "workspace smaller than moe_ctx_workspace_bytes()");
    STMOE_CHECK(reinterpret_cast<uintptr_t>(dev_ws) % 256 == 0, "workspace must be 256-byte aligned");
    if (pred) {
        int pL, pE, pK, pB;
        stmoe_shape(pred, &pL, &pE, &pK, &pB);
        STMOE_CHECK(pL == d->L && pE == d->E && pK == d->K && pB == d->B,
                    "the predictor was created for another L/E/K/B");
    }
    if (cache) {
        int cL, cE;
        size_t cblob;
        expert_cache_shape(cache, &cL, &cE, &cblob);
        STMOE_CHECK(cL == d->L && cE == d->E, "the cache was created for another L/E");
        STMOE_CHECK(cblob >= moe_blob_bytes(d->H, d->I, d->dtype), "the cache's blobs are smaller than an expert");
    }
    auto* c = new moe_ctx();
    c->L = d->L; c->E = d->E; c->K = d->K; c->B = d->B; c->H = d->H; c->I = d->I;
    c->n_shared = d->n_shared; c->dtype = d->dtype; c->renorm = d->renorm;
    c->esz = d->dtype == STMOE_BF16 ? 2 : 4;
    c->router.assign(d->router_w, d->router_w + d->L);
    c->pred = pred;
    c->cache = cache;
    c->s = as_stream(compute_stream);
    c->host_table.assign(c->E, nullptr);
    if (d->resident_w) {
        auto at = [&](int l, int x) { return reinterpret_cast<uintptr_t>(d->resident_w[size_t(l) * d->E + x]); };
        const uintptr_t stride = d->E > 1 ? at(0, 1) - at(0, 0) : 0;
        bool strided = d->E == 1 || at(0, 1) > at(0, 0);
        for (int l = 0; strided && l < d->L; ++l)
            for (int x = 0; strided && x < d->E; ++x) strided = at(l, x) == at(l, 0) + uintptr_t(x) * stride;
        if (strided) {
            c->rstride = size_t(stride);
            for (int l = 0; l < d->L; ++l) c->rbase.push_back(reinterpret_cast<const char*>(at(l, 0)));
        }
    }
    char* base = static_cast<char*>(dev_ws);
    c->idx = reinterpret_cast<int32_t*>(base + y.idx);
    c->w = reinterpret_cast<float*>(base + y.w);
    c->ranked = reinterpret_cast<int32_t*>(base + y.ranked);
    c->route_ws = base + y.route_ws;
    c->route_ws_bytes = y.route_ws_bytes;
    c->ffn_ws = base + y.ffn_ws;
    c->ffn_ws_bytes = y.ffn_ws_bytes;
    c->tables = reinterpret_cast<const void**>(base + y.tables);
    c->shared = c->n_shared ? reinterpret_cast<const void**>(base + y.shared) : nullptr;
    c->n_experts = reinterpret_cast<unsigned long long*>(base + y.n_experts);
    c->seq_args[0] = base + y.seq_args;
    c->seq_args[1] = base + y.seq_args + y.seq_bytes;
    c->x_stage = base + y.x_stage;
    c->y_stage = reinterpret_cast<float*>(base + y.y_stage);
    c->tok = reinterpret_cast<int64_t*>(base + y.tok);
    hipError_t e = hipHostMalloc(&c->rec, size_t(c->B * c->K) * sizeof(int32_t) + ranked_bytes(c->E));
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->rec_ev, hipEventDisableTiming);
    if (e == hipSuccess && !cache && pred) {
        // the side stream's events only order kernels of this device (the
        // kernel boundaries make their writes visible): no system-scope fence,
        // which would write back the caches at every record
        e = hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&c->ev_sel, hipEventDisableTiming | hipEventDisableSystemFence);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&c->ev_side, hipEventDisableTiming | hipEventDisableSystemFence);
    }
    if (e == hipSuccess) e = hipMemset(dev_ws, 0, y.total);
    if (e == hipSuccess && d->resident_w)
        e = hipMemcpy(c->tables, d->resident_w, size_t(c->L) * c->E * sizeof(void*), hipMemcpyHostToDevice);
    if (e == hipSuccess && c->n_shared)
        e = hipMemcpy(c->shared, d->shared_w, size_t(c->L) * c->n_shared * sizeof(void*),
                      hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        set_error(std::string("moe_ctx_create: ") + hipGetErrorString(e));
        free_ctx(c);
        return e == hipErrorOutOfMemory ? STMOE_ENOMEM : STMOE_EHIP;
    }
    // the per-token predictor launch reads each parity's selections through
    // arguments built once here
    if (pred) {
        const size_t LBK = size_t(c->L) * c->B * c->K;
        for (int par = 0; par < 2; ++par)
            if (int rc = update_predict_seq_args(pred, c->idx + par * LBK, c->seq_args[par])) {
                free_ctx(c);
                return rc;
            }
    }
    *out = c;
    return STMOE_OK;
}

extern "C" int moe_ctx_destroy(moe_ctx* c) {
    free_ctx(c);
    return STMOE_OK;
}

namespace {

bool timed_token(const moe_ctx* c, int token) { return c->timing_every > 0 && token % c->timing_every == 0; }

// Verify/update and the next layer's prediction on the side stream; the
// ranked prediction is kept only when a layer report asks for it.
int side_update_predict(moe_ctx* c, int layer, const int32_t* prev, const int32_t* idx_l, int use) {
    const int E = c->E;
    if (c->want_ranked)
        return update_predict(c->pred, layer, prev, idx_l, use, c->online, c->ranked, c->ranked + E,
                              max_scores(c->ranked, E), c->side);
    return update_predict(c->pred, layer, prev, idx_l, use, c->online, nullptr, nullptr, nullptr, c->side);
}

// One layer; `timing` permits the FFN events of timed tokens (off while a
// graph is captured).  Arguments are checked by the callers.
int decode_layer(moe_ctx* c, int token, int layer, const void* x, float* y, int mode, bool timing,
                 bool defer_side = false) {
    const int use = use_bits(mode);
    STMOE_CHECK(use == 0 || c->pred, "prediction modes need a predictor");
    const int L = c->L, B = c->B, K = c->K, E = c->E;
    const int64_t stamp = int64_t(token) * L + layer + 1;
    const size_t pbase = size_t(c->cur_par) * L * B * K;
    int32_t* idx_l = c->idx + pbase + size_t(layer) * B * K;
    float* w_l = c->w + pbase + size_t(layer) * B * K;
    c->last_par = c->cur_par;
    // device decisions stamp with the token held on the device (a graph
    // replay advances it); eager calls set it when it differs
    DeviceCache* dcache = c->cache ? expert_cache_device(c->cache) : nullptr;
    if (dcache && !c->capturing && c->tok_value != token) {
        hipLaunchKernelGGL(set_token_kernel, dim3(1), dim3(1), 0, c->s, c->tok, int64_t(token));
        STMOE_LAUNCHED();
        c->tok_value = token;
    }

    // first call: layer 0's prediction comes from the profiled HT[0]
    if (!c->started) {
        c->started = true;
        if (use) {
            if (int rc = stmoe_predict(c->pred, -1, nullptr, use & STMOE_USE_HT, nullptr, nullptr,
                                       max_scores(c->ranked, E), c->ranked, c->ranked + E, c->s))
                return rc;
            if (DeviceCache* dc = c->cache ? expert_cache_device(c->cache) : nullptr) {
                if (int rc = device_cache_decide(dc, 0, 0, nullptr, 0, c->ranked, c->ranked + E,
                                                 max_scores(c->ranked, E), c->pf_min_score, c->pf_max,
                                                 c->tok, layer, c->tables, c->s))
                    return rc;
                if (int rc = device_cache_prefetch(dc, 0, c->s)) return rc;
            } else if (c->cache) {
                if (int rc = fetch_record(c, idx_l, true)) return rc;
                if (int rc = prefetch_from_record(c, 0, stamp - 1)) return rc;
            }
        }
    }

    // R + V + P.  Without a cache: the router on the compute stream (for
    // B*E <= 128 only its logits: the FFN's gate/up kernel does softmax and
    // top-K), then verify/update and prediction on the side stream, off the
    // FFN's path.
    // Side work still queued reads selections of this token's layers and the
    // next one's; in the usual layer order it can only collide with this
    // call from layer 0 on, so the compute stream waits for it once per token.
    const bool in_order = layer == (c->last_layer + 1) % L;
    if (c->side_pending && (layer == 0 || !in_order || !(use && c->side))) {
        STMOE_HIP(hipEventRecord(c->ev_side, c->side));
        STMOE_HIP(hipStreamWaitEvent(c->s, c->ev_side, 0));
        c->side_pending = false;
    }
    const bool route_in_ffn = !c->cache && B * E <= kRouteInFfnMax;
    float* zbuf = reinterpret_cast<float*>(c->route_ws);
    const bool timed = timing && timed_token(c, token);
    moe_ctx::TimedLayer tl;
    auto stamp_event = [&](int& slot, hipStream_t st) -> int {
        hipEvent_t ev = next_event(c);
        if (!ev) {
            set_error("moe_decode_layer: hipEventCreate failed");
            return STMOE_EHIP;
        }
        slot = int(c->ev_used - 1);
        STMOE_HIP(hipEventRecord(ev, st));
        return STMOE_OK;
    };
    if (timed)
        if (int rc = stamp_event(tl.route0, c->s)) return rc;
    if (route_in_ffn) {
        if (int rc = route_logits(x, c->router[layer], B, c->H, E, c->dtype, zbuf, c->s)) return rc;
    } else if (use && c->side) {
        if (int rc = moe_route_topk(x, c->router[layer], B, c->H, E, K, c->dtype, c->renorm, idx_l, w_l,
                                    nullptr, c->route_ws, c->route_ws_bytes, c->s))
            return rc;
        if (!defer_side) {
            STMOE_HIP(hipEventRecord(c->ev_sel, c->s));
            STMOE_HIP(hipStreamWaitEvent(c->side, c->ev_sel, 0));
            const int32_t* prev = layer > 0 ? c->idx + pbase + size_t(layer - 1) * B * K : nullptr;
            if (timed)
                if (int rc = stamp_event(tl.pred0, c->side)) return rc;
            if (int rc = side_update_predict(c, layer, prev, idx_l, use)) return rc;
            if (timed)
                if (int rc = stamp_event(tl.pred1, c->side)) return rc;
            c->side_pending = true;
        }
    } else if (use) {
        // with a cache the host reads the prediction: one fused launch pair
        const int32_t* prev = layer > 0 ? c->idx + pbase + size_t(layer - 1) * B * K : nullptr;
        if (int rc = fused_route_predict(x, c->router[layer], c->H, c->dtype, c->renorm, idx_l, w_l,
                                         c->route_ws, c->pred, layer, prev, use, c->online, c->ranked,
                                         c->ranked + E, max_scores(c->ranked, E), c->s))
            return rc;
    } else {
        if (int rc = moe_route_topk(x, c->router[layer], B, c->H, E, K, c->dtype, c->renorm, idx_l, w_l,
                                    nullptr, c->route_ws, c->route_ws_bytes, c->s))
            return rc;
    }
    // with a cache the routing record wait and the missed loads come next;
    // without one the FFN follows directly and its first event ends routing
    if (timed && c->cache)
        if (int rc = stamp_event(tl.route1, c->s)) return rc;
    // ML: make the selection resident
    DeviceCache* dc = c->cache ? expert_cache_device(c->cache) : nullptr;
    const bool pf_now = dc && use && L > 1;          // L == 1: after the FFN, which reads the same slots
    if (dc) {
        // device decisions: no host wait; the FFN reads the table they write
        if (int rc = device_cache_decide(dc, layer, (layer + 1) % L, idx_l, B * K, use ? c->ranked : nullptr,
                                         c->ranked + E, max_scores(c->ranked, E), c->pf_min_score, c->pf_max,
                                         c->tok, layer + 1, c->tables + size_t(layer) * E, c->s))
            return rc;
        const bool after_demand = expert_cache_after_demand(c->cache);
        if (pf_now && !after_demand)
            if (int rc = device_cache_prefetch(dc, (layer + 1) % L, c->s)) return rc;
        if (int rc = device_cache_demand(dc, layer, c->s)) return rc;
        if (pf_now && after_demand)
            if (int rc = device_cache_prefetch(dc, (layer + 1) % L, c->s)) return rc;
    } else if (c->cache) {
        if (int rc = fetch_record(c, idx_l, use != 0)) return rc;
        int needed[kMaxE];
        int n = 0;
        {
            std::vector<char> seen(E, 0);
            for (int i = 0; i < B * K; ++i) {
                const int e = c->rec[i];
                if (e < 0 || e >= E) {
                    set_error("moe_decode_layer: routing produced an invalid expert index");
                    return STMOE_ESTATE;
                }
                if (!seen[e]) { seen[e] = 1; needed[n++] = e; }
            }
            std::sort(needed, needed + n);
        }
        const int rc = expert_cache_acquire(c->cache, layer, needed, n, stamp, c->host_table.data(), c->s);
        if (rc < 0) return rc;
        if (int rc2 = set_table(c, layer, c->host_table)) return rc2;
    }
    // Com.: expert FFN (timed with events before, between and after its two kernels)
    hipEvent_t e1 = nullptr;
    if (timed) {
        if (int rc = stamp_event(tl.up0, c->s)) return rc;
        if (!c->cache) tl.route1 = tl.up0;
        e1 = next_event(c);
        if (!e1) { set_error("moe_decode_layer: hipEventCreate failed"); return STMOE_EHIP; }
        tl.mid = int(c->ev_used - 1);
    }
    if (int rc = ffn_launch(x, idx_l, w_l, B, K, c->H, c->I, E, c->dtype, c->tables + size_t(layer) * E,
                            c->n_shared ? c->shared + size_t(layer) * c->n_shared : nullptr, c->n_shared,
                            y, c->ffn_ws, c->s, timed ? c->n_experts : nullptr, e1,
                            route_in_ffn ? zbuf : nullptr, c->renorm,
                            c->rbase.empty() ? nullptr : c->rbase[size_t(layer)], c->rstride))
        return rc;
    if (timed) {
        if (int rc = stamp_event(tl.down1, c->s)) return rc;
        ++c->n_calls;
    }
    if (route_in_ffn && use && c->side && !defer_side) {
        // the selection exists once the FFN has run
        STMOE_HIP(hipEventRecord(c->ev_sel, c->s));
        STMOE_HIP(hipStreamWaitEvent(c->side, c->ev_sel, 0));
        const int32_t* prev = layer > 0 ? c->idx + pbase + size_t(layer - 1) * B * K : nullptr;
        if (timed)
            if (int rc = stamp_event(tl.pred0, c->side)) return rc;
        if (int rc = side_update_predict(c, layer, prev, idx_l, use)) return rc;
        if (timed)
            if (int rc = stamp_event(tl.pred1, c->side)) return rc;
        c->side_pending = true;
    }
    if (timed) c->timed_layers.push_back(tl);
    // EP: prefetch the next layer's predicted experts, overlapping the FFN
    if (dc) {
        if (use && !pf_now)
            if (int rc = device_cache_prefetch(dc, (layer + 1) % L, c->s)) return rc;
    } else if (c->cache) {
        if (int rc = expert_cache_release(c->cache, layer, c->s)) return rc;
        if (use) {
            if (int rc = prefetch_from_record(c, (layer + 1) % L, stamp)) return rc;
        }
    }
    c->last_token = token;
    c->last_layer = layer;
    return STMOE_OK;
}

// The compute stream waits for side work still queued (it reads selections
// that the next work rewrites).
int join_side(moe_ctx* c) {
    if (!c->side_pending) return STMOE_OK;
    STMOE_HIP(hipEventRecord(c->ev_side, c->side));
    STMOE_HIP(hipStreamWaitEvent(c->s, c->ev_side, 0));
    c->side_pending = false;
    return STMOE_OK;
}

// The compute stream waits for the per-token predictor launch that still
// reads the selection buffer of parity `par`.
int wait_token_side(moe_ctx* c, int par) {
    if (!c->tok_pending[par]) return STMOE_OK;
    STMOE_HIP(hipStreamWaitEvent(c->s, c->ev_tok[par], 0));
    c->tok_pending[par] = false;
    return STMOE_OK;
}

// One token's predictor work in one side-stream launch (after its last
// layer): every layer's verify/update and next-layer prediction, in layer
// order, on the selections of parity c->cur_par.
int token_side(moe_ctx* c, int token, int use) {
    const int par = c->cur_par;
    STMOE_HIP(hipEventRecord(c->ev_sel, c->s));
    STMOE_HIP(hipStreamWaitEvent(c->side, c->ev_sel, 0));
    const bool timed = c->timing_every > 0 && token % c->timing_every == 0 && !c->timed_layers.empty();
    int p0 = -1, p1 = -1;
    auto stamp = [&](int& slot) -> int {
        hipEvent_t ev = next_event(c);
        if (!ev) {
            set_error("moe_decode_token: hipEventCreate failed");
            return STMOE_EHIP;
        }
        slot = int(c->ev_used - 1);
        STMOE_HIP(hipEventRecord(ev, c->side));
        return STMOE_OK;
    };
    if (timed)
        if (int rc = stamp(p0)) return rc;
    if (int rc = update_predict_seq(c->pred, c->seq_args[par], use, c->online, c->side)) return rc;
    if (timed) {
        if (int rc = stamp(p1)) return rc;
        // the token's predictor time, reported with its last layer
        c->timed_layers.back().pred0 = p0;
        c->timed_layers.back().pred1 = p1;
    }
    STMOE_HIP(hipEventRecord(c->ev_tok[par], c->side));
    c->tok_pending[par] = true;
    return STMOE_OK;
}

// A captured graph bakes in the context's knobs and the cache's
// configuration: it is stale once either changed.
bool graph_stale(const moe_ctx* c) {
    return c->graph_settings != c->settings ||
           (c->cache && c->graph_cache_version != expert_cache_version(c->cache));
}

// Capture all L layers of one token, reading x_stage and writing y_stage,
// into c->graph_exec.  The capture runs on the graph stream (the compute
// stream may be the null stream, which cannot be captured).
int capture_token(moe_ctx* c, int token, int mode) {
    if (c->graph_exec) (void)hipGraphExecDestroy(c->graph_exec);
    if (c->graph) (void)hipGraphDestroy(c->graph);
    c->graph_exec = nullptr;
    c->graph = nullptr;
    hipStream_t user = c->s;
    c->s = c->gs;
    DeviceCache* dc = c->cache ? expert_cache_device(c->cache) : nullptr;
    if (dc) {
        // the graph starts from a state with every earlier copy done: the
        // graph stream waits for the cache's side work, and the capture does
        // not refer to completion events recorded outside it
        if (int rc = device_cache_join(dc, c->gs)) { c->s = user; return rc; }
        device_cache_forget_waits(dc);
    }
    STMOE_HIP(hipStreamBeginCapture(c->gs, hipStreamCaptureModeThreadLocal));
    c->capturing = true;
    int rc = STMOE_OK;
    for (int l = 0; l < c->L && rc == STMOE_OK; ++l) {
        const char* x = reinterpret_cast<const char*>(c->x_stage) + size_t(l) * c->B * c->H * c->esz;
        rc = decode_layer(c, token, l, x, c->y_stage + size_t(l) * c->B * c->H, mode, false);
    }
    if (rc == STMOE_OK) rc = join_side(c);      // the side branch rejoins inside the graph
    if (rc == STMOE_OK && dc) {
        // the next replay stamps the next token; the prefetch copies rejoin
        hipLaunchKernelGGL(next_token_kernel, dim3(1), dim3(1), 0, c->gs, c->tok);
        if (hipGetLastError() != hipSuccess) rc = STMOE_EHIP;
        if (rc == STMOE_OK) rc = device_cache_join(dc, c->gs);
    }
    c->capturing = false;
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(c->gs, &g);
    c->s = user;
    c->side_pending = false;
    if (dc) device_cache_forget_waits(dc);     // events recorded in the capture are graph nodes
    if (rc != STMOE_OK || e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        if (rc == STMOE_OK) set_error(std::string("moe_decode_token: capture: ") + hipGetErrorString(e));
        return rc != STMOE_OK ? rc : STMOE_EHIP;
    }
    const hipError_t ei = hipGraphInstantiate(&c->graph_exec, g, nullptr, nullptr, 0);
    if (ei != hipSuccess) {
        (void)hipGraphDestroy(g);
        c->graph_exec = nullptr;
        set_error(std::string("moe_decode_token: instantiate: ") + hipGetErrorString(ei));
        return STMOE_EHIP;
    }
    c->graph = g;
    c->graph_mode = mode;
    c->graph_settings = c->settings;
    c->graph_cache_version = c->cache ? expert_cache_version(c->cache) : 0;
    return STMOE_OK;
}

int decode_token_graph(moe_ctx* c, int token, const void* xs, float* ys, int mode) {
    if (int rc = join_side(c)) return rc;
    c->cur_par = 0;
    DeviceCache* dc = c->cache ? expert_cache_device(c->cache) : nullptr;
    if (c->cache && !dc) {
        set_error("moe_decode_token: graph replay with a cache needs device-side decisions");
        return STMOE_ESTATE;
    }
    if (!c->graph_exec || c->graph_mode != mode || graph_stale(c))
        if (int rc = capture_token(c, token, mode)) return rc;
    const size_t n = size_t(c->L) * c->B * c->H;
    STMOE_HIP(hipEventRecord(c->ev_in, c->s));
    STMOE_HIP(hipStreamWaitEvent(c->gs, c->ev_in, 0));
    if (dc) {
        // earlier eager work of the cache's side stream, and the token stamp
        if (int rc = device_cache_join(dc, c->gs)) return rc;
        device_cache_forget_waits(dc);
        if (c->tok_value != token) {
            hipLaunchKernelGGL(set_token_kernel, dim3(1), dim3(1), 0, c->gs, c->tok, int64_t(token));
            STMOE_LAUNCHED();
        }
        c->tok_value = token + 1;      // the graph advances the device token
    }
    if (xs != c->x_stage)
        STMOE_HIP(hipMemcpyAsync(c->x_stage, xs, n * c->esz, hipMemcpyDeviceToDevice, c->gs));
    STMOE_HIP(hipGraphLaunch(c->graph_exec, c->gs));
    if (ys != c->y_stage)
        STMOE_HIP(hipMemcpyAsync(ys, c->y_stage, n * sizeof(float), hipMemcpyDeviceToDevice, c->gs));
    STMOE_HIP(hipEventRecord(c->ev_out, c->gs));
    STMOE_HIP(hipStreamWaitEvent(c->s, c->ev_out, 0));
    c->last_token = token;
    c->last_layer = c->L - 1;
    return STMOE_OK;
}

}  // namespace

namespace {
// The report of the layer just issued: waits for its work on every stream.
int fill_report(moe_ctx* c, int layer, int mode, moe_layer_report* rep) {
    STMOE_HIP(hipStreamSynchronize(c->s));
    if (c->side) STMOE_HIP(hipStreamSynchronize(c->side));
    const size_t bk = size_t(c->B) * c->K;
    *rep = moe_layer_report{};
    rep->B = c->B;
    rep->K = c->K;
    STMOE_HIP(hipMemcpy(rep->idx, c->idx + size_t(layer) * bk, bk * sizeof(int32_t), hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(rep->w, c->w + size_t(layer) * bk, bk * sizeof(float), hipMemcpyDeviceToHost));
    for (int e = 0; e < kMaxE; ++e) rep->ranked[e] = -1;
    rep->n_ranked = -1;
    if (use_bits(mode) && c->pred) {
        std::vector<int32_t> r(size_t(c->E) + 1);
        STMOE_HIP(hipMemcpy(r.data(), c->ranked, r.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
        rep->n_ranked = r[size_t(c->E)];
        for (int e = 0; e < c->E; ++e) rep->ranked[e] = r[size_t(e)];
    }
    if (c->pred) {
        std::vector<int64_t> st(size_t(c->L) * 3);
        if (int rc = stmoe_stats(c->pred, st.data())) return rc;
        for (int i = 0; i < 3; ++i) rep->pred_stats[i] = st[size_t(layer) * 3 + i];
    }
    if (c->cache)
        if (int rc = expert_cache_stats(c->cache, &rep->cache)) return rc;
    return STMOE_OK;
}
}  // namespace

extern "C" int moe_decode_layer(moe_ctx* c, int token, int layer, const void* x, float* y, int mode,
                                moe_layer_report* rep) {
    clear_error();
    STMOE_CHECK(c && x && y, "null pointer");
    STMOE_CHECK(layer >= 0 && layer < c->L, "layer out of range");
    STMOE_CHECK(token >= 0, "token must be >= 0");
    STMOE_CHECK(mode >= MOE_MODE_ON_DEMAND && mode <= MOE_MODE_CCT_ONLY, "bad mode");
    // single layers use the parity-0 selection buffer and per-layer predictor work
    c->cur_par = 0;
    if (int rc = wait_token_side(c, 0)) return rc;
    c->want_ranked = rep != nullptr;
    const int rc = decode_layer(c, token, layer, x, y, mode, true);
    c->want_ranked = false;
    if (rc != STMOE_OK || !rep) return rc;
    return fill_report(c, layer, mode, rep);
}

extern "C" int moe_ctx_set_predictor_batch(moe_ctx* c, int on) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_CHECK(on == 0 || on == 1, "on must be 0 or 1");
    STMOE_CHECK(!on || (!c->cache && c->side), "per-token predictor launches need a context without a cache "
                                               "and with a predictor");
    STMOE_CHECK(!on || !c->graph_on, "per-token predictor launches and graph replay exclude each other");
    STMOE_HIP(hipDeviceSynchronize());
    if (on && !c->ev_tok[0]) {
        for (int i = 0; i < 2; ++i)
            STMOE_HIP(hipEventCreateWithFlags(&c->ev_tok[i], hipEventDisableTiming | hipEventDisableSystemFence));
    }
    c->tok_pending[0] = c->tok_pending[1] = false;
    c->side_pending = false;
    c->pred_batch = on != 0;
    c->cur_par = 0;
    return STMOE_OK;
}

extern "C" int moe_ctx_set_graph(moe_ctx* c, int on) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_CHECK(!on || !c->cache || expert_cache_device(c->cache),
                "graph replay with a cache needs device-side decisions");
    STMOE_CHECK(!on || !c->pred_batch, "per-token predictor launches and graph replay exclude each other");
    STMOE_HIP(hipStreamSynchronize(c->s));
    if (c->gs) STMOE_HIP(hipStreamSynchronize(c->gs));
    if (c->graph_exec) (void)hipGraphExecDestroy(c->graph_exec);
    if (c->graph) (void)hipGraphDestroy(c->graph);
    c->graph_exec = nullptr;
    c->graph = nullptr;
    c->graph_mode = -1;
    if (on && !c->gs) {
        // the staging buffers are part of the context's workspace
        hipError_t e = hipStreamCreateWithFlags(&c->gs, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_in, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_out, hipEventDisableTiming);
        if (e != hipSuccess) {
            set_error(std::string("moe_ctx_set_graph: ") + hipGetErrorString(e));
            return STMOE_EHIP;
        }
    }
    c->graph_on = on != 0;
    return STMOE_OK;
}

extern "C" int moe_ctx_graph_buffers(moe_ctx* c, void** x_stage, float** y_stage) {
    clear_error();
    STMOE_CHECK(c && x_stage && y_stage, "null pointer");
    STMOE_CHECK(c->graph_on, "graph replay is off");
    *x_stage = c->x_stage;
    *y_stage = c->y_stage;
    return STMOE_OK;
}

extern "C" int moe_ctx_set_prefetch(moe_ctx* c, int min_score, int max_per_layer) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_CHECK(min_score >= 0 && max_per_layer >= 0, "knobs must be >= 0");
    c->pf_min_score = min_score;
    c->pf_max = max_per_layer;
    ++c->settings;
    return STMOE_OK;
}

extern "C" int moe_ctx_set_online_update(moe_ctx* c, int on) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    c->online = on ? 1 : 0;
    ++c->settings;
    return STMOE_OK;
}

extern "C" int moe_decode_token(moe_ctx* c, int token, const void* xs, float* ys, int mode) {
    clear_error();
    STMOE_CHECK(c && xs && ys, "null pointer");
    STMOE_CHECK(token >= 0, "token must be >= 0");
    STMOE_CHECK(mode >= MOE_MODE_ON_DEMAND && mode <= MOE_MODE_CCT_ONLY, "bad mode");
    // graph replay once the first call has run (it seeds layer 0's
    // prediction); event-timed tokens run eagerly
    if (c->graph_on && c->started && !timed_token(c, token)) return decode_token_graph(c, token, xs, ys, mode);
    // per-token predictor work: this token's selections go to its parity's
    // buffer, which the launch of two tokens ago may still be reading
    const int use = use_bits(mode);
    const bool batch = c->pred_batch && use != 0;
    c->cur_par = batch ? (token & 1) : 0;
    if (int rc = wait_token_side(c, c->cur_par)) return rc;
    for (int l = 0; l < c->L; ++l) {
        const char* x = reinterpret_cast<const char*>(xs) + size_t(l) * c->B * c->H * c->esz;
        if (int rc = decode_layer(c, token, l, x, ys + size_t(l) * c->B * c->H, mode, true, batch)) return rc;
    }
    if (batch)
        if (int rc = token_side(c, token, use)) return rc;
    return STMOE_OK;
}

extern "C" int moe_ctx_last_routing(moe_ctx* c, int32_t* idx, float* w) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_HIP(hipStreamSynchronize(c->s));
    const size_t n = size_t(c->L) * c->B * c->K;
    const size_t off = size_t(c->last_par) * n;
    if (idx) STMOE_HIP(hipMemcpy(idx, c->idx + off, n * sizeof(int32_t), hipMemcpyDeviceToHost));
    if (w) STMOE_HIP(hipMemcpy(w, c->w + off, n * sizeof(float), hipMemcpyDeviceToHost));
    return STMOE_OK;
}

extern "C" int moe_ctx_set_timing(moe_ctx* c, int every) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_CHECK(every >= 0, "every must be >= 0");
    // the side stream may still have to record events of earlier timed layers
    STMOE_HIP(hipDeviceSynchronize());
    c->timing_every = every;
    c->ev_used = 0;
    c->n_calls = 0;
    c->timed_layers.clear();
    STMOE_HIP(hipMemset(c->n_experts, 0, sizeof(unsigned long long)));
    return STMOE_OK;
}

namespace {
// Summed milliseconds between two recorded events of each timed layer.
int sum_pairs(moe_ctx* c, int moe_ctx::TimedLayer::*a, int moe_ctx::TimedLayer::*b, double& out) {
    out = 0.0;
    for (const auto& t : c->timed_layers) {
        if (t.*a < 0 || t.*b < 0) continue;
        float ms = 0.f;
        STMOE_HIP(hipEventElapsedTime(&ms, c->ev_pool[size_t(t.*a)], c->ev_pool[size_t(t.*b)]));
        out += ms;
    }
    return STMOE_OK;
}
}  // namespace

extern "C" int moe_ctx_timing(moe_ctx* c, double* up_ms, double* down_ms, int64_t* n_calls,
                              int64_t* n_experts) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_HIP(hipDeviceSynchronize());
    double a = 0.0, b = 0.0;
    if (int rc = sum_pairs(c, &moe_ctx::TimedLayer::up0, &moe_ctx::TimedLayer::mid, a)) return rc;
    if (int rc = sum_pairs(c, &moe_ctx::TimedLayer::mid, &moe_ctx::TimedLayer::down1, b)) return rc;
    unsigned long long ne = 0;
    STMOE_HIP(hipMemcpy(&ne, c->n_experts, sizeof(ne), hipMemcpyDeviceToHost));
    if (up_ms) *up_ms = a;
    if (down_ms) *down_ms = b;
    if (n_calls) *n_calls = c->n_calls;
    if (n_experts) *n_experts = int64_t(ne);
    return STMOE_OK;
}

extern "C" int moe_ctx_stage_timing(moe_ctx* c, double* route_ms, double* miss_ms, double* ffn_ms,
                                    double* predict_ms, int64_t* n_calls) {
    clear_error();
    STMOE_CHECK(c, "null ctx");
    STMOE_HIP(hipDeviceSynchronize());
    double r = 0.0, m = 0.0, f = 0.0, p = 0.0;
    if (int rc = sum_pairs(c, &moe_ctx::TimedLayer::route0, &moe_ctx::TimedLayer::route1, r)) return rc;
    if (int rc = sum_pairs(c, &moe_ctx::TimedLayer::route1, &moe_ctx::TimedLayer::up0, m)) return rc;
    if (int rc = sum_pairs(c, &moe_ctx::TimedLayer::up0, &moe_ctx::TimedLayer::down1, f)) return rc;
    if (int rc = sum_pairs(c, &moe_ctx::TimedLayer::pred0, &moe_ctx::TimedLayer::pred1, p)) return rc;
    if (route_ms) *route_ms = r;
    if (miss_ms) *miss_ms = m;
    if (ffn_ms) *ffn_ms = f;
    if (predict_ms) *predict_ms = p;
    if (n_calls) *n_calls = c->n_calls;
    return STMOE_OK;
}
