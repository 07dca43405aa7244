// HBM expert cache: the staging buffer that predicted experts are prefetched
// into (Section 4.1; Section 4.3.4, "EP" and "ML" stages of the pipelined
// workflow).  On the GPU the slow link is PCIe from pinned host memory and
// the fast memory is HBM; one hipMemcpyAsync moves one packed expert.
//
// stmoe_policy is the pure decision logic (no HIP calls): per-layer slot
// partitions, least recently used with protection of the current ranked or
// selected set (or, frequency-aware, least used first, then least recently),
// residency counted from copy issue so decisions never depend on timing.  expert_cache wraps it with slots in an HBM arena, a demand and
// a side stream, and two events per slot (last copy into it, last reader of
// it) that order every reuse.
#include <algorithm>
#include <string>
#include <vector>

#include "cache_device.h"
#include "common.h"

struct stmoe_policy {
    int L, E, C;
    std::vector<int> slot;          // [L*C] expert in slot or -1
    std::vector<int64_t> last;      // [L*C] last use stamp
    std::vector<int> where;         // [L*E] slot of expert or -1
    std::vector<char> pending;      // [L*E] prefetched, not yet verified
    std::vector<int64_t> freq;      // [L*E] use counts (frequency-aware eviction)
    int use_freq = 0;               // 1: victims by (uses, last use, slot); 0: (last use, slot)
    stmoe_cache_stats st{};

    int64_t uses(int l, int c) const {
        const int e = slot[l * C + c];
        return e >= 0 ? freq[size_t(l) * E + e] : -1;
    }
    int victim(int l, const std::vector<char>& keep) const {
        int best = -1;
        for (int c = 0; c < C; ++c) {
            const int e = slot[l * C + c];
            if (e >= 0 && keep[e]) continue;
            if (best < 0) {
                best = c;
                continue;
            }
            if (use_freq) {
                const int64_t u = uses(l, c), ub = uses(l, best);
                if (u != ub) {
                    if (u < ub) best = c;
                    continue;
                }
            }
            if (last[l * C + c] < last[l * C + best]) best = c;
        }
        return best;
    }
    void place(int l, int c, int e) {
        const int old = slot[l * C + c];
        if (old >= 0) where[l * E + old] = -1;
        slot[l * C + c] = e;
        where[l * E + e] = c;
    }
};

namespace stmoe {
namespace {

int check_list(const int32_t* v, int n, int E, bool distinct) {
    STMOE_CHECK(n >= 0 && n <= E, "list length must be in [0, E]");
    STMOE_CHECK(n == 0 || v, "null list");
    std::vector<char> seen(E, 0);
    for (int i = 0; i < n; ++i) {
        STMOE_CHECK(v[i] >= 0 && v[i] < E, "expert index out of range");
        if (distinct) STMOE_CHECK(!seen[v[i]], "repeated expert in list");
        seen[v[i]] = 1;
    }
    return STMOE_OK;
}

int policy_prefetch(stmoe_policy* p, int l, const int32_t* ranked, int n, int64_t stamp,
                    int32_t* pairs) {
    const int m = std::min(n, p->C);
    std::vector<char> keep(p->E, 0);
    for (int i = 0; i < m; ++i) keep[ranked[i]] = 1;
    int copies = 0;
    for (int i = 0; i < m; ++i) {
        const int f = ranked[i];
        if (p->where[l * p->E + f] >= 0) continue;
        const int c = p->victim(l, keep);
        if (c < 0) break;
        p->place(l, c, f);
        p->last[l * p->C + c] = stamp;
        p->pending[l * p->E + f] = 1;
        if (pairs) {
            pairs[2 * copies] = f;
            pairs[2 * copies + 1] = c;
        }
        ++copies;
    }
    p->st.prefetch += copies;
    return copies;
}

int policy_acquire(stmoe_policy* p, int l, const int32_t* needed, int n, int64_t stamp,
                   int32_t* pairs, int32_t* n_hits) {
    std::vector<int> U(needed, needed + n);
    std::sort(U.begin(), U.end());
    std::vector<char> keep(p->E, 0);
    for (int f : U) keep[f] = 1;
    int out = 0, hits = 0;
    std::vector<int> used;
    for (int f : U) {
        int c = p->where[l * p->E + f];
        if (c >= 0) {
            ++hits;
            used.push_back(c);
            continue;
        }
        c = p->victim(l, keep);
        if (c < 0) {
            if (pairs) { pairs[2 * out] = f; pairs[2 * out + 1] = -1; }
            ++out;
            ++p->st.overflow;
            continue;
        }
        p->place(l, c, f);
        used.push_back(c);
        if (pairs) { pairs[2 * out] = f; pairs[2 * out + 1] = c; }
        ++out;
        ++p->st.demand;
    }
    for (int c : used) p->last[l * p->C + c] = stamp;
    if (p->use_freq)
        for (int f : U) ++p->freq[size_t(l) * p->E + f];
    for (int e = 0; e < p->E; ++e) {
        if (!p->pending[l * p->E + e]) continue;
        if (keep[e]) ++p->st.useful; else ++p->st.wasted;
        p->pending[l * p->E + e] = 0;
    }
    p->st.hits += hits;
    if (n_hits) *n_hits = hits;
    return out;
}

}  // namespace
}  // namespace stmoe

using namespace stmoe;

extern "C" int stmoe_policy_create(int L, int E, int C, const int32_t* warm, stmoe_policy** out) {
    clear_error();
    STMOE_CHECK(out, "null output");
    STMOE_CHECK(L >= 1 && E >= 1 && E <= kMaxE && C >= 1 && C <= kMaxE, "bad L/E/C");
    auto* p = new stmoe_policy();
    p->L = L; p->E = E; p->C = C;
    p->slot.assign(size_t(L) * C, -1);
    p->last.assign(size_t(L) * C, 0);
    p->where.assign(size_t(L) * E, -1);
    p->pending.assign(size_t(L) * E, 0);
    p->freq.assign(size_t(L) * E, 0);
    if (warm) {
        for (int l = 0; l < L; ++l)
            for (int c = 0; c < C; ++c) {
                const int e = warm[l * C + c];
                if (e < 0) continue;
                if (e >= E || p->where[l * E + e] >= 0) {
                    delete p;
                    set_error("stmoe_policy_create: warm set has an invalid or repeated expert");
                    return STMOE_EINVAL;
                }
                p->place(l, c, e);
            }
    }
    *out = p;
    return STMOE_OK;
}

extern "C" int expert_cache_warm_sets(const int32_t* sel, int P, int B, int L, int K, int E, int C,
                                     int32_t* out) {
    clear_error();
    STMOE_CHECK(sel && out, "null pointer");
    STMOE_CHECK(P >= 1 && B >= 1 && L >= 1 && K >= 1 && E >= 1 && E <= kMaxE && C >= 1, "bad shape");
    std::vector<int64_t> cnt(E);
    std::vector<int> order(E);
    for (int l = 0; l < L; ++l) {
        std::fill(cnt.begin(), cnt.end(), 0);
        for (int p = 0; p < P; ++p)
            for (int b = 0; b < B; ++b)
                for (int k = 0; k < K; ++k) {
                    const int e = sel[((size_t(p) * B + b) * L + l) * K + k];
                    STMOE_CHECK(e >= 0 && e < E, "selection index out of range");
                    ++cnt[e];
                }
        for (int e = 0; e < E; ++e) order[e] = e;
        std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return cnt[x] > cnt[y]; });
        for (int c = 0; c < C; ++c) out[size_t(l) * C + c] = c < E ? order[c] : -1;
    }
    return STMOE_OK;
}

namespace stmoe {
namespace {
int policy_set_counts(stmoe_policy* p, const int64_t* counts) {
    if (counts)
        for (size_t i = 0; i < size_t(p->L) * p->E; ++i)
            STMOE_CHECK(counts[i] >= 0, "use counts must be >= 0");
    p->use_freq = counts != nullptr;
    if (counts) std::copy(counts, counts + size_t(p->L) * p->E, p->freq.begin());
    else std::fill(p->freq.begin(), p->freq.end(), 0);
    return STMOE_OK;
}
}  // namespace
}  // namespace stmoe

extern "C" int stmoe_policy_set_counts(stmoe_policy* p, const int64_t* counts) {
    clear_error();
    STMOE_CHECK(p, "null policy");
    return policy_set_counts(p, counts);
}

extern "C" int expert_cache_use_counts(const int32_t* sel, int P, int B, int L, int K, int E, int64_t* out) {
    clear_error();
    STMOE_CHECK(sel && out, "null pointer");
    STMOE_CHECK(P >= 1 && B >= 1 && L >= 1 && K >= 1 && E >= 1 && E <= kMaxE, "bad shape");
    std::fill(out, out + size_t(L) * E, int64_t(0));
    std::vector<int> seen(E, -1);
    for (int l = 0; l < L; ++l)
        for (int p = 0; p < P; ++p)
            for (int b = 0; b < B; ++b)
                for (int k = 0; k < K; ++k) {
                    const int e = sel[((size_t(p) * B + b) * L + l) * K + k];
                    STMOE_CHECK(e >= 0 && e < E, "selection index out of range");
                    const int key = l * P + p;              // once per (layer, token)
                    if (seen[e] == key) continue;
                    seen[e] = key;
                    ++out[size_t(l) * E + e];
                }
    return STMOE_OK;
}

extern "C" int stmoe_policy_destroy(stmoe_policy* p) {
    delete p;
    return STMOE_OK;
}

extern "C" int stmoe_policy_prefetch(stmoe_policy* p, int layer, const int32_t* ranked, int n,
                                     int64_t stamp, int32_t* pairs) {
    clear_error();
    STMOE_CHECK(p, "null policy");
    STMOE_CHECK(layer >= 0 && layer < p->L, "layer out of range");
    if (int rc = check_list(ranked, n, p->E, true)) return rc;
    return policy_prefetch(p, layer, ranked, n, stamp, pairs);
}

extern "C" int stmoe_policy_acquire(stmoe_policy* p, int layer, const int32_t* needed, int n,
                                    int64_t stamp, int32_t* pairs, int32_t* n_hits) {
    clear_error();
    STMOE_CHECK(p, "null policy");
    STMOE_CHECK(layer >= 0 && layer < p->L, "layer out of range");
    if (int rc = check_list(needed, n, p->E, true)) return rc;
    return policy_acquire(p, layer, needed, n, stamp, pairs, n_hits);
}

extern "C" int stmoe_policy_slots(const stmoe_policy* p, int32_t* slot_expert) {
    clear_error();
    STMOE_CHECK(p && slot_expert, "null pointer");
    std::copy(p->slot.begin(), p->slot.end(), slot_expert);
    return STMOE_OK;
}

extern "C" int stmoe_policy_stats(const stmoe_policy* p, stmoe_cache_stats* out) {
    clear_error();
    STMOE_CHECK(p && out, "null pointer");
    *out = p->st;
    return STMOE_OK;
}

// ---------------------------------------------------------------------------
// device-backed cache
// ---------------------------------------------------------------------------

// The arena holds L*C + n_stage blocks of one blob each.  Slot s of layer l
// lives in block blk[l*C + s] (block l*C + s until staged prefetches swap
// blocks).  The last 2*ns staging blocks hold staged prefetches (two sets
// that alternate between consecutive layers); the others form the ring that
// overflow experts stream through.  Events are per block.
struct expert_cache {
    stmoe_policy* pol = nullptr;
    int L = 0, E = 0, C = 0, n_stage = 0;
    size_t blob = 0;
    char* arena = nullptr;
    std::vector<const void*> host;       // [L*E]
    hipStream_t demand = nullptr, side = nullptr;
    std::vector<hipEvent_t> loaded, released;   // [L*C + n_stage] per block
    std::vector<char> loaded_set, released_set;
    std::vector<int> blk;                // [L*C] block of each slot
    int stage_next = 0;
    std::vector<std::vector<int>> held;  // per layer: blocks read by the last acquire
    hipEvent_t demand_done = nullptr;    // after the last acquire's demand copies
    bool demand_done_set = false;
    int after_demand = 0;                // prefetch copies wait for demand_done
    stmoe::DeviceCache* dev = nullptr;   // device-side decisions (null: the host decides)
    // staged prefetch with host decisions: ns positions per set, the first
    // `head` bytes of a staged expert copied when it is staged, the rest once
    // the next layer selects it
    int ns = 0;
    size_t head = 0;
    std::vector<int> sblk, sexp;         // [2][ns] block and staged expert of each position
    int cur = 0, stg_layer[2] = {-1, -1}, stg_n[2] = {0, 0};
    bool permuted = false;               // some slot lives outside its home block
    uint64_t version = 0;                // bumped by every change of the cache's settings
    int copy_wgs[2] = {0, 0};            // device decisions: copy kernel workgroups (0: defaults)

    char* block_ptr(int b) const { return arena + size_t(b) * blob; }
    int ring() const { return n_stage - 2 * ns; }
};

namespace stmoe {
// Internal: the shape a cache was created with (checked by moe_ctx_create).
void expert_cache_shape(const expert_cache* c, int* L, int* E, size_t* blob_bytes) {
    *L = c->L;
    *E = c->E;
    *blob_bytes = c->blob;
}
// Internal: the device decisions when switched on, and the prefetch order.
DeviceCache* expert_cache_device(expert_cache* c) { return c->dev; }
// Internal: changes whenever a setting that a captured decode graph bakes in
// may have changed (residency, decision site, staged count, link order).
uint64_t expert_cache_version(const expert_cache* c) { return c->version; }
int expert_cache_after_demand(const expert_cache* c) {
    // staged prefetches only take the link once the missed loads are in
    return c->after_demand || (c->dev && device_cache_staged(c->dev) > 0);
}

namespace {
PolicyState policy_state(expert_cache* c) {
    stmoe_policy* p = c->pol;
    return PolicyState{p->L, p->E, p->C, p->slot.data(), p->last.data(), p->where.data(), p->pending.data(),
                       p->freq.data(), &p->use_freq, &p->st};
}
}  // namespace
}  // namespace stmoe


namespace stmoe {
namespace {

// Order a copy of bytes [off, off + n) of a blob into block `b` on stream
// `s` after the block's previous copy and its last reader, then issue it and
// record the block's loaded event.
int copy_into(expert_cache* c, int b, const void* src, hipStream_t s, size_t off = 0, size_t n = 0) {
    if (n == 0) n = c->blob - off;
    if (c->loaded_set[b]) STMOE_HIP(hipStreamWaitEvent(s, c->loaded[b], 0));
    if (c->released_set[b]) STMOE_HIP(hipStreamWaitEvent(s, c->released[b], 0));
    STMOE_HIP(hipMemcpyAsync(c->block_ptr(b) + off, static_cast<const char*>(src) + off, n, hipMemcpyDefault, s));
    STMOE_HIP(hipEventRecord(c->loaded[b], s));
    c->loaded_set[b] = 1;
    return STMOE_OK;
}

void reset_blocks(expert_cache* c) {
    for (size_t i = 0; i < c->blk.size(); ++i) c->blk[i] = int(i);
    c->sblk.assign(size_t(2) * c->ns, 0);
    c->sexp.assign(size_t(2) * c->ns, -1);
    for (int p = 0; p < 2; ++p)
        for (int j = 0; j < c->ns; ++j) c->sblk[size_t(p) * c->ns + j] = c->L * c->C + c->ring() + p * c->ns + j;
    c->cur = 0;
    c->stg_layer[0] = c->stg_layer[1] = -1;
    c->stg_n[0] = c->stg_n[1] = 0;
    c->stage_next = 0;
    c->permuted = false;
}

}  // namespace
}  // namespace stmoe

namespace {
size_t slots_bytes(int L, int C, size_t blob_bytes, int n_stage) {
    return ((size_t(L) * C + n_stage) * blob_bytes + 255) / 256 * 256;
}
}  // namespace

extern "C" size_t expert_cache_arena_bytes(int L, int E, int C, size_t blob_bytes, int n_stage) {
    if (L < 1 || E < 1 || E > kMaxE || C < 1 || C > E || n_stage < 0) return 0;
    return slots_bytes(L, C, blob_bytes, n_stage) + stmoe::device_cache_state_bytes(L, E, C);
}

extern "C" int expert_cache_create(int L, int E, int C, size_t blob_bytes, int n_stage, void* arena,
                                   size_t arena_bytes, const void* const* host_blobs,
                                   void* demand_stream, void* side_stream, expert_cache** out) {
    clear_error();
    STMOE_CHECK(out && arena && host_blobs, "null pointer");
    STMOE_CHECK(L >= 1 && E >= 1 && E <= kMaxE && C >= 1 && C <= E, "bad L/E/C");
    STMOE_CHECK(n_stage >= 0 && n_stage <= kMaxE, "n_stage must be in [0, 256]");
    STMOE_CHECK(blob_bytes > 0 && blob_bytes % 16 == 0, "blob_bytes must be a positive multiple of 16");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(arena) & 255) == 0, "arena must be 256-byte aligned");
    if (arena_bytes < expert_cache_arena_bytes(L, E, C, blob_bytes, n_stage)) {
        set_error("expert_cache_create: arena smaller than expert_cache_arena_bytes()");
        return STMOE_ECAPACITY;
    }
    for (size_t i = 0; i < size_t(L) * E; ++i) STMOE_CHECK(host_blobs[i], "null host blob pointer");
    auto* c = new expert_cache();
    if (int rc = stmoe_policy_create(L, E, C, nullptr, &c->pol)) {
        delete c;
        return rc;
    }
    c->L = L; c->E = E; c->C = C; c->n_stage = n_stage;
    c->blob = blob_bytes;
    c->arena = reinterpret_cast<char*>(arena);
    c->host.assign(host_blobs, host_blobs + size_t(L) * E);
    c->demand = as_stream(demand_stream);
    c->side = as_stream(side_stream);
    const size_t n = size_t(L) * C + n_stage;
    c->loaded.assign(n, nullptr);
    c->released.assign(n, nullptr);
    c->loaded_set.assign(n, 0);
    c->released_set.assign(n, 0);
    c->held.assign(L, {});
    c->blk.assign(size_t(L) * C, 0);
    reset_blocks(c);
    for (size_t i = 0; i < n; ++i) {
        if (hipEventCreateWithFlags(&c->loaded[i], hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&c->released[i], hipEventDisableTiming) != hipSuccess) {
            expert_cache_destroy(c);
            set_error("expert_cache_create: hipEventCreateWithFlags failed");
            return STMOE_EHIP;
        }
    }
    if (hipEventCreateWithFlags(&c->demand_done, hipEventDisableTiming) != hipSuccess) {
        expert_cache_destroy(c);
        set_error("expert_cache_create: hipEventCreateWithFlags failed");
        return STMOE_EHIP;
    }
    *out = c;
    return STMOE_OK;
}

extern "C" int expert_cache_destroy(expert_cache* c) {
    if (!c) return STMOE_OK;
    if (c->demand) (void)hipStreamSynchronize(c->demand);
    if (c->side) (void)hipStreamSynchronize(c->side);
    if (c->dev) stmoe::device_cache_destroy(c->dev);
    for (auto e : c->loaded)
        if (e) (void)hipEventDestroy(e);
    for (auto e : c->released)
        if (e) (void)hipEventDestroy(e);
    if (c->demand_done) (void)hipEventDestroy(c->demand_done);
    stmoe_policy_destroy(c->pol);
    delete c;
    return STMOE_OK;
}

extern "C" int expert_cache_warm(expert_cache* c, const int32_t* warm) {
    clear_error();
    STMOE_CHECK(c && warm, "null pointer");
    ++c->version;
    if (c->dev) {
        set_error("expert_cache_warm: device decisions are on");
        return STMOE_ESTATE;
    }
    stmoe_policy* np = nullptr;
    if (int rc = stmoe_policy_create(c->L, c->E, c->C, warm, &np)) return rc;
    STMOE_HIP(hipStreamSynchronize(c->demand));
    STMOE_HIP(hipStreamSynchronize(c->side));
    np->use_freq = c->pol->use_freq;       // the replacement rule and its counts stay
    np->freq = c->pol->freq;
    stmoe_policy_destroy(c->pol);
    c->pol = np;
    reset_blocks(c);
    for (int l = 0; l < c->L; ++l)
        for (int s = 0; s < c->C; ++s) {
            const int e = warm[l * c->C + s];
            if (e < 0) continue;
            STMOE_HIP(hipMemcpyAsync(c->block_ptr(c->blk[l * c->C + s]), c->host[size_t(l) * c->E + e], c->blob,
                                     hipMemcpyDefault, c->demand));
        }
    STMOE_HIP(hipStreamSynchronize(c->demand));
    std::fill(c->loaded_set.begin(), c->loaded_set.end(), 0);
    std::fill(c->released_set.begin(), c->released_set.end(), 0);
    for (auto& h : c->held) h.clear();
    return STMOE_OK;
}

extern "C" int expert_cache_prefetch(expert_cache* c, int layer, const int32_t* ranked, int n,
                                     int64_t stamp) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    if (c->dev) {
        set_error("expert_cache_prefetch: device decisions are on");
        return STMOE_ESTATE;
    }
    STMOE_CHECK(layer >= 0 && layer < c->L, "layer out of range");
    if (int rc = check_list(ranked, n, c->E, true)) return rc;
    if (c->ns > 0) {
        // staged: the first ns ranked experts not resident, into the other set
        // of staging blocks; no slot changes hands.  They take the link only
        // once the latest missed loads are in.
        const int nx = c->cur ^ 1;
        int k = 0;
        for (int i = 0; i < n && k < c->ns; ++i) {
            const int f = ranked[i];
            if (c->pol->where[layer * c->E + f] >= 0) continue;
            if (k == 0 && c->demand_done_set) STMOE_HIP(hipStreamWaitEvent(c->side, c->demand_done, 0));
            const int b = c->sblk[size_t(nx) * c->ns + k];
            c->sexp[size_t(nx) * c->ns + k] = f;
            const size_t first = c->head > 0 && c->head < c->blob ? c->head : c->blob;
            if (int rc = copy_into(c, b, c->host[size_t(layer) * c->E + f], c->side, 0, first)) return rc;
            ++k;
        }
        c->stg_layer[nx] = layer;
        c->stg_n[nx] = k;
        c->cur = nx;
        c->pol->st.prefetch += k;
        (void)stamp;
        return k;
    }
    int32_t pairs[2 * kMaxE];
    const int m = policy_prefetch(c->pol, layer, ranked, n, stamp, pairs);
    if (m > 0 && c->after_demand && c->demand_done_set)
        STMOE_HIP(hipStreamWaitEvent(c->side, c->demand_done, 0));
    for (int i = 0; i < m; ++i) {
        const int e = pairs[2 * i], s = pairs[2 * i + 1];
        if (int rc = copy_into(c, c->blk[layer * c->C + s], c->host[size_t(layer) * c->E + e], c->side)) return rc;
    }
    return m;
}

extern "C" int expert_cache_acquire(expert_cache* c, int layer, const int32_t* needed, int n,
                                    int64_t stamp, const void** dev_table_out, void* compute) {
    clear_error();
    STMOE_CHECK(c && dev_table_out, "null pointer");
    STMOE_CHECK(layer >= 0 && layer < c->L, "layer out of range");
    if (c->dev) {
        set_error("expert_cache_acquire: device decisions are on");
        return STMOE_ESTATE;
    }
    if (int rc = check_list(needed, n, c->E, true)) return rc;
    hipStream_t cs = as_stream(compute);
    int32_t pairs[2 * kMaxE];
    int32_t n_hits = 0;
    // overflow must fit the staging ring: count before committing
    {
        int missing = 0;
        for (int i = 0; i < n; ++i) missing += c->pol->where[layer * c->E + needed[i]] < 0;
        int evictable = 0;
        std::vector<char> keep(c->E, 0);
        for (int i = 0; i < n; ++i) keep[needed[i]] = 1;
        for (int s = 0; s < c->C; ++s) {
            const int e = c->pol->slot[layer * c->C + s];
            evictable += (e < 0 || !keep[e]);
        }
        const int overflow = missing > evictable ? missing - evictable : 0;
        if (overflow > c->ring()) {
            set_error("expert_cache_acquire: more overflow experts than staging slots");
            return STMOE_ECAPACITY;
        }
    }
    // the staged set issued for this layer (if the last one targets it)
    std::vector<int> spos(c->E, -1);
    const int cur = c->cur;
    const int n_cons = c->ns > 0 && c->stg_layer[cur] == layer ? c->stg_n[cur] : 0;
    for (int j = 0; j < n_cons; ++j) spos[c->sexp[size_t(cur) * c->ns + j]] = j;
    const int m = policy_acquire(c->pol, layer, needed, n, stamp, pairs, &n_hits);
    auto& held = c->held[layer];
    held.clear();
    // demand copies, overflow staging and used staged copies
    std::vector<int> blk_of(c->E, -1);
    for (int i = 0; i < m; ++i) {
        const int e = pairs[2 * i], s = pairs[2 * i + 1];
        const int j = spos[e];
        if (j >= 0) {
            // a staged copy serves this miss: its remaining bytes follow on the
            // side stream; with a slot, the staging block becomes the slot's
            int& pos = c->sblk[size_t(cur) * c->ns + j];
            const int b = pos;
            if (c->head > 0 && c->head < c->blob)
                if (int rc = copy_into(c, b, c->host[size_t(layer) * c->E + e], c->side, c->head)) return rc;
            if (s >= 0) {
                pos = c->blk[layer * c->C + s];
                c->blk[layer * c->C + s] = b;
                c->permuted = true;
                --c->pol->st.demand;
            } else {
                --c->pol->st.overflow;
            }
            ++c->pol->st.useful;
            blk_of[e] = b;
            continue;
        }
        int b;
        if (s >= 0) {
            b = c->blk[layer * c->C + s];
        } else {
            b = c->L * c->C + c->stage_next;
            c->stage_next = (c->stage_next + 1) % c->ring();
        }
        if (int rc = copy_into(c, b, c->host[size_t(layer) * c->E + e], c->demand)) return rc;
        blk_of[e] = b;
    }
    if (n_cons > 0) {
        std::vector<char> keep(c->E, 0);
        for (int i = 0; i < n; ++i) keep[needed[i]] = 1;
        for (int j = 0; j < n_cons; ++j) c->pol->st.wasted += !keep[c->sexp[size_t(cur) * c->ns + j]];
        c->stg_layer[cur] = -1;
    }
    if (m > 0) {
        STMOE_HIP(hipEventRecord(c->demand_done, c->demand));
        c->demand_done_set = true;
    }
    // every needed expert: the compute stream waits for its block's last copy
    for (int i = 0; i < n; ++i) {
        const int e = needed[i];
        const int s = c->pol->where[layer * c->E + e];
        const int b = blk_of[e] >= 0 ? blk_of[e] : (s >= 0 ? c->blk[layer * c->C + s] : -1);
        if (b < 0) {
            set_error("expert_cache_acquire: internal error, expert without a block");
            return STMOE_ESTATE;
        }
        dev_table_out[e] = c->block_ptr(b);
        if (c->loaded_set[b]) STMOE_HIP(hipStreamWaitEvent(cs, c->loaded[b], 0));
        held.push_back(b);
    }
    return n_hits;
}

extern "C" int expert_cache_set_device_policy(expert_cache* c, int on) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    STMOE_CHECK(on == 0 || on == 1, "on must be 0 or 1");
    ++c->version;
    if (bool(on) == (c->dev != nullptr)) return STMOE_OK;
    STMOE_HIP(hipStreamSynchronize(c->demand));
    STMOE_HIP(hipStreamSynchronize(c->side));
    if (on) {
        if (c->permuted || c->ns > 0) {
            set_error("expert_cache_set_device_policy: staged prefetches with host decisions are on, or have "
                      "moved slots to other arena blocks; device decisions cannot take the cache over");
            return STMOE_ESTATE;
        }
        for (auto& h : c->held) h.clear();
        const int rc = stmoe::device_cache_create(stmoe::policy_state(c), c->arena, c->blob, c->n_stage,
                                                  c->host.data(), c->arena + slots_bytes(c->L, c->C, c->blob,
                                                                                         c->n_stage),
                                                  c->side, &c->dev);
        if (rc == STMOE_OK) stmoe::device_cache_set_copy_workgroups(c->dev, c->copy_wgs[0], c->copy_wgs[1]);
        return rc;
    }
    const int rc = stmoe::device_cache_download(c->dev, stmoe::policy_state(c));
    if (rc != STMOE_OK) return rc;       // the device keeps deciding
    stmoe::device_cache_destroy(c->dev);
    c->dev = nullptr;
    // every slot was last written and read on the device streams, now idle
    std::fill(c->loaded_set.begin(), c->loaded_set.end(), 0);
    std::fill(c->released_set.begin(), c->released_set.end(), 0);
    return rc;
}

extern "C" int expert_cache_set_staged_prefetch(expert_cache* c, int n_per_layer, size_t head_bytes) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    ++c->version;
    STMOE_CHECK(n_per_layer >= 0 && n_per_layer <= kMaxE, "n_per_layer must be in [0, 256]");
    if (c->dev) {
        STMOE_CHECK(2 * n_per_layer <= c->n_stage, "n_per_layer must be in [0, n_stage / 2]");
        return stmoe::device_cache_set_staged(c->dev, n_per_layer);
    }
    // host decisions: the overflow ring keeps what the staged sets leave
    STMOE_CHECK(2 * n_per_layer <= c->n_stage, "n_per_layer must be in [0, n_stage / 2]");
    if (c->permuted && n_per_layer != c->ns) {
        set_error("expert_cache_set_staged_prefetch: staged prefetches have moved slots to other arena blocks; "
                  "reload the cache with expert_cache_warm before changing the staged count");
        return STMOE_ESTATE;
    }
    STMOE_HIP(hipStreamSynchronize(c->demand));
    STMOE_HIP(hipStreamSynchronize(c->side));
    if (n_per_layer != c->ns) {
        c->ns = n_per_layer;
        reset_blocks(c);       // nothing is permuted: slots stay in their home blocks
    }
    c->head = head_bytes;
    return STMOE_OK;
}

extern "C" int expert_cache_set_counts(expert_cache* c, const int64_t* counts) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    ++c->version;
    if (counts)
        for (size_t i = 0; i < size_t(c->L) * c->E; ++i) STMOE_CHECK(counts[i] >= 0, "use counts must be >= 0");
    if (c->dev) return stmoe::device_cache_set_counts(c->dev, counts);
    return policy_set_counts(c->pol, counts);
}

extern "C" int expert_cache_set_copy_workgroups(expert_cache* c, int demand, int prefetch) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    STMOE_CHECK(demand >= 0 && demand <= 1024 && prefetch >= 0 && prefetch <= 1024,
                "workgroup counts must be in [0, 1024]");
    ++c->version;
    c->copy_wgs[0] = demand;
    c->copy_wgs[1] = prefetch;
    if (c->dev) stmoe::device_cache_set_copy_workgroups(c->dev, demand, prefetch);
    return STMOE_OK;
}

extern "C" int expert_cache_set_prefetch_order(expert_cache* c, int after_demand) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    STMOE_CHECK(after_demand == 0 || after_demand == 1, "after_demand must be 0 or 1");
    ++c->version;
    c->after_demand = after_demand;
    return STMOE_OK;
}

extern "C" int expert_cache_release(expert_cache* c, int layer, void* compute) {
    clear_error();
    STMOE_CHECK(c, "null cache");
    STMOE_CHECK(layer >= 0 && layer < c->L, "layer out of range");
    for (int gid : c->held[layer]) {
        STMOE_HIP(hipEventRecord(c->released[gid], as_stream(compute)));
        c->released_set[gid] = 1;
    }
    c->held[layer].clear();
    return STMOE_OK;
}

extern "C" int expert_cache_stats(const expert_cache* c, stmoe_cache_stats* out) {
    clear_error();
    STMOE_CHECK(c && out, "null pointer");
    if (c->dev) return stmoe::device_cache_stats(c->dev, out);
    *out = c->pol->st;
    return STMOE_OK;
}
