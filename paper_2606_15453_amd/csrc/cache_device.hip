// Device-side cache decisions (see cache_device.h).  The policy is the host
// policy's (expert_cache.cpp): per-layer slot partitions; a missed expert
// takes the evictable slot (empty, or holding an expert outside the current
// selection) with the smallest (last use, slot), or, frequency-aware, the
// smallest (use count, last use, slot) with an empty slot counting -1; a
// prefetch walks the admitted ranking and takes victims the same way among
// slots outside the ranked set, stopping when none is left; residency counts
// from copy issue.  Evictions within one call never change the other
// candidates' keys, so the k-th missed (or non-resident ranked) expert takes
// the k-th victim in key order: the kernel ranks slots and experts in
// parallel instead of searching once per copy.
//
// Staged prefetch (an alternative to prefetching into evicted slots): the
// predicted experts of the next layer are copied into spare staging blocks,
// evicting nothing, after the layer's missed loads.  At the next layer's
// decisions a staged expert that was selected is served from its block: if
// it takes a slot, the slot's block and the staging block swap places (no
// copy); staged experts that were not selected are cancelled, and their copy
// kernel stops at its next check.  Residency therefore evolves exactly as
// with on-demand loading; the staged copies only move bytes earlier, while
// the link would otherwise idle during the layer's computation.
#include <algorithm>
#include <vector>

#include "cache_device.h"

namespace stmoe {
namespace {

constexpr int kT = 256;          // threads of the decision kernel (E, C <= 256)
constexpr int kBlitWgs = 64;     // copy kernel workgroups (enough to fill the host link)
// Prefetch copies run beside the FFN, and a copy kernel reading pinned host
// memory slows a concurrent FFN several-fold; fewer workgroups leave it most
// of the chip (staged prefetch on Mixtral shapes: 10.4 tokens/s with 64,
// 13.7 with 16, 12.0 with 4; missed loads, which the FFN waits for, keep 64).
constexpr int kPrefetchWgs = 16;

struct Copy {
    const char* src;             // device-accessible host blob
    char* dst;                   // HBM block
    const int32_t* cancel;       // null, or a flag that stops the copy once set
};

constexpr int kStageMax = kMaxE;  // staging positions per parity

struct DecideArgs {
    int L, E, C, layer, next, BK, pf_min, pf_max;
    int demand_on;               // 0: only the prefetch decisions (no selection yet)
    const int64_t* tok;          // device: the decode token (stamps are tok * L + stamp_add)
    int64_t stamp_add;
    int64_t stamp;               // set in the kernel
    int32_t* slot;
    int64_t* last;
    int32_t* where;
    int32_t* pending;
    long long* stats;            // hits, demand, overflow, prefetch, useful, wasted
    const int32_t* idx;
    const int32_t* ranked;       // null: no prefetch
    const int32_t* n_ranked;
    const uint8_t* max_score;
    const char* const* host;     // [L*E]
    char* arena;
    size_t blob;
    const void** table;          // [E] for `layer`
    Copy* demand;                // [kMaxE]
    int32_t* n_demand;
    Copy* pf;                    // [kMaxE] for `next`
    int32_t* n_pf;               // for `next`
    int32_t* blk;                // [L*C] arena block of each slot
    // staged prefetch (ns > 0): two parities of ns positions; ctl = {parity
    // issued last, target layer of parity 0 and 1, count of parity 0 and 1}
    int ns;
    int32_t* sblk;               // [2][kStageMax] arena block of each position
    int32_t* sexp;               // [2][kStageMax] staged expert
    int32_t* cancel;             // [2][kStageMax]
    int32_t* ctl;                // [5]
    int64_t* freq;               // [L*E] use counts
    const int32_t* use_freq;     // 1: frequency-aware eviction (read on the device, so a
                                 // captured graph follows later changes)
};

// Exclusive rank of a flag among the workgroup's threads (thread order) and
// the number of set flags.  Whole workgroup calls it; ends with a barrier.
__device__ int flag_rank(bool f, int* wsum, int& total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const unsigned long long m = __ballot(f);
    const int below = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    int off = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kT / 64; ++w) {
        if (w < wave) off += wsum[w];
        total += wsum[w];
    }
    __syncthreads();
    return off + below;
}

// Victims of layer l given the protected set `keep`: vic[r] = the slot of
// rank r among evictable slots by (last use, slot), or (uses, last use,
// slot) when frequency-aware; returns their number.  occ[c] receives each
// slot's occupant.  Ends with a barrier.
__device__ int rank_victims(const DecideArgs& a, int l, const unsigned char* keep, int* occ,
                            int64_t* lastl, int64_t* usel, unsigned char* evl, int* vic, int* wsum) {
    const int t = threadIdx.x;
    const bool by_uses = *a.use_freq != 0;
    if (t < a.C) {
        const int e = a.slot[l * a.C + t];
        occ[t] = e;
        lastl[t] = a.last[l * a.C + t];
        usel[t] = !by_uses ? 0 : e >= 0 ? a.freq[size_t(l) * a.E + e] : -1;
        evl[t] = e < 0 || !keep[e];
    }
    __syncthreads();
    if (t < a.C && evl[t]) {
        const int64_t lt = lastl[t], ut = usel[t];
        int r = 0;
        for (int c = 0; c < a.C; ++c)
            r += evl[c] && (usel[c] < ut || (usel[c] == ut && (lastl[c] < lt || (lastl[c] == lt && c < t))));
        vic[r] = t;
    }
    int n;
    (void)flag_rank(t < a.C && evl[t], wsum, n);
    return n;
}

// Slot c of layer l takes expert f: the old occupant (if any) leaves.
__device__ void place(const DecideArgs& a, int l, int c, int f, int old) {
    if (old >= 0) a.where[l * a.E + old] = -1;
    a.slot[l * a.C + c] = f;
    a.where[l * a.E + f] = c;
}

__device__ char* block_ptr(const DecideArgs& a, int b) { return a.arena + size_t(b) * a.blob; }

__device__ char* slot_ptr(const DecideArgs& a, int l, int c) { return block_ptr(a, a.blk[l * a.C + c]); }

__global__ __launch_bounds__(kT) void decide_kernel(DecideArgs a) {
    __shared__ unsigned char keep[kMaxE];
    __shared__ unsigned char evl[kMaxE];
    __shared__ int occ[kMaxE];
    __shared__ int vic[kMaxE];
    __shared__ int64_t lastl[kMaxE];
    __shared__ int64_t usel[kMaxE];
    __shared__ int wsum[kT / 64];
    __shared__ int cnt[3];               // used prefetches, wasted prefetches, staged overflow
    __shared__ int n_adm;
    __shared__ int spos[kMaxE];          // staging position of a staged expert of this layer, or -1
    const int t = threadIdx.x;
    const int l = a.layer;
    const bool staged = a.ns > 0;
    a.stamp = *a.tok * a.L + a.stamp_add;
    // the staged list consumed here is the last one issued, if it targets this layer
    const int cur = staged ? a.ctl[0] : 0;
    const int n_cons = staged && a.demand_on && a.ctl[1 + cur] == l ? a.ctl[3 + cur] : 0;

    // ---- missed experts of layer l (the selection U = distinct idx)
    if (a.demand_on) {
        if (t < a.E) {
            keep[t] = 0;
            spos[t] = -1;
        }
        if (t < 3) cnt[t] = 0;
        __syncthreads();
        for (int i = t; i < a.BK; i += kT) {
            const int e = a.idx[i];
            if (e >= 0 && e < a.E) keep[e] = 1;
        }
        for (int j = t; j < n_cons; j += kT) spos[a.sexp[cur * kStageMax + j]] = j;
        __syncthreads();
        const bool inU = t < a.E && keep[t];
        const int wh = t < a.E ? a.where[l * a.E + t] : -1;
        const bool hit = inU && wh >= 0, miss = inU && wh < 0;
        const int sj = t < a.E ? spos[t] : -1;           // staged for this layer
        const int nV = rank_victims(a, l, keep, occ, lastl, usel, evl, vic, wsum);
        int n_hit, n_miss, n_dem;
        (void)flag_rank(hit, wsum, n_hit);
        const int mr = flag_rank(miss, wsum, n_miss);      // ascending expert order
        const bool dem = miss && mr < nV && sj < 0;        // a copy of its own
        const int dr = flag_rank(dem, wsum, n_dem);
        int c = hit ? wh : -1;
        if (miss && mr < nV) {
            c = vic[mr];
            place(a, l, c, t, occ[c]);
            if (sj >= 0) {
                // the staged block becomes the slot's block; the slot's old block is the position's
                const int old = a.blk[l * a.C + c];
                a.blk[l * a.C + c] = a.sblk[cur * kStageMax + sj];
                a.sblk[cur * kStageMax + sj] = old;
            } else {
                a.demand[dr] = Copy{a.host[l * a.E + t], slot_ptr(a, l, c), nullptr};
            }
        }
        if (miss && mr >= nV && sj >= 0) atomicAdd(&cnt[2], 1);
        if (c >= 0) a.last[l * a.C + c] = a.stamp;
        if (inU && *a.use_freq) a.freq[size_t(l) * a.E + t] += 1;   // after this layer's victims
        // the FFN reads resident experts from their slot, staged overflow from its
        // staging block, other overflow from host memory
        if (inU)
            a.table[t] = c >= 0    ? static_cast<const void*>(slot_ptr(a, l, c))
                         : sj >= 0 ? static_cast<const void*>(block_ptr(a, a.sblk[cur * kStageMax + sj]))
                                   : static_cast<const void*>(a.host[l * a.E + t]);
        if (!staged && t < a.E && a.pending[l * a.E + t]) {
            atomicAdd(&cnt[keep[t] ? 0 : 1], 1);
            a.pending[l * a.E + t] = 0;
        }
        // staged experts: selected ones were used; the others are cancelled
        for (int j = t; j < n_cons; j += kT) {
            const int e = a.sexp[cur * kStageMax + j];
            if (keep[e]) {
                atomicAdd(&cnt[0], 1);
            } else {
                atomicAdd(&cnt[1], 1);
                __hip_atomic_store(a.cancel + cur * kStageMax + j, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        __syncthreads();
        if (t == 0) {
            const int n_placed = n_miss < nV ? n_miss : nV;
            *a.n_demand = n_dem;
            a.stats[0] += n_hit;
            a.stats[1] += n_dem;
            a.stats[4] += cnt[0];
            a.stats[5] += cnt[1];
            // overflow: misses without a slot that were not staged
            a.stats[2] += n_miss - n_placed - cnt[2];
        }
    }
    if (!a.ranked) return;

    // ---- prefetch for layer `next`: admitted prefix of the ranking
    const int lp = a.next;
    if (t == 0) n_adm = a.E;
    __syncthreads();
    const int total_r = *a.n_ranked;
    int f = -1;
    if (t < a.E) {
        f = t < total_r ? a.ranked[t] : -1;
        const bool adm = f >= 0 && f < a.E && t < a.pf_max && a.max_score[f] >= a.pf_min;
        if (!adm) atomicMin(&n_adm, t);
    }
    if (t < a.E) keep[t] = 0;
    __syncthreads();
    if (staged) {
        // the first ns admitted experts not resident in `next`, into the other parity
        const int nx = cur ^ 1;
        const bool nonres = t < n_adm && a.where[lp * a.E + f] < 0;
        int n_nonres;
        const int j = flag_rank(nonres, wsum, n_nonres);
        const int n_st = n_nonres < a.ns ? n_nonres : a.ns;
        if (nonres && j < a.ns) {
            a.sexp[nx * kStageMax + j] = f;
            __hip_atomic_store(a.cancel + nx * kStageMax + j, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.pf[j] = Copy{a.host[lp * a.E + f], block_ptr(a, a.sblk[nx * kStageMax + j]),
                           a.cancel + nx * kStageMax + j};
        }
        if (t == 0) {
            *a.n_pf = n_st;
            a.stats[3] += n_st;
            a.ctl[1 + nx] = lp;
            a.ctl[3 + nx] = n_st;
            a.ctl[0] = nx;
        }
        return;
    }
    const int m = n_adm < a.C ? n_adm : a.C;
    const bool ranked_in = t < m;                       // f is valid here
    if (ranked_in) keep[f] = 1;
    __syncthreads();
    const int nV2 = rank_victims(a, lp, keep, occ, lastl, usel, evl, vic, wsum);
    const bool nonres = ranked_in && a.where[lp * a.E + f] < 0;
    int n_nonres;
    const int j = flag_rank(nonres, wsum, n_nonres);    // ranking order
    const int copies = n_nonres < nV2 ? n_nonres : nV2;
    if (nonres && j < nV2) {
        const int cs = vic[j];
        place(a, lp, cs, f, occ[cs]);
        a.last[lp * a.C + cs] = a.stamp;
        a.pending[lp * a.E + f] = 1;
        a.pf[j] = Copy{a.host[lp * a.E + f], slot_ptr(a, lp, cs), nullptr};
    }
    if (t == 0) {
        *a.n_pf = copies;
        a.stats[3] += copies;
    }
}

// Copy the listed blobs (16-byte chunks, four in flight per thread).  A copy
// with a cancel flag stops at the first check after the flag is set (every
// 4 x 16 bytes per thread); the kernel never waits on the flag.
__global__ __launch_bounds__(256) void blit_kernel(const Copy* list, const int32_t* n, size_t chunks) {
    typedef const __attribute__((address_space(1))) u32x4 gsrc;
    typedef __attribute__((address_space(1))) u32x4 gdst;
    const int nc = *n;
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    for (int i = 0; i < nc; ++i) {
        gsrc* src = (gsrc*)(list[i].src);
        gdst* dst = (gdst*)(list[i].dst);
        const int32_t* cancel = list[i].cancel;
        size_t k = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
        for (; k + 3 * stride < chunks; k += 4 * stride) {
            if (cancel && __hip_atomic_load(cancel, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
            u32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + k + u * stride);
#pragma unroll
            for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + k + u * stride);
        }
        if (cancel && __hip_atomic_load(cancel, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) continue;
        for (; k < chunks; k += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + k), dst + k);
    }
}

}  // namespace

struct DeviceCache {
    int L = 0, E = 0, C = 0;
    size_t blob = 0;
    char* arena = nullptr;
    hipStream_t side = nullptr;
    // device state
    int32_t* slot = nullptr;
    int64_t* last = nullptr;
    int32_t* where = nullptr;
    int32_t* pending = nullptr;
    long long* stats = nullptr;
    const char** host = nullptr;     // [L*E]
    Copy* demand = nullptr;          // [kMaxE]
    int32_t* n_demand = nullptr;
    Copy* pf = nullptr;              // [L][kMaxE]
    int32_t* n_pf = nullptr;         // [L]
    int32_t* blk = nullptr;          // [L*C]
    int32_t* sblk = nullptr;         // [2][kStageMax]
    int32_t* sexp = nullptr;         // [2][kStageMax]
    int32_t* cancel = nullptr;       // [2][kStageMax]
    int32_t* ctl = nullptr;          // [5]
    int64_t* freq = nullptr;         // [L*E]
    int32_t* use_freq = nullptr;     // [1]
    int demand_wgs = kBlitWgs;       // copy kernel workgroups: missed loads ...
    int prefetch_wgs = kPrefetchWgs; // ... and prefetches
    int n_blocks = 0;                // arena blocks: L*C slots + staging
    int ns = 0;                      // staged positions per parity (0: prefetch into slots)
    bool permuted = false;           // staged prefetches have swapped slot blocks
    // ordering: decisions made (compute stream), prefetch of layer l done (side),
    // all side work joined back (graph capture and replay)
    hipEvent_t ev_decided = nullptr, ev_join = nullptr;
    std::vector<hipEvent_t> pf_done;
    std::vector<char> pf_set;
};

namespace {

void free_dc(DeviceCache* d) {
    if (!d) return;
    if (d->side) (void)hipStreamSynchronize(d->side);
    if (d->ev_decided) (void)hipEventDestroy(d->ev_decided);
    if (d->ev_join) (void)hipEventDestroy(d->ev_join);
    for (auto e : d->pf_done)
        if (e) (void)hipEventDestroy(e);
    delete d;       // the state lives in the cache's arena
}

// Layout of the decision state inside the cache arena (256-byte aligned).
struct StateLayout {
    size_t slot, last, where, pending, stats, host, demand, n_demand, pf, n_pf, blk, sblk, sexp, cancel, ctl,
        freq, use_freq, total;
};

StateLayout state_layout(int L, int E, int C) {
    StateLayout y{};
    const size_t LC = size_t(L) * C, LE = size_t(L) * E;
    size_t off = 0;
    auto take = [&](size_t n) { const size_t at = off; off = (off + n + 255) / 256 * 256; return at; };
    y.slot = take(LC * 4);
    y.last = take(LC * 8);
    y.where = take(LE * 4);
    y.pending = take(LE * 4);
    y.stats = take(6 * sizeof(long long));
    y.host = take(LE * sizeof(char*));
    y.demand = take(kMaxE * sizeof(Copy));
    y.n_demand = take(4);
    y.pf = take(size_t(L) * kMaxE * sizeof(Copy));
    y.n_pf = take(size_t(L) * 4);
    y.blk = take(LC * 4);
    y.sblk = take(2 * kStageMax * 4);
    y.sexp = take(2 * kStageMax * 4);
    y.cancel = take(2 * kStageMax * 4);
    y.ctl = take(5 * 4);
    y.freq = take(LE * 8);
    y.use_freq = take(4);
    y.total = off;
    return y;
}

}  // namespace

size_t device_cache_state_bytes(int L, int E, int C) { return state_layout(L, E, C).total; }

int device_cache_create(const PolicyState& ps, char* arena, size_t blob, int n_stage,
                        const void* const* host_blobs, char* state, hipStream_t side, DeviceCache** out) {
    STMOE_CHECK(ps.E <= kMaxE && ps.C <= kMaxE && blob % 16 == 0, "bad cache shape for device decisions");
    // every pool blob must be reachable from kernels at its own address:
    // pinned host memory mapped at the same address, or device memory
    std::vector<const char*> hp(size_t(ps.L) * ps.E);
    for (size_t i = 0; i < hp.size(); ++i) {
        hipPointerAttribute_t at{};
        if (hipPointerGetAttributes(&at, host_blobs[i]) != hipSuccess ||
            (at.type != hipMemoryTypeHost && at.type != hipMemoryTypeDevice) ||
            at.devicePointer != host_blobs[i]) {
            (void)hipGetLastError();
            set_error("expert_cache_set_device_policy: pool blob " + std::to_string(i) +
                      " is neither device memory nor pinned host memory mapped at its own address");
            return STMOE_EINVAL;
        }
        hp[i] = static_cast<const char*>(host_blobs[i]);
    }
    auto* d = new DeviceCache();
    d->L = ps.L; d->E = ps.E; d->C = ps.C; d->blob = blob; d->arena = arena; d->side = side;
    const size_t LC = size_t(ps.L) * ps.C, LE = size_t(ps.L) * ps.E;
    const StateLayout y = state_layout(ps.L, ps.E, ps.C);
    d->slot = reinterpret_cast<int32_t*>(state + y.slot);
    d->last = reinterpret_cast<int64_t*>(state + y.last);
    d->where = reinterpret_cast<int32_t*>(state + y.where);
    d->pending = reinterpret_cast<int32_t*>(state + y.pending);
    d->stats = reinterpret_cast<long long*>(state + y.stats);
    d->host = reinterpret_cast<const char**>(state + y.host);
    d->demand = reinterpret_cast<Copy*>(state + y.demand);
    d->n_demand = reinterpret_cast<int32_t*>(state + y.n_demand);
    d->pf = reinterpret_cast<Copy*>(state + y.pf);
    d->n_pf = reinterpret_cast<int32_t*>(state + y.n_pf);
    d->blk = reinterpret_cast<int32_t*>(state + y.blk);
    d->sblk = reinterpret_cast<int32_t*>(state + y.sblk);
    d->sexp = reinterpret_cast<int32_t*>(state + y.sexp);
    d->cancel = reinterpret_cast<int32_t*>(state + y.cancel);
    d->ctl = reinterpret_cast<int32_t*>(state + y.ctl);
    d->freq = reinterpret_cast<int64_t*>(state + y.freq);
    d->use_freq = reinterpret_cast<int32_t*>(state + y.use_freq);
    d->n_blocks = int(LC) + n_stage;
    std::vector<int32_t> blk(LC);
    for (size_t i = 0; i < LC; ++i) blk[i] = int32_t(i);
    const int32_t ctl[5] = {0, -1, -1, 0, 0};
    hipError_t e = hipEventCreateWithFlags(&d->ev_decided, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&d->ev_join, hipEventDisableTiming);
    d->pf_done.assign(ps.L, nullptr);
    d->pf_set.assign(ps.L, 0);
    for (int l = 0; e == hipSuccess && l < ps.L; ++l) e = hipEventCreateWithFlags(&d->pf_done[l], hipEventDisableTiming);
    std::vector<int32_t> pend(LE);
    for (size_t i = 0; i < LE; ++i) pend[i] = ps.pending[i];
    const long long st[6] = {ps.st->hits, ps.st->demand, ps.st->overflow, ps.st->prefetch, ps.st->useful,
                             ps.st->wasted};
    if (e == hipSuccess) e = hipMemcpy(d->slot, ps.slot, LC * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->last, ps.last, LC * 8, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->where, ps.where, LE * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->pending, pend.data(), LE * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->stats, st, sizeof(st), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->host, hp.data(), LE * sizeof(char*), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(d->n_demand, 0, 4);
    if (e == hipSuccess) e = hipMemset(d->n_pf, 0, size_t(ps.L) * 4);
    if (e == hipSuccess) e = hipMemcpy(d->blk, blk.data(), LC * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->ctl, ctl, sizeof(ctl), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(d->cancel, 0, 2 * kStageMax * 4);
    const int32_t uf = *ps.use_freq;
    if (e == hipSuccess) e = hipMemcpy(d->freq, ps.freq, LE * 8, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d->use_freq, &uf, 4, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        set_error(std::string("expert_cache_set_device_policy: ") + hipGetErrorString(e));
        free_dc(d);
        return STMOE_EHIP;
    }
    *out = d;
    return STMOE_OK;
}

int device_cache_download(DeviceCache* d, const PolicyState& ps) {
    STMOE_HIP(hipStreamSynchronize(d->side));
    STMOE_HIP(hipDeviceSynchronize());
    if (d->permuted) {
        set_error("expert_cache_set_device_policy: staged prefetches have moved slots to other arena blocks; "
                  "the host policy cannot take the cache over");
        return STMOE_ESTATE;
    }
    const size_t LC = size_t(d->L) * d->C, LE = size_t(d->L) * d->E;
    std::vector<int32_t> pend(LE);
    long long st[6];
    STMOE_HIP(hipMemcpy(ps.slot, d->slot, LC * 4, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(ps.last, d->last, LC * 8, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(ps.where, d->where, LE * 4, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(pend.data(), d->pending, LE * 4, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(st, d->stats, sizeof(st), hipMemcpyDeviceToHost));
    int32_t uf = 0;
    STMOE_HIP(hipMemcpy(ps.freq, d->freq, LE * 8, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(&uf, d->use_freq, 4, hipMemcpyDeviceToHost));
    *ps.use_freq = uf;
    for (size_t i = 0; i < LE; ++i) ps.pending[i] = char(pend[i] != 0);
    *ps.st = stmoe_cache_stats{st[0], st[1], st[2], st[3], st[4], st[5]};
    return STMOE_OK;
}

void device_cache_destroy(DeviceCache* d) { free_dc(d); }

int device_cache_set_staged(DeviceCache* d, int ns) {
    STMOE_CHECK(ns >= 0 && ns <= kStageMax && d->n_blocks - d->L * d->C >= 2 * ns,
                "staged prefetch needs 2 * n staging slots in the cache arena");
    STMOE_HIP(hipStreamSynchronize(d->side));
    STMOE_HIP(hipDeviceSynchronize());
    if (ns > 0) {
        // the staging positions of both parities take the blocks no slot
        // holds (staged prefetches may have swapped blocks between slots and
        // staging positions before)
        const size_t LC = size_t(d->L) * d->C;
        std::vector<int32_t> blk(LC);
        STMOE_HIP(hipMemcpy(blk.data(), d->blk, LC * 4, hipMemcpyDeviceToHost));
        std::vector<char> held(size_t(d->n_blocks), 0);
        for (int32_t b : blk) held[size_t(b)] = 1;
        std::vector<int32_t> spare;
        for (int b = 0; b < d->n_blocks; ++b)
            if (!held[size_t(b)]) spare.push_back(b);
        if (spare.size() < size_t(2 * ns)) {
            set_error("expert_cache_set_staged_prefetch: internal error, too few spare blocks");
            return STMOE_ESTATE;
        }
        std::vector<int32_t> sblk(2 * kStageMax, -1);
        for (int p = 0; p < 2; ++p)
            for (int j = 0; j < ns; ++j) sblk[size_t(p) * kStageMax + j] = spare[size_t(p) * ns + j];
        const int32_t ctl[5] = {0, -1, -1, 0, 0};
        STMOE_HIP(hipMemcpy(d->sblk, sblk.data(), sblk.size() * 4, hipMemcpyHostToDevice));
        STMOE_HIP(hipMemcpy(d->ctl, ctl, sizeof(ctl), hipMemcpyHostToDevice));
        d->permuted = true;
    }
    d->ns = ns;
    return STMOE_OK;
}

int device_cache_staged(const DeviceCache* d) { return d->ns; }

void device_cache_set_copy_workgroups(DeviceCache* d, int demand, int prefetch) {
    d->demand_wgs = demand > 0 ? demand : kBlitWgs;
    d->prefetch_wgs = prefetch > 0 ? prefetch : kPrefetchWgs;
}

int device_cache_set_counts(DeviceCache* d, const int64_t* counts) {
    STMOE_HIP(hipStreamSynchronize(d->side));
    STMOE_HIP(hipDeviceSynchronize());
    const size_t LE = size_t(d->L) * d->E;
    std::vector<int64_t> v(LE, 0);
    if (counts) std::copy(counts, counts + LE, v.begin());
    const int32_t uf = counts != nullptr;
    STMOE_HIP(hipMemcpy(d->freq, v.data(), LE * 8, hipMemcpyHostToDevice));
    STMOE_HIP(hipMemcpy(d->use_freq, &uf, 4, hipMemcpyHostToDevice));
    return STMOE_OK;
}

int device_cache_stats(DeviceCache* d, stmoe_cache_stats* out) {
    STMOE_HIP(hipStreamSynchronize(d->side));
    STMOE_HIP(hipDeviceSynchronize());
    long long st[6];
    STMOE_HIP(hipMemcpy(st, d->stats, sizeof(st), hipMemcpyDeviceToHost));
    *out = stmoe_cache_stats{st[0], st[1], st[2], st[3], st[4], st[5]};
    return STMOE_OK;
}

int device_cache_join(DeviceCache* d, hipStream_t s) {
    STMOE_HIP(hipEventRecord(d->ev_join, d->side));
    STMOE_HIP(hipStreamWaitEvent(s, d->ev_join, 0));
    return STMOE_OK;
}

void device_cache_forget_waits(DeviceCache* d) { std::fill(d->pf_set.begin(), d->pf_set.end(), char(0)); }

int device_cache_decide(DeviceCache* d, int layer, int next, const int32_t* idx, int BK,
                        const int32_t* ranked, const int32_t* n_ranked, const uint8_t* max_score,
                        int pf_min, int pf_max, const int64_t* tok, int64_t stamp_add, const void** table,
                        hipStream_t s) {
    STMOE_CHECK(layer >= 0 && layer < d->L && next >= 0 && next < d->L && BK >= 0 && BK <= kT,
                "bad layer or selection size");
    STMOE_CHECK(BK > 0 || ranked, "nothing to decide");
    // the prefetch list of `next` is rewritten below: its previous copy kernel must be done
    if (ranked && d->pf_set[next]) STMOE_HIP(hipStreamWaitEvent(s, d->pf_done[next], 0));
    DecideArgs a{};
    a.L = d->L; a.E = d->E; a.C = d->C; a.layer = layer; a.next = next; a.BK = BK;
    a.pf_min = pf_min; a.pf_max = pf_max; a.tok = tok; a.stamp_add = stamp_add; a.demand_on = BK > 0;
    a.slot = d->slot; a.last = d->last; a.where = d->where; a.pending = d->pending; a.stats = d->stats;
    a.idx = idx; a.ranked = ranked; a.n_ranked = n_ranked; a.max_score = max_score;
    a.host = d->host; a.arena = d->arena; a.blob = d->blob; a.table = table;
    a.demand = d->demand; a.n_demand = d->n_demand;
    a.pf = d->pf + size_t(next) * kMaxE; a.n_pf = d->n_pf + next;
    a.blk = d->blk; a.ns = d->ns; a.sblk = d->sblk; a.sexp = d->sexp; a.cancel = d->cancel; a.ctl = d->ctl;
    a.freq = d->freq; a.use_freq = d->use_freq;
    hipLaunchKernelGGL(decide_kernel, dim3(1), dim3(kT), 0, s, a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

int device_cache_demand(DeviceCache* d, int layer, hipStream_t s) {
    // slots of `layer` written by an earlier prefetch are read from here on
    if (d->pf_set[layer]) STMOE_HIP(hipStreamWaitEvent(s, d->pf_done[layer], 0));
    hipLaunchKernelGGL(blit_kernel, dim3(unsigned(d->demand_wgs)), dim3(256), 0, s, d->demand, d->n_demand,
                       d->blob / 16);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

int device_cache_prefetch(DeviceCache* d, int next, hipStream_t s) {
    // starts after the work enqueued so far on `s`: the decisions, and every
    // earlier reader of `next`'s slots (the caller enqueues the FFN first
    // when it reads them too)
    STMOE_HIP(hipEventRecord(d->ev_decided, s));
    STMOE_HIP(hipStreamWaitEvent(d->side, d->ev_decided, 0));
    hipLaunchKernelGGL(blit_kernel, dim3(unsigned(d->prefetch_wgs)), dim3(256), 0, d->side, d->pf + size_t(next) * kMaxE,
                       d->n_pf + next, d->blob / 16);
    STMOE_LAUNCHED();
    STMOE_HIP(hipEventRecord(d->pf_done[next], d->side));
    d->pf_set[next] = 1;
    return STMOE_OK;
}

}  // namespace stmoe
