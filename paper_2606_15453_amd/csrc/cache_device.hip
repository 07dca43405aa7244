// Device-side cache decisions (see cache_device.h).  The policy is the host
// policy's (expert_cache.cpp): per-layer slot partitions; a missed expert
// takes the evictable slot (empty, or holding an expert outside the current
// selection) with the smallest (last use, slot); a prefetch walks the
// admitted ranking and takes victims the same way among slots outside the
// ranked set, stopping when none is left; residency counts from copy issue.
// Evictions within one call never change the other candidates' keys, so the
// k-th missed (or non-resident ranked) expert takes the k-th victim in
// (last use, slot) order: the kernel ranks slots and experts in parallel
// instead of searching once per copy.
#include <vector>

#include "cache_device.h"

namespace stmoe {
namespace {

constexpr int kT = 256;          // threads of the decision kernel (E, C <= 256)
constexpr int kBlitWgs = 64;     // copy kernel workgroups (enough to fill the host link)

struct Copy {
    const char* src;             // device-accessible host blob
    char* dst;                   // HBM slot
};

struct DecideArgs {
    int L, E, C, layer, next, BK, pf_min, pf_max;
    int demand_on;               // 0: only the prefetch decisions (no selection yet)
    int64_t stamp;
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
    Copy* pf;                    // [C] for `next`
    int32_t* n_pf;               // for `next`
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
// rank r among evictable slots by (last use, slot); returns their number.
// occ[c] receives each slot's occupant.  Ends with a barrier.
__device__ int rank_victims(const DecideArgs& a, int l, const unsigned char* keep, int* occ,
                            int64_t* lastl, unsigned char* evl, int* vic, int* wsum) {
    const int t = threadIdx.x;
    if (t < a.C) {
        const int e = a.slot[l * a.C + t];
        occ[t] = e;
        lastl[t] = a.last[l * a.C + t];
        evl[t] = e < 0 || !keep[e];
    }
    __syncthreads();
    if (t < a.C && evl[t]) {
        const int64_t lt = lastl[t];
        int r = 0;
        for (int c = 0; c < a.C; ++c) r += evl[c] && (lastl[c] < lt || (lastl[c] == lt && c < t));
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

__device__ char* slot_ptr(const DecideArgs& a, int l, int c) {
    return a.arena + (size_t(l) * a.C + c) * a.blob;
}

__global__ __launch_bounds__(kT) void decide_kernel(DecideArgs a) {
    __shared__ unsigned char keep[kMaxE];
    __shared__ unsigned char evl[kMaxE];
    __shared__ int occ[kMaxE];
    __shared__ int vic[kMaxE];
    __shared__ int64_t lastl[kMaxE];
    __shared__ int wsum[kT / 64];
    __shared__ int cnt[2];
    __shared__ int n_adm;
    const int t = threadIdx.x;
    const int l = a.layer;

    // ---- missed experts of layer l (the selection U = distinct idx)
    if (a.demand_on) {
        if (t < a.E) keep[t] = 0;
        if (t < 2) cnt[t] = 0;
        __syncthreads();
        for (int i = t; i < a.BK; i += kT) {
            const int e = a.idx[i];
            if (e >= 0 && e < a.E) keep[e] = 1;
        }
        __syncthreads();
        const bool inU = t < a.E && keep[t];
        const int wh = t < a.E ? a.where[l * a.E + t] : -1;
        const bool hit = inU && wh >= 0, miss = inU && wh < 0;
        const int nV = rank_victims(a, l, keep, occ, lastl, evl, vic, wsum);
        int n_hit, n_miss;
        (void)flag_rank(hit, wsum, n_hit);
        const int mr = flag_rank(miss, wsum, n_miss);      // ascending expert order
        const int n_placed = n_miss < nV ? n_miss : nV;
        int c = hit ? wh : -1;
        if (miss && mr < nV) {
            c = vic[mr];
            place(a, l, c, t, occ[c]);
            a.demand[mr] = Copy{a.host[l * a.E + t], slot_ptr(a, l, c)};
        }
        if (c >= 0) a.last[l * a.C + c] = a.stamp;
        // the FFN reads resident experts from their slot, overflow from host memory
        if (inU) a.table[t] = c >= 0 ? static_cast<const void*>(slot_ptr(a, l, c)) : a.host[l * a.E + t];
        if (t < a.E && a.pending[l * a.E + t]) {
            atomicAdd(&cnt[keep[t] ? 0 : 1], 1);
            a.pending[l * a.E + t] = 0;
        }
        __syncthreads();
        if (t == 0) {
            *a.n_demand = n_placed;
            a.stats[0] += n_hit;
            a.stats[1] += n_placed;
            a.stats[2] += n_miss - n_placed;
            a.stats[4] += cnt[0];
            a.stats[5] += cnt[1];
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
    const int m = n_adm < a.C ? n_adm : a.C;
    const bool ranked_in = t < m;                       // f is valid here
    if (ranked_in) keep[f] = 1;
    __syncthreads();
    const int nV2 = rank_victims(a, lp, keep, occ, lastl, evl, vic, wsum);
    const bool nonres = ranked_in && a.where[lp * a.E + f] < 0;
    int n_nonres;
    const int j = flag_rank(nonres, wsum, n_nonres);    // ranking order
    const int copies = n_nonres < nV2 ? n_nonres : nV2;
    if (nonres && j < nV2) {
        const int cs = vic[j];
        place(a, lp, cs, f, occ[cs]);
        a.last[lp * a.C + cs] = a.stamp;
        a.pending[lp * a.E + f] = 1;
        a.pf[j] = Copy{a.host[lp * a.E + f], slot_ptr(a, lp, cs)};
    }
    if (t == 0) {
        *a.n_pf = copies;
        a.stats[3] += copies;
    }
}

// Copy the listed blobs (16-byte chunks, four in flight per thread).
__global__ __launch_bounds__(256) void blit_kernel(const Copy* list, const int32_t* n, size_t chunks) {
    typedef const __attribute__((address_space(1))) u32x4 gsrc;
    typedef __attribute__((address_space(1))) u32x4 gdst;
    const int nc = *n;
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    for (int i = 0; i < nc; ++i) {
        gsrc* src = (gsrc*)(list[i].src);
        gdst* dst = (gdst*)(list[i].dst);
        size_t k = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
        for (; k + 3 * stride < chunks; k += 4 * stride) {
            u32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + k + u * stride);
#pragma unroll
            for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + k + u * stride);
        }
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
    Copy* pf = nullptr;              // [L][C]
    int32_t* n_pf = nullptr;         // [L]
    // ordering: decisions made (compute stream), prefetch of layer l done (side)
    hipEvent_t ev_decided = nullptr;
    std::vector<hipEvent_t> pf_done;
    std::vector<char> pf_set;
};

namespace {

void free_dc(DeviceCache* d) {
    if (!d) return;
    if (d->side) (void)hipStreamSynchronize(d->side);
    for (void* p : {(void*)d->slot, (void*)d->last, (void*)d->where, (void*)d->pending, (void*)d->stats,
                    (void*)d->host, (void*)d->demand, (void*)d->n_demand, (void*)d->pf, (void*)d->n_pf})
        if (p) (void)hipFree(p);
    if (d->ev_decided) (void)hipEventDestroy(d->ev_decided);
    for (auto e : d->pf_done)
        if (e) (void)hipEventDestroy(e);
    delete d;
}

}  // namespace

int device_cache_create(const PolicyState& ps, char* arena, size_t blob, const void* const* host_blobs,
                        hipStream_t side, DeviceCache** out) {
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
    hipError_t e = hipMalloc(&d->slot, LC * 4);
    if (e == hipSuccess) e = hipMalloc(&d->last, LC * 8);
    if (e == hipSuccess) e = hipMalloc(&d->where, LE * 4);
    if (e == hipSuccess) e = hipMalloc(&d->pending, LE * 4);
    if (e == hipSuccess) e = hipMalloc(&d->stats, 6 * sizeof(long long));
    if (e == hipSuccess) e = hipMalloc(&d->host, LE * sizeof(char*));
    if (e == hipSuccess) e = hipMalloc(&d->demand, kMaxE * sizeof(Copy));
    if (e == hipSuccess) e = hipMalloc(&d->n_demand, 4);
    if (e == hipSuccess) e = hipMalloc(&d->pf, LC * sizeof(Copy));
    if (e == hipSuccess) e = hipMalloc(&d->n_pf, size_t(ps.L) * 4);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&d->ev_decided, hipEventDisableTiming);
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
    const size_t LC = size_t(d->L) * d->C, LE = size_t(d->L) * d->E;
    std::vector<int32_t> pend(LE);
    long long st[6];
    STMOE_HIP(hipMemcpy(ps.slot, d->slot, LC * 4, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(ps.last, d->last, LC * 8, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(ps.where, d->where, LE * 4, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(pend.data(), d->pending, LE * 4, hipMemcpyDeviceToHost));
    STMOE_HIP(hipMemcpy(st, d->stats, sizeof(st), hipMemcpyDeviceToHost));
    for (size_t i = 0; i < LE; ++i) ps.pending[i] = char(pend[i] != 0);
    *ps.st = stmoe_cache_stats{st[0], st[1], st[2], st[3], st[4], st[5]};
    return STMOE_OK;
}

void device_cache_destroy(DeviceCache* d) { free_dc(d); }

int device_cache_stats(DeviceCache* d, stmoe_cache_stats* out) {
    STMOE_HIP(hipStreamSynchronize(d->side));
    STMOE_HIP(hipDeviceSynchronize());
    long long st[6];
    STMOE_HIP(hipMemcpy(st, d->stats, sizeof(st), hipMemcpyDeviceToHost));
    *out = stmoe_cache_stats{st[0], st[1], st[2], st[3], st[4], st[5]};
    return STMOE_OK;
}

int device_cache_decide(DeviceCache* d, int layer, int next, const int32_t* idx, int BK,
                        const int32_t* ranked, const int32_t* n_ranked, const uint8_t* max_score,
                        int pf_min, int pf_max, int64_t stamp, const void** table, hipStream_t s) {
    STMOE_CHECK(layer >= 0 && layer < d->L && next >= 0 && next < d->L && BK >= 0 && BK <= kT,
                "bad layer or selection size");
    STMOE_CHECK(BK > 0 || ranked, "nothing to decide");
    // the prefetch list of `next` is rewritten below: its previous copy kernel must be done
    if (ranked && d->pf_set[next]) STMOE_HIP(hipStreamWaitEvent(s, d->pf_done[next], 0));
    DecideArgs a{};
    a.L = d->L; a.E = d->E; a.C = d->C; a.layer = layer; a.next = next; a.BK = BK;
    a.pf_min = pf_min; a.pf_max = pf_max; a.stamp = stamp; a.demand_on = BK > 0;
    a.slot = d->slot; a.last = d->last; a.where = d->where; a.pending = d->pending; a.stats = d->stats;
    a.idx = idx; a.ranked = ranked; a.n_ranked = n_ranked; a.max_score = max_score;
    a.host = d->host; a.arena = d->arena; a.blob = d->blob; a.table = table;
    a.demand = d->demand; a.n_demand = d->n_demand;
    a.pf = d->pf + size_t(next) * d->C; a.n_pf = d->n_pf + next;
    hipLaunchKernelGGL(decide_kernel, dim3(1), dim3(kT), 0, s, a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

int device_cache_demand(DeviceCache* d, int layer, hipStream_t s) {
    // slots of `layer` written by an earlier prefetch are read from here on
    if (d->pf_set[layer]) STMOE_HIP(hipStreamWaitEvent(s, d->pf_done[layer], 0));
    hipLaunchKernelGGL(blit_kernel, dim3(kBlitWgs), dim3(256), 0, s, d->demand, d->n_demand, d->blob / 16);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

int device_cache_prefetch(DeviceCache* d, int next, hipStream_t s) {
    // starts after the work enqueued so far on `s`: the decisions, and every
    // earlier reader of `next`'s slots (the caller enqueues the FFN first
    // when it reads them too)
    STMOE_HIP(hipEventRecord(d->ev_decided, s));
    STMOE_HIP(hipStreamWaitEvent(d->side, d->ev_decided, 0));
    hipLaunchKernelGGL(blit_kernel, dim3(kBlitWgs), dim3(256), 0, d->side, d->pf + size_t(next) * d->C,
                       d->n_pf + next, d->blob / 16);
    STMOE_LAUNCHED();
    STMOE_HIP(hipEventRecord(d->pf_done[next], d->side));
    d->pf_set[next] = 1;
    return STMOE_OK;
}

}  // namespace stmoe
