// Device-side cache decisions: the expert cache's policy state lives in HBM
// and a one-workgroup kernel per layer makes the missed-loading and prefetch
// decisions from the routing and the prediction already on the device
// (Section 4.3.4's "ML" and "EP" stages without a host round trip).  Copies
// from pinned host memory run as copy kernels on the compute stream (missed
// experts) and on the cache's side stream (prefetches); experts beyond the
// layer's slots are read by the FFN straight from host memory.
#pragma once

#include "common.h"

namespace stmoe {

struct DeviceCache;

// Host policy state handed over when device decisions are switched on and
// taken back when they are switched off (both [sync]).
struct PolicyState {
    int L, E, C;
    int32_t* slot;              // [L*C] expert in slot or -1
    int64_t* last;              // [L*C] last use stamp
    int32_t* where;             // [L*E] slot of expert or -1
    char* pending;              // [L*E] prefetched, not yet verified
    int64_t* freq;              // [L*E] use counts
    int* use_freq;              // 1: frequency-aware eviction
    stmoe_cache_stats* st;
};

// Bytes of device decision state for a cache of L layers, E experts and C
// slots per layer (part of the cache arena).
size_t device_cache_state_bytes(int L, int E, int C);
// `state`: device_cache_state_bytes(L, E, C) bytes of the cache arena,
// 256-byte aligned; the decisions keep their state there.
int device_cache_create(const PolicyState& ps, char* arena, size_t blob, int n_stage,
                        const void* const* host_blobs, char* state, hipStream_t side, DeviceCache** out);
// Staged prefetch with ns positions per parity (0: prefetch into slots).  [sync]
int device_cache_set_staged(DeviceCache* d, int ns);
// Frequency-aware eviction with these use counts ([L*E] host), or least
// recently used (counts null).  [sync]
int device_cache_set_counts(DeviceCache* d, const int64_t* counts);
// Workgroups of the copy kernels for missed loads and prefetches (0: the
// defaults, 64 and 16).  Takes effect for copies launched afterwards.
void device_cache_set_copy_workgroups(DeviceCache* d, int demand, int prefetch);
int device_cache_staged(const DeviceCache* d);
int device_cache_download(DeviceCache* d, const PolicyState& ps);
void device_cache_destroy(DeviceCache* d);
int device_cache_stats(DeviceCache* d, stmoe_cache_stats* st);

// One layer on `s` (the compute stream).  decide: the decisions for `layer`
// (missed experts; none when BK == 0) and, with `ranked`, for `next`
// (prefetch under the admission knobs), and the pointer table the FFN reads
// (table [E]).
// demand: the missed experts' copies.  prefetch: the copies for `next` on
// the side stream, after everything enqueued on `s` so far.
// Stamps are read on the device: *tok * L + stamp_add (tok: device int64).
int device_cache_decide(DeviceCache* d, int layer, int next, const int32_t* idx, int BK,
                        const int32_t* ranked, const int32_t* n_ranked, const uint8_t* max_score,
                        int pf_min, int pf_max, const int64_t* tok, int64_t stamp_add, const void** table,
                        hipStream_t s);
// `s` waits for all work queued so far on the side stream.
int device_cache_join(DeviceCache* d, hipStream_t s);
// Forget the prefetch completion events (all side work is known to be
// ordered before what follows: a joined graph replay or capture).
void device_cache_forget_waits(DeviceCache* d);
int device_cache_demand(DeviceCache* d, int layer, hipStream_t s);
int device_cache_prefetch(DeviceCache* d, int next, hipStream_t s);

}  // namespace stmoe
