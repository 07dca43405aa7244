/*
 * stmoe.h -- C ABI of the MI355X (gfx950) decode-step MoE layer with
 * spatio-temporal expert prefetching (ST-MoE).
 *
 * The calls follow the paper's problem statement:
 *   gating                      Section 2 (z_j = w_j^T x, softmax, top-K, weighted sum)
 *   profile / predict / update  Section 4.2, Algorithms 1-3 and Eq. 1
 *   prefetch, verify, missed    Section 4.1 and Section 4.3.4 (pipelined workflow)
 *   loading
 *   expert computation          Section 2 (experts are feed-forward networks; SwiGLU form)
 *
 * Conventions
 *   - Every int-returning call returns STMOE_OK (0) or a negative status code;
 *     stmoe_last_error() then returns a thread-local message.  No C++
 *     exception crosses this boundary.
 *   - Arguments are validated before any device work; an invalid call does
 *     nothing on the device.
 *   - "device" pointers are HIP device allocations of the current device;
 *     "host" pointers are ordinary (or pinned, where stated) host memory.
 *   - The caller owns every device buffer and every stream.  Device memory a
 *     handle needs (predictor tables, decode-context buffers, cache slots and
 *     the cache's decision state) comes from a caller workspace sized by the
 *     matching *_workspace_bytes / *_arena_bytes query and passed to the
 *     create call; the library never allocates or frees device memory.  It
 *     owns only the opaque host-side handles (and, for the decode context,
 *     one small pinned host record, events and internal streams), released
 *     by the matching destroy call.  A workspace must stay allocated, and
 *     must not be touched by the caller, until the handle is destroyed.
 *   - `stream` arguments are hipStream_t values passed as void* (NULL is the
 *     default stream).  Calls are asynchronous on that stream unless marked
 *     [sync].
 *   - Limits: 1 <= E <= 256 (8-bit expert indices in the tables),
 *     1 <= K <= min(E, 16), 1 <= B <= 16, H and I multiples of 8, H <= 16384.
 *   - Data types: STMOE_BF16 (weights and activations bfloat16, fp32
 *     accumulation) or STMOE_F32.  Outputs of the FFN are fp32.
 */
#ifndef STMOE_H
#define STMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    STMOE_OK = 0,
    STMOE_EINVAL = -1,     /* invalid argument */
    STMOE_EHIP = -2,       /* a HIP runtime call failed */
    STMOE_ENOMEM = -3,     /* allocation failed or workspace too small */
    STMOE_ECAPACITY = -4,  /* cache arena too small for the requested slots */
    STMOE_ESTATE = -5      /* call out of order (e.g. predict before profile) */
};

typedef enum { STMOE_F32 = 0, STMOE_BF16 = 1 } stmoe_dtype;

/* Message of the last failed call on this thread ("" if none). */
const char* stmoe_last_error(void);
/* ABI version of this header: 2. */
int stmoe_abi_version(void);

/* Pinned host memory for the expert pool (exact size, hipHostMalloc; not
 * rounded up the way caching allocators do).  The caller owns the block
 * and releases it with stmoe_host_free.  [sync] */
int stmoe_host_alloc(size_t bytes, void** out);
int stmoe_host_free(void* p);

/* ------------------------------------------------------------------------
 * Gating (Section 2): z[b][e] = sum_h x[b][h] * w_gate[e][h] (fp32
 * accumulation), s = softmax(z[b]), top-K experts by logit (descending,
 * equal logits -> lower index), weight = s of the selected expert (the
 * paper weights expert outputs by their gating probabilities), or, with
 * renorm = 1, that probability divided by the sum over the K selected.
 *
 *   x        device [B][H] row-major, dtype
 *   w_gate   device [E][H] row-major, dtype
 *   topk_idx device out [B][K] int32, in descending-logit order
 *   topk_w   device out [B][K] fp32
 *   logits   device out [B][E] fp32, or NULL
 *   ws       device workspace of moe_route_workspace_bytes(B, E) bytes (the
 *            logits; no initial contents required)
 *   Two launches on `stream`: logits (one workgroup per expert), then the
 *   softmax / top-K tail.  Calls sharing one workspace must be ordered on
 *   one stream.
 * ---------------------------------------------------------------------- */
size_t moe_route_workspace_bytes(int B, int E);
int moe_route_topk(const void* x, const void* w_gate, int B, int H, int E, int K,
                   int dtype, int renorm, int32_t* topk_idx, float* topk_w, float* logits,
                   void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Spatio-temporal predictor (Section 4.2).
 *
 * Device state per predictor: for every adjacent layer pair i (0..L-2) a
 * Cross-layer Correlation Table CCT_i[E][K] of (expert index, 2-bit
 * confidence) slots; for every layer l and batch row b a History Table entry
 * HT[l][b][K] holding the previous token's selection (kept sorted ascending;
 * its confidence is fixed at 2, "10").  Batch rows share the CCTs.
 * ---------------------------------------------------------------------- */
typedef struct stmoe_predictor stmoe_predictor;

/* Prediction sources, for the ablation of Section 5 (temporal / spatial). */
enum { STMOE_USE_CCT = 1, STMOE_USE_HT = 2, STMOE_USE_BOTH = 3 };

/* Device bytes of a predictor's workspace (its tables, hit statistics and
 * the staging area of the profiling selections); 0 for an invalid shape. */
size_t stmoe_workspace_bytes(int L, int E, int K, int B);
/* Create a predictor whose tables live in dev_ws (device, 256-byte aligned,
 * at least stmoe_workspace_bytes(L, E, K, B) bytes; zeroed here).  [sync] */
int stmoe_create(int L, int E, int K, int B, void* dev_ws, size_t ws_bytes, stmoe_predictor** out);
/* Release the handle (the workspace stays the caller's). */
int stmoe_destroy(stmoe_predictor* p);

/* Algorithm 1 and the HT initialisation (Section 4.1).  [sync]
 *   sel  host [P][B][L][K] int32: the profiling tokens' selections (distinct
 *        within each [K] row, each < E).
 * For each pair i, Co_i[e][f] counts tokens and rows that selected e at
 * layer i and f at layer i+1; CCT_i[e] takes the K largest counts (equal
 * counts -> lower index) with confidence 2; HT[l][b] <- sel[P-1][b][l].
 * Resets the hit statistics.  The selections pass through the workspace's
 * staging area in chunks of whole tokens. */
int stmoe_profile(stmoe_predictor* p, const int32_t* sel, int P);

/* Verify + table update at `layer` (Algorithm 3; Section 4.3.4).
 *   sel_prev device [B][K] int32: selection at layer-1 (ignored at layer 0)
 *   sel_cur  device [B][K] int32: selection at layer
 * For b = 0..B-1 in order, every CCT_{layer-1} entry e in sel_prev[b] is
 * updated against F = sel_cur[b]: a slot whose expert is in F gains 1
 * (saturating at 3); otherwise it loses 1 while above 0, and at 0 it is
 * replaced by the next expert (ascending) of F that the entry did not hold
 * before this update, with confidence 2.  Then HT[layer][b] <- sel_cur[b].
 * If `online` is 0 the CCT is left unchanged (HT is still overwritten).
 * Also counts |sel_cur[b] intersect P_layer[b]| against the last prediction
 * made for this layer, into the statistics. */
int stmoe_update(stmoe_predictor* p, int layer, const int32_t* sel_prev,
                 const int32_t* sel_cur, int online, void* stream);

/* Expert prediction for layer+1 (Algorithm 2 with Eq. 1).
 *   layer    0..L-2 predicts layer+1 from sel_cur; -1 predicts layer 0 from
 *            HT[0] alone (sel_cur ignored).
 *   sel_cur  device [B][K] int32
 *   use      STMOE_USE_* bit set
 *   score    device out [B][E] uint8 or NULL:
 *            score[b][f] = sum_{e in sel_cur[b]} conf of f in CCT_layer[e]
 *                          + 2 * [f in HT[layer+1][b]]
 *   mask     device out [E] uint8 or NULL: 1 where any row scores >= 2
 *   max_score device out [E] uint8 or NULL: max over rows of score[b][f]
 *   ranked   device out [E] int32 or NULL: experts with mask = 1 ordered by
 *            (max over rows of score desc, index asc), then -1 padding
 *   n_ranked device out [1] int32 or NULL: number of such experts */
int stmoe_predict(stmoe_predictor* p, int layer, const int32_t* sel_cur, int use,
                  uint8_t* score, uint8_t* mask, uint8_t* max_score, int32_t* ranked,
                  int32_t* n_ranked, void* stream);

/* Copy the tables to host memory (any pointer may be NULL).  [sync]
 *   co [L-1][E][E] int32, cct_idx / cct_conf [L-1][E][K] uint8,
 *   ht [L][B][K] int32 (rows ascending) */
int stmoe_export(stmoe_predictor* p, int32_t* co, uint8_t* cct_idx, uint8_t* cct_conf,
                 int32_t* ht);
/* Replace the CCT and HT with host copies (same layouts).  Every CCT entry
 * must name K distinct experts < E with confidences in 0..3, and every HT
 * row K distinct experts < E (stored sorted); otherwise STMOE_EINVAL and
 * nothing changes.  Distinct entries bound every Eq. 1 score by 3K + 2.
 * [sync] */
int stmoe_import(stmoe_predictor* p, const uint8_t* cct_idx, const uint8_t* cct_conf,
                 const int32_t* ht);

/* Hit statistics per layer since stmoe_profile, host out [L][3] int64:
 * (sum |A intersect P|, sum |A|, sum |P|) over batch rows.  [sync] */
int stmoe_stats(stmoe_predictor* p, int64_t* out);

/* ------------------------------------------------------------------------
 * Expert packing.  A packed expert ("blob") is one contiguous buffer:
 * W_gate [I][H], then W_up [I][H], then W_down [H][I], each row-major in
 * the storage dtype; 3*H*I elements.  One blob moves with one copy.
 * ---------------------------------------------------------------------- */
size_t moe_blob_bytes(int H, int I, int dtype);
/* [sync, host] blob_out: host, moe_blob_bytes(H, I, dtype) bytes. */
int moe_pack_expert(const void* w_gate, const void* w_up, const void* w_down, int H, int I,
                    int dtype, void* blob_out);

/* ------------------------------------------------------------------------
 * Expert FFN (Section 2): for every batch row b
 *   y[b] = sum_k topk_w[b][k] * W_down e (silu(W_gate e x[b]) * (W_up e x[b]))
 *        + sum_s  W_down s (silu(W_gate s x[b]) * (W_up s x[b]))   (shared, weight 1)
 * with e = topk_idx[b][k] and silu(g) = g / (1 + exp(-g)).
 * Each distinct selected expert's weights are read once per call.  The sum
 * over experts runs in ascending expert index (shared experts last), so the
 * result does not depend on where the blobs live.
 *
 *   x            device [B][H] dtype
 *   topk_idx     device [B][K] int32 (< E), topk_w device [B][K] fp32; an
 *                entry outside [0, E) is ignored, and an expert repeated
 *                within a row counts once, with its first entry's weight
 *   expert_ptrs  device array [E] of device blob pointers; only selected
 *                experts' entries are read
 *   shared_ptrs  device array [n_shared] of device blob pointers, or NULL
 *   y            device out [B][H] fp32 (overwritten)
 *   ws           device workspace of moe_expert_ffn_workspace_bytes(...) bytes,
 *                256-byte aligned (activations and partial sums; no initial
 *                contents required); calls sharing it must be ordered on one
 *                stream
 *   B < 8 runs the GEMV kernels; B >= 8 with bf16 and H, I multiples of 64
 *   runs the MFMA grouped-GEMM kernels (the SwiGLU activation then passes
 *   through bf16); other shapes fall back to the GEMV kernels.
 * ---------------------------------------------------------------------- */
size_t moe_expert_ffn_workspace_bytes(int B, int K, int E, int H, int I, int n_shared, int dtype);
int moe_expert_ffn(const void* x, const int32_t* topk_idx, const float* topk_w, int B, int K,
                   int H, int I, int E, int dtype, const void* const* expert_ptrs,
                   const void* const* shared_ptrs, int n_shared, float* y, void* ws,
                   size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * expert FFN as moe_expert_ffn, with the workspace taken from a 16 MiB
 * scratch array that the library holds on each GPU it runs on (until the
 * process ends) instead of a caller buffer.  It allocates nothing and calls
 * no allocating routine.  Shapes whose moe_expert_ffn_workspace_bytes exceeds
 * 16 MiB (16777216 bytes) return STMOE_ENOMEM before any device work; every
 * configuration named in this library's documentation fits (the largest,
 * batch 16 x top-8 of 128 experts, hidden 4096, intermediate 1536, needs
 * 14.7 MB).  All calls on one GPU share its scratch array: calls that overlap
 * in time on that GPU (different streams, different threads) race and must
 * be serialised by the caller; the array keeps the last call's contents and
 * needs no initial contents.  Arguments as moe_expert_ffn. */
int moe_expert_ffn_noalloc(const void* x, const int32_t* topk_idx, const float* topk_w, int B, int K,
                           int H, int I, int E, int dtype, const void* const* expert_ptrs,
                           const void* const* shared_ptrs, int n_shared, float* y, void* stream);

/* ------------------------------------------------------------------------
 * Expert cache policy (host only, no HIP calls): per-layer partition of C
 * slots, least recently used with protection of the current set.
 *   prefetch(layer, ranked, n, stamp): for each of the first min(n, C)
 *     ranked experts not resident, evict the slot whose expert is not among
 *     them with the smallest (last use, slot); stop when none is left.
 *   acquire(layer, needed, n, stamp): for each needed expert (ascending) not
 *     resident, evict the slot whose expert is not needed with the smallest
 *     (last use, slot); with no such slot the expert is "overflow" (served
 *     from staging, not admitted).  Then needed resident experts get
 *     last use = stamp.
 * Decisions are returned as (expert, slot) pairs; overflow experts as slot -1.
 * ---------------------------------------------------------------------- */
typedef struct stmoe_policy stmoe_policy;
typedef struct {
    int64_t hits, demand, overflow, prefetch, useful, wasted;
} stmoe_cache_stats;

/* Initial residency of a cache (Section 4.1 stages experts before decode;
 * the paper names no choice): per layer the C experts most often selected by
 * the profiling tokens, count desc then index asc, -1 padding when C > E.
 *   sel host [P][B][L][K] int32 (each < E); out host [L][C] int32.  [host] */
int expert_cache_warm_sets(const int32_t* sel, int P, int B, int L, int K, int E, int C, int32_t* out);
/* Seeds of frequency-aware eviction (this implementation's alternative to
 * least recently used; the paper's buffer has no replacement rule): per layer
 * the number of profiling tokens whose selection (any batch row) contains
 * each expert.  sel host [P][B][L][K] int32 (each < E); out host [L][E]
 * int64.  [host] */
int expert_cache_use_counts(const int32_t* sel, int P, int B, int L, int K, int E, int64_t* out);

int stmoe_policy_create(int L, int E, int C, const int32_t* warm /* host [L][C], -1 = empty */,
                        stmoe_policy** out);
int stmoe_policy_destroy(stmoe_policy* p);
/* returns the number of copies (>= 0); pairs host out [2*C] (expert, slot) */
int stmoe_policy_prefetch(stmoe_policy* p, int layer, const int32_t* ranked, int n,
                          int64_t stamp, int32_t* pairs);
/* returns the number of entries written to pairs (host out [2*n]):
 * (expert, slot) for each needed expert that was not resident, slot -1 for
 * overflow; *n_hits receives the number of resident experts. */
int stmoe_policy_acquire(stmoe_policy* p, int layer, const int32_t* needed, int n,
                         int64_t stamp, int32_t* pairs, int32_t* n_hits);
/* slot_expert host out [L][C] (-1 = empty) */
int stmoe_policy_slots(const stmoe_policy* p, int32_t* slot_expert);
int stmoe_policy_stats(const stmoe_policy* p, stmoe_cache_stats* out);
/* Replacement rule.  counts host [L][E] int64 (each >= 0, else STMOE_EINVAL):
 * frequency-aware eviction seeded with these use counts; victims are taken
 * by the smallest (use count of the slot's expert, last use, slot), an empty
 * slot counting -1, and every acquire adds 1 to the count of each expert it
 * is given.  counts NULL: least recently used (the default).  [host] */
int stmoe_policy_set_counts(stmoe_policy* p, const int64_t* counts);

/* ------------------------------------------------------------------------
 * HBM expert cache (Section 4.1 prefetch staging; Section 4.3.4 missed
 * loading).  Routed experts of layer l live either in one of the layer's C
 * HBM slots or only in the pinned host pool; copies are one hipMemcpyAsync
 * per blob.  Prefetches run on `side`, demand copies on `demand`; slot
 * reuse is ordered by events (a slot is overwritten only after its last
 * reader and its previous copy have completed).
 *
 *   arena       device, 256-byte aligned, at least
 *               expert_cache_arena_bytes(L, E, C, blob, n_stage): the L*C slots and
 *               n_stage staging slots, then the state of device-side decisions
 *   host_blobs  host array [L*E] of pinned host blob pointers.  Device
 *               pointers are accepted too (the copies then run device to
 *               device: a pool in another HBM region models a backing tier
 *               much faster than the host link)
 *   n_stage     staging slots for overflow experts (>= 1 when a layer can
 *               select more distinct experts than C)
 * ---------------------------------------------------------------------- */
typedef struct expert_cache expert_cache;

size_t expert_cache_arena_bytes(int L, int E, int C, size_t blob_bytes, int n_stage);
int expert_cache_create(int L, int E, int C, size_t blob_bytes, int n_stage, void* arena,
                        size_t arena_bytes, const void* const* host_blobs, void* demand_stream,
                        void* side_stream, expert_cache** out);
int expert_cache_destroy(expert_cache* c);
/* Load the initial residency warm [L][C] (host, -1 = empty).  [sync] */
int expert_cache_warm(expert_cache* c, const int32_t* warm);
/* Issue prefetch copies on the side stream; returns the number of copies. */
int expert_cache_prefetch(expert_cache* c, int layer, const int32_t* ranked, int n,
                          int64_t stamp);
/* Link order of prefetch copies (Section 4.3.4 overlaps them with the
 * current layer's work; the paper leaves their order against the missed
 * loads open).  after_demand = 0 (default): they start when issued and share
 * the host link with demand copies still in flight.  1: they wait for the
 * demand copies of the latest acquire, so they only take the link once the
 * current layer's missed experts are in.  Which copies happen, and the
 * counts, do not change.  Returns STMOE_EINVAL for other values. */
int expert_cache_set_prefetch_order(expert_cache* c, int after_demand);
/* The cache's replacement rule, as stmoe_policy_set_counts (host decisions;
 * with device decisions the counts move to device memory and the decision
 * kernel keeps them, also under graph replay).  expert_cache_warm keeps the
 * rule and the counts.  [sync] with device decisions, [host] otherwise. */
int expert_cache_set_counts(expert_cache* c, const int64_t* counts);
/* Workgroups of the copy kernels that move experts with device decisions:
 * missed loads (default 64, enough to fill the host link) and prefetches
 * (default 16: fewer leave the concurrent FFN most of the chip); 0 restores
 * a default, values above 1024 return STMOE_EINVAL.  Fewer workgroups lower
 * the achieved copy rate (a throttled link for bandwidth sweeps); more raise
 * it for a pool in device memory.  Kept across device-policy switches; host
 * decisions copy with DMA and ignore it.  [host] */
int expert_cache_set_copy_workgroups(expert_cache* c, int demand, int prefetch);
/* Device-side decisions (Section 4.3.4's missed loading and prefetch
 * without a host round trip).  on = 1: the policy state moves to device
 * memory and moe_decode_layer takes its decisions in a one-workgroup kernel
 * from the routing and the prediction on the device: the same policy and
 * the same decisions and counts as the host path.  Missed experts are copied
 * by a copy kernel on the compute stream, prefetches by one on the side
 * stream; experts beyond the layer's slots (the host path's staging
 * overflow) are read by the FFN straight from host memory, so the staging
 * slots are not used.  Every pool blob must be device memory or pinned host
 * memory that the device maps at the same address (hipHostMalloc, torch
 * pin_memory); otherwise STMOE_EINVAL and nothing changes.  While on,
 * expert_cache_acquire / _prefetch / _warm return STMOE_ESTATE and
 * expert_cache_stats reads the device counters.  on = 0 moves the state
 * back to the host policy.  [sync] */
int expert_cache_set_device_policy(expert_cache* c, int on);
/* Staged prefetch (Section 4.1 prefetches predicted experts, Section 4.3.4
 * overlaps the transfer with computation).  n > 0: instead of evicting
 * slots, the next layer's admitted predicted experts that are not resident
 * (at most n, ranked order) are copied into spare staging blocks of the
 * arena (2n of the n_stage staging slots: two sets alternate between
 * consecutive layers) once the layer's missed loads are in.  At the next
 * layer's decisions a staged expert that was selected is used from its
 * block: when it takes a slot (the slot the missed load would take) the two
 * blocks swap places, with no copy; otherwise the FFN reads the staging
 * block.  Residency evolves exactly as with on-demand loading; counts:
 * prefetch = staged experts, useful = staged experts selected, wasted = the
 * others, demand and overflow = the other misses.
 *   Device decisions: the staged copy kernel stops an unselected copy at its
 *   next check once the next layer's decisions cancel it (head_bytes unused).
 *   Host decisions: the first head_bytes of each staged expert are copied
 *   (hipMemcpyAsync on the side stream) when it is staged, the rest only once
 *   the next layer selects it; head_bytes = 0 or >= the blob copies it whole.
 *   The remaining overflow ring is n_stage - 2n slots.
 * n = 0 returns to prefetching into slots.  Once staged prefetches have moved
 * slots to other arena blocks, switching between host and device decisions
 * returns STMOE_ESTATE (and, with host decisions, so does changing n until
 * expert_cache_warm reloads the cache).  STMOE_EINVAL if 2n > n_stage.
 * [sync] */
int expert_cache_set_staged_prefetch(expert_cache* c, int n_per_layer, size_t head_bytes);
/* Make `needed` (host, n distinct experts) resident for a kernel on
 * `compute`: demand copies on the demand stream, `compute` waits for every
 * copy it needs; dev_table_out (host [E]) receives the device blob pointer
 * of each needed expert (other entries untouched). */
int expert_cache_acquire(expert_cache* c, int layer, const int32_t* needed, int n,
                         int64_t stamp, const void** dev_table_out, void* compute);
/* Mark the slots handed out by the last acquire of `layer` as read by work
 * enqueued so far on `compute`. */
int expert_cache_release(expert_cache* c, int layer, void* compute);
int expert_cache_stats(const expert_cache* c, stmoe_cache_stats* out);

/* ------------------------------------------------------------------------
 * One decode-step MoE layer (Section 4.3.4): route, verify/update, predict
 * the next layer, fetch missed experts, expert FFN, prefetch the next
 * layer's predicted experts.
 * ---------------------------------------------------------------------- */
enum { MOE_MODE_ON_DEMAND = 0, MOE_MODE_STMOE = 1, MOE_MODE_HT_ONLY = 2, MOE_MODE_CCT_ONLY = 3 };

typedef struct {
    int L, E, K, B, H, I, n_shared, dtype, renorm;
    const void* const* router_w;   /* host [L] device pointers to W_g [E][H] */
    const void* const* shared_w;   /* host [L*n_shared] device blob pointers, or NULL */
    const void* const* resident_w; /* host [L*E] device blob pointers when every routed
                                      expert is in HBM (cache must then be NULL).  Read
                                      once at create: when every layer's E pointers are
                                      equally spaced (one stride for all layers), the FFN
                                      computes blob addresses from the layer's first
                                      pointer and the stride */
} moe_model_desc;

typedef struct moe_ctx moe_ctx;

/* Device bytes of a context's workspace: routing records, the routing and
 * FFN workspaces, expert pointer tables, the per-token predictor arguments
 * and the graph-replay staging buffers; 0 for an invalid description. */
size_t moe_ctx_workspace_bytes(const moe_model_desc* desc);
/* cache may be NULL only when desc->resident_w is given.  pred (if given)
 * and cache must have been created for the same L, E (and, for pred, K and
 * B) as desc, and the cache's blob size must hold one expert
 * (moe_blob_bytes(H, I, dtype)); otherwise STMOE_EINVAL.  dev_ws: device,
 * 256-byte aligned, at least moe_ctx_workspace_bytes(desc) bytes (zeroed
 * here).  [sync] */
int moe_ctx_create(const moe_model_desc* desc, stmoe_predictor* pred, expert_cache* cache,
                   void* compute_stream, void* dev_ws, size_t ws_bytes, moe_ctx** out);
int moe_ctx_destroy(moe_ctx* ctx);
/* One MoE layer for decode token `token`:
 *   x device [B][H] dtype; y device out [B][H] fp32.
 * With a cache, this call waits once on the host for the layer's routing
 * record (selected and predicted experts).  Without one it never waits, and
 * in the prediction modes the table update and the next layer's prediction
 * run on a stream of the context's own that waits for the layer's router
 * and overlaps the FFN (the compute stream waits for that stream once per
 * token, before selections it still reads are rewritten).  Layers are
 * expected in order 0..L-1 per token; other orders are correct but wait.
 * Layer-0 predictions come from HT[0]; the prefetch for layer 0 of the next
 * token is issued at layer L-1.
 * rep (host, or NULL): when given, the call waits for the layer's work on
 * every stream and fills the report below. */
typedef struct {
    int32_t B, K;
    int32_t idx[16 * 16];       /* [B][K] the layer's selection, descending logit */
    float w[16 * 16];           /* [B][K] its gate weights */
    int32_t n_ranked;           /* experts predicted for the next layer (score >= 2),
                                   -1 when the mode predicts nothing */
    int32_t ranked[256];        /* their ranking (max score over rows desc, index asc),
                                   -1 padding */
    int64_t pred_stats[3];      /* this layer's predictor statistics since profiling:
                                   sum |A n P|, sum |A|, sum |P| (0 without a predictor) */
    stmoe_cache_stats cache;    /* cache counters so far (0 without a cache) */
} moe_layer_report;
int moe_decode_layer(moe_ctx* ctx, int token, int layer, const void* x, float* y, int mode,
                     moe_layer_report* rep);
/* Prefetch admission (cache only).  A predicted expert is prefetched only if
 * its prediction score (max over rows, Eq. 1) is at least min_score, and at
 * most max_per_layer experts are prefetched per layer (the ranked order
 * decides which).  Defaults: min_score = 2 (the paper's threshold) and
 * max_per_layer = the cache's slots per layer. */
int moe_ctx_set_prefetch(moe_ctx* ctx, int min_score, int max_per_layer);
/* Online CCT update (Algorithm 3, Section 4.2) during decode: on (1, the
 * default) or frozen after profiling (0; HT rows are still overwritten with
 * each selection).  An ablation switch. */
int moe_ctx_set_online_update(moe_ctx* ctx, int on);
/* All L layers of one token: xs device [L][B][H], ys device out [L][B][H].
 * With graph replay on (moe_ctx_set_graph), every call after the first whose
 * token is not event-timed replays one HIP graph of the whole token: xs is
 * copied into the context's input staging buffer, the graph runs, and the
 * output staging buffer is copied to ys (a copy is skipped when the pointer
 * is the staging buffer itself).  The graph is captured at the first such
 * call and again when `mode`, a setting of the context (moe_ctx_set_prefetch,
 * moe_ctx_set_online_update) or the cache's configuration (warm start,
 * decision site, staged prefetch, prefetch order, replacement rule) has
 * changed since; results equal the eager calls. */
int moe_decode_token(moe_ctx* ctx, int token, const void* xs, float* ys, int mode);
/* Per-token predictor launches for moe_decode_token (contexts without a
 * cache, with a predictor; on = 1 or 0, default 0).  Without a cache the
 * prediction feeds no copy, so the verify/update of every layer and its
 * next-layer prediction (Algorithm 3, Eq. 1, in layer order) can run as one
 * side-stream launch after the token's last layer instead of one launch per
 * layer: the same tables and hit statistics, three host calls per token
 * instead of three per layer.  Each token's selections go to a buffer of its
 * parity, so the launch overlaps the next token; the compute stream waits
 * for it two tokens later.  moe_decode_layer keeps per-layer launches.
 * STMOE_EINVAL with a cache, without a predictor or with graph replay on.
 * [sync] */
int moe_ctx_set_predictor_batch(moe_ctx* ctx, int on);
/* Graph replay of moe_decode_token on (1) or off (0): contexts without a
 * cache, or with a cache whose decisions are on the device
 * (expert_cache_set_device_policy); a host-decision cache returns
 * STMOE_EINVAL here (and STMOE_ESTATE at a replay, if its decisions moved
 * back to the host).  With a cache the graph holds the whole token: routing,
 * predictor, the cache's decisions, its copy kernels and the side stream's
 * prefetch copies, which rejoin before the graph ends; the cache policy's
 * stamps come from a device copy of the token that each replay advances (an
 * eager call, or a replay for a token that does not follow the last one,
 * sets it first).  The staging buffers (L*B*H elements of the storage dtype
 * and L*B*H fp32) are part of the context's workspace; turning replay on
 * creates an internal stream.  The graph launch is ordered after earlier
 * work on the compute stream (and, with a cache, on its side stream) and
 * before later work on the compute stream by events.  [sync] */
int moe_ctx_set_graph(moe_ctx* ctx, int on);
/* The staging buffers of graph replay (device, owned by the context):
 * x_stage [L][B][H] storage dtype, y_stage [L][B][H] fp32.  Writing the
 * inputs there and passing these pointers avoids the two copies. */
int moe_ctx_graph_buffers(moe_ctx* ctx, void** x_stage, float** y_stage);
/* Last routing of each layer: host out idx [L][B][K] int32, w [L][B][K] fp32.  [sync] */
int moe_ctx_last_routing(moe_ctx* ctx, int32_t* idx, float* w);
/* Event timing of the expert-FFN kernels.  every > 0 starts recording (and
 * resets the totals): the FFN of every layer of each token whose index is a
 * multiple of `every` is bracketed by events on the compute stream (before,
 * between and after its two kernels); every = 0 stops.  moe_ctx_timing syncs
 * and returns the summed milliseconds of the gate/up kernel and of the down
 * kernel over the timed calls, the number of timed FFN calls and the summed
 * number of distinct routed experts over those calls. */
int moe_ctx_set_timing(moe_ctx* ctx, int every);
int moe_ctx_timing(moe_ctx* ctx, double* up_ms, double* down_ms, int64_t* n_calls,
                   int64_t* n_experts);
/* Stage times over the same timed layers (summed milliseconds, [sync]):
 *   route_ms    the routing launches (with a cache: router + update + predict)
 *   miss_ms     from routing to the FFN: the host's wait for the routing
 *               record and the missed-expert loads (0 without a cache)
 *   ffn_ms      both FFN kernels
 *   predict_ms  update + predict on the side stream (no cache; overlaps the
 *               FFN and the next layer's router, so it is not on the layer's
 *               critical path)
 * Any argument may be NULL. */
int moe_ctx_stage_timing(moe_ctx* ctx, double* route_ms, double* miss_ms, double* ffn_ms,
                         double* predict_ms, int64_t* n_calls);

/* ------------------------------------------------------------------------
 * Measurement kernels of known traffic (not part of the decode path).
 *   stmoe_calib_copy: dst[i] = src[i] over `bytes` (multiple of 16, 16-byte
 *     aligned): reads and writes exactly `bytes`; used to turn the
 *     FETCH_SIZE / WRITE_SIZE hardware counters into bytes.
 *   stmoe_calib_read: streams `bytes` with the expert FFN's non-temporal
 *     16-byte loads; out (device, stmoe_calib_read_out_words(bytes, pattern)
 *     words) receives one checksum word per workgroup.  pattern 0: a
 *     grid-stride sweep; 1: every workgroup reads one contiguous 256 KiB
 *     region (the way the FFN's workgroups read an expert's rows); 2: the
 *     same with 32 KiB regions, one round of eight loads per thread (the
 *     shortest time one launch needs to stream `bytes`).  Other patterns
 *     return STMOE_EINVAL.
 * ---------------------------------------------------------------------- */
int stmoe_calib_copy(const void* src, void* dst, size_t bytes, void* stream);
/* The same copy on `workgroups` workgroups (1..1024, else STMOE_EINVAL) with
 * the expert cache's copy-kernel access pattern (four 16-byte chunks in
 * flight per thread, non-temporal): the copy rate that workgroup count
 * reaches, from pinned host memory or device memory. */
int stmoe_calib_copy_grid(const void* src, void* dst, size_t bytes, int workgroups, void* stream);
size_t stmoe_calib_read_out_words(size_t bytes, int pattern);
int stmoe_calib_read(const void* src, size_t bytes, int pattern, unsigned* out, void* stream);
/* Handoff between workgroups, the step a single gate/up + down launch would
 * need (Section 2's FFN: the down projection reads every activation the
 * gate/up projection writes).  `producers` workgroups each read their chunk1
 * bytes of w1 (device, producers x chunk1, 16-byte aligned) and write one
 * word, the wrapping sum of the 32-bit words read, to act[p] (device
 * [producers]); `consumers` workgroups each read their chunk2 bytes of w2
 * (device, consumers x chunk2; chunk2 of 4, 8, 16, 24 or 32 KiB) into
 * registers and then write out[c] (device [consumers]) = the sum of those
 * words plus every act word.  mode 0: two launches (the kernel boundary
 * orders them).  modes 1-4: one launch of producers + consumers workgroups
 * whose consumers wait until the count of published producers, sync[0],
 * reaches `target` (the caller zeroes sync once and adds `producers` to the
 * target at every launch): 1 publishes with a write-through store and a
 * relaxed increment and every consumer polls sync[0]; 2 the same with a
 * release increment and acquire polls; 3 as 1, and the producer whose
 * increment reaches the target writes it to 64 flag words (sync[64 + 1024 r],
 * r < 64, on different memory channels), consumer c polling copy c mod 64;
 * 4 as 3, but producer p counts itself in group word sync[576 + 1024 (p mod
 * 64)], the last of each group in sync[2], and the last group (which sets
 * those words back to 0 and adds `producers` to sync[0]) writes the flags.
 * Modes 3 and 4 need at least STMOE_HANDOFF_SYNC_WORDS words of sync.  A
 * consumer that polls 32768 times in vain sets sync[1] (its output is then
 * not meaningful) instead of waiting on; producers take the lower workgroup
 * indices.  Every mode gives the same out.  Errors: STMOE_EINVAL. */
#define STMOE_HANDOFF_SYNC_WORDS (64 + 64 * 1024)
int stmoe_calib_handoff(const void* w1, size_t chunk1, int producers, const void* w2, size_t chunk2,
                        int consumers, int mode, unsigned* act, unsigned* out, unsigned* sync,
                        unsigned target, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* STMOE_H */
