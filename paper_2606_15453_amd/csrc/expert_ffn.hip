// Expert FFN of the decode-step MoE layer (Section 2; SwiGLU experts):
//   y[b] = sum over selected experts e of w[b][e] * W_down_e (silu(W_gate_e x_b) * (W_up_e x_b))
//        + the same with weight 1 for shared experts.
//
// Decode is bandwidth-bound (about 2 flops per weight byte per token), so
// every kernel here streams each selected expert's weights from HBM exactly
// once, as 16-byte non-temporal loads, and is priced against 8 TB/s.
//
// Two phases, two launches:
//   gate/up  one workgroup = (expert slot, block of rows of W_gate and W_up):
//            a[slot][b][i] = w_b * silu(W_gate[i] . x_b) * (W_up[i] . x_b)
//   down     sum over slots (ascending expert index, shared experts last)
//            of W_down_slot[h] . a[slot][b].  The GEMV kernels give each
//            workgroup a block of output rows and split the slots (or the row
//            length) over its four waves, combining them through LDS; the MFMA
//            kernel splits slots over workgroups into partial sums that a
//            third small kernel adds in group order.  No workgroup waits on
//            another (device-scope fences between workgroups would write back
//            the L2 of every XCD), and the summation order depends only on the
//            routing, never on where the blobs live.
//
// Batch < 8: GEMV kernels.  A group of G lanes (64, 32 or 16, by row length)
// owns R rows and strides over their 16-byte chunks; the activations come
// from L1/L2; DPP / shuffle segment sums reduce.  For long down rows the
// whole workgroup strides one row block (split-K over its four waves).
// Batch >= 8: MFMA kernels (v_mfma_f32_16x16x32_bf16).  The tokens form the
// 16-row A operand (padded with zeros), 16 weight rows the B operand.  In
// each 64-element step lane (n, q) loads elements 8q..8q+7 and 32+8q..32+8q+7
// of row n, so every load instruction reads 16 full 64-byte row segments.
// The SwiGLU activation goes through bf16.
//
// Every kernel rebuilds the slot plan (distinct selected experts ascending,
// token masks) from topk_idx/topk_w in LDS: no host round trip, no planning
// launch.
#include <mutex>
#include <type_traits>

#include "common.h"
#include "gating_dev.h"

// Workspace of moe_expert_ffn_noalloc: one copy per GPU, held until the
// process ends.  In host code this name is a stand-in, not a device address;
// the device address comes from hipGetSymbolAddress (see noalloc_scratch).
static __device__ __align__(256) unsigned char scratch[size_t(16) << 20];

namespace stmoe {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxShared = 8;
constexpr int kMaxSlots = kMaxE + kMaxShared;
constexpr int kDownWgTarget = 256;    // workgroups the MFMA down phase aims for
constexpr int kMfmaMinB = 8;          // batch from which the MFMA kernels run
constexpr int kUpInFlight = 2;        // 16-byte chunks per row in flight per lane (GEMV gate/up)
constexpr bool kUpB1 = true;           // batch 1: the gate/up kernel that finds its slot in registers
constexpr int kUpB1RouteMaxE = 128;    // ... and routes up to this many experts (in registers up to 64)
constexpr int kShortRowChunks = 4;    // down rows with at most this many chunks per lane are short: ...
constexpr int kDownInFlightShort = 4; // ... the lane-group down kernel loads a slot's chunks in one step
constexpr bool kStageX = true;        // GEMV gate/up: token activations staged in LDS ...
constexpr int kXStageMax = 32768;     // ... when B*H*esz fits in this many bytes
constexpr int kStageXMaskedFromNB = 4;  // ... and from this many token columns only the slot's tokens
constexpr int kDownInFlight = 2;      // ... per row per lane in the whole-workgroup down kernel
constexpr int kDownCarryMaxNB = 4;    // lane-group down, one row per group: activations loaded with the
                                      // weights up to this many tokens (more rows: the registers cost more)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct FfnArgs {
    const void* x;                   // [B][H]
    const int32_t* idx;              // [B][K]
    const float* w;                  // [B][K]
    const void* const* eptr;         // [E] device blob pointers
    const char* ebase;               // or, when not null, expert e's blob at ebase + e * estride
    size_t estride;
    const void* const* sptr;         // [n_shared] or null
    int B, K, H, I, E, n_shared;
    void* act;                       // [slots][B][I]: bf16 (MFMA; GEMV per act_bf16) or fp32
    float* part;                     // [ng][B][H] partial sums of the MFMA down phase (ng > 1)
    float* y;                        // [B][H]
    unsigned long long* n_experts;   // optional: += distinct routed experts (block 0)
    int ng, spg;                     // expert-slot groups of the down phase, slots per group
    // optional routing prologue of the gate/up kernels: softmax + top-K of
    // these router logits [B][E] (B*E <= kRouteInFfnMax); block 0 writes the
    // selection to idx/w for the down kernel and the caller
    const float* logits;
    int renorm;
};

struct Plan {
    int32_t idx[kMaxB * kMaxK];
    float w[kMaxB * kMaxK];
    unsigned sel[kMaxE / 32];
    int expert[kMaxSlots];           // routed slots: expert index; shared slots: -1 - s
    unsigned tok[kMaxSlots];         // token bit mask per slot
    int n_routed, n_slots;
};

// The plan of kernels whose waves walk many slots: each slot's blob pointer
// is resolved once while the plan is built, so a slot's first weight loads
// do not wait behind a table lookup.  Kernels that take one slot per
// workgroup keep the smaller plan (LDS decides their occupancy).
struct PlanB : Plan {
    const char* blob[kMaxSlots];
};

// Gating (Section 2) inside a gate/up workgroup: the same steps and
// arithmetic as the router tail, on rows of E rounded up to 4, into the
// plan's idx/w; block 0 also publishes them.
__device__ void route_into_plan(const FfnArgs& a, Plan& p) {
    constexpr int kRouteRows = kRouteInFfnMax + 3 * kMaxB;
    __shared__ __align__(16) uint32_t keys[kRouteRows];
    __shared__ float zl[kRouteRows];
    __shared__ int32_t win[kMaxB * kMaxK];
    __shared__ float rowmax[kMaxB];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int row = (a.E + 3) & ~3;
    gating::stage_keys(a.logits, a.B, a.E, row, keys, zl);
    gating::rank_winners(keys, zl, a.B, a.E, a.K, row, win, rowmax);
    for (int b = wave; b < a.B; b += kWaves) {
        int e;
        float wt;
        gating::row_weights(zl, win, rowmax, b, a.E, a.K, row, a.renorm, e, wt);
        if (lane < a.K) {
            p.idx[b * a.K + lane] = e;
            p.w[b * a.K + lane] = wt;
            if (blockIdx.x == 0) {
                const_cast<int32_t*>(a.idx)[b * a.K + lane] = e;
                const_cast<float*>(a.w)[b * a.K + lane] = wt;
            }
        }
    }
}

// Routed expert e's blob: computed from a base and stride where the caller's
// blobs are laid out that way (no dependent load from the pointer table).
__device__ __forceinline__ const char* routed_blob(const FfnArgs& a, int e) {
    return a.ebase ? a.ebase + size_t(e) * a.estride : reinterpret_cast<const char*>(a.eptr[e]);
}

// Build the slot plan in LDS (all threads participate; ends with a barrier).
// Slot order: selected routed experts ascending, then shared experts.  With
// `route` and router logits in the arguments the selection is computed here
// (gate/up kernels); otherwise it is read from idx/w.
template <class P>
__device__ void build_plan(const FfnArgs& a, P& p, bool route = false) {
    constexpr bool kBlobs = std::is_same<P, PlanB>::value;
    const int tid = threadIdx.x;
    const int BK = a.B * a.K;
    if (route && a.logits) {
        route_into_plan(a, p);
    } else {
        for (int t = tid; t < BK; t += kThreads) {
            const int e = a.idx[t];
            p.idx[t] = (e >= 0 && e < a.E) ? e : -1;   // out-of-range entries are ignored
            p.w[t] = a.w[t];
        }
    }
    if (tid < kMaxE / 32) p.sel[tid] = 0u;
    for (int s = tid; s < kMaxSlots; s += kThreads) p.tok[s] = 0u;
    __syncthreads();
    for (int t = tid; t < BK; t += kThreads)
        if (p.idx[t] >= 0) atomicOr(&p.sel[p.idx[t] >> 5], 1u << (p.idx[t] & 31));
    __syncthreads();
    int total = 0;
#pragma unroll
    for (int q = 0; q < kMaxE / 32; ++q) total += __popc(p.sel[q]);
    for (int t = tid; t < BK; t += kThreads) {
        const int e = p.idx[t], b = t / a.K;
        if (e < 0) continue;
        int rank = __popc(p.sel[e >> 5] & ((1u << (e & 31)) - 1u));
        for (int q = 0; q < (e >> 5); ++q) rank += __popc(p.sel[q]);
        atomicOr(&p.tok[rank], 1u << b);
        p.expert[rank] = e;
        if constexpr (kBlobs) p.blob[rank] = routed_blob(a, e);   // equal per rank
    }
    for (int s = tid; s < a.n_shared; s += kThreads) {
        p.expert[total + s] = -1 - s;
        if constexpr (kBlobs) p.blob[total + s] = reinterpret_cast<const char*>(a.sptr[s]);
        p.tok[total + s] = (1u << a.B) - 1u;
    }
    if (tid == 0) {
        p.n_routed = total;
        p.n_slots = total + a.n_shared;
    }
    __syncthreads();
}

// Gate weight of token b for slot j (1 for shared experts, 0 if not routed).
__device__ __forceinline__ float slot_weight(const FfnArgs& a, const Plan& p, int j, int b) {
    const int e = p.expert[j];
    if (e < 0) return 1.f;
    for (int k = 0; k < a.K; ++k)
        if (p.idx[b * a.K + k] == e) return p.w[b * a.K + k];
    return 0.f;
}

__device__ __forceinline__ const char* slot_blob(const FfnArgs& a, const Plan& p, int j) {
    const int e = p.expert[j];
    return e >= 0 ? routed_blob(a, e) : reinterpret_cast<const char*>(a.sptr[-1 - e]);
}
__device__ __forceinline__ const char* slot_blob(const FfnArgs&, const PlanB& p, int j) { return p.blob[j]; }

template <bool BF>
struct Chunk {
    static constexpr int N = BF ? 8 : 4;   // elements per 16 bytes
    float v[N];
    __device__ __forceinline__ void unpack(const uint4 q) {
        if constexpr (BF) {
            v[0] = bf16_lo(q.x); v[1] = bf16_hi(q.x); v[2] = bf16_lo(q.y); v[3] = bf16_hi(q.y);
            v[4] = bf16_lo(q.z); v[5] = bf16_hi(q.z); v[6] = bf16_lo(q.w); v[7] = bf16_hi(q.w);
        } else {
            v[0] = __uint_as_float(q.x); v[1] = __uint_as_float(q.y);
            v[2] = __uint_as_float(q.z); v[3] = __uint_as_float(q.w);
        }
    }
    __device__ __forceinline__ void load_f32(const float* p) {
#pragma unroll
        for (int q = 0; q < N / 4; ++q) {
            const float4 f = reinterpret_cast<const float4*>(p)[q];
            v[4 * q + 0] = f.x; v[4 * q + 1] = f.y; v[4 * q + 2] = f.z; v[4 * q + 3] = f.w;
        }
    }
};

// Dot product of a packed 16-byte weight chunk with an unpacked chunk,
// unpacking each weight as it is used (fewer live registers than unpacking
// R rows up front).
template <bool BF>
__device__ __forceinline__ float dotq(const uint4& w, const Chunk<BF>& x, float acc) {
    if constexpr (BF) {
        acc = fmaf(bf16_lo(w.x), x.v[0], acc); acc = fmaf(bf16_hi(w.x), x.v[1], acc);
        acc = fmaf(bf16_lo(w.y), x.v[2], acc); acc = fmaf(bf16_hi(w.y), x.v[3], acc);
        acc = fmaf(bf16_lo(w.z), x.v[4], acc); acc = fmaf(bf16_hi(w.z), x.v[5], acc);
        acc = fmaf(bf16_lo(w.w), x.v[6], acc); acc = fmaf(bf16_hi(w.w), x.v[7], acc);
    } else {
        acc = fmaf(__uint_as_float(w.x), x.v[0], acc); acc = fmaf(__uint_as_float(w.y), x.v[1], acc);
        acc = fmaf(__uint_as_float(w.z), x.v[2], acc); acc = fmaf(__uint_as_float(w.w), x.v[3], acc);
    }
    return acc;
}

template <bool BF>
__device__ __forceinline__ float dotc(const Chunk<BF>& w, const Chunk<BF>& x, float acc) {
#pragma unroll
    for (int i = 0; i < Chunk<BF>::N; ++i) acc = fmaf(w.v[i], x.v[i], acc);
    return acc;
}

// Weight rows are addressed through pointers read from memory (expert
// tables, the slot plan), which the compiler cannot place in an address
// space: loads through them would be FLAT instructions, which count against
// the LDS wait counter too, so every LDS read behind them would wait for all
// weight loads in flight.  They point into device memory: say so.
typedef const __attribute__((address_space(1))) u32x4 gu32x4;
__device__ __forceinline__ gu32x4* gmem(const char* p) { return (gu32x4*)(p); }

__device__ __forceinline__ uint4 ld_stream(const char* p) {
    const u32x4 v = __builtin_nontemporal_load(gmem(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint4 ld_cached(const char* p) {
    const u32x4 v = *gmem(p);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ bf16x8 ld_bf8_stream(const char* p) {
    return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(gmem(p)));
}
__device__ __forceinline__ bf16x8 ld_bf8(const char* p) {
    return __builtin_bit_cast(bf16x8, *gmem(p));
}

// Sum over a segment of G consecutive lanes (G = 16, 32 or 64); every lane
// of the segment returns the segment's sum.
template <int G>
__device__ __forceinline__ float seg_sum(float v) {
    if constexpr (G == 64) {
        return wave_sum(v);
    } else {
#pragma unroll
        for (int o = G / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
        return v;
    }
}

__device__ __forceinline__ float silu(float g) { return g / (1.f + expf(-g)); }

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return uint16_t((u + (((u >> 16) & 1u) + 0x7fffu)) >> 16);
}

// The SwiGLU activations of the GEMV path are stored as bf16 (rounded to
// nearest even, as the MFMA path does) where the down kernel reading them
// has the registers to unpack them (see act_bf16): one 16-byte chunk of
// bf16 activations then matches one 16-byte chunk of a W_down row, and every
// down workgroup, which re-reads them all, moves half the bytes.
__device__ __forceinline__ void store_act(void* act, int act16, size_t i, float v) {
    if (act16) reinterpret_cast<uint16_t*>(act)[i] = f32_to_bf16_rne(v);
    else reinterpret_cast<float*>(act)[i] = v;
}

// ============================================================================
// GEMV path (batch < 8)
// ============================================================================

// XL: the B token rows of x are staged in LDS (dynamic shared memory of
// B*H*esz bytes) by the whole workgroup, their loads issued before the
// routing prologue so both latencies overlap; every wave then reads x from
// LDS instead of L1/L2.
template <bool BF, int G, int R, int NB, bool XL>
__global__ __launch_bounds__(kThreads) void ffn_gate_up(FfnArgs a, int blocks_per_slot, int act16) {
    __shared__ Plan p;
    extern __shared__ uint4 x_lds[];
    constexpr int esz = BF ? 2 : 4;
    constexpr int kXRegs = kXStageMax / 16 / kThreads;
    // few token columns: every token, loads issued before the routing
    // prologue; more: only the tokens routed to this workgroup's slot
    // (typically one or two), after the plan names them
    constexpr bool kMasked = XL && NB >= kStageXMaskedFromNB;
    const int nx = XL ? a.B * a.H * esz / 16 : 0;
    const int cpx = a.H * esz / 16;
    const char* xsrc = reinterpret_cast<const char*>(a.x);
    uint4 xr[kXRegs];
    if (XL && !kMasked) {
#pragma unroll
        for (int u = 0; u < kXRegs; ++u) {
            const int i = u * kThreads + int(threadIdx.x);
            if (i < nx) xr[u] = ld_cached(xsrc + size_t(i) * 16);
        }
    }
    build_plan(a, p, true);
    const int j = blockIdx.x / blocks_per_slot;
    if (XL) {
        const unsigned tx = kMasked ? (j < p.n_slots ? p.tok[j] : 0u) : ~0u;
        if (kMasked) {
#pragma unroll
            for (int u = 0; u < kXRegs; ++u) {
                const int i = u * kThreads + int(threadIdx.x);
                if (i < nx && ((tx >> (i / cpx)) & 1u)) xr[u] = ld_cached(xsrc + size_t(i) * 16);
            }
        }
#pragma unroll
        for (int u = 0; u < kXRegs; ++u) {
            const int i = u * kThreads + int(threadIdx.x);
            if (i < nx && ((tx >> (i / cpx)) & 1u)) x_lds[i] = xr[u];
        }
        __syncthreads();
    }
    if (j >= p.n_slots) return;
    const int rows_per_block = kWaves * (64 / G) * R;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int grp = lane / G, g = lane % G;
    const int i0 = (blockIdx.x % blocks_per_slot) * rows_per_block + (wave * (64 / G) + grp) * R;
    if (i0 >= a.I) return;   // I is a multiple of R: the group's rows are all valid
    const unsigned tm = p.tok[j];
    const size_t rowb = size_t(a.H) * esz;
    const char* blob = slot_blob(a, p, j);
    const char* wg = blob + size_t(i0) * rowb;
    const char* wu = blob + size_t(a.I) * rowb + size_t(i0) * rowb;
    const char* xs = reinterpret_cast<const char*>(a.x);
    const int cpr = int(rowb / 16);

    float accg[R][NB], accu[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) accg[r][b] = accu[r][b] = 0.f;

    auto compute = [&](int c, const uint4 (&qg)[R], const uint4 (&qu)[R]) {
        Chunk<BF> cg[R], cu[R];
#pragma unroll
        for (int r = 0; r < R; ++r) { cg[r].unpack(qg[r]); cu[r].unpack(qu[r]); }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (!((tm >> b) & 1u)) continue;
            Chunk<BF> cx;
            cx.unpack(XL ? x_lds[b * cpr + c] : ld_cached(xs + b * rowb + size_t(c) * 16));
#pragma unroll
            for (int r = 0; r < R; ++r) {
                accg[r][b] = dotc<BF>(cg[r], cx, accg[r][b]);
                accu[r][b] = dotc<BF>(cu[r], cx, accu[r][b]);
            }
        }
    };
    // U chunks per row in flight; the fewer than U left over go in one
    // guarded step.  Chunks are summed in ascending order either way.
    constexpr int U = kUpInFlight;
    int c = g;
    for (; c + (U - 1) * G < cpr; c += U * G) {
        uint4 qg[U][R], qu[U][R];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r) {
                qg[u][r] = ld_stream(wg + r * rowb + size_t(c + u * G) * 16);
                qu[u][r] = ld_stream(wu + r * rowb + size_t(c + u * G) * 16);
            }
#pragma unroll
        for (int u = 0; u < U; ++u) compute(c + u * G, qg[u], qu[u]);
    }
    if (c < cpr) {
        uint4 qg[U][R], qu[U][R];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * G < cpr)
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    qg[u][r] = ld_stream(wg + r * rowb + size_t(c + u * G) * 16);
                    qu[u][r] = ld_stream(wu + r * rowb + size_t(c + u * G) * 16);
                }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * G < cpr) compute(c + u * G, qg[u], qu[u]);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (!((tm >> b) & 1u)) continue;
        const float wb = slot_weight(a, p, j, b);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float gs = seg_sum<G>(accg[r][b]);
            const float us = seg_sum<G>(accu[r][b]);
            if (g == 0) store_act(a.act, act16, (size_t(j) * a.B + b) * a.I + i0 + r, wb * silu(gs) * us);
        }
    }
}

// gate/up, whole workgroup per block of R rows: the 256 lanes stride the
// rows' chunks together (every lane issues all its loads of an iteration at
// once), then the four waves' sums combine through LDS.
template <bool BF, int R, int NB>
__global__ __launch_bounds__(kThreads) void ffn_gate_up_wg(FfnArgs a, int blocks_per_slot, int act16) {
    __shared__ Plan p;
    __shared__ float red[kWaves][2][R][NB];
    build_plan(a, p, true);
    const int j = blockIdx.x / blocks_per_slot;
    if (j >= p.n_slots) return;
    const int i0 = (blockIdx.x % blocks_per_slot) * R;
    if (i0 >= a.I) return;   // I is a multiple of R
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const unsigned tm = p.tok[j];
    constexpr int esz = BF ? 2 : 4;
    const size_t rowb = size_t(a.H) * esz;
    const char* blob = slot_blob(a, p, j);
    const char* wg = blob + size_t(i0) * rowb;
    const char* wu = blob + size_t(a.I) * rowb + size_t(i0) * rowb;
    const char* xs = reinterpret_cast<const char*>(a.x);
    const int cpr = int(rowb / 16);

    float accg[R][NB], accu[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) accg[r][b] = accu[r][b] = 0.f;

    auto compute = [&](int c, const uint4 (&qg)[R], const uint4 (&qu)[R]) {
        Chunk<BF> cg[R], cu[R];
#pragma unroll
        for (int r = 0; r < R; ++r) { cg[r].unpack(qg[r]); cu[r].unpack(qu[r]); }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (!((tm >> b) & 1u)) continue;
            Chunk<BF> cx;
            cx.unpack(ld_cached(xs + b * rowb + size_t(c) * 16));
#pragma unroll
            for (int r = 0; r < R; ++r) {
                accg[r][b] = dotc<BF>(cg[r], cx, accg[r][b]);
                accu[r][b] = dotc<BF>(cu[r], cx, accu[r][b]);
            }
        }
    };
    int c = tid;
    for (; c + kThreads < cpr; c += 2 * kThreads) {
        uint4 ga[R], ua[R], gb[R], ub[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            ga[r] = ld_stream(wg + r * rowb + size_t(c) * 16);
            ua[r] = ld_stream(wu + r * rowb + size_t(c) * 16);
            gb[r] = ld_stream(wg + r * rowb + size_t(c + kThreads) * 16);
            ub[r] = ld_stream(wu + r * rowb + size_t(c + kThreads) * 16);
        }
        compute(c, ga, ua);
        compute(c + kThreads, gb, ub);
    }
    if (c < cpr) {
        uint4 ga[R], ua[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            ga[r] = ld_stream(wg + r * rowb + size_t(c) * 16);
            ua[r] = ld_stream(wu + r * rowb + size_t(c) * 16);
        }
        compute(c, ga, ua);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (!((tm >> b) & 1u)) continue;
            const float gs = wave_sum(accg[r][b]);
            const float us = wave_sum(accu[r][b]);
            if (lane == 0) { red[wave][0][r][b] = gs; red[wave][1][r][b] = us; }
        }
    __syncthreads();
    if (tid < R * NB) {
        const int r = tid / NB, b = tid % NB;
        if ((tm >> b) & 1u) {
            float gs = 0.f, us = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) { gs += red[w][0][r][b]; us += red[w][1][r][b]; }
            store_act(a.act, act16, (size_t(j) * a.B + b) * a.I + i0 + r, slot_weight(a, p, j, b) * silu(gs) * us);
        }
    }
}

// ---------------------------------------------------------------- batch 1
// One token: every routed slot serves it, so the slot plan reduces to the
// selection ordered by expert index.  The batch-1 gate/up kernel finds its
// slot in registers, each wave on its own (no LDS plan; with the selection
// given or up to 64 experts to route, no barrier either), and loads the
// token's activation chunks beside the weight chunks; chunks are summed in
// the lane-group kernel's order, so the activations are bit-identical to
// that kernel's.

// Value of lane `src` (uniform) of v: a scalar read, no LDS traffic.
__device__ __forceinline__ int lane_i(int v, int src) { return __builtin_amdgcn_readlane(v, src); }
__device__ __forceinline__ float lane_f(float v, int src) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
}

// n-th set bit (n >= 0) of a uniform 64-bit mask, or -1.
__device__ __forceinline__ int nth_bit(unsigned long long m, int n) {
    for (int q = 0; q < n && m; ++q) m &= m - 1ull;
    return m ? __ffsll(m) - 1 : -1;
}

// Selection given: lane k < K holds idx[k].  Slots are the row's distinct
// valid experts ascending; a repeated expert takes the weight of its first
// entry (build_plan and slot_weight do the same).  Returns slot j's expert
// (or -1 when j is not a routed slot) and the routed slot count.
__device__ __forceinline__ int b1_given(const FfnArgs& a, int j, float& wj, int& n_routed) {
    const int K = a.K, lane = threadIdx.x & 63;
    int v = -1;
    float wv = 0.f;
    if (lane < K) {
        v = a.idx[lane];
        wv = a.w[lane];
    }
    const bool valid = lane < K && v >= 0 && v < a.E;
    bool first = valid;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) first &= !(r < lane && lane_i(v, r) == v);
    const unsigned long long fm = __ballot(first);
    int place = 0;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) place += ((fm >> r) & 1ull) && lane_i(v, r) < v;
    n_routed = __popcll(fm);
    if (j >= n_routed) return -1;
    const int src = __ffsll(__ballot(first && place == j)) - 1;
    wj = lane_f(wv, src);
    return lane_i(v, src);
}

// Router logits given (used up to 64 experts, correct up to 128): the router
// tail's softmax / top-K in registers, lanes f and f + 64 holding expert f
// and f + 64.  The same order
// keys and the same count of the keys that beat each expert (larger key, or
// equal key at a lower index) give the same winners; the softmax sum takes
// each lane's terms in the tail's order into the same wave sum, and lane k
// holds the probability of the position-k winner as in the tail, so the
// weights are bit-identical too.  Block 0 publishes idx/w.
__device__ __forceinline__ int b1_routed(const FfnArgs& a, int j, float& wj, int& n_routed) {
    const int E = a.E, K = a.K, lane = threadIdx.x & 63;
    const float z0 = lane < E ? a.logits[lane] : 0.f;
    const float z1 = lane + 64 < E ? a.logits[lane + 64] : 0.f;
    const uint32_t k0 = lane < E ? gating::order_key(z0) : 0u;
    const uint32_t k1 = lane + 64 < E ? gating::order_key(z1) : 0u;
    int c0 = 0, c1 = 0;
    const int e0 = E < 64 ? E : 64;
#pragma unroll 8
    for (int g = 0; g < e0; ++g) {
        const uint32_t kg = uint32_t(lane_i(int(k0), g));
        c0 += kg > k0 || (kg == k0 && g < lane);
        c1 += kg > k1;
    }
#pragma unroll 8
    for (int g = 64; g < E; ++g) {
        const uint32_t kg = uint32_t(lane_i(int(k1), g - 64));
        c0 += kg > k0;
        c1 += kg > k1 || (kg == k1 && g < lane + 64);
    }
    const bool w0 = lane < E && c0 < K, w1 = lane + 64 < E && c1 < K;
    const unsigned long long W0 = __ballot(w0), W1 = __ballot(w1);
    // the row max is the logit of the position-0 winner
    const unsigned long long t0 = __ballot(w0 && c0 == 0), t1 = __ballot(w1 && c1 == 0);
    const float m = t0 ? lane_f(z0, __ffsll(t0) - 1) : lane_f(z1, __ffsll(t1) - 1);
    float s = 0.f;
    if (lane < E) s += expf(z0 - m);
    if (lane + 64 < E) s += expf(z1 - m);
    s = wave_sum(s);
    // lane k < K: expert and probability of the position-k winner
    int ek = 0;
    for (int k = 0; k < K; ++k) {
        const unsigned long long q0 = __ballot(w0 && c0 == k), q1 = __ballot(w1 && c1 == k);
        const int f = q0 ? __ffsll(q0) - 1 : 64 + __ffsll(q1) - 1;
        if (lane == k) ek = f;
    }
    const float zk0 = __shfl(z0, ek & 63, 64), zk1 = __shfl(z1, ek & 63, 64);
    float p = 0.f;
    if (lane < K) p = expf((ek < 64 ? zk0 : zk1) - m) / s;
    const float wsum = wave_sum(p);
    const float wt = a.renorm ? p / wsum : p;
    if (blockIdx.x == 0 && threadIdx.x < K) {
        const_cast<int32_t*>(a.idx)[lane] = ek;
        const_cast<float*>(a.w)[lane] = wt;
    }
    n_routed = __popcll(W0) + __popcll(W1);
    if (j >= n_routed) return -1;
    const int n0 = __popcll(W0);
    const int e = j < n0 ? nth_bit(W0, j) : 64 + nth_bit(W1, j - n0);
    const int pos = e < 64 ? lane_i(c0, e) : lane_i(c1, e - 64);
    wj = lane_f(wt, pos);
    return e;
}

// Router logits given, 64 < E <= 128: too many experts for every wave to
// rank on its own, so the workgroup runs the lane-group kernel's gating
// (route_into_plan: the router tail's steps, bit-identical) and only skips
// the slot plan after it: slot j is the j-th smallest of the K winners,
// found in registers.
__device__ __forceinline__ int b1_routed_lds(const FfnArgs& a, int j, float& wj, int& n_routed, Plan& p) {
    const int K = a.K, lane = threadIdx.x & 63;
    route_into_plan(a, p);
    __syncthreads();
    const int ek = lane < K ? p.idx[lane] : 0;
    const float wk = lane < K ? p.w[lane] : 0.f;
    n_routed = K;
    if (j >= K) return -1;
    int place = 0;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) place += r < K && lane_i(ek, r) < ek;
    const int src = __ffsll(__ballot(lane < K && place == j)) - 1;
    wj = lane_f(wk, src);
    return lane_i(ek, src);
}

template <bool BF, int G, int R>
__global__ __launch_bounds__(kThreads) void ffn_gate_up_b1(FfnArgs a, int blocks_per_slot, int act16) {
    constexpr int esz = BF ? 2 : 4;
    constexpr int U = kUpInFlight;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = blockIdx.x / blocks_per_slot;
    __shared__ Plan p;
    float wj = 1.f;
    int n_routed = 0;
    const int e = !a.logits      ? b1_given(a, j, wj, n_routed)
                  : a.E <= 64    ? b1_routed(a, j, wj, n_routed)
                                 : b1_routed_lds(a, j, wj, n_routed, p);
    const char* blob;
    if (e >= 0) {
        blob = routed_blob(a, e);
    } else if (j < n_routed + a.n_shared) {
        wj = 1.f;
        blob = reinterpret_cast<const char*>(a.sptr[j - n_routed]);
    } else {
        return;
    }
    const int grp = lane / G, g = lane % G;
    const int i0 = (blockIdx.x % blocks_per_slot) * (kWaves * (64 / G) * R) + (wave * (64 / G) + grp) * R;
    if (i0 >= a.I) return;   // I is a multiple of R
    const size_t rowb = size_t(a.H) * esz;
    const char* wg = blob + size_t(i0) * rowb;
    const char* wu = blob + size_t(a.I) * rowb + size_t(i0) * rowb;
    const char* xs = reinterpret_cast<const char*>(a.x);
    const int cpr = int(rowb / 16);
    float accg[R], accu[R];
#pragma unroll
    for (int r = 0; r < R; ++r) accg[r] = accu[r] = 0.f;
    auto compute = [&](const uint4 (&qg)[R], const uint4 (&qu)[R], const uint4& qx) {
        Chunk<BF> cx;
        cx.unpack(qx);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            Chunk<BF> cg, cu;
            cg.unpack(qg[r]);
            cu.unpack(qu[r]);
            accg[r] = dotc<BF>(cg, cx, accg[r]);
            accu[r] = dotc<BF>(cu, cx, accu[r]);
        }
    };
    int c = g;
    for (; c + (U - 1) * G < cpr; c += U * G) {
        uint4 qg[U][R], qu[U][R], qx[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int r = 0; r < R; ++r) {
                qg[u][r] = ld_stream(wg + r * rowb + size_t(c + u * G) * 16);
                qu[u][r] = ld_stream(wu + r * rowb + size_t(c + u * G) * 16);
            }
            qx[u] = ld_cached(xs + size_t(c + u * G) * 16);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) compute(qg[u], qu[u], qx[u]);
    }
    if (c < cpr) {
        uint4 qg[U][R], qu[U][R], qx[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * G < cpr) {
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    qg[u][r] = ld_stream(wg + r * rowb + size_t(c + u * G) * 16);
                    qu[u][r] = ld_stream(wu + r * rowb + size_t(c + u * G) * 16);
                }
                qx[u] = ld_cached(xs + size_t(c + u * G) * 16);
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * G < cpr) compute(qg[u], qu[u], qx[u]);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float gs = seg_sum<G>(accg[r]);
        const float us = seg_sum<G>(accu[r]);
        if (g == 0) store_act(a.act, act16, size_t(j) * a.I + i0 + r, wj * silu(gs) * us);
    }
}

// One slot's contribution to R down rows: chunk steps c0, c0 + S, ... of
// the rows, U steps in flight.  With CARRY the activation chunks of the
// slot's tokens are loaded together with the weight chunks, so a step costs
// one memory round trip; otherwise they are loaded when the step is summed
// (after its weights have arrived: two round trips, fewer registers).
template <bool BF, int R, int NB, int U, bool CARRY>
__device__ __forceinline__ void down_slot(const char* wd, size_t rowb, int cpr, int c0, int S,
                                          const float* act, int B, int I, unsigned tm,
                                          float (&acc)[R][NB]) {
    constexpr int N = Chunk<BF>::N;
    constexpr int NX = N / 4;                  // float4 per chunk and token
    constexpr int NBX = CARRY ? NB : 1;
    const float4* act4 = reinterpret_cast<const float4*>(act);
    auto load_x = [&](int c, float4 (&xv)[NBX][NX]) {
        if constexpr (CARRY) {
#pragma unroll
            for (int b = 0; b < NB; ++b)
                if ((tm >> b) & 1u)
#pragma unroll
                    for (int q = 0; q < NX; ++q) xv[b][q] = act4[(size_t(b) * I + size_t(c) * N) / 4 + q];
        }
    };
    auto compute = [&](int c, const uint4 (&w)[R], const float4 (&xv)[NBX][NX]) {
        Chunk<BF> cw[R];
#pragma unroll
        for (int r = 0; r < R; ++r) cw[r].unpack(w[r]);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (!((tm >> b) & 1u)) continue;
            Chunk<BF> cx;
            if constexpr (CARRY) {
#pragma unroll
                for (int q = 0; q < NX; ++q) {
                    cx.v[4 * q + 0] = xv[b][q].x; cx.v[4 * q + 1] = xv[b][q].y;
                    cx.v[4 * q + 2] = xv[b][q].z; cx.v[4 * q + 3] = xv[b][q].w;
                }
            } else {
                cx.load_f32(act + size_t(b) * I + c * N);
            }
#pragma unroll
            for (int r = 0; r < R; ++r) acc[r][b] = dotc<BF>(cw[r], cx, acc[r][b]);
        }
    };
    int c = c0;
    for (; c + (U - 1) * S < cpr; c += U * S) {
        uint4 q[U][R];
        float4 xv[U][NBX][NX];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r) q[u][r] = ld_stream(wd + r * rowb + size_t(c + u * S) * 16);
#pragma unroll
        for (int u = 0; u < U; ++u) load_x(c + u * S, xv[u]);
#pragma unroll
        for (int u = 0; u < U; ++u) compute(c + u * S, q[u], xv[u]);
    }
    if (c < cpr) {      // fewer than U steps left: one guarded step
        uint4 q[U][R];
        float4 xv[U][NBX][NX];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * S < cpr)
#pragma unroll
                for (int r = 0; r < R; ++r) q[u][r] = ld_stream(wd + r * rowb + size_t(c + u * S) * 16);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * S < cpr) load_x(c + u * S, xv[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * S < cpr) compute(c + u * S, q[u], xv[u]);
    }
}

// down_slot for bf16 activations (16 bytes per chunk and token, the same
// chunk layout as a W_down row; weights unpacked as they are used).  With
// TOKENS (and no CARRY) the step's weight chunks are loaded first and then,
// token by token, all of that token's activation chunks of the step
// together: one wait per token instead of one per chunk (an activation load
// waits for every load issued before it).  Every accumulator still adds its
// chunks in ascending order, so the order of the token loop does not change a
// sum.  Lane-group kernel, DeepSeek-V2-Lite shapes at batch 4: 30.6 -> 29.2 us
// per launch; the whole-workgroup kernel (Mixtral shapes) keeps the per-chunk
// loads, about 1% faster there.
template <bool BF, int R, int NB, int U, bool CARRY, bool TOKENS = false>
__device__ __forceinline__ void down_slot16(const char* wd, size_t rowb, int cpr, int c0, int S,
                                            const char* act, unsigned tm, float (&acc)[R][NB]) {
    static_assert(BF, "bf16 activations go with bf16 weights");
    constexpr int NBX = CARRY ? NB : 1;
    // token b's activation row: rowb bytes, like a W_down row
    auto load_x = [&](int c, uint4 (&xv)[NBX]) {
        if constexpr (CARRY) {
#pragma unroll
            for (int b = 0; b < NB; ++b)
                if ((tm >> b) & 1u) xv[b] = ld_cached(act + size_t(b) * rowb + size_t(c) * 16);
        }
    };
    auto compute = [&](int c, const uint4 (&w)[R], const uint4 (&xv)[NBX]) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (!((tm >> b) & 1u)) continue;
            Chunk<BF> cx;
            if constexpr (CARRY) cx.unpack(xv[b]);
            else cx.unpack(ld_cached(act + size_t(b) * rowb + size_t(c) * 16));
#pragma unroll
            for (int r = 0; r < R; ++r) acc[r][b] = dotq<BF>(w[r], cx, acc[r][b]);
        }
    };
    // TOKENS: token-outer over a step whose weights are in registers
    auto tokens = [&](int c, const uint4 (&q)[U][R], bool guarded) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (!((tm >> b) & 1u)) continue;
            uint4 xv[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (!guarded || c + u * S < cpr) xv[u] = ld_cached(act + size_t(b) * rowb + size_t(c + u * S) * 16);
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (!guarded || c + u * S < cpr) {
                    Chunk<BF> cx;
                    cx.unpack(xv[u]);
#pragma unroll
                    for (int r = 0; r < R; ++r) acc[r][b] = dotq<BF>(q[u][r], cx, acc[r][b]);
                }
        }
    };
    int c = c0;
    for (; c + (U - 1) * S < cpr; c += U * S) {
        uint4 q[U][R];
        uint4 xv[U][NBX];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r) q[u][r] = ld_stream(wd + r * rowb + size_t(c + u * S) * 16);
        if constexpr (TOKENS && !CARRY) {
            tokens(c, q, false);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) load_x(c + u * S, xv[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) compute(c + u * S, q[u], xv[u]);
        }
    }
    if (c < cpr) {      // fewer than U steps left: one guarded step
        uint4 q[U][R];
        uint4 xv[U][NBX];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c + u * S < cpr)
#pragma unroll
                for (int r = 0; r < R; ++r) q[u][r] = ld_stream(wd + r * rowb + size_t(c + u * S) * 16);
        if constexpr (TOKENS && !CARRY) {
            tokens(c, q, true);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (c + u * S < cpr) load_x(c + u * S, xv[u]);
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (c + u * S < cpr) compute(c + u * S, q[u], xv[u]);
        }
    }
}

// Down, rows owned by lane groups: every wave covers the workgroup's rows
// (R per lane group); the four waves split the slots (wave w takes slots w,
// w+4, ...) and their sums are added in wave order through LDS.  Each
// activation chunk a lane loads serves its R rows: every workgroup reads all
// activations, so R sets how much L2 traffic the weight rows carry along.
template <bool BF, int G, int R, int NB, int U>
__global__ __launch_bounds__(kThreads) void ffn_down_rows(FfnArgs a) {
    constexpr int kRows = (64 / G) * R;
    __shared__ PlanB p;
    __shared__ float red[kWaves][kRows][NB];
    build_plan(a, p);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lg = lane / G, g = lane % G;
    const int hb = blockIdx.x * kRows;
    const int h0 = hb + lg * R;
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.n_experts)
        atomicAdd(a.n_experts, (unsigned long long)p.n_routed);
    const bool live = h0 < a.H;   // H is a multiple of R
    constexpr int esz = BF ? 2 : 4;
    constexpr int N = Chunk<BF>::N;
    const size_t rowb = size_t(a.I) * esz;
    const int cpr = int(rowb / 16);

    float acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[r][b] = 0.f;

    for (int j = wave; live && j < p.n_slots; j += kWaves) {
        if constexpr (BF && R < 4)
            down_slot16<BF, R, NB, U, (R == 1 && NB <= kDownCarryMaxNB), true>(
                slot_blob(a, p, j) + 2 * size_t(a.I) * a.H * esz + size_t(h0) * rowb, rowb, cpr, g, G,
                reinterpret_cast<const char*>(a.act) + size_t(j) * a.B * rowb, p.tok[j], acc);
        else
            down_slot<BF, R, NB, U, (R == 1 && NB <= kDownCarryMaxNB)>(
                slot_blob(a, p, j) + 2 * size_t(a.I) * a.H * esz + size_t(h0) * rowb, rowb, cpr, g, G,
                reinterpret_cast<const float*>(a.act) + size_t(j) * a.B * a.I, a.B, a.I, p.tok[j], acc);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float s = seg_sum<G>(acc[r][b]);
            if (g == 0) red[wave][lg * R + r][b] = s;
        }
    __syncthreads();
    for (int t = threadIdx.x; t < kRows * NB; t += kThreads) {
        const int q = t / NB, b = t % NB, h = hb + q;
        if (b < a.B && h < a.H) {
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) s += red[w][q][b];
            a.y[size_t(b) * a.H + h] = s;
        }
    }
}

// Down, long rows: the whole workgroup strides one block of R rows (split-K
// over the four waves) for every slot, then combines the waves' sums
// through LDS.
template <bool BF, int R, int NB>
__global__ __launch_bounds__(kThreads) void ffn_down_wg(FfnArgs a) {
    __shared__ PlanB p;
    __shared__ float red[kWaves][R][NB];
    build_plan(a, p);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h0 = blockIdx.x * R;   // H is a multiple of R
    if (blockIdx.x == 0 && tid == 0 && a.n_experts)
        atomicAdd(a.n_experts, (unsigned long long)p.n_routed);
    constexpr int esz = BF ? 2 : 4;
    constexpr int N = Chunk<BF>::N;
    const size_t rowb = size_t(a.I) * esz;
    const int cpr = int(rowb / 16);

    float acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[r][b] = 0.f;

    for (int j = 0; j < p.n_slots; ++j) {
        const char* wd = slot_blob(a, p, j) + 2 * size_t(a.I) * a.H * esz + size_t(h0) * rowb;
        if constexpr (BF && NB <= 2)
            down_slot16<BF, R, NB, kDownInFlight, false>(
                wd, rowb, cpr, tid, kThreads, reinterpret_cast<const char*>(a.act) + size_t(j) * a.B * rowb,
                p.tok[j], acc);
        else
            down_slot<BF, R, NB, kDownInFlight, false>(
                wd, rowb, cpr, tid, kThreads, reinterpret_cast<const float*>(a.act) + size_t(j) * a.B * a.I,
                a.B, a.I, p.tok[j], acc);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const float s = wave_sum(acc[r][b]);
            if (lane == 0) red[wave][r][b] = s;
        }
    __syncthreads();
    if (tid < R * NB) {
        const int r = tid / NB, b = tid % NB;
        if (b < a.B) {
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) s += red[w][r][b];
            a.y[size_t(b) * a.H + h0 + r] = s;
        }
    }
}

// ============================================================================
// MFMA path (batch >= 8, bf16, H and I multiples of 64)
// ============================================================================

// gate/up: each wave computes NT tiles of 16 rows x 16 tokens for W_gate and
// W_up over the whole hidden dimension, then writes the bf16 activation
// (zero for tokens not routed to the slot).
template <int NT>
__global__ __launch_bounds__(kThreads) void ffn_gate_up_mfma(FfnArgs a, int blocks_per_slot) {
    __shared__ Plan p;
    build_plan(a, p, true);
    const int j = blockIdx.x / blocks_per_slot;
    if (j >= p.n_slots) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, q = lane >> 4;
    const int i0 = (blockIdx.x % blocks_per_slot) * (kWaves * NT * 16) + wave * NT * 16;
    if (i0 >= a.I) return;   // I is a multiple of 16
    const unsigned tm = p.tok[j];
    const size_t rowb = size_t(a.H) * 2;
    const char* blob = slot_blob(a, p, j);
    const bool xrow = n < a.B;     // A operand row n = token n
    const char* xs = reinterpret_cast<const char*>(a.x) + size_t(xrow ? n : 0) * rowb + q * 16;
    const char* wg[NT];
    const char* wu[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        wg[t] = blob + size_t(i0 + t * 16 + n) * rowb + q * 16;
        wu[t] = blob + size_t(a.I + i0 + t * 16 + n) * rowb + q * 16;
    }
    f32x4 dg[NT], du[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dg[t] = du[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    // two 64-element steps in flight: all loads of both steps issue before
    // the first MFMA waits on them (H is a multiple of 64; an odd last step
    // runs alone)
    auto step = [&](const bf16x8 (&g0)[NT], const bf16x8 (&g1)[NT], const bf16x8 (&u0)[NT],
                    const bf16x8 (&u1)[NT], const bf16x8& x0, const bf16x8& x1) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            dg[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, g0[t], dg[t], 0, 0, 0);
            dg[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, g1[t], dg[t], 0, 0, 0);
            du[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x0, u0[t], du[t], 0, 0, 0);
            du[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x1, u1[t], du[t], 0, 0, 0);
        }
    };
    int h = 0;
    for (; h + 64 < a.H; h += 128) {
        const size_t o0 = size_t(h) * 2, o1 = o0 + 128;
        bf16x8 ga0[NT], gb0[NT], ua0[NT], ub0[NT], ga1[NT], gb1[NT], ua1[NT], ub1[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            ga0[t] = ld_bf8_stream(wg[t] + o0);
            gb0[t] = ld_bf8_stream(wg[t] + o0 + 64);
            ua0[t] = ld_bf8_stream(wu[t] + o0);
            ub0[t] = ld_bf8_stream(wu[t] + o0 + 64);
            ga1[t] = ld_bf8_stream(wg[t] + o1);
            gb1[t] = ld_bf8_stream(wg[t] + o1 + 64);
            ua1[t] = ld_bf8_stream(wu[t] + o1);
            ub1[t] = ld_bf8_stream(wu[t] + o1 + 64);
        }
        const bf16x8 xa0 = xrow ? ld_bf8(xs + o0) : zero, xb0 = xrow ? ld_bf8(xs + o0 + 64) : zero;
        const bf16x8 xa1 = xrow ? ld_bf8(xs + o1) : zero, xb1 = xrow ? ld_bf8(xs + o1 + 64) : zero;
        step(ga0, gb0, ua0, ub0, xa0, xb0);
        step(ga1, gb1, ua1, ub1, xa1, xb1);
    }
    if (h < a.H) {
        const size_t o0 = size_t(h) * 2;
        bf16x8 ga0[NT], gb0[NT], ua0[NT], ub0[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            ga0[t] = ld_bf8_stream(wg[t] + o0);
            gb0[t] = ld_bf8_stream(wg[t] + o0 + 64);
            ua0[t] = ld_bf8_stream(wu[t] + o0);
            ub0[t] = ld_bf8_stream(wu[t] + o0 + 64);
        }
        const bf16x8 xa0 = xrow ? ld_bf8(xs + o0) : zero, xb0 = xrow ? ld_bf8(xs + o0 + 64) : zero;
        step(ga0, gb0, ua0, ub0, xa0, xb0);
    }
    // D layout: lane holds rows m = 4q + r (tokens) of column n (weight row)
    uint16_t* act = reinterpret_cast<uint16_t*>(a.act) + size_t(j) * a.B * a.I;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int b = 4 * q + r;
        if (b >= a.B) continue;
        const bool routed = (tm >> b) & 1u;
        const float wb = routed ? slot_weight(a, p, j, b) : 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float v = routed ? wb * silu(dg[t][r]) * du[t][r] : 0.f;
            act[size_t(b) * a.I + i0 + t * 16 + n] = f32_to_bf16_rne(v);
        }
    }
}

// gate/up through LDS: each wave stages its rows (NT 16-row tiles of W_gate,
// then the same of W_up) 128 elements at a time.  The loads read 256
// contiguous bytes of a row per 16 lanes (four rows per instruction), which
// streams better than loading the MFMA operand layout straight from HBM (16
// rows x 64 bytes per instruction); the wave writes the segment to its own
// padded LDS rows and reads the operands back in the layout of
// v_mfma_f32_16x16x32_bf16 while the next segment's loads are in flight.
// Waves never wait on each other (each owns its LDS region).
constexpr int kLdsSegU4 = 16;         // 128 bf16 = 16 uint4 per row per step
constexpr int kLdsPadU4 = 17;         // padded row stride in uint4: conflict-free reads

// SK (split-K, NT = 1): the workgroup's four waves share the same 16 rows
// and each covers a quarter of the hidden dimension; the partial tiles add
// up in LDS (for shapes whose row count alone gives too few workgroups).
template <int NT, bool SK>
__global__ __launch_bounds__(kThreads) void ffn_gate_up_mfma_lds(FfnArgs a, int blocks_per_slot) {
    static_assert(!SK || NT == 1, "split-K runs one tile per wave");
    __shared__ Plan p;
    __shared__ float red[SK ? kWaves : 1][2][64][4];
    extern __shared__ uint4 stage[];
    build_plan(a, p, true);
    const int j = blockIdx.x / blocks_per_slot;
    if (j >= p.n_slots) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, q = lane >> 4;
    const int i0 = SK ? (blockIdx.x % blocks_per_slot) * 16
                      : (blockIdx.x % blocks_per_slot) * (kWaves * NT * 16) + wave * NT * 16;
    if (!SK && i0 >= a.I) return;   // I is a multiple of 16
    constexpr int kRows = 2 * NT * 16;       // staged rows per wave: gate tiles, then up tiles
    constexpr int kLoads = kRows / 4;        // load instructions per step (four rows each)
    const int h_lo = SK ? wave * (a.H / kWaves) : 0;           // SK: H is a multiple of 512
    const int h_hi = SK ? h_lo + a.H / kWaves : a.H;
    const unsigned tm = p.tok[j];
    const size_t rowb = size_t(a.H) * 2;
    const char* blob = slot_blob(a, p, j);
    uint4* my = stage + size_t(wave) * kRows * kLdsPadU4;
    // loader mapping: lane (g, e) loads uint4 e of the segment of row 4r + g
    const int g = lane >> 4, e = lane & 15;
    const char* src[kLoads];
#pragma unroll
    for (int r = 0; r < kLoads; ++r) {
        const int rr = 4 * r + g, m = rr / (NT * 16), t = rr % (NT * 16);
        src[r] = blob + size_t(m * a.I + i0 + t) * rowb + size_t(h_lo + 8 * e) * 2;
    }
    const bool xrow = n < a.B;     // A operand row n = token n
    const char* xs = reinterpret_cast<const char*>(a.x) + size_t(xrow ? n : 0) * rowb + q * 16;
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    f32x4 dg[NT], du[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dg[t] = du[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    // A operand of a step, loaded one step ahead and issued before that
    // step's weight rows: waiting for it never waits for a weight prefetch
    bf16x8 xa[4], xn[4];
    auto load_x = [&](int h, bf16x8 (&xv)[4]) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) xv[kb] = ld_bf8(xs + size_t(h + 32 * kb) * 2);
    };
    load_x(h_lo, xa);
    uint4 ld[kLoads];
#pragma unroll
    for (int r = 0; r < kLoads; ++r) ld[r] = ld_stream(src[r]);
    for (int h = h_lo; h < h_hi; h += 128) {
        // the previous step's operand reads are done before its rows are overwritten
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < kLoads; ++r) my[(4 * r + g) * kLdsPadU4 + e] = ld[r];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const bool more = h + 128 < h_hi;
        if (more) {
            load_x(h + 128, xn);
            const size_t o = size_t(h + 128 - h_lo) * 2;
#pragma unroll
            for (int r = 0; r < kLoads; ++r) ld[r] = ld_stream(src[r] + o);
        }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            const bf16x8 xv = xrow ? xa[kb] : zero;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const bf16x8 gv = __builtin_bit_cast(bf16x8, my[(t * 16 + n) * kLdsPadU4 + kb * 4 + q]);
                const bf16x8 uv = __builtin_bit_cast(bf16x8, my[((NT + t) * 16 + n) * kLdsPadU4 + kb * 4 + q]);
                dg[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv, gv, dg[t], 0, 0, 0);
                du[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv, uv, du[t], 0, 0, 0);
            }
        }
        if (more) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) xa[kb] = xn[kb];
        }
    }
    if (SK) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            red[SK ? wave : 0][0][lane][r] = dg[0][r];
            red[SK ? wave : 0][1][lane][r] = du[0][r];
        }
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float gs = 0.f, us = 0.f;
#pragma unroll
            for (int w = 0; w < (SK ? kWaves : 1); ++w) { gs += red[w][0][lane][r]; us += red[w][1][lane][r]; }
            dg[0][r] = gs;
            du[0][r] = us;
        }
    }
    // D layout: lane holds rows m = 4q + r (tokens) of column n (weight row)
    uint16_t* act = reinterpret_cast<uint16_t*>(a.act) + size_t(j) * a.B * a.I;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int b = 4 * q + r;
        if (b >= a.B) continue;
        const bool routed = (tm >> b) & 1u;
        const float wb = routed ? slot_weight(a, p, j, b) : 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float v = routed ? wb * silu(dg[t][r]) * du[t][r] : 0.f;
            act[size_t(b) * a.I + i0 + t * 16 + n] = f32_to_bf16_rne(v);
        }
    }
}

// down through LDS: as the gate/up kernel, with W_down rows (length I) as the
// staged operand and the slot's bf16 activations as the A operand, summing
// the slots of the workgroup's group.
template <int NT>
__global__ __launch_bounds__(kThreads) void ffn_down_mfma_lds(FfnArgs a) {
    __shared__ PlanB p;
    extern __shared__ uint4 stage[];
    build_plan(a, p);
    const int rb = blockIdx.x / a.ng, grp = blockIdx.x % a.ng;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, q = lane >> 4;
    const int rows_per_block = kWaves * NT * 16;
    const int h0 = rb * rows_per_block + wave * NT * 16;
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.n_experts)
        atomicAdd(a.n_experts, (unsigned long long)p.n_routed);
    const bool live = h0 < a.H;   // H is a multiple of 64 * NT
    constexpr int kRows = NT * 16;
    constexpr int kLoads = kRows / 4;
    const size_t rowb = size_t(a.I) * 2;
    const bool arow = n < a.B;
    const int g = lane >> 4, e = lane & 15;
    uint4* my = stage + size_t(wave) * kRows * kLdsPadU4;
    // the selected slots split evenly over the groups (an empty group writes zeros)
    const int j0 = grp * p.n_slots / a.ng, j1 = (grp + 1) * p.n_slots / a.ng;
    f32x4 d[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) d[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    // the group's (slot, 128-column step) pairs as one stream: the next
    // step's activations and weight rows (the next slot's first ones at a
    // slot's end) are in flight while the current step runs, activations
    // issued first so that waiting for them never waits for weights
    const int steps = a.I / 128;                   // I is a multiple of 128
    const int total = live ? (j1 - j0) * steps : 0;
    uint4 ld[kLoads];
    bf16x8 av[4], an[4];
    auto issue = [&](int j, int k, bf16x8 (&ax)[4]) {
        const char* wd = slot_blob(a, p, j) + 2 * size_t(a.I) * a.H * 2 + size_t(k) * 2;
        const char* ar = reinterpret_cast<const char*>(a.act) + (size_t(j) * a.B + (arow ? n : 0)) * rowb +
                         q * 16 + size_t(k) * 2;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) ax[kb] = ld_bf8(ar + size_t(32 * kb) * 2);
#pragma unroll
        for (int r = 0; r < kLoads; ++r) ld[r] = ld_stream(wd + size_t(h0 + 4 * r + g) * rowb + size_t(e) * 16);
    };
    int jn = j0, kn = 0;                            // next step to issue
    if (total > 0) {
        issue(jn, kn, av);
        if ((kn += 128) == a.I) { kn = 0; ++jn; }
    }
    for (int s = 0; s < total; ++s) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < kLoads; ++r) my[(4 * r + g) * kLdsPadU4 + e] = ld[r];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const bool more = s + 1 < total;
        if (more) {
            issue(jn, kn, an);
            if ((kn += 128) == a.I) { kn = 0; ++jn; }
        }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            const bf16x8 ax = arow ? av[kb] : zero;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const bf16x8 wv = __builtin_bit_cast(bf16x8, my[(t * 16 + n) * kLdsPadU4 + kb * 4 + q]);
                d[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ax, wv, d[t], 0, 0, 0);
            }
        }
        if (more) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) av[kb] = an[kb];
        }
    }
    float* out = a.ng == 1 ? a.y : a.part + size_t(grp) * a.B * a.H;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int b = 4 * q + r;
        if (!live || b >= a.B) continue;
#pragma unroll
        for (int t = 0; t < NT; ++t) out[size_t(b) * a.H + h0 + t * 16 + n] = d[t][r];
    }
}

// gate/up, split-K: one workgroup = 16 rows of one slot; wave w covers the
// w-th quarter of the hidden dimension and the four partial tiles add up in
// LDS (for shapes whose row count alone gives too few workgroups).
__global__ __launch_bounds__(kThreads) void ffn_gate_up_mfma_sk(FfnArgs a, int blocks_per_slot) {
    __shared__ Plan p;
    __shared__ float red[kWaves][2][64][4];
    build_plan(a, p, true);
    const int j = blockIdx.x / blocks_per_slot;
    if (j >= p.n_slots) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, q = lane >> 4;
    const int i0 = (blockIdx.x % blocks_per_slot) * 16;   // I is a multiple of 16
    const unsigned tm = p.tok[j];
    const size_t rowb = size_t(a.H) * 2;
    const char* blob = slot_blob(a, p, j);
    const bool xrow = n < a.B;
    const int hq = a.H / kWaves;                            // H is a multiple of 256
    const size_t kbase = size_t(wave) * hq * 2 + q * 16;
    const char* xs = reinterpret_cast<const char*>(a.x) + size_t(xrow ? n : 0) * rowb + kbase;
    const char* wg = blob + size_t(i0 + n) * rowb + kbase;
    const char* wu = blob + size_t(a.I + i0 + n) * rowb + kbase;
    f32x4 dg = f32x4{0.f, 0.f, 0.f, 0.f}, du = dg;
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    int h = 0;
    for (; h + 64 < hq; h += 128) {
        const size_t o0 = size_t(h) * 2, o1 = o0 + 128;
        const bf16x8 ga0 = ld_bf8_stream(wg + o0), gb0 = ld_bf8_stream(wg + o0 + 64);
        const bf16x8 ua0 = ld_bf8_stream(wu + o0), ub0 = ld_bf8_stream(wu + o0 + 64);
        const bf16x8 ga1 = ld_bf8_stream(wg + o1), gb1 = ld_bf8_stream(wg + o1 + 64);
        const bf16x8 ua1 = ld_bf8_stream(wu + o1), ub1 = ld_bf8_stream(wu + o1 + 64);
        const bf16x8 xa0 = xrow ? ld_bf8(xs + o0) : zero, xb0 = xrow ? ld_bf8(xs + o0 + 64) : zero;
        const bf16x8 xa1 = xrow ? ld_bf8(xs + o1) : zero, xb1 = xrow ? ld_bf8(xs + o1 + 64) : zero;
        dg = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa0, ga0, dg, 0, 0, 0);
        dg = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb0, gb0, dg, 0, 0, 0);
        du = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa0, ua0, du, 0, 0, 0);
        du = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb0, ub0, du, 0, 0, 0);
        dg = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa1, ga1, dg, 0, 0, 0);
        dg = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb1, gb1, dg, 0, 0, 0);
        du = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa1, ua1, du, 0, 0, 0);
        du = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb1, ub1, du, 0, 0, 0);
    }
    if (h < hq) {
        const size_t o0 = size_t(h) * 2;
        const bf16x8 ga0 = ld_bf8_stream(wg + o0), gb0 = ld_bf8_stream(wg + o0 + 64);
        const bf16x8 ua0 = ld_bf8_stream(wu + o0), ub0 = ld_bf8_stream(wu + o0 + 64);
        const bf16x8 xa0 = xrow ? ld_bf8(xs + o0) : zero, xb0 = xrow ? ld_bf8(xs + o0 + 64) : zero;
        dg = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa0, ga0, dg, 0, 0, 0);
        dg = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb0, gb0, dg, 0, 0, 0);
        du = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa0, ua0, du, 0, 0, 0);
        du = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb0, ub0, du, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) { red[wave][0][lane][r] = dg[r]; red[wave][1][lane][r] = du[r]; }
    __syncthreads();
    if (wave != 0) return;
    uint16_t* act = reinterpret_cast<uint16_t*>(a.act) + size_t(j) * a.B * a.I;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int b = 4 * q + r;
        if (b >= a.B) continue;
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) { g += red[w][0][lane][r]; u += red[w][1][lane][r]; }
        const bool routed = (tm >> b) & 1u;
        const float v = routed ? slot_weight(a, p, j, b) * silu(g) * u : 0.f;
        act[size_t(b) * a.I + i0 + n] = f32_to_bf16_rne(v);
    }
}

// down: each wave computes NT tiles of 16 output rows x 16 tokens, summing
// the slots of its group (A operand = the slot's bf16 activations).
template <int NT>
__global__ __launch_bounds__(kThreads) void ffn_down_mfma(FfnArgs a) {
    __shared__ Plan p;
    build_plan(a, p);
    const int rb = blockIdx.x / a.ng, grp = blockIdx.x % a.ng;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, q = lane >> 4;
    const int rows_per_block = kWaves * NT * 16;
    const int h0 = rb * rows_per_block + wave * NT * 16;
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.n_experts)
        atomicAdd(a.n_experts, (unsigned long long)p.n_routed);
    const bool live = h0 < a.H;   // H is a multiple of 64 * NT
    const size_t rowb = size_t(a.I) * 2;
    const bool arow = n < a.B;
    // the selected slots split evenly over the groups (an empty group writes zeros)
    const int j0 = grp * p.n_slots / a.ng, j1 = (grp + 1) * p.n_slots / a.ng;
    f32x4 d[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) d[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    for (int j = j0; live && j < j1; ++j) {
        const char* wd = slot_blob(a, p, j) + 2 * size_t(a.I) * a.H * 2 + q * 16;
        const char* wr[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) wr[t] = wd + size_t(h0 + t * 16 + n) * rowb;
        const char* ar = reinterpret_cast<const char*>(a.act) +
                         (size_t(j) * a.B + (arow ? n : 0)) * rowb + q * 16;
        auto step = [&](const bf16x8 (&w0)[NT], const bf16x8 (&w1)[NT], const bf16x8& a0, const bf16x8& a1) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                d[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, w0[t], d[t], 0, 0, 0);
                d[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, w1[t], d[t], 0, 0, 0);
            }
        };
        int k = 0;
        for (; k + 64 < a.I; k += 128) {
            const size_t o0 = size_t(k) * 2, o1 = o0 + 128;
            bf16x8 wa0[NT], wb0[NT], wa1[NT], wb1[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                wa0[t] = ld_bf8_stream(wr[t] + o0);
                wb0[t] = ld_bf8_stream(wr[t] + o0 + 64);
                wa1[t] = ld_bf8_stream(wr[t] + o1);
                wb1[t] = ld_bf8_stream(wr[t] + o1 + 64);
            }
            const bf16x8 aa0 = arow ? ld_bf8(ar + o0) : zero, ab0 = arow ? ld_bf8(ar + o0 + 64) : zero;
            const bf16x8 aa1 = arow ? ld_bf8(ar + o1) : zero, ab1 = arow ? ld_bf8(ar + o1 + 64) : zero;
            step(wa0, wb0, aa0, ab0);
            step(wa1, wb1, aa1, ab1);
        }
        if (k < a.I) {
            const size_t o0 = size_t(k) * 2;
            bf16x8 wa0[NT], wb0[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                wa0[t] = ld_bf8_stream(wr[t] + o0);
                wb0[t] = ld_bf8_stream(wr[t] + o0 + 64);
            }
            const bf16x8 aa0 = arow ? ld_bf8(ar + o0) : zero, ab0 = arow ? ld_bf8(ar + o0 + 64) : zero;
            step(wa0, wb0, aa0, ab0);
        }
    }
    float* out = a.ng == 1 ? a.y : a.part + size_t(grp) * a.B * a.H;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int b = 4 * q + r;
        if (!live || b >= a.B) continue;
#pragma unroll
        for (int t = 0; t < NT; ++t) out[size_t(b) * a.H + h0 + t * 16 + n] = d[t][r];
    }
}

// y = sum over slot groups of the MFMA down phase's partial sums, in group
// order; four outputs per thread, eight groups' loads in flight.
__global__ __launch_bounds__(kThreads) void ffn_reduce(const float* part, int ng, int n4, float* y) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= n4) return;
    const float4* p4 = reinterpret_cast<const float4*>(part);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    int g = 0;
    for (; g + 8 <= ng; g += 8) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = p4[size_t(g + u) * n4 + i];
#pragma unroll
        for (int u = 0; u < 8; ++u) { s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w; }
    }
    for (; g < ng; ++g) {
        const float4 v = p4[size_t(g) * n4 + i];
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    reinterpret_cast<float4*>(y)[i] = s;
}

// ============================================================================
// host side
// ============================================================================

// lanes per row: the widest of 64/32/16 that divides the row's chunk count
int pick_group(int chunks) {
    if (chunks % 64 == 0 || chunks > 512) return 64;
    if (chunks % 32 == 0) return 32;
    if (chunks % 16 == 0) return 16;
    return 64;
}

struct Shape {
    bool mfma;          // MFMA path
    int slots;          // slot capacity
    int gu_G;           // GEMV gate/up lanes per row
    int dn_kind;        // 0: rows (lane groups, slots split over waves), 1: whole-workgroup rows, 2: MFMA
    int dn_G;           // lanes per row for kind 0
    int dn_rows;        // rows per down workgroup
    int n_rb;           // down row blocks
    int ng, spg;        // slot groups of the MFMA down phase
    int dn_nt;          // 16-row tiles per wave of the MFMA down kernel
    int dn_R;           // rows per lane group of the GEMV down kernel
};

constexpr int kDownRowsWgTarget = 1024;  // lane-group down: fewest workgroups more rows per group may leave
constexpr int kDownWgR = 4;   // rows per workgroup (whole-workgroup down)
constexpr int kUpWgR = 0;     // rows per workgroup of the whole-workgroup gate/up kernel (0: lane groups)
constexpr int kDownForceG = 0;  // lanes per down row (0: by row length)
constexpr int kMfmaNT = 0;      // 1: force one 16-row tile per wave in the MFMA gate/up kernel
constexpr int kMfmaDownNT = 2;  // 16-row tiles per wave of the MFMA down kernel (1, 2 or 4)
constexpr int kMfmaSplitKBelow = 2048;  // split-K MFMA gate/up when the tiled grid has fewer workgroups
constexpr bool kMfmaUpLds = true;       // MFMA gate/up stages weight rows through LDS (H % 128 == 0;
                                        // split-K: H % 512 == 0)
constexpr bool kMfmaDownLds = true;     // MFMA down stages W_down rows through LDS (I % 128 == 0)
constexpr int kUpWgMinChunks = 512;   // ... used when a row has at least this many chunks

Shape plan_shape(int B, int K, int H, int I, int E, int n_shared, int dtype) {
    Shape s{};
    const int esz = dtype == STMOE_BF16 ? 2 : 4;
    s.slots = (B * K < E ? B * K : E) + n_shared;
    s.mfma = dtype == STMOE_BF16 && B >= kMfmaMinB && H % 64 == 0 && I % 64 == 0;
    s.gu_G = pick_group(H * esz / 16);
    const int cpr_i = I * esz / 16;
    s.ng = s.spg = 1;
    s.dn_nt = 1;
    if (s.mfma) {
        s.dn_kind = 2;
        // several row tiles per wave share each activation load
        s.dn_nt = (H % (kWaves * 16 * kMfmaDownNT) == 0) ? kMfmaDownNT : 1;
        s.dn_rows = kWaves * 16 * s.dn_nt;
    } else if (cpr_i >= 512 && H % kDownWgR == 0 && s.slots < kWaves) {
        s.dn_kind = 1;
        s.dn_rows = kDownWgR;
    } else {
        s.dn_kind = 0;
        // 64 lanes per row once a row has 128 chunks: one row per wave pass
        // gives more workgroups than lane groups of 16 or 32
        s.dn_G = kDownForceG ? kDownForceG : (cpr_i >= 128 ? 64 : pick_group(cpr_i));
        // rows per lane group: as many as keep kDownRowsWgTarget workgroups
        // (every workgroup re-reads all activations; more rows amortise them)
        const int rmax = s.dn_G == 64 ? 4 : (s.dn_G == 32 ? 2 : 1);
        s.dn_R = 1;
        while (s.dn_R < rmax && H % ((64 / s.dn_G) * s.dn_R * 2) == 0 &&
               H / ((64 / s.dn_G) * s.dn_R * 2) >= kDownRowsWgTarget)
            s.dn_R *= 2;
        s.dn_rows = (64 / s.dn_G) * s.dn_R;
    }
    s.n_rb = (H + s.dn_rows - 1) / s.dn_rows;
    if (s.mfma) {
        int ng = (kDownWgTarget + s.n_rb - 1) / s.n_rb;
        if (ng > s.slots) ng = s.slots;
        if (ng < 1) ng = 1;
        s.ng = ng;
        s.spg = (s.slots + ng - 1) / ng;
    }
    return s;
}

struct WsLayout {
    size_t act, part, total;
};

WsLayout ws_layout(int B, int H, int I, const Shape& s) {
    auto up = [](size_t v) { return (v + 255) / 256 * 256; };
    WsLayout w{};
    w.act = 0;
    w.part = up(size_t(s.slots) * B * I * sizeof(float));
    w.total = w.part + (s.ng > 1 ? up(size_t(s.ng) * B * H * sizeof(float)) : 0);
    return w;
}

// GEMV activations are bf16 for the lane-group down kernel below four rows
// per group and the whole-workgroup one up to two token columns, fp32
// otherwise (there the unpacking registers cost more than the traffic
// saves); the gate/up launch writes what its down kernel reads.
template <bool BF>
int act_bf16(const Shape& s, int B) { return BF && (s.dn_kind == 1 ? B <= 2 : s.dn_R < 4); }

template <bool BF, int G, int NB, int R>
int launch_gate_up_r(const FfnArgs& a, const Shape& s, hipStream_t st) {
    const int rows = kWaves * (64 / G) * R;
    const int bps = (a.I + rows - 1) / rows;
    const size_t xbytes = size_t(a.B) * a.H * (BF ? 2 : 4);
    const int act16 = act_bf16<BF>(s, a.B);
    if constexpr (kUpB1 && NB == 1) {
        if (a.B == 1 && (!a.logits || a.E <= kUpB1RouteMaxE)) {
            hipLaunchKernelGGL((ffn_gate_up_b1<BF, G, R>), dim3(unsigned(bps * s.slots)), dim3(kThreads), 0, st, a,
                               bps, act16);
            STMOE_LAUNCHED();
            return STMOE_OK;
        }
    }
    if (kStageX && xbytes <= size_t(kXStageMax))
        hipLaunchKernelGGL((ffn_gate_up<BF, G, R, NB, true>), dim3(unsigned(bps * s.slots)), dim3(kThreads),
                           unsigned(xbytes), st, a, bps, act16);
    else
        hipLaunchKernelGGL((ffn_gate_up<BF, G, R, NB, false>), dim3(unsigned(bps * s.slots)), dim3(kThreads), 0,
                           st, a, bps, act16);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

template <bool BF, int G, int NB>
int launch_gate_up(const FfnArgs& a, const Shape& s, hipStream_t st) {
    if constexpr (kUpWgR > 0) {
        if (a.H * (BF ? 2 : 4) / 16 >= kUpWgMinChunks && a.I % kUpWgR == 0) {
            const int bps = a.I / kUpWgR;
            hipLaunchKernelGGL((ffn_gate_up_wg<BF, kUpWgR, NB>), dim3(unsigned(bps * s.slots)),
                               dim3(kThreads), 0, st, a, bps, act_bf16<BF>(s, a.B));
            STMOE_LAUNCHED();
            return STMOE_OK;
        }
    }
    // every workgroup stages all token activations; from 4 token columns on
    // two rows per lane group halve that traffic, below it one row per group
    // gives more workgroups in flight (I is a multiple of 8)
    if constexpr (NB >= 4) return launch_gate_up_r<BF, G, NB, 2>(a, s, st);
    else return launch_gate_up_r<BF, G, NB, 1>(a, s, st);
}

template <bool BF, int NB, int U>
void launch_down_rows_u(const FfnArgs& a, const Shape& s, hipStream_t st) {
    const dim3 grid(unsigned(s.n_rb));
    if (s.dn_G == 16)
        hipLaunchKernelGGL((ffn_down_rows<BF, 16, 1, NB, U>), grid, dim3(kThreads), 0, st, a);
    else if (s.dn_G == 32 && s.dn_R == 2)
        hipLaunchKernelGGL((ffn_down_rows<BF, 32, 2, NB, U>), grid, dim3(kThreads), 0, st, a);
    else if (s.dn_G == 32)
        hipLaunchKernelGGL((ffn_down_rows<BF, 32, 1, NB, U>), grid, dim3(kThreads), 0, st, a);
    else if (s.dn_R == 4)
        hipLaunchKernelGGL((ffn_down_rows<BF, 64, 4, NB, U>), grid, dim3(kThreads), 0, st, a);
    else if (s.dn_R == 2)
        hipLaunchKernelGGL((ffn_down_rows<BF, 64, 2, NB, U>), grid, dim3(kThreads), 0, st, a);
    else
        hipLaunchKernelGGL((ffn_down_rows<BF, 64, 1, NB, U>), grid, dim3(kThreads), 0, st, a);
}

// short rows (at most kShortRowChunks chunks per lane) load a slot's chunks in one step
template <bool BF, int NB>
void launch_down_rows(const FfnArgs& a, const Shape& s, hipStream_t st) {
    if ((a.I * (BF ? 2 : 4) / 16 + s.dn_G - 1) / s.dn_G <= kShortRowChunks)
        launch_down_rows_u<BF, NB, kDownInFlightShort>(a, s, st);
    else
        launch_down_rows_u<BF, NB, 2>(a, s, st);
}

template <bool BF, int NB>
int launch_down(const FfnArgs& a, const Shape& s, hipStream_t st) {
    const dim3 grid(unsigned(s.n_rb));
    if (s.dn_kind == 1) {
        hipLaunchKernelGGL((ffn_down_wg<BF, kDownWgR, NB>), grid, dim3(kThreads), 0, st, a);
    } else {
        launch_down_rows<BF, NB>(a, s, st);
    }
    STMOE_LAUNCHED();
    return STMOE_OK;
}

template <bool BF, int NB>
int launch_gemv(const FfnArgs& a, const Shape& s, hipStream_t st, hipEvent_t ev_mid) {
    int rc;
    if (s.gu_G == 16) rc = launch_gate_up<BF, 16, NB>(a, s, st);
    else if (s.gu_G == 32) rc = launch_gate_up<BF, 32, NB>(a, s, st);
    else rc = launch_gate_up<BF, 64, NB>(a, s, st);
    if (rc) return rc;
    if (ev_mid) STMOE_HIP(hipEventRecord(ev_mid, st));
    return launch_down<BF, NB>(a, s, st);
}

template <bool BF>
int launch_gemv_b(const FfnArgs& a, const Shape& s, hipStream_t st, hipEvent_t ev_mid) {
    if (a.B <= 1) return launch_gemv<BF, 1>(a, s, st, ev_mid);
    if (a.B <= 2) return launch_gemv<BF, 2>(a, s, st, ev_mid);
    if (a.B <= 4) return launch_gemv<BF, 4>(a, s, st, ev_mid);
    if (a.B <= 8) return launch_gemv<BF, 8>(a, s, st, ev_mid);
    return launch_gemv<BF, 16>(a, s, st, ev_mid);
}

int launch_mfma(const FfnArgs& a, const Shape& s, hipStream_t st, hipEvent_t ev_mid) {
    // two 16-row tiles per wave when that still leaves >= 1024 workgroups
    constexpr int NT = 2;
    const int rows = kWaves * NT * 16;
    if ((a.I / (kWaves * 16)) * s.slots < kMfmaSplitKBelow && a.H % 256 == 0) {
        const int bps = a.I / 16;
        if (kMfmaUpLds && a.H % 512 == 0) {
            const unsigned lds = unsigned(kWaves * 2 * 16 * kLdsPadU4 * sizeof(uint4));
            hipLaunchKernelGGL((ffn_gate_up_mfma_lds<1, true>), dim3(unsigned(bps * s.slots)), dim3(kThreads), lds,
                               st, a, bps);
        } else {
            hipLaunchKernelGGL(ffn_gate_up_mfma_sk, dim3(unsigned(bps * s.slots)), dim3(kThreads), 0, st, a, bps);
        }
    } else if (a.I % rows != 0 || (a.I / rows) * s.slots < 1024 || kMfmaNT == 1) {
        const int bps = a.I / (kWaves * 16);
        if (kMfmaUpLds && a.H % 128 == 0) {
            const unsigned lds = unsigned(kWaves * 2 * 16 * kLdsPadU4 * sizeof(uint4));
            hipLaunchKernelGGL((ffn_gate_up_mfma_lds<1, false>), dim3(unsigned(bps * s.slots)), dim3(kThreads), lds, st,
                               a, bps);
        } else {
            hipLaunchKernelGGL((ffn_gate_up_mfma<1>), dim3(unsigned(bps * s.slots)), dim3(kThreads), 0, st, a,
                               bps);
        }
    } else {
        const int bps = a.I / rows;
        if (kMfmaUpLds && a.H % 128 == 0) {
            const unsigned lds = unsigned(kWaves * 2 * NT * 16 * kLdsPadU4 * sizeof(uint4));
            hipLaunchKernelGGL((ffn_gate_up_mfma_lds<NT, false>), dim3(unsigned(bps * s.slots)), dim3(kThreads), lds, st,
                               a, bps);
        } else {
            hipLaunchKernelGGL((ffn_gate_up_mfma<NT>), dim3(unsigned(bps * s.slots)), dim3(kThreads), 0, st, a,
                               bps);
        }
    }
    STMOE_LAUNCHED();
    if (ev_mid) STMOE_HIP(hipEventRecord(ev_mid, st));
    const dim3 dgrid(unsigned(s.n_rb * s.ng));
    const unsigned dlds = unsigned(kWaves * s.dn_nt * 16 * kLdsPadU4 * sizeof(uint4));
    const bool dn_lds = kMfmaDownLds && a.I % 128 == 0;
    if (s.dn_nt == 4) {
        if (dn_lds) hipLaunchKernelGGL((ffn_down_mfma_lds<4>), dgrid, dim3(kThreads), dlds, st, a);
        else hipLaunchKernelGGL((ffn_down_mfma<4>), dgrid, dim3(kThreads), 0, st, a);
    } else if (s.dn_nt == 2) {
        if (dn_lds) hipLaunchKernelGGL((ffn_down_mfma_lds<2>), dgrid, dim3(kThreads), dlds, st, a);
        else hipLaunchKernelGGL((ffn_down_mfma<2>), dgrid, dim3(kThreads), 0, st, a);
    } else {
        if (dn_lds) hipLaunchKernelGGL((ffn_down_mfma_lds<1>), dgrid, dim3(kThreads), dlds, st, a);
        else hipLaunchKernelGGL((ffn_down_mfma<1>), dgrid, dim3(kThreads), 0, st, a);
    }
    STMOE_LAUNCHED();
    if (s.ng > 1) {
        const int n4 = a.B * a.H / 4;   // H is a multiple of 64
        hipLaunchKernelGGL(ffn_reduce, dim3(unsigned((n4 + kThreads - 1) / kThreads)), dim3(kThreads), 0, st,
                           a.part, s.ng, n4, a.y);
        STMOE_LAUNCHED();
    }
    return STMOE_OK;
}

}  // namespace

size_t ffn_workspace_bytes(int B, int K, int E, int H, int I, int n_shared, int dtype) {
    const Shape s = plan_shape(B, K, H, I, E, n_shared, dtype);
    return ws_layout(B, H, I, s).total;
}

// Internal entry used by the decode-layer orchestration (no argument checks).
// With `logits` (B*E <= kRouteInFfnMax) the gate/up kernel routes first and
// idx/w are outputs, written before the down kernel reads them.
int ffn_launch(const void* x, const int32_t* idx, const float* w, int B, int K, int H, int I, int E,
               int dtype, const void* const* eptr, const void* const* sptr, int n_shared,
               float* y, void* ws, hipStream_t st, unsigned long long* n_experts, hipEvent_t ev_mid,
               const float* logits, int renorm, const void* ebase, size_t estride) {
    if (logits && B * E > kRouteInFfnMax) {
        set_error("ffn_launch: routing inside the FFN needs B*E <= 128");
        return STMOE_EINVAL;
    }
    const Shape s = plan_shape(B, K, H, I, E, n_shared, dtype);
    const WsLayout L = ws_layout(B, H, I, s);
    char* base = reinterpret_cast<char*>(ws);
    FfnArgs a;
    a.x = x;
    a.idx = idx;
    a.w = w;
    a.eptr = eptr;
    a.ebase = reinterpret_cast<const char*>(ebase);
    a.estride = estride;
    a.sptr = sptr;
    a.B = B;
    a.K = K;
    a.H = H;
    a.I = I;
    a.E = E;
    a.n_shared = n_shared;
    a.act = base + L.act;
    a.part = reinterpret_cast<float*>(base + L.part);
    a.y = y;
    a.n_experts = n_experts;
    a.ng = s.ng;
    a.spg = s.spg;
    a.logits = logits;
    a.renorm = renorm;
    if (s.mfma) return launch_mfma(a, s, st, ev_mid);
    return dtype == STMOE_BF16 ? launch_gemv_b<true>(a, s, st, ev_mid)
                               : launch_gemv_b<false>(a, s, st, ev_mid);
}

}  // namespace stmoe

using namespace stmoe;

extern "C" size_t moe_expert_ffn_workspace_bytes(int B, int K, int E, int H, int I, int n_shared,
                                                 int dtype) {
    if (B < 1 || K < 1 || E < 1 || H < 1 || I < 1 || n_shared < 0) return 0;
    if (dtype != STMOE_BF16 && dtype != STMOE_F32) return 0;
    return ffn_workspace_bytes(B, K, E, H, I, n_shared, dtype);
}

extern "C" int moe_expert_ffn(const void* x, const int32_t* topk_idx, const float* topk_w, int B,
                              int K, int H, int I, int E, int dtype, const void* const* expert_ptrs,
                              const void* const* shared_ptrs, int n_shared, float* y, void* ws,
                              size_t ws_bytes, void* stream) {
    clear_error();
    STMOE_CHECK(x && topk_idx && topk_w && expert_ptrs && y && ws, "null pointer");
    STMOE_CHECK(B >= 1 && B <= kMaxB, "B must be in [1, 16]");
    STMOE_CHECK(E >= 1 && E <= kMaxE, "E must be in [1, 256]");
    STMOE_CHECK(K >= 1 && K <= E && K <= kMaxK, "K must be in [1, min(E, 16)]");
    STMOE_CHECK(H >= 8 && H % 8 == 0 && H <= kMaxH, "H must be a multiple of 8 in [8, 16384]");
    STMOE_CHECK(I >= 8 && I % 8 == 0, "I must be a positive multiple of 8");
    STMOE_CHECK(n_shared >= 0 && n_shared <= kMaxShared, "n_shared must be in [0, 8]");
    STMOE_CHECK(n_shared == 0 || shared_ptrs, "shared_ptrs is required when n_shared > 0");
    STMOE_CHECK(dtype == STMOE_BF16 || dtype == STMOE_F32, "dtype must be STMOE_BF16 or STMOE_F32");
    STMOE_CHECK(ws_bytes >= moe_expert_ffn_workspace_bytes(B, K, E, H, I, n_shared, dtype),
                "workspace too small");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(x) & 15) == 0 && (reinterpret_cast<uintptr_t>(ws) & 255) == 0,
                "x must be 16-byte and ws 256-byte aligned");
    return ffn_launch(x, topk_idx, topk_w, B, K, H, I, E, dtype, expert_ptrs, shared_ptrs, n_shared, y,
                      ws, as_stream(stream), nullptr, nullptr, nullptr, 0, nullptr, 0);
}

namespace {

constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];      // device address of `scratch` per device (null until resolved)

// The current device's address of `scratch`, resolved once per device with
// that device current.
int noalloc_scratch(void** out) {
    int dev = -1;
    STMOE_HIP(hipGetDevice(&dev));
    STMOE_CHECK(dev >= 0 && dev < kMaxDevices, "device ordinal beyond the library's table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        STMOE_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        STMOE_CHECK(p != nullptr, "hipGetSymbolAddress returned no address");
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return STMOE_OK;
}

}  // namespace

extern "C" int moe_expert_ffn_noalloc(const void* x, const int32_t* topk_idx, const float* topk_w, int B,
                                      int K, int H, int I, int E, int dtype, const void* const* expert_ptrs,
                                      const void* const* shared_ptrs, int n_shared, float* y, void* stream) {
    clear_error();
    STMOE_CHECK(x && topk_idx && topk_w && expert_ptrs && y, "null pointer");
    STMOE_CHECK(B >= 1 && B <= kMaxB, "B must be in [1, 16]");
    STMOE_CHECK(E >= 1 && E <= kMaxE, "E must be in [1, 256]");
    STMOE_CHECK(K >= 1 && K <= E && K <= kMaxK, "K must be in [1, min(E, 16)]");
    STMOE_CHECK(H >= 8 && H % 8 == 0 && H <= kMaxH, "H must be a multiple of 8 in [8, 16384]");
    STMOE_CHECK(I >= 8 && I % 8 == 0, "I must be a positive multiple of 8");
    STMOE_CHECK(n_shared >= 0 && n_shared <= kMaxShared, "n_shared must be in [0, 8]");
    STMOE_CHECK(n_shared == 0 || shared_ptrs, "shared_ptrs is required when n_shared > 0");
    STMOE_CHECK(dtype == STMOE_BF16 || dtype == STMOE_F32, "dtype must be STMOE_BF16 or STMOE_F32");
    const size_t need = moe_expert_ffn_workspace_bytes(B, K, E, H, I, n_shared, dtype);
    if (need > kNoAllocScratchBytes) {
        set_error("moe_expert_ffn_noalloc: this shape needs " + std::to_string(need) +
                  " bytes of workspace; the library's scratch holds " + std::to_string(kNoAllocScratchBytes) +
                  " (use moe_expert_ffn with a caller workspace)");
        return STMOE_ENOMEM;
    }
    STMOE_CHECK((reinterpret_cast<uintptr_t>(x) & 15) == 0, "x must be 16-byte aligned");
    void* ws = nullptr;
    if (int rc = noalloc_scratch(&ws)) return rc;
    return ffn_launch(x, topk_idx, topk_w, B, K, H, I, E, dtype, expert_ptrs, shared_ptrs, n_shared, y, ws,
                      as_stream(stream), nullptr, nullptr, nullptr, 0, nullptr, 0);
}
