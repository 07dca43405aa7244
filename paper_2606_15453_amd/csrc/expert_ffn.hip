// Expert FFN of the decode-step MoE layer (Section 2; SwiGLU experts):
//   y[b] = sum over selected experts e of w[b][e] * W_down_e (silu(W_gate_e x_b) * (W_up_e x_b))
//        + the same with weight 1 for shared experts.
//
// Decode is bandwidth-bound: every selected expert's weights are streamed
// from HBM once per call, at about 2 flops per weight byte per token.  Two
// kernels, both reading 16-byte weight chunks with non-temporal loads:
//
//   ffn_gate_up  one workgroup = (expert slot, 8*R rows of W_gate and W_up).
//                A group of G lanes owns R rows; each lane strides over the
//                row's 16-byte chunks, dots them with the tokens' activations
//                (cache-resident), and the G-lane segment sums give g and u.
//                a = w_b * silu(g) * u goes to the workspace [slot][b][I].
//   ffn_down     one workgroup = a block of output rows h.  For each slot in
//                ascending expert order (shared experts last) it streams row h
//                of W_down and dots it with a[slot][b][*]; partial sums stay in
//                registers across slots, so y is written once, with a fixed
//                summation order (the result does not depend on where the
//                blobs live).
//
// Both kernels rebuild the slot plan (distinct selected experts ascending,
// their token masks and weights) from topk_idx/topk_w in LDS; no host
// round trip and no separate planning launch.
#include "common.h"

namespace stmoe {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxShared = 8;
constexpr int kMaxSlots = kMaxE + kMaxShared;

struct FfnArgs {
    const void* x;               // [B][H]
    const int32_t* idx;          // [B][K]
    const float* w;              // [B][K]
    const void* const* eptr;     // [E] device blob pointers
    const void* const* sptr;     // [n_shared] or null
    int B, K, H, I, E, n_shared;
    float* act;                  // [slots][B][I]
    float* y;                    // [B][H]
    unsigned long long* n_experts;   // optional: += distinct routed experts (block 0)
};

struct Plan {
    int32_t idx[kMaxB * kMaxK];
    float w[kMaxB * kMaxK];
    unsigned sel[kMaxE / 32];
    int expert[kMaxSlots];       // routed slots: expert index; shared slots: -1 - s
    unsigned tok[kMaxSlots];     // token bit mask per slot
    float wt[kMaxSlots][kMaxB];  // gate weight per slot and token (valid where tok is set)
    int n_routed, n_slots;
};

// Build the slot plan in LDS (all threads participate; ends with a barrier).
// Slot order: selected routed experts ascending, then shared experts.
__device__ void build_plan(const FfnArgs& a, Plan& p) {
    const int tid = threadIdx.x;
    const int BK = a.B * a.K;
    for (int t = tid; t < BK; t += kThreads) {
        const int e = a.idx[t];
        p.idx[t] = (e >= 0 && e < a.E) ? e : -1;   // out-of-range entries are ignored
        p.w[t] = a.w[t];
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
        p.wt[rank][b] = p.w[t];
        p.expert[rank] = e;
    }
    for (int s = tid; s < a.n_shared; s += kThreads) {
        p.expert[total + s] = -1 - s;
        p.tok[total + s] = (1u << a.B) - 1u;
        for (int b = 0; b < a.B; ++b) p.wt[total + s][b] = 1.f;
    }
    if (tid == 0) {
        p.n_routed = total;
        p.n_slots = total + a.n_shared;
    }
    __syncthreads();
}

__device__ __forceinline__ const char* slot_blob(const FfnArgs& a, const Plan& p, int j) {
    const int e = p.expert[j];
    return reinterpret_cast<const char*>(e >= 0 ? a.eptr[e] : a.sptr[-1 - e]);
}

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
};

template <bool BF>
__device__ __forceinline__ float dotc(const Chunk<BF>& w, const Chunk<BF>& x, float acc) {
#pragma unroll
    for (int i = 0; i < Chunk<BF>::N; ++i) acc = fmaf(w.v[i], x.v[i], acc);
    return acc;
}

__device__ __forceinline__ uint4 ld_stream(const char* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint4 ld_cached(const char* p) {
    return *reinterpret_cast<const uint4*>(p);
}

// Sum over a segment of G consecutive lanes (G = 16, 32 or 64); every lane
// of the segment returns the segment's sum.
template <int G>
__device__ __forceinline__ float seg_sum(float v) {
    if (G == 64) return wave_sum(v);
#pragma unroll
    for (int o = G / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ float silu(float g) { return g / (1.f + expf(-g)); }

// ----------------------------------------------------------------------------
// gate/up: rows of W_gate and W_up of one slot -> a = w * silu(g) * u
// ----------------------------------------------------------------------------
template <bool BF, int G, int R, int NB>
__global__ __launch_bounds__(kThreads) void ffn_gate_up(FfnArgs a, int blocks_per_slot) {
    __shared__ Plan p;
    build_plan(a, p);
    const int j = blockIdx.x / blocks_per_slot;
    if (j >= p.n_slots) return;
    const int rows_per_block = kWaves * (64 / G) * R;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int grp = lane / G, g = lane % G;
    const int i0 = (blockIdx.x % blocks_per_slot) * rows_per_block + (wave * (64 / G) + grp) * R;
    if (i0 >= a.I) return;   // I is a multiple of R: the group's rows are all valid
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

    for (int c = g; c < cpr; c += G) {
        uint4 qg[R], qu[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            qg[r] = ld_stream(wg + r * rowb + size_t(c) * 16);
            qu[r] = ld_stream(wu + r * rowb + size_t(c) * 16);
        }
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
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (!((tm >> b) & 1u)) continue;
        const float wb = p.wt[j][b];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float gs = seg_sum<G>(accg[r][b]);
            const float us = seg_sum<G>(accu[r][b]);
            if (g == 0) a.act[(size_t(j) * a.B + b) * a.I + i0 + r] = wb * silu(gs) * us;
        }
    }
}

// ----------------------------------------------------------------------------
// down: y[b][h] = sum over slots j (ascending) of W_down_j[h] . a[j][b]
// ----------------------------------------------------------------------------
template <bool BF, int G, int R, int NB>
__global__ __launch_bounds__(kThreads) void ffn_down(FfnArgs a) {
    __shared__ Plan p;
    build_plan(a, p);
    const int rows_per_block = kWaves * (64 / G) * R;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int grp = lane / G, g = lane % G;
    const int h0 = blockIdx.x * rows_per_block + (wave * (64 / G) + grp) * R;
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.n_experts)
        atomicAdd(a.n_experts, (unsigned long long)p.n_routed);
    if (h0 >= a.H) return;   // H is a multiple of R
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
        const unsigned tm = p.tok[j];
        const char* wd = slot_blob(a, p, j) + 2 * size_t(a.I) * a.H * esz + size_t(h0) * rowb;
        const float* act = a.act + size_t(j) * a.B * a.I;
        for (int c = g; c < cpr; c += G) {
            uint4 q[R];
#pragma unroll
            for (int r = 0; r < R; ++r) q[r] = ld_stream(wd + r * rowb + size_t(c) * 16);
            Chunk<BF> cw[R];
#pragma unroll
            for (int r = 0; r < R; ++r) cw[r].unpack(q[r]);
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                if (!((tm >> b) & 1u)) continue;
                const float4* ap = reinterpret_cast<const float4*>(act + size_t(b) * a.I + c * N);
                Chunk<BF> cx;
#pragma unroll
                for (int q4 = 0; q4 < N / 4; ++q4) {
                    const float4 f = ap[q4];
                    cx.v[q4 * 4 + 0] = f.x; cx.v[q4 * 4 + 1] = f.y;
                    cx.v[q4 * 4 + 2] = f.z; cx.v[q4 * 4 + 3] = f.w;
                }
#pragma unroll
                for (int r = 0; r < R; ++r) acc[r][b] = dotc<BF>(cw[r], cx, acc[r][b]);
            }
        }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (b >= a.B) break;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float s = seg_sum<G>(acc[r][b]);
            if (g == 0) a.y[size_t(b) * a.H + h0 + r] = s;
        }
    }
}

// lanes per row: the widest of 64/32/16 that divides the row's chunk count
int pick_group(int chunks) {
    if (chunks % 64 == 0 || chunks > 512) return 64;
    if (chunks % 32 == 0) return 32;
    if (chunks % 16 == 0) return 16;
    return 64;
}

template <bool BF, int G, int NB>
int launch_g(const FfnArgs& a, int slots, hipStream_t s, int G_down, hipEvent_t ev_mid) {
    constexpr int R = 2;
    const int rows_up = kWaves * (64 / G) * R;
    const int bps = (a.I + rows_up - 1) / rows_up;
    hipLaunchKernelGGL((ffn_gate_up<BF, G, R, NB>), dim3(unsigned(bps * slots)), dim3(kThreads), 0, s,
                       a, bps);
    STMOE_LAUNCHED();
    if (ev_mid) STMOE_HIP(hipEventRecord(ev_mid, s));
    // the down kernel's row length is I (its own lane grouping)
    switch (G_down) {
        case 16: {
            const int rows = kWaves * 4 * R;
            hipLaunchKernelGGL((ffn_down<BF, 16, R, NB>), dim3(unsigned((a.H + rows - 1) / rows)),
                               dim3(kThreads), 0, s, a);
            break;
        }
        case 32: {
            const int rows = kWaves * 2 * R;
            hipLaunchKernelGGL((ffn_down<BF, 32, R, NB>), dim3(unsigned((a.H + rows - 1) / rows)),
                               dim3(kThreads), 0, s, a);
            break;
        }
        default: {
            const int rows = kWaves * 1 * R;
            hipLaunchKernelGGL((ffn_down<BF, 64, R, NB>), dim3(unsigned((a.H + rows - 1) / rows)),
                               dim3(kThreads), 0, s, a);
        }
    }
    STMOE_LAUNCHED();
    return STMOE_OK;
}

template <bool BF, int NB>
int launch_nb(const FfnArgs& a, int slots, hipStream_t s, hipEvent_t ev_mid) {
    constexpr int esz = BF ? 2 : 4;
    const int gu = pick_group(a.H * esz / 16);
    const int gd = pick_group(a.I * esz / 16);
    switch (gu) {
        case 16: return launch_g<BF, 16, NB>(a, slots, s, gd, ev_mid);
        case 32: return launch_g<BF, 32, NB>(a, slots, s, gd, ev_mid);
        default: return launch_g<BF, 64, NB>(a, slots, s, gd, ev_mid);
    }
}

template <bool BF>
int launch_gemv(const FfnArgs& a, int slots, hipStream_t s, hipEvent_t ev_mid) {
    if (a.B <= 1) return launch_nb<BF, 1>(a, slots, s, ev_mid);
    if (a.B <= 2) return launch_nb<BF, 2>(a, slots, s, ev_mid);
    if (a.B <= 4) return launch_nb<BF, 4>(a, slots, s, ev_mid);
    if (a.B <= 8) return launch_nb<BF, 8>(a, slots, s, ev_mid);
    return launch_nb<BF, 16>(a, slots, s, ev_mid);
}

}  // namespace

// Internal entry used by the decode-layer orchestration (no argument checks).
int ffn_launch(const void* x, const int32_t* idx, const float* w, int B, int K, int H, int I, int E,
               int dtype, const void* const* eptr, const void* const* sptr, int n_shared,
               float* y, void* ws, hipStream_t s, unsigned long long* n_experts, hipEvent_t ev_mid) {
    FfnArgs a;
    a.x = x;
    a.idx = idx;
    a.w = w;
    a.eptr = eptr;
    a.sptr = sptr;
    a.B = B;
    a.K = K;
    a.H = H;
    a.I = I;
    a.E = E;
    a.n_shared = n_shared;
    a.act = reinterpret_cast<float*>(ws);
    a.y = y;
    a.n_experts = n_experts;
    const int slots = (B * K < E ? B * K : E) + n_shared;
    return dtype == STMOE_BF16 ? launch_gemv<true>(a, slots, s, ev_mid)
                                : launch_gemv<false>(a, slots, s, ev_mid);
}

}  // namespace stmoe

using namespace stmoe;

extern "C" size_t moe_expert_ffn_workspace_bytes(int B, int K, int E, int I, int n_shared) {
    if (B < 1 || K < 1 || E < 1 || I < 1 || n_shared < 0) return 0;
    const size_t slots = size_t(B * K < E ? B * K : E) + n_shared;
    return slots * B * I * sizeof(float);
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
    STMOE_CHECK(ws_bytes >= moe_expert_ffn_workspace_bytes(B, K, E, I, n_shared), "workspace too small");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(x) & 15) == 0, "x must be 16-byte aligned");
    return ffn_launch(x, topk_idx, topk_w, B, K, H, I, E, dtype, expert_ptrs, shared_ptrs, n_shared, y,
                      ws, as_stream(stream), nullptr, nullptr);
}
