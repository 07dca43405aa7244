// Gating (Section 2): logits z = x W_g^T, softmax, top-K by logit.
//
// One launch.  Each workgroup computes the logits of one expert row for all
// B tokens (256 lanes split H into 16-byte chunks, DPP wave sums, one LDS
// combine), writes them to the workspace and takes a completion ticket.  The
// workgroup that takes the last ticket runs softmax and top-K: one wave per
// batch row, K rounds of a wave-wide arg-max (value desc, index asc).  That
// workgroup also resets the ticket, so the workspace is zero again on exit.
#include "common.h"

namespace stmoe {
namespace {

constexpr int kThreads = 256;

struct RouteArgs {
    const void* x;
    const void* wg;
    int B, H, E, K, renorm, bf16;
    int32_t* idx;
    float* w;
    float* logits;
    float* zbuf;        // [B][E] workspace
    unsigned* ticket;   // workspace, zero between launches
};

template <bool BF16>
__device__ __forceinline__ void dot_chunk(const void* wrow, const void* xrow, int c, float& acc) {
    // one 16-byte chunk: 8 bf16 or 4 fp32 values of the row and of x
    const uint4 wv = reinterpret_cast<const uint4*>(wrow)[c];
    const uint4 xv = reinterpret_cast<const uint4*>(xrow)[c];
    if (BF16) {
        acc += bf16_lo(wv.x) * bf16_lo(xv.x) + bf16_hi(wv.x) * bf16_hi(xv.x);
        acc += bf16_lo(wv.y) * bf16_lo(xv.y) + bf16_hi(wv.y) * bf16_hi(xv.y);
        acc += bf16_lo(wv.z) * bf16_lo(xv.z) + bf16_hi(wv.z) * bf16_hi(xv.z);
        acc += bf16_lo(wv.w) * bf16_lo(xv.w) + bf16_hi(wv.w) * bf16_hi(xv.w);
    } else {
        acc += __uint_as_float(wv.x) * __uint_as_float(xv.x);
        acc += __uint_as_float(wv.y) * __uint_as_float(xv.y);
        acc += __uint_as_float(wv.z) * __uint_as_float(xv.z);
        acc += __uint_as_float(wv.w) * __uint_as_float(xv.w);
    }
}

// Better candidate: larger logit, or equal logit and lower index.  NaN logits
// rank below every number.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    if (bi < 0) return i >= 0;
    if (i < 0) return false;
    const bool vn = v != v, bn = bv != bv;
    if (vn != bn) return bn;
    if (v != bv) return v > bv;
    return i < bi;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void route_topk_kernel(RouteArgs a) {
    __shared__ float part[kMaxB][kThreads / 64];
    __shared__ bool last;
    const int e = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int esz = BF16 ? 2 : 4;
    const int chunks = a.H * esz / 16;
    const char* wrow = reinterpret_cast<const char*>(a.wg) + size_t(e) * a.H * esz;

    for (int b = 0; b < a.B; ++b) {
        const char* xrow = reinterpret_cast<const char*>(a.x) + size_t(b) * a.H * esz;
        float acc = 0.f;
        for (int c = tid; c < chunks; c += kThreads) dot_chunk<BF16>(wrow, xrow, c, acc);
        acc = wave_sum(acc);
        if (lane == 0) part[b][wave] = acc;
    }
    __syncthreads();
    if (tid < a.B) {
        float z = 0.f;
        for (int w = 0; w < kThreads / 64; ++w) z += part[tid][w];
        a.zbuf[tid * a.E + e] = z;
        if (a.logits) a.logits[tid * a.E + e] = z;
    }
    // publish the logits, then take a ticket
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const unsigned t = atomicAdd(a.ticket, 1u);
        last = (t == unsigned(gridDim.x) - 1);
    }
    __syncthreads();
    if (!last) return;
    __threadfence();   // acquire: see every workgroup's logits

    // softmax + top-K, one wave per batch row
    for (int b = wave; b < a.B; b += kThreads / 64) {
        float v[kMaxE / 64];
        int id[kMaxE / 64];
#pragma unroll
        for (int j = 0; j < kMaxE / 64; ++j) {
            const int ee = lane + 64 * j;
            id[j] = ee < a.E ? ee : -1;
            v[j] = ee < a.E ? a.zbuf[b * a.E + ee] : 0.f;
        }
        // max for the softmax (NaN-free inputs assumed for the weights)
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < kMaxE / 64; ++j)
            if (id[j] >= 0) m = fmaxf(m, v[j]);
        for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < kMaxE / 64; ++j)
            if (id[j] >= 0) s += expf(v[j] - m);
        s = wave_sum(s);

        // after the butterfly every lane holds the winner; lane k keeps round k
        float my_w = 0.f, wsum = 0.f;
        int my_i = 0;
        for (int k = 0; k < a.K; ++k) {
            float bv = 0.f;
            int bi = -1;
#pragma unroll
            for (int j = 0; j < kMaxE / 64; ++j)
                if (better(v[j], id[j], bv, bi)) { bv = v[j]; bi = id[j]; }
            for (int o = 32; o > 0; o >>= 1) {
                const float ov = __shfl_xor(bv, o, 64);
                const int oi = __shfl_xor(bi, o, 64);
                if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
            }
#pragma unroll
            for (int j = 0; j < kMaxE / 64; ++j)
                if (id[j] == bi) id[j] = -1;
            const float p = expf(bv - m) / s;
            wsum += p;
            if (lane == k) { my_w = p; my_i = bi; }
        }
        if (lane < a.K) {
            a.idx[b * a.K + lane] = my_i;
            a.w[b * a.K + lane] = a.renorm ? my_w / wsum : my_w;
        }
    }
    if (tid == 0) atomicExch(a.ticket, 0u);
}

}  // namespace
}  // namespace stmoe

using namespace stmoe;

extern "C" size_t moe_route_workspace_bytes(int B, int E) {
    if (B < 1 || E < 1) return 0;
    return (size_t(B) * E * sizeof(float) + 255) / 256 * 256 + 256;
}

extern "C" int moe_route_topk(const void* x, const void* w_gate, int B, int H, int E, int K,
                              int dtype, int renorm, int32_t* topk_idx, float* topk_w,
                              float* logits, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    STMOE_CHECK(x && w_gate && topk_idx && topk_w && ws, "null pointer");
    STMOE_CHECK(B >= 1 && B <= kMaxB, "B must be in [1, 16]");
    STMOE_CHECK(E >= 1 && E <= kMaxE, "E must be in [1, 256]");
    STMOE_CHECK(K >= 1 && K <= E && K <= kMaxK, "K must be in [1, min(E, 16)]");
    STMOE_CHECK(H >= 8 && H % 8 == 0 && H <= kMaxH, "H must be a multiple of 8 in [8, 16384]");
    STMOE_CHECK(dtype == STMOE_BF16 || dtype == STMOE_F32, "dtype must be STMOE_BF16 or STMOE_F32");
    STMOE_CHECK(ws_bytes >= moe_route_workspace_bytes(B, E), "workspace too small");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                    (reinterpret_cast<uintptr_t>(w_gate) & 15) == 0,
                "x and w_gate must be 16-byte aligned");
    RouteArgs a;
    a.x = x;
    a.wg = w_gate;
    a.B = B;
    a.H = H;
    a.E = E;
    a.K = K;
    a.renorm = renorm ? 1 : 0;
    a.bf16 = dtype == STMOE_BF16;
    a.idx = topk_idx;
    a.w = topk_w;
    a.logits = logits;
    a.zbuf = reinterpret_cast<float*>(ws);
    a.ticket = reinterpret_cast<unsigned*>(reinterpret_cast<char*>(ws) +
                                           (size_t(B) * E * sizeof(float) + 255) / 256 * 256);
    if (a.bf16)
        hipLaunchKernelGGL(route_topk_kernel<true>, dim3(E), dim3(kThreads), 0, as_stream(stream), a);
    else
        hipLaunchKernelGGL(route_topk_kernel<false>, dim3(E), dim3(kThreads), 0, as_stream(stream), a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}
