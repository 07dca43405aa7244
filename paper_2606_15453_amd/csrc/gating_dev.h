// Gating device code (Section 2): per-expert logits, a completion ticket,
// and the softmax / top-K tail that the last workgroup runs.  Shared by the
// standalone router kernel and the fused router + predictor kernel.
#pragma once

#include "common.h"

namespace stmoe {
namespace gating {

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

// Logits of expert row blockIdx.x for every token, written to the
// workspace, then a completion ticket.  Returns true only in the workgroup
// that took the last ticket (after an acquire fence); all its threads agree.
template <bool BF16>
__device__ bool logits_and_ticket(const RouteArgs& a, float (*part)[kThreads / 64], bool& last) {
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
    if (!last) return false;
    __threadfence();   // acquire: see every workgroup's logits
    return true;
}

// Softmax and top-K of every batch row (one wave per row) in the last
// workgroup.  Writes idx/w (and the selection to s_idx in LDS when given),
// resets the ticket, and ends with a barrier.
__device__ void softmax_topk_tail(const RouteArgs& a, int32_t* s_idx) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
            if (s_idx) s_idx[b * a.K + lane] = my_i;
        }
    }
    if (tid == 0) atomicExch(a.ticket, 0u);
    __syncthreads();
}

}  // namespace gating
}  // namespace stmoe
