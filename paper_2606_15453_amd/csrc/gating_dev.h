// Gating device code (Section 2): per-expert logits (one workgroup per
// expert row) and the softmax / top-K tail (one workgroup).  They run as two
// launches: the kernel boundary orders the logits before the tail, where a
// device-scope fence per workgroup would write back the L2 of every XCD.
// Shared by the standalone router and the decode path's router + predictor.
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

// Total order on logits as unsigned keys: larger logit -> larger key; -0
// and +0 are one value; NaN ranks below every number.  Equal keys are
// broken by the lower expert index.
__device__ __forceinline__ uint32_t order_key(float v) {
    if (v != v) return 0u;
    const uint32_t u = v == 0.f ? 0u : __float_as_uint(v);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Logits of expert row blockIdx.x for every token, written to the workspace.
template <bool BF16>
__device__ void expert_logits(const RouteArgs& a, float (*part)[kThreads / 64]) {
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
}

// Softmax and top-K of every batch row in one workgroup, from the logits z
// ([B][E], global or LDS).  For each (row, expert) pair, T lanes split the
// row and count the experts that beat it (larger key, or equal key and
// lower index): a count below K is its output position, so the selection
// comes out ordered (logit desc, index asc) with no serial rounds.  The row
// max is the winner at position 0; one wave per row then forms the softmax
// sum and the K weights.  Writes idx/w (and the selection to s_idx in LDS
// when given) and ends with a barrier.
__device__ void softmax_topk_tail(const RouteArgs& a, const float* z, int32_t* s_idx) {
    constexpr int kRow = kMaxE;                   // LDS row stride
    __shared__ __align__(16) uint32_t keys[kMaxB * kRow];
    __shared__ float zl[kMaxB * kRow];
    __shared__ int32_t win[kMaxB * kMaxK];
    __shared__ float rowmax[kMaxB];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int K = a.K, E = a.E, BE = a.B * a.E;
    const int E4 = (E + 3) & ~3;
    // keys padded with 0 up to a multiple of 4: a pad never beats a real key
    // and never ties with a lower index
    for (int i = tid; i < a.B * E4; i += kThreads) {
        const int b = i / E4, f = i - b * E4;
        const float v = f < E ? z[b * E + f] : 0.f;
        keys[b * kRow + f] = f < E ? order_key(v) : 0u;
        zl[b * kRow + f] = v;
    }
    __syncthreads();
    int T = 1;                                    // lanes per pair (power of two)
    while (T < 16 && BE * T * 2 <= kThreads) T *= 2;
    const int n4 = E4 / 4;
    for (int base = 0; base < BE * T; base += kThreads) {
        const int t = base + tid, i = t / T, part = t & (T - 1);
        const int b = i / E, f = i - b * E;
        int cnt = 0;
        if (i < BE) {
            const uint32_t* row = keys + b * kRow;
            const uint32_t mine = row[f];
            for (int c = part; c < n4; c += T) {
                const uint4 k = *reinterpret_cast<const uint4*>(row + 4 * c);
                const int g = 4 * c;
                cnt += (k.x > mine) + (k.y > mine) + (k.z > mine) + (k.w > mine);
                cnt += (k.x == mine && g < f) + (k.y == mine && g + 1 < f) + (k.z == mine && g + 2 < f) +
                       (k.w == mine && g + 3 < f);
            }
        }
        for (int o = 1; o < T; o <<= 1) cnt += __shfl_xor(cnt, o, 64);
        if (i < BE && part == 0 && cnt < K) {
            win[b * K + cnt] = f;
            if (cnt == 0) rowmax[b] = zl[b * kRow + f];
        }
    }
    __syncthreads();
    for (int b = wave; b < a.B; b += kThreads / 64) {
        // softmax sum (NaN-free inputs assumed for the weights)
        const float m = rowmax[b];
        float s = 0.f;
        for (int f = lane; f < E; f += 64) s += expf(zl[b * kRow + f] - m);
        s = wave_sum(s);
        float p = 0.f;
        int e = 0;
        if (lane < K) {
            e = win[b * K + lane];
            p = expf(zl[b * kRow + e] - m) / s;
        }
        const float wsum = wave_sum(p);
        if (lane < K) {
            a.idx[b * K + lane] = e;
            a.w[b * K + lane] = a.renorm ? p / wsum : p;
            if (s_idx) s_idx[b * K + lane] = e;
        }
    }
    __syncthreads();
}

}  // namespace gating
}  // namespace stmoe
