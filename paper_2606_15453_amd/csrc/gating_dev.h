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
__device__ __forceinline__ void dot_chunk(const uint4 wv, const uint4 xv, float& acc) {
    // one 16-byte chunk: 8 bf16 or 4 fp32 values of the row and of x
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

// Logits of expert row blockIdx.x for the tokens of row group blockIdx.y
// (NB tokens per group), written to the workspace.  The 256 lanes split H
// into 16-byte chunks, two chunks per step, and every chunk of the group's
// tokens is loaded before any is used, so a workgroup costs one round of load
// latency per step.  Each lane adds its chunks in ascending order, then a DPP
// wave sum and an LDS combine in wave order: a token's logit does not depend
// on NB or on the grid.
template <bool BF16, int NB>
__device__ void expert_logits(const RouteArgs& a, float (*part)[kThreads / 64]) {
    const int e = blockIdx.x, b0 = blockIdx.y * NB;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int esz = BF16 ? 2 : 4;
    const int chunks = a.H * esz / 16;
    const uint4* wrow = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(a.wg) + size_t(e) * a.H * esz);
    const uint4* x = reinterpret_cast<const uint4*>(a.x);
    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
    float acc[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) acc[u] = 0.f;
    for (int c = tid; c < chunks; c += 2 * kThreads) {
        const bool two = c + kThreads < chunks;
        const uint4 w0 = wrow[c];
        const uint4 w1 = two ? wrow[c + kThreads] : zero;
        uint4 x0[NB], x1[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const bool in = b0 + u < a.B;
            x0[u] = in ? x[size_t(b0 + u) * chunks + c] : zero;
            x1[u] = in && two ? x[size_t(b0 + u) * chunks + c + kThreads] : zero;
        }
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            dot_chunk<BF16>(w0, x0[u], acc[u]);
            if (two) dot_chunk<BF16>(w1, x1[u], acc[u]);
        }
    }
#pragma unroll
    for (int u = 0; u < NB; ++u) {
        const float v = wave_sum(acc[u]);
        if (lane == 0) part[u][wave] = v;
    }
    __syncthreads();
    if (tid < NB && b0 + tid < a.B) {
        const int b = b0 + tid;
        float z = 0.f;
        for (int w = 0; w < kThreads / 64; ++w) z += part[tid][w];
        a.zbuf[b * a.E + e] = z;
        if (a.logits) a.logits[b * a.E + e] = z;
    }
}

// Softmax and top-K of every batch row in one workgroup, in three steps
// that share LDS buffers passed by the caller (rows of `row` >= E rounded up
// to 4 entries):
//   stage_keys   logits -> order keys and values in LDS
//   rank_winners for each (row, expert) pair, T lanes split the row and count
//                the experts that beat it (larger key, or equal key and lower
//                index): a count below K is its output position, so the
//                selection comes out ordered (logit desc, index asc) with no
//                serial rounds; the winner at position 0 gives the row max
//   row_weights  one wave per row: softmax sum and the K weights.
// The router tail and the expert FFN's routing prologue both run these, so
// their selections and weights are bit-identical.

// Keys padded with 0 up to a multiple of 4: a pad never beats a real key
// and never ties with a lower index.  Ends with a barrier.
__device__ void stage_keys(const float* z, int B, int E, int row, uint32_t* keys, float* zl) {
    const int E4 = (E + 3) & ~3;
    for (int i = threadIdx.x; i < B * E4; i += kThreads) {
        const int b = i / E4, f = i - b * E4;
        const float v = f < E ? z[b * E + f] : 0.f;
        keys[b * row + f] = f < E ? order_key(v) : 0u;
        zl[b * row + f] = v;
    }
    __syncthreads();
}

// win [B][K]: selected experts by position; rowmax [B].  Ends with a barrier.
// The scan counts greater and equal keys (four row entries per LDS read,
// four reads in flight); only a lane that met an equal key other than its
// own rescans its row for equal keys at lower indices.
__device__ void rank_winners(const uint32_t* keys, const float* zl, int B, int E, int K, int row,
                             int32_t* win, float* rowmax) {
    const int tid = threadIdx.x, BE = B * E;
    int T = 1;                                    // lanes per pair (power of two)
    while (T < 16 && BE * T * 2 <= kThreads) T *= 2;
    const int n4 = ((E + 3) & ~3) / 4;
    for (int base = 0; base < BE * T; base += kThreads) {
        const int t = base + tid, i = t / T, part = t & (T - 1);
        const int b = i / E, f = i - b * E;
        int gt = 0, eq = 0;
        const uint32_t* rk = keys + b * row;
        const uint32_t mine = i < BE ? rk[f] : 0u;
        if (i < BE) {
            int c = part;
            for (; c + 3 * T < n4; c += 4 * T) {
                uint4 k[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) k[u] = *reinterpret_cast<const uint4*>(rk + 4 * (c + u * T));
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    gt += int(k[u].x > mine) + int(k[u].y > mine) + int(k[u].z > mine) + int(k[u].w > mine);
                    eq += int(k[u].x == mine) + int(k[u].y == mine) + int(k[u].z == mine) + int(k[u].w == mine);
                }
            }
            for (; c < n4; c += T) {
                const uint4 k = *reinterpret_cast<const uint4*>(rk + 4 * c);
                gt += int(k.x > mine) + int(k.y > mine) + int(k.z > mine) + int(k.w > mine);
                eq += int(k.x == mine) + int(k.y == mine) + int(k.z == mine) + int(k.w == mine);
            }
        }
        for (int o = 1; o < T; o <<= 1) {
            gt += __shfl_xor(gt, o, 64);
            eq += __shfl_xor(eq, o, 64);
        }
        if (i < BE && part == 0) {
            int cnt = gt;
            if (eq > 1)                           // ties: equal keys at lower indices rank higher
                for (int g = 0; g < f; ++g) cnt += rk[g] == mine;
            if (cnt < K) {
                win[b * K + cnt] = f;
                if (cnt == 0) rowmax[b] = zl[b * row + f];
            }
        }
    }
    __syncthreads();
}

// Softmax weights of the winners (NaN-free logits assumed): lanes k < K of
// the row's wave get (expert, weight) of position k.  Whole wave calls it.
__device__ __forceinline__ void row_weights(const float* zl, const int32_t* win, const float* rowmax, int b,
                                            int E, int K, int row, int renorm, int& e, float& wt) {
    const int lane = threadIdx.x & 63;
    const float m = rowmax[b];
    float s = 0.f;
    for (int f = lane; f < E; f += 64) s += expf(zl[b * row + f] - m);
    s = wave_sum(s);
    float p = 0.f;
    e = 0;
    if (lane < K) {
        e = win[b * K + lane];
        p = expf(zl[b * row + e] - m) / s;
    }
    const float wsum = wave_sum(p);
    wt = renorm ? p / wsum : p;
}

// The router tail: writes idx/w (and the selection to s_idx in LDS when
// given) and ends with a barrier.
__device__ void softmax_topk_tail(const RouteArgs& a, const float* z, int32_t* s_idx) {
    constexpr int kRow = kMaxE;
    __shared__ __align__(16) uint32_t keys[kMaxB * kRow];
    __shared__ float zl[kMaxB * kRow];
    __shared__ int32_t win[kMaxB * kMaxK];
    __shared__ float rowmax[kMaxB];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    stage_keys(z, a.B, a.E, kRow, keys, zl);
    rank_winners(keys, zl, a.B, a.E, a.K, kRow, win, rowmax);
    for (int b = wave; b < a.B; b += kThreads / 64) {
        int e;
        float wt;
        row_weights(zl, win, rowmax, b, a.E, a.K, kRow, a.renorm, e, wt);
        if (lane < a.K) {
            a.idx[b * a.K + lane] = e;
            a.w[b * a.K + lane] = wt;
            if (s_idx) s_idx[b * a.K + lane] = e;
        }
    }
    __syncthreads();
}

}  // namespace gating
}  // namespace stmoe
