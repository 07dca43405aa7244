// Measurement kernels of known traffic, for pricing the hot-path kernels:
//   stmoe_calib_copy   reads n bytes and writes n bytes (16-byte vector copy);
//                      its FETCH_SIZE / WRITE_SIZE counter readings give the
//                      factor that turns those counters into bytes.
//   stmoe_calib_copy_grid  the same copy on a given number of workgroups,
//                      four 16-byte chunks in flight per thread, non-temporal
//                      (the access pattern of the expert cache's copy kernels):
//                      the copy rate a given workgroup count reaches.
//   stmoe_calib_read   reads n bytes with the same non-temporal 16-byte loads
//                      as the expert FFN and writes one word per workgroup:
//                      the achievable streaming-read bandwidth of the chip,
//                      for two access patterns: a grid-stride sweep (every
//                      load instruction of the grid covers consecutive
//                      bytes), or each workgroup reading one contiguous
//                      region (256 KiB, or 32 KiB as one round of eight
//                      loads per thread) as an expert's rows are read.
//   stmoe_calib_handoff  workgroups that stream a chunk and publish one word
//                      each, and workgroups that stream their own chunk and
//                      then read every published word: as two launches, or
//                      as one launch whose consumers wait for the producers
//                      (the handoff a fused gate/up + down launch would need).
#include "common.h"

namespace stmoe {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void calib_copy_kernel(const uint4* src, uint4* dst, size_t n) {
    const size_t stride = size_t(gridDim.x) * kThreads;
    for (size_t i = size_t(blockIdx.x) * kThreads + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(kThreads) void calib_copy4_kernel(const u32x4* src, u32x4* dst, size_t n) {
    const size_t stride = size_t(gridDim.x) * kThreads;
    size_t k = size_t(blockIdx.x) * kThreads + threadIdx.x;
    for (; k + 3 * stride < n; k += 4 * stride) {
        u32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + k + u * stride);
#pragma unroll
        for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + k + u * stride);
    }
    for (; k < n; k += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + k), dst + k);
}

__global__ __launch_bounds__(kThreads) void calib_read_kernel(const char* src, size_t n, unsigned* out) {
    const size_t stride = size_t(gridDim.x) * kThreads;
    unsigned acc = 0;
    size_t i = size_t(blockIdx.x) * kThreads + threadIdx.x;
    for (; i + stride < n; i += 2 * stride) {
        const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + i);
        const u32x4 b = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + i + stride);
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w;
    }
    if (i < n) {
        const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + i);
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    // keep the loads live: one word per workgroup
    for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
    __shared__ unsigned w[kThreads / 64];
    if ((threadIdx.x & 63) == 0) w[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = w[0] ^ w[1] ^ w[2] ^ w[3];
}

// Workgroup w reads the contiguous 16-byte chunks [w*kBlockChunks,
// (w+1)*kBlockChunks): eight loads per thread in flight, each instruction
// covering 4 KiB of consecutive bytes.
template <size_t kBlockChunks>
__global__ __launch_bounds__(kThreads) void calib_read_blocked_kernel(const char* src, size_t n, unsigned* out) {
    const u32x4* base = reinterpret_cast<const u32x4*>(src);
    const size_t lo = size_t(blockIdx.x) * kBlockChunks;
    const size_t hi = lo + kBlockChunks < n ? lo + kBlockChunks : n;
    unsigned acc = 0;
    size_t i = lo + threadIdx.x;
    for (; i + 7 * kThreads < hi; i += 8 * kThreads) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(base + i + u * kThreads);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < hi; i += kThreads) {
        const u32x4 a = __builtin_nontemporal_load(base + i);
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
    __shared__ unsigned w[kThreads / 64];
    if ((threadIdx.x & 63) == 0) w[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = w[0] ^ w[1] ^ w[2] ^ w[3];
}

// ------------------------------------------------------------- handoff
constexpr unsigned kHandoffSpin = 1u << 15;   // polls before a consumer gives up (each one memory round trip)
// modes 3 and 4: the target is published to kFlagCopies words kFlagStride
// words apart (on different memory channels), from word kFlagBase of sync
// on; mode 4 counts producer p first in group counter p mod kFlagCopies
// (kGroupOffset words after flag copy p mod kFlagCopies), then once per
// complete group in sync[2]
constexpr int kFlagBase = 64, kFlagCopies = 64, kFlagStride = 1024, kGroupOffset = 512;

__device__ unsigned block_sum_u32(unsigned v) {
    __shared__ unsigned red[kThreads / 64];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    unsigned s = 0;
    for (int w = 0; w < kThreads / 64; ++w) s += red[w];
    __syncthreads();
    return s;
}

// Sum of the 32-bit words of this producer's chunk (n16 16-byte chunks),
// eight loads per thread in flight.
__device__ unsigned produce_sum(const u32x4* base, size_t n16) {
    unsigned acc = 0;
    size_t i = threadIdx.x;
    for (; i + 7 * kThreads < n16; i += 8 * kThreads) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(base + i + u * kThreads);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += v[u].x + v[u].y + v[u].z + v[u].w;
    }
    for (; i < n16; i += kThreads) {
        const u32x4 a = __builtin_nontemporal_load(base + i);
        acc += a.x + a.y + a.z + a.w;
    }
    return block_sum_u32(acc);
}

__global__ __launch_bounds__(kThreads) void handoff_produce_kernel(const char* w1, size_t n1, unsigned* act) {
    const unsigned s = produce_sum(reinterpret_cast<const u32x4*>(w1) + size_t(blockIdx.x) * n1, n1);
    if (threadIdx.x == 0) act[blockIdx.x] = s;
}

// A consumer's chunk is NX 16-byte loads per thread, held in registers.
template <int NX>
__device__ __forceinline__ void consume_load(const char* w2, int c, u32x4 (&q)[NX]) {
    const u32x4* base = reinterpret_cast<const u32x4*>(w2) + size_t(c) * NX * kThreads;
#pragma unroll
    for (int u = 0; u < NX; ++u) q[u] = __builtin_nontemporal_load(base + u * kThreads + threadIdx.x);
}

template <int NX, bool COHERENT>
__device__ __forceinline__ void consume_finish(const unsigned* act, int producers, const u32x4 (&q)[NX],
                                               unsigned* out, int c) {
    unsigned s = 0;
    for (int i = threadIdx.x; i < producers; i += kThreads)
        s += COHERENT ? __hip_atomic_load(act + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : act[i];
#pragma unroll
    for (int u = 0; u < NX; ++u) s += q[u].x + q[u].y + q[u].z + q[u].w;
    s = block_sum_u32(s);
    if (threadIdx.x == 0) out[c] = s;
}

template <int NX>
__global__ __launch_bounds__(kThreads) void handoff_consume_kernel(const char* w2, const unsigned* act, int producers,
                                                                   unsigned* out) {
    u32x4 q[NX];
    consume_load<NX>(w2, blockIdx.x, q);
    consume_finish<NX, false>(act, producers, q, out, blockIdx.x);
}

// One launch: workgroups below `producers` produce; the others load their
// chunk, wait (bounded) until the counter reaches `target`, then consume.
// MODE 1: the word is stored write-through (an agent-scope store), the store
// is waited for, then a relaxed counter increment; consumers poll relaxed and
// read the words with agent-scope loads.  MODE 2: plain store and a release
// increment; consumers poll with acquire loads and read plainly.
template <int NX, int MODE>
__global__ __launch_bounds__(kThreads) void handoff_fused_kernel(const char* w1, size_t n1, const char* w2,
                                                                 int producers, unsigned* act, unsigned* out,
                                                                 unsigned* sync, unsigned target) {
    if (int(blockIdx.x) < producers) {
        const unsigned s = produce_sum(reinterpret_cast<const u32x4*>(w1) + size_t(blockIdx.x) * n1, n1);
        if (threadIdx.x == 0) {
            if (MODE == 1 || MODE == 3) {
                __hip_atomic_store(act + blockIdx.x, s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
                const unsigned before = __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                // mode 3: the producer that completes the count tells every flag copy
                if (MODE == 3 && before + 1u == target)
                    for (int r = 0; r < kFlagCopies; ++r)
                        __hip_atomic_store(sync + kFlagBase + r * kFlagStride, target, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
            } else if (MODE == 4) {
                __hip_atomic_store(act + blockIdx.x, s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
                const int g = int(blockIdx.x) % kFlagCopies;
                const unsigned in_group = unsigned((producers - 1 - g) / kFlagCopies + 1);
                const unsigned groups = unsigned(producers < kFlagCopies ? producers : kFlagCopies);
                unsigned* gc = sync + kFlagBase + g * kFlagStride + kGroupOffset;
                if (__hip_atomic_fetch_add(gc, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u == in_group) {
                    // every producer of the group has counted: ready for the next launch
                    __hip_atomic_store(gc, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (__hip_atomic_fetch_add(sync + 2, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u ==
                        groups) {
                        __hip_atomic_store(sync + 2, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        __hip_atomic_fetch_add(sync, unsigned(producers), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        for (int r = 0; r < kFlagCopies; ++r)
                            __hip_atomic_store(sync + kFlagBase + r * kFlagStride, target, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            } else {
                act[blockIdx.x] = s;
                __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        return;
    }
    const int c = int(blockIdx.x) - producers;
    u32x4 q[NX];
    consume_load<NX>(w2, c, q);
    if (threadIdx.x == 0) {
        // mode 3 polls this consumer's flag copy; modes 1 and 2 the count itself
        const unsigned* w = MODE >= 3 ? sync + kFlagBase + (c % kFlagCopies) * kFlagStride : sync;
        unsigned it = 0;
        for (; it < kHandoffSpin; ++it) {
            const unsigned v = MODE == 2 ? __hip_atomic_load(w, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT)
                                         : __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (int(v - target) >= 0) break;
            __builtin_amdgcn_s_sleep(1);
        }
        if (it == kHandoffSpin) atomicOr(sync + 1, 1u);
    }
    __syncthreads();
    consume_finish<NX, MODE != 2>(act, producers, q, out, c);
}

template <int NX>
void launch_handoff(const char* w1, size_t n1, int producers, const char* w2, int consumers, int mode,
                    unsigned* act, unsigned* out, unsigned* sync, unsigned target, hipStream_t s) {
    if (mode == 0) {
        hipLaunchKernelGGL(handoff_produce_kernel, dim3(unsigned(producers)), dim3(kThreads), 0, s, w1, n1, act);
        hipLaunchKernelGGL((handoff_consume_kernel<NX>), dim3(unsigned(consumers)), dim3(kThreads), 0, s, w2, act,
                           producers, out);
    } else if (mode == 1) {
        hipLaunchKernelGGL((handoff_fused_kernel<NX, 1>), dim3(unsigned(producers + consumers)), dim3(kThreads), 0,
                           s, w1, n1, w2, producers, act, out, sync, target);
    } else if (mode == 2) {
        hipLaunchKernelGGL((handoff_fused_kernel<NX, 2>), dim3(unsigned(producers + consumers)), dim3(kThreads), 0,
                           s, w1, n1, w2, producers, act, out, sync, target);
    } else if (mode == 3) {
        hipLaunchKernelGGL((handoff_fused_kernel<NX, 3>), dim3(unsigned(producers + consumers)), dim3(kThreads), 0,
                           s, w1, n1, w2, producers, act, out, sync, target);
    } else {
        hipLaunchKernelGGL((handoff_fused_kernel<NX, 4>), dim3(unsigned(producers + consumers)), dim3(kThreads), 0,
                           s, w1, n1, w2, producers, act, out, sync, target);
    }
}

constexpr size_t kBigBlockChunks = (size_t(256) << 10) / 16;    // pattern 1
constexpr size_t kSmallBlockChunks = (size_t(32) << 10) / 16;   // pattern 2

size_t block_chunks(int pattern) { return pattern == 1 ? kBigBlockChunks : kSmallBlockChunks; }

unsigned blocked_grid_for(size_t n16, int pattern) {
    const size_t c = block_chunks(pattern);
    const size_t g = (n16 + c - 1) / c;
    return unsigned(g < 1 ? 1 : g);
}

unsigned grid_for(size_t n16) {
    size_t g = (n16 + kThreads - 1) / kThreads;
    if (g > 8192) g = 8192;
    return unsigned(g < 1 ? 1 : g);
}

}  // namespace
}  // namespace stmoe

using namespace stmoe;

extern "C" int stmoe_calib_copy(const void* src, void* dst, size_t bytes, void* stream) {
    clear_error();
    STMOE_CHECK(src && dst && bytes > 0 && bytes % 16 == 0, "null pointer or size not a multiple of 16");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(src) & 15) == 0 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0,
                "pointers must be 16-byte aligned");
    const size_t n = bytes / 16;
    hipLaunchKernelGGL(calib_copy_kernel, dim3(grid_for(n)), dim3(kThreads), 0, as_stream(stream),
                       reinterpret_cast<const uint4*>(src), reinterpret_cast<uint4*>(dst), n);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

extern "C" int stmoe_calib_copy_grid(const void* src, void* dst, size_t bytes, int workgroups, void* stream) {
    clear_error();
    STMOE_CHECK(src && dst && bytes > 0 && bytes % 16 == 0, "null pointer or size not a multiple of 16");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(src) & 15) == 0 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0,
                "pointers must be 16-byte aligned");
    STMOE_CHECK(workgroups >= 1 && workgroups <= 1024, "workgroups must be in [1, 1024]");
    hipLaunchKernelGGL(calib_copy4_kernel, dim3(unsigned(workgroups)), dim3(kThreads), 0, as_stream(stream),
                       reinterpret_cast<const u32x4*>(src), reinterpret_cast<u32x4*>(dst), bytes / 16);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

extern "C" size_t stmoe_calib_read_out_words(size_t bytes, int pattern) {
    return pattern == 1 || pattern == 2 ? blocked_grid_for(bytes / 16, pattern) : grid_for(bytes / 16);
}

extern "C" int stmoe_calib_read(const void* src, size_t bytes, int pattern, unsigned* out, void* stream) {
    clear_error();
    STMOE_CHECK(src && out && bytes > 0 && bytes % 16 == 0, "null pointer or size not a multiple of 16");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(src) & 15) == 0, "src must be 16-byte aligned");
    STMOE_CHECK(pattern >= 0 && pattern <= 2,
                "pattern must be 0 (grid stride), 1 (256 KiB per workgroup) or 2 (32 KiB per workgroup)");
    const size_t n = bytes / 16;
    STMOE_CHECK(pattern == 0 || blocked_grid_for(n, pattern) < (1u << 31), "too many workgroups");
    if (pattern == 1)
        hipLaunchKernelGGL(calib_read_blocked_kernel<kBigBlockChunks>, dim3(blocked_grid_for(n, 1)), dim3(kThreads),
                           0, as_stream(stream), reinterpret_cast<const char*>(src), n, out);
    else if (pattern == 2)
        hipLaunchKernelGGL(calib_read_blocked_kernel<kSmallBlockChunks>, dim3(blocked_grid_for(n, 2)),
                           dim3(kThreads), 0, as_stream(stream), reinterpret_cast<const char*>(src), n, out);
    else
        hipLaunchKernelGGL(calib_read_kernel, dim3(grid_for(n)), dim3(kThreads), 0, as_stream(stream),
                           reinterpret_cast<const char*>(src), n, out);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

extern "C" int stmoe_calib_handoff(const void* w1, size_t chunk1, int producers, const void* w2, size_t chunk2,
                                   int consumers, int mode, unsigned* act, unsigned* out, unsigned* sync,
                                   unsigned target, void* stream) {
    clear_error();
    STMOE_CHECK(w1 && w2 && act && out && (mode == 0 || sync), "null pointer");
    STMOE_CHECK((reinterpret_cast<uintptr_t>(w1) & 15) == 0 && (reinterpret_cast<uintptr_t>(w2) & 15) == 0,
                "w1 and w2 must be 16-byte aligned");
    STMOE_CHECK(mode >= 0 && mode <= 4, "mode must be 0 (two launches), 1 (write-through), 2 (release/acquire), "
                                        "3 (flag copies) or 4 (group counters and flag copies)");
    STMOE_CHECK(producers >= 1 && consumers >= 1 && producers + consumers <= (1 << 20), "workgroup counts out of range");
    STMOE_CHECK(chunk1 >= 16 && chunk1 % 16 == 0, "chunk1 must be a positive multiple of 16");
    const size_t nx = chunk2 / (16 * kThreads);
    STMOE_CHECK(chunk2 % (16 * kThreads) == 0 && (nx == 1 || nx == 2 || nx == 4 || nx == 6 || nx == 8),
                "chunk2 must be 4, 8, 16, 24 or 32 KiB");
    const char* a = reinterpret_cast<const char*>(w1);
    const char* b = reinterpret_cast<const char*>(w2);
    const size_t n1 = chunk1 / 16;
    hipStream_t s = as_stream(stream);
    if (nx == 1) launch_handoff<1>(a, n1, producers, b, consumers, mode, act, out, sync, target, s);
    else if (nx == 2) launch_handoff<2>(a, n1, producers, b, consumers, mode, act, out, sync, target, s);
    else if (nx == 4) launch_handoff<4>(a, n1, producers, b, consumers, mode, act, out, sync, target, s);
    else if (nx == 6) launch_handoff<6>(a, n1, producers, b, consumers, mode, act, out, sync, target, s);
    else launch_handoff<8>(a, n1, producers, b, consumers, mode, act, out, sync, target, s);
    STMOE_LAUNCHED();
    return STMOE_OK;
}
