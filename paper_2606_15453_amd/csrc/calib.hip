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
