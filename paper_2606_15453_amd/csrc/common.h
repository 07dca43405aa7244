// Internal helpers shared by the library's translation units: status
// handling, argument checks, bf16 decoding and wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/stmoe.h"

namespace stmoe {

void set_error(const std::string& msg);
void clear_error();

// Report a failed HIP call and return STMOE_EHIP from the enclosing function.
#define STMOE_HIP(call)                                                                  \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess) {                                                          \
            ::stmoe::set_error(std::string(#call) + ": " + hipGetErrorString(e_));       \
            return STMOE_EHIP;                                                           \
        }                                                                                \
    } while (0)

#define STMOE_CHECK(cond, msg)                                                           \
    do {                                                                                 \
        if (!(cond)) {                                                                   \
            ::stmoe::set_error(std::string(__func__) + ": " + (msg));                    \
            return STMOE_EINVAL;                                                         \
        }                                                                                \
    } while (0)

// Kernel launches: check the launch itself (configuration errors).
#define STMOE_LAUNCHED()                                                                 \
    do {                                                                                 \
        hipError_t e_ = hipGetLastError();                                               \
        if (e_ != hipSuccess) {                                                          \
            ::stmoe::set_error(std::string(__func__) + ": launch: " + hipGetErrorString(e_)); \
            return STMOE_EHIP;                                                           \
        }                                                                                \
    } while (0)

constexpr int kMaxE = 256;
constexpr int kMaxK = 16;
constexpr int kMaxB = 16;
constexpr int kMaxH = 16384;
// batch x experts up to which the expert FFN's gate/up kernel runs the
// gating itself (every gate/up workgroup ranks the logits, so beyond this the
// separate router tail costs less than the larger prologue)
constexpr int kRouteInFfnMax = 128;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ----------------------------------------------------------------------------
// device helpers
// ----------------------------------------------------------------------------

// Two bf16 values packed in a 32-bit word -> two floats (exact).
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// Sum over the 64 lanes of a wave: DPP row shifts inside each 16-lane row,
// then cross-row broadcasts; every lane returns the full sum.
__device__ __forceinline__ float wave_sum(float v) {
    // within 16-lane rows
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x111, 0xf, 0xf, false)); // row_shr:1
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x112, 0xf, 0xf, false)); // row_shr:2
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x114, 0xf, 0xf, false)); // row_shr:4
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x118, 0xf, 0xf, false)); // row_shr:8
    // lane 15 of each row now holds that row's sum; combine rows
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xa, 0xf, false)); // row_bcast:15
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xc, 0xf, false)); // row_bcast:31
    // lane 63 holds the total
    return __shfl(v, 63, 64);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

}  // namespace stmoe
