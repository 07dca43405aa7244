// Status reporting, ABI version and the expert packer.
#include <cstring>
#include <string>

#include "common.h"

namespace stmoe {
namespace {
thread_local std::string g_last_error;
}
void set_error(const std::string& msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }
}  // namespace stmoe

using namespace stmoe;

extern "C" const char* stmoe_last_error(void) { return g_last_error.c_str(); }

extern "C" int stmoe_abi_version(void) { return 2; }

extern "C" int stmoe_host_alloc(size_t bytes, void** out) {
    clear_error();
    STMOE_CHECK(out && bytes > 0, "null output or zero size");
    *out = nullptr;
    const hipError_t e = hipHostMalloc(out, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        set_error(std::string("stmoe_host_alloc: ") + hipGetErrorString(e));
        return e == hipErrorOutOfMemory ? STMOE_ENOMEM : STMOE_EHIP;
    }
    return STMOE_OK;
}

extern "C" int stmoe_host_free(void* p) {
    clear_error();
    if (p) STMOE_HIP(hipHostFree(p));
    return STMOE_OK;
}

extern "C" size_t moe_blob_bytes(int H, int I, int dtype) {
    if (H < 1 || I < 1 || (dtype != STMOE_BF16 && dtype != STMOE_F32)) return 0;
    return size_t(3) * H * I * (dtype == STMOE_BF16 ? 2 : 4);
}

extern "C" int moe_pack_expert(const void* w_gate, const void* w_up, const void* w_down, int H, int I,
                               int dtype, void* blob_out) {
    clear_error();
    STMOE_CHECK(w_gate && w_up && w_down && blob_out, "null pointer");
    STMOE_CHECK(H >= 8 && H % 8 == 0 && I >= 8 && I % 8 == 0, "H and I must be positive multiples of 8");
    STMOE_CHECK(dtype == STMOE_BF16 || dtype == STMOE_F32, "bad dtype");
    const size_t m = size_t(H) * I * (dtype == STMOE_BF16 ? 2 : 4);
    char* o = reinterpret_cast<char*>(blob_out);
    std::memcpy(o, w_gate, m);
    std::memcpy(o + m, w_up, m);
    std::memcpy(o + 2 * m, w_down, m);
    return STMOE_OK;
}
