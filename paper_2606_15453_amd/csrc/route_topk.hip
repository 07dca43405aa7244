// Gating (Section 2): logits z = x W_g^T, softmax, top-K by logit.
//
// Two launches.  route_logits_kernel: one workgroup per expert row computes
// its logits for all B tokens (256 lanes split H into 16-byte chunks, up to
// eight tokens per round of loads, DPP wave sums, one LDS combine) into the
// workspace.  route_tail_kernel: one workgroup per batch row ranks every
// expert by counting the logits that beat it (value desc, index asc) and
// forms the softmax weights of the winners.
#include "gating_dev.h"

namespace stmoe {
namespace {

using namespace gating;

template <bool BF16, int NB>
__global__ __launch_bounds__(kThreads) void route_logits_kernel(RouteArgs a) {
    __shared__ float part[NB][kThreads / 64];
    expert_logits<BF16, NB>(a, part);
}

// Tokens per workgroup: four (one load round each, E x ceil(B/4)
// workgroups), fewer for smaller batches.
template <bool BF16>
void launch_logits(const RouteArgs& a, hipStream_t s) {
    if (a.B <= 1)
        hipLaunchKernelGGL((route_logits_kernel<BF16, 1>), dim3(a.E), dim3(kThreads), 0, s, a);
    else if (a.B <= 2)
        hipLaunchKernelGGL((route_logits_kernel<BF16, 2>), dim3(a.E), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL((route_logits_kernel<BF16, 4>), dim3(a.E, (a.B + 3) / 4), dim3(kThreads), 0, s, a);
}

// One workgroup per batch row (blockIdx.x): the tail's steps on that row
// alone.  Ranking, softmax sum and weights of a row do not depend on the
// other rows, so the results equal a one-workgroup tail over all rows.
__global__ __launch_bounds__(kThreads) void route_tail_kernel(RouteArgs a) {
    const int b = blockIdx.x;
    RouteArgs r = a;
    r.B = 1;
    r.idx = a.idx + size_t(b) * a.K;
    r.w = a.w + size_t(b) * a.K;
    softmax_topk_tail(r, a.zbuf + size_t(b) * a.E, nullptr);
}

}  // namespace
}  // namespace stmoe

using namespace stmoe;
using stmoe::gating::RouteArgs;
using stmoe::gating::kThreads;

extern "C" size_t moe_route_workspace_bytes(int B, int E) {
    if (B < 1 || E < 1) return 0;
    return (size_t(B) * E * sizeof(float) + 255) / 256 * 256;
}

namespace stmoe {
// Launch the per-expert logits kernel (the first of the router's two launches).
int launch_route_logits(const RouteArgs& a, hipStream_t s) {
    if (a.bf16)
        launch_logits<true>(a, s);
    else
        launch_logits<false>(a, s);
    STMOE_LAUNCHED();
    return STMOE_OK;
}
}  // namespace stmoe

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
    if (int rc = launch_route_logits(a, as_stream(stream))) return rc;
    hipLaunchKernelGGL(route_tail_kernel, dim3(B), dim3(kThreads), 0, as_stream(stream), a);
    STMOE_LAUNCHED();
    return STMOE_OK;
}

namespace stmoe {
// Internal: the router's logits alone, z [B][E] fp32 (for callers that run
// softmax / top-K elsewhere).  Shapes are validated by the caller.
int route_logits(const void* x, const void* w_gate, int B, int H, int E, int dtype, float* z, hipStream_t s) {
    RouteArgs a{};
    a.x = x;
    a.wg = w_gate;
    a.B = B;
    a.H = H;
    a.E = E;
    a.K = 1;
    a.bf16 = dtype == STMOE_BF16;
    a.zbuf = z;
    return launch_route_logits(a, s);
}
}  // namespace stmoe
