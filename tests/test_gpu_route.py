"""GPU parity of moe_route_topk (Section 2 gating) against the oracle."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _case(B, H, E, K, dtype, seed, planted=False):
    from paper_2606_15453_amd import workload as W
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((E, H))
    g /= np.linalg.norm(g, axis=1, keepdims=True)
    if planted:
        x = np.zeros((B, H))
        for b in range(B):
            x[b] = 3 * g[rng.choice(E, size=K, replace=False)].sum(0) + rng.normal(0, 1 / 16, H)
    else:
        x = rng.normal(0, 1, (B, H))
    conv = (lambda a: W.f32_to_bf16_bits(a.astype(np.float32))) if dtype == "bf16" else \
        (lambda a: a.astype(np.float32))
    return conv(x), conv(g)


CASES = [
    # B, H, E, K, dtype, planted
    (1, 256, 8, 2, "f32", True),        # tiny stack shape
    (1, 4096, 8, 2, "bf16", True),      # Mixtral-8x7B shape
    (1, 2048, 128, 8, "bf16", True),    # Qwen3-30B-A3B shape, batch 1
    (8, 2048, 128, 8, "bf16", True),    # ... batch 8
    (4, 2048, 64, 6, "bf16", True),     # DeepSeek-V2-Lite shape
    (16, 4096, 128, 8, "bf16", True),   # Qwen3-235B-A22B shape
    (3, 2056, 60, 4, "bf16", False),    # E not a multiple of 64, ragged H
    (2, 64, 256, 16, "bf16", False),    # maximum E and K
    (5, 8, 1, 1, "f32", False),         # degenerate: one expert
    (16, 16384, 200, 16, "f32", False), # maximum H and B
]


@pytest.mark.parametrize("B,H,E,K,dtype,planted", CASES)
@pytest.mark.parametrize("renorm", [False, True])
def test_route_parity(B, H, E, K, dtype, planted, renorm):
    import torch
    from gpuhelp import DEV, to_dev
    from oracle.stmoe_oracle import decode_storage, route
    from paper_2606_15453_amd import stmoe as S
    xs, gs = _case(B, H, E, K, dtype, seed=B * 1000 + E + H, planted=planted)
    ref = route(decode_storage(xs), decode_storage(gs), K, renorm=renorm)
    x, g = to_dev(xs), to_dev(gs)
    idx = torch.full((B, K), -7, dtype=torch.int32, device=DEV)
    w = torch.zeros((B, K), dtype=torch.float32, device=DEV)
    z = torch.zeros((B, E), dtype=torch.float32, device=DEV)
    ws = torch.zeros(S.route_workspace_bytes(B, E), dtype=torch.uint8, device=DEV)
    for rep in range(2):          # the workspace is reusable
        S.route_topk(x, g, K, idx, w, ws, renorm=renorm, logits=z)
        torch.cuda.synchronize()
    gi, gw, gz = idx.cpu().numpy(), w.cpu().numpy(), z.cpu().numpy()
    # logits: fp32 accumulation error bound
    mag = np.abs(decode_storage(xs)) @ np.abs(decode_storage(gs)).T
    assert np.all(np.abs(gz - ref["z"]) <= 1e-5 * mag + 1e-6)
    exact = order_ties = 0
    for b in range(B):
        if ref["tie_boundary"][b]:
            continue                     # the set itself may legitimately differ
        if ref["tie_order"][b]:
            assert sorted(gi[b]) == sorted(ref["idx"][b])   # only the order may differ
            order_ties += 1
        else:
            assert gi[b].tolist() == ref["idx"][b].tolist()
            exact += 1
        order = np.argsort(ref["idx"][b])
        gorder = np.argsort(gi[b])
        assert np.allclose(gw[b][gorder], ref["w"][b][order], rtol=2e-5, atol=1e-7)
    if planted:
        # planted rows have a wide gap between rank K and K+1: never a boundary tie
        assert exact + order_ties == B


def test_route_reports_near_ties_consistently():
    """Two experts with identical rows tie exactly: the lower index wins."""
    import torch
    from gpuhelp import DEV, to_dev
    from paper_2606_15453_amd import stmoe as S
    H, E, K = 64, 8, 1
    g = np.zeros((E, H), np.float32)
    g[3, 0] = g[5, 0] = 1.0
    x = np.ones((1, H), np.float32)
    idx = torch.zeros((1, K), dtype=torch.int32, device=DEV)
    w = torch.zeros((1, K), dtype=torch.float32, device=DEV)
    ws = torch.zeros(S.route_workspace_bytes(1, E), dtype=torch.uint8, device=DEV)
    S.route_topk(to_dev(x), to_dev(g), K, idx, w, ws)
    assert idx.item() == 3
