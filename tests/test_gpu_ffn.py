"""GPU parity of moe_expert_ffn (SwiGLU experts weighted by gating
probabilities, Section 2) against the fp64 oracle: relative L2 <= 1e-2."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TOL = 1e-2


def _gpu_ffn(cfg, layer, idx, w, x_store, n_shared=0):
    """moe_expert_ffn on seeded blobs of the row's valid experts."""
    import torch
    from gpuhelp import DEV, blob_dev, i32, ptr_array, storage_dtype, to_dev
    from paper_2606_15453_amd import stmoe as S
    B, K = idx.shape
    sel = sorted(e for e in set(idx.ravel().tolist()) if 0 <= e < cfg.E)
    blobs = {e: blob_dev(cfg, layer, e) for e in sel}
    ptrs = [blobs[e].data_ptr() if e in blobs else 0 for e in range(cfg.E)]
    shared = [blob_dev(cfg, layer, s, shared=True) for s in range(n_shared)]
    y = torch.full((B, cfg.H), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.zeros(S.ffn_workspace_bytes(B, K, cfg.E, cfg.H, cfg.I, n_shared, storage_dtype(cfg)),
                     dtype=torch.uint8, device=DEV)
    S.expert_ffn(to_dev(x_store), i32(idx), torch.from_numpy(w.astype(np.float32)).to(DEV), cfg.H,
                 cfg.I, cfg.E, storage_dtype(cfg), ptr_array(ptrs), y, ws,
                 shared_ptrs=ptr_array([s.data_ptr() for s in shared]) if n_shared else None,
                 n_shared=n_shared)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def _run_ffn(cfg, layer, idx, w, x_store, n_shared=0):
    from gpuhelp import expert_f64, rel_l2
    from oracle.stmoe_oracle import decode_storage, moe_ffn
    got = _gpu_ffn(cfg, layer, idx, w, x_store, n_shared)
    ref = moe_ffn(decode_storage(x_store), idx, w, lambda e: expert_f64(cfg, layer, e),
                  shared=[expert_f64(cfg, layer, s, shared=True) for s in range(n_shared)])
    return got, ref, rel_l2(got, ref)


def _inputs(cfg, B, K, seed, distinct_rows=True):
    from paper_2606_15453_amd import workload as W
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.choice(cfg.E, K, replace=False) for _ in range(B)]).astype(np.int32)
    w = rng.dirichlet(np.ones(cfg.E), size=B)[:, :K].astype(np.float32) + 0.05
    x = rng.normal(0, 1, (B, cfg.H))
    return idx, w, W.to_storage(cfg, x)


@pytest.mark.parametrize("name,B", [("tiny", 1), ("qwen30b", 1), ("dsv2lite", 1), ("qwen30b", 3), ("qwen30b-b8", 8),
                                    ("qwen30b-b8", 12), ("dsv2lite", 4), ("dsv2lite", 9),
                                    ("qwen235b", 16), ("qwen235b", 9), ("qwen235b", 2), ("qwen235b", 4),
                                    ("mixtral", 4), ("mixtral", 8)])
def test_ffn_parity(name, B):
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(B=B)
    idx, w, x = _inputs(cfg, B, cfg.K, seed=B + len(name))
    got, ref, err = _run_ffn(cfg, 1, idx, w, x, n_shared=cfg.n_shared)
    print(f"{name} B={B}: rel L2 {err:.3e}")
    assert np.isfinite(got).all()
    assert err <= TOL


@pytest.mark.parametrize("H,I", [(4096, 1536), (4096, 1472), (4032, 1536)])
def test_ffn_mfma_tiled_shapes(H, I):
    """Batch 16 over 128 experts takes the tiled MFMA gate/up: through LDS with
    two 16-row tiles per wave (H % 128 == 0, I % 128 == 0), with one tile
    (I % 128 != 0), and the direct-load kernel (H % 128 != 0)."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen235b"].scaled(H=H, I=I, B=16)
    idx, w, x = _inputs(cfg, 16, cfg.K, seed=H + I)
    got, ref, err = _run_ffn(cfg, 2, idx, w, x)
    print(f"H={H} I={I}: rel L2 {err:.3e}")
    assert np.isfinite(got).all()
    assert err <= TOL


def test_ffn_parity_mixtral_shape():
    """Full Mixtral-8x7B expert shape (H 4096, I 14336), batch 1, top-2."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["mixtral"]
    idx, w, x = _inputs(cfg, 1, 2, seed=5)
    got, ref, err = _run_ffn(cfg, 0, idx, w, x)
    print(f"mixtral: rel L2 {err:.3e}")
    assert err <= TOL


def test_ffn_shared_tokens_overlap():
    """Several rows selecting the same experts: each expert is read once and
    its tokens are grouped; ragged sizes (H and I not multiples of 64 chunks)."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(H=264, I=40, E=10, K=3, B=6)
    idx = np.array([[0, 1, 2], [2, 1, 0], [9, 0, 4], [4, 9, 1], [3, 5, 7], [0, 2, 1]], np.int32)
    w = np.random.default_rng(2).random((6, 3)).astype(np.float32)
    x = W.to_storage(cfg, np.random.default_rng(3).normal(0, 1, (6, cfg.H)))
    got, ref, err = _run_ffn(cfg, 0, idx, w, x)
    assert err <= TOL


@pytest.mark.parametrize("B", [8, 11])
def test_ffn_batch8_fallback_shapes(B):
    """Batch >= 8 with H, I not multiples of 64 runs the GEMV kernels."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(H=264, I=40, E=12, K=3, B=B)
    idx, w, x = _inputs(cfg, B, 3, seed=B)
    got, ref, err = _run_ffn(cfg, 0, idx, w, x)
    assert err <= TOL


def test_ffn_repeated_calls_reuse_workspace():
    """Completion tickets in the workspace are reset by every call."""
    import torch
    from gpuhelp import DEV, blob_dev, expert_f64, i32, ptr_array, rel_l2, storage_dtype, to_dev
    from oracle.stmoe_oracle import decode_storage, moe_ffn
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    for name, B in (("qwen30b", 1), ("qwen235b", 16)):
        cfg = W.CONFIGS[name].scaled(B=B, E=24)
        blobs = [blob_dev(cfg, 0, e) for e in range(cfg.E)]
        ptrs = ptr_array([b.data_ptr() for b in blobs])
        ws = torch.zeros(S.ffn_workspace_bytes(B, cfg.K, cfg.E, cfg.H, cfg.I, 0, storage_dtype(cfg)),
                         dtype=torch.uint8, device=DEV)
        y = torch.empty((B, cfg.H), dtype=torch.float32, device=DEV)
        for rep in range(3):
            idx, w, x = _inputs(cfg, B, cfg.K, seed=100 + rep)
            S.expert_ffn(to_dev(x), i32(idx), torch.from_numpy(w).to(DEV), cfg.H, cfg.I, cfg.E,
                         storage_dtype(cfg), ptrs, y, ws)
            ref = moe_ffn(decode_storage(x), idx, w, lambda e: expert_f64(cfg, 0, e))
            assert rel_l2(y.cpu().numpy(), ref) <= TOL


def test_ffn_zero_input_and_linearity():
    import torch
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(B=2)
    idx, w, x = _inputs(cfg, 2, cfg.K, seed=9)
    got0, _, _ = _run_ffn(cfg, 0, idx, w, np.zeros_like(x))
    assert np.all(got0 == 0)
    g1, _, _ = _run_ffn(cfg, 0, idx, w, x)
    g2, _, _ = _run_ffn(cfg, 0, idx, 2 * w, x)
    assert np.allclose(g2, 2 * g1, rtol=1e-5, atol=1e-7)


def test_ffn_deterministic():
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(B=4)
    idx, w, x = _inputs(cfg, 4, cfg.K, seed=11)
    a, _, _ = _run_ffn(cfg, 2, idx, w, x)
    b, _, _ = _run_ffn(cfg, 2, idx, w, x)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("name,row", [("qwen30b", [5, 9, 5, -1, 17, 9, 3, 130]), ("tiny", [3, 3]),
                                      ("dsv2lite", [7, 200, 7, 1, 63, -5])])
def test_ffn_repeated_and_out_of_range_entries(name, row):
    """A selection row that repeats an expert or holds an index outside
    [0, E): out-of-range entries are ignored and a repeated expert counts once,
    with the weight of its first entry (batch 1 takes the register slot
    lookup; batch 2 repeats the row and takes the slot plan).  Checked against
    the oracle on the row's distinct valid entries."""
    from paper_2606_15453_amd import workload as W
    base = W.CONFIGS[name]
    K = len(row)
    for B in (1, 2):
        cfg = base.scaled(B=B, K=K, E=max(base.E, K))
        rng = np.random.default_rng(K + B)
        idx = np.array([row] * B, dtype=np.int32)
        w = (rng.random((B, K)) + 0.1).astype(np.float32)
        x = W.to_storage(cfg, rng.normal(0, 1, (B, cfg.H)))
        keep = [k for k in range(K) if 0 <= row[k] < cfg.E and row[k] not in row[:k]]
        got = _gpu_ffn(cfg, 1, idx, w, x, n_shared=cfg.n_shared)
        _, ref, _ = _run_ffn(cfg, 1, idx[:, keep].copy(), w[:, keep].copy(), x, n_shared=cfg.n_shared)
        from gpuhelp import rel_l2
        err = rel_l2(got, ref)
        print(f"{name} B={B} row {row}: rel L2 against the oracle on {len(keep)} entries {err:.3e}")
        assert np.isfinite(got).all() and err <= TOL

