"""The allocation-free expert FFN entry point (moe_expert_ffn_noalloc): the
same outputs as moe_expert_ffn with a caller workspace, bit for bit, on two
calls in a row (the second with a smaller input), through the C ABI; shapes
beyond its scratch are refused before any device work."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _case(cfg_name, B, seed):
    import torch
    from gpuhelp import DEV
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[cfg_name].scaled(B=B)
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.choice(cfg.E, cfg.K, replace=False) for _ in range(cfg.B)]).astype(np.int32)
    w = rng.random((cfg.B, cfg.K)).astype(np.float32)
    sel = sorted(set(idx.ravel().tolist()))
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    store = torch.empty((len(sel) + cfg.n_shared, cfg.blob_elems), dtype=tdt, device=DEV)
    for k, e in enumerate(sel):
        W.expert_blob_torch(cfg, 0, e, store[k])
    for sh in range(cfg.n_shared):
        W.expert_blob_torch(cfg, 0, sh, store[len(sel) + sh], shared=True)
    ptrs = [store[0].data_ptr()] * cfg.E
    for k, e in enumerate(sel):
        ptrs[e] = store[k].data_ptr()
    eptr = torch.tensor(ptrs, dtype=torch.int64, device=DEV)
    sptr = (torch.tensor([store[len(sel) + s].data_ptr() for s in range(cfg.n_shared)], dtype=torch.int64,
                         device=DEV) if cfg.n_shared else None)
    dt = S.BF16 if cfg.dtype == "bf16" else S.F32
    x = torch.from_numpy(W.to_storage(cfg, rng.normal(0, 1, (cfg.B, cfg.H))).view(
        np.int16 if cfg.dtype == "bf16" else np.float32)).to(DEV)
    if cfg.dtype == "bf16":
        x = x.view(torch.bfloat16)
    return cfg, dt, x, torch.from_numpy(idx).to(DEV), torch.from_numpy(w).to(DEV), eptr, sptr, store


@pytest.mark.parametrize("first,second", [(("qwen235b", 16), ("dsv2lite", 4)),
                                          (("qwen30b-b8", 8), ("qwen30b", 1)),
                                          (("mixtral", 4), ("tiny", 1))])
def test_noalloc_matches_workspace_entry(first, second):
    import torch
    from gpuhelp import DEV
    from paper_2606_15453_amd import stmoe as S
    for name, B in (first, second):
        print(f"[noalloc] {name} B={B}", flush=True)
        cfg, dt, x, ti, tw, eptr, sptr, store = _case(name, B, 31 + B)
        y_ref = torch.empty((cfg.B, cfg.H), dtype=torch.float32, device=DEV)
        ws = torch.zeros(S.ffn_workspace_bytes(cfg.B, cfg.K, cfg.E, cfg.H, cfg.I, cfg.n_shared, dt),
                         dtype=torch.uint8, device=DEV)
        S.expert_ffn(x, ti, tw, cfg.H, cfg.I, cfg.E, dt, eptr, y_ref, ws, shared_ptrs=sptr, n_shared=cfg.n_shared)
        y = torch.full((cfg.B, cfg.H), float("nan"), dtype=torch.float32, device=DEV)
        S.expert_ffn_noalloc(x, ti, tw, cfg.H, cfg.I, cfg.E, dt, eptr, y, shared_ptrs=sptr, n_shared=cfg.n_shared)
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), name
        del store, ws


def test_noalloc_refuses_beyond_scratch():
    import torch
    from gpuhelp import DEV
    from paper_2606_15453_amd import stmoe as S
    B, K, E, H, I = 16, 16, 256, 16384, 16384
    assert S.ffn_workspace_bytes(B, K, E, H, I, 0, S.BF16) > (16 << 20)
    dummy = torch.zeros(64, dtype=torch.int64, device=DEV)
    rc = S._lib.moe_expert_ffn_noalloc(dummy.data_ptr(), dummy.data_ptr(), dummy.data_ptr(), B, K, H, I, E,
                                       S.BF16, dummy.data_ptr(), None, 0, dummy.data_ptr(), None)
    assert rc == S.ENOMEM
    assert "scratch" in S._lib.stmoe_last_error().decode()
