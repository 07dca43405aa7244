"""Parity at the full workload sizes, in the launch configuration the decode
benchmark times: every expert of the whole stack resident in HBM, one
moe_decode_token call per token (router logits, gate/up with its routing
prologue, down, the predictor's update and prediction of every layer in one
side-stream launch per token, HIP events around the FFN), for the first
decode tokens of the seeded workload.

Checked against the oracle: the selection of every (token, layer, row)
(bit-exact, rows with an fp64 near-tie excluded and counted), the predictor's
per-layer hit and prediction counts (Algorithm 3, Eq. 1) and its final tables,
and the FFN output y of sampled (token, layer) pairs within relative L2 1e-2
(Section 2; the oracle widens the generated bf16 weights to fp64)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TOL = 1e-2
N_TOKENS = 3


class FullStack:
    """One workload at its full size in HBM: one tensor of all L*E expert blobs
    (and the shared experts), router rows, and hidden states for n decode tokens."""

    def __init__(self, cfg, n_tokens):
        import torch
        from gpuhelp import DEV, to_dev
        from paper_2606_15453_amd import workload as W
        self.cfg = cfg
        self.sel = W.planted_trace(cfg)
        self.prof = W.profiling_selections(cfg, self.sel)
        self.wg = [W.router_rows(cfg, l) for l in range(cfg.L)]
        self.wg_dev = [to_dev(g) for g in self.wg]
        self.x_store = [[W.to_storage(cfg, W.hidden_f64(cfg, self.sel, cfg.P + t, l)) for l in range(cfg.L)]
                        for t in range(n_tokens)]
        self.x_dev = [to_dev(np.stack(xs)) for xs in self.x_store]
        dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        self.blobs = torch.empty((cfg.L * cfg.E, cfg.blob_elems), dtype=dt, device=DEV)
        for i in range(cfg.L * cfg.E):
            W.expert_blob_torch(cfg, i // cfg.E, i % cfg.E, self.blobs[i])
        self.shared = None
        if cfg.n_shared:
            self.shared = torch.empty((cfg.L * cfg.n_shared, cfg.blob_elems), dtype=dt, device=DEV)
            for i in range(cfg.L * cfg.n_shared):
                W.expert_blob_torch(cfg, i // cfg.n_shared, i % cfg.n_shared, self.shared[i], shared=True)
        torch.cuda.synchronize()

    def mats_f64(self, blob):
        """(W_gate [I][H], W_up [I][H], W_down [H][I]) of a generated blob as float64."""
        cfg = self.cfg
        b = blob.to("cpu").double().numpy()
        n = cfg.H * cfg.I
        return b[:n].reshape(cfg.I, cfg.H), b[n:2 * n].reshape(cfg.I, cfg.H), b[2 * n:].reshape(cfg.H, cfg.I)


def _gpu_decode(st, n_tokens, cache=None, mode=None):
    import torch
    from gpuhelp import DEV, storage_dtype
    from paper_2606_15453_amd import stmoe as S
    cfg = st.cfg
    mode = S.MODE_STMOE if mode is None else mode
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(st.prof)
    resident = None if cache else [st.blobs[i].data_ptr() for i in range(cfg.L * cfg.E)]
    shared = None if st.shared is None else [st.shared[i].data_ptr() for i in range(st.shared.shape[0])]
    ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                          [g.data_ptr() for g in st.wg_dev], predictor=pred, cache=cache,
                          resident_ptrs=resident, shared_ptrs=shared, n_shared=cfg.n_shared)
    ctx.set_timing(1)
    if cache is None:
        ctx.set_predictor_batch(True)    # as the bench's resident runs
    idx_hist, ys = [], []
    for t in range(n_tokens):
        y = torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device=DEV)
        ctx.token(t, st.x_dev[t], y, mode=mode)
        idx, _ = ctx.last_routing()
        idx_hist.append(idx)
        ys.append(y)
    torch.cuda.synchronize()
    stats = pred.stats()
    tables = pred.export()
    ctx.close()
    pred.close()
    return idx_hist, ys, stats, tables


@pytest.mark.parametrize("name", ["mixtral", "qwen30b", "qwen30b-b8", "dsv2lite"])
def test_full_size_decode_matches_oracle(name):
    import torch
    from gpuhelp import rel_l2
    from oracle.stmoe_oracle import MODE_STMOE, decode_reference, decode_storage, moe_ffn, route
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name]
    print(f"[full-size] {cfg.name}: generating the stack", flush=True)
    st = FullStack(cfg, N_TOKENS)
    try:
        idx_hist, ys, stats, tables = _gpu_decode(st, N_TOKENS)
        print(f"[full-size] {cfg.name}: {N_TOKENS} tokens decoded; running the oracle", flush=True)
        x_of = lambda t, l: decode_storage(st.x_store[t][l])
        wg_of = lambda l: decode_storage(st.wg[l])
        ref = decode_reference(cfg.L, cfg.E, cfg.K, cfg.B, x_of, wg_of, st.prof, N_TOKENS, mode=MODE_STMOE)
        # selections: every (token, layer, row), near-ties excluded and counted
        ties = 0
        for t in range(N_TOKENS):
            for l in range(cfg.L):
                r = route(x_of(t, l), wg_of(l), cfg.K)
                for b in range(cfg.B):
                    if r["tie_boundary"][b]:
                        ties += 1
                        continue
                    assert sorted(idx_hist[t][l][b].tolist()) == sorted(r["idx"][b].tolist()), (t, l, b)
        print(f"[full-size] {cfg.name}: near-tie rows {ties} of {N_TOKENS * cfg.L * cfg.B}", flush=True)
        if ties == 0:
            # with identical selections the predictor state is determined exactly
            assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
            assert np.array_equal(stats[:, 2], ref["npred"].sum(axis=0))
            _, rci, rcc, rht = ref["predictor"].tables()
            _, ci, cc, ht = tables
            assert np.array_equal(ci, rci) and np.array_equal(cc, rcc) and np.array_equal(ht, rht)
        # FFN outputs of sampled (token, layer) pairs
        for t, l in [(0, 0), (1, cfg.L // 2), (N_TOKENS - 1, cfg.L - 1)]:
            r = ref["idx"][t * cfg.L + l], ref["w"][t * cfg.L + l]
            experts = {e: st.mats_f64(st.blobs[l * cfg.E + e]) for e in sorted(set(r[0].ravel().tolist()))}
            shared = [st.mats_f64(st.shared[l * cfg.n_shared + s]) for s in range(cfg.n_shared)]
            y_ref = moe_ffn(x_of(t, l), r[0], r[1], lambda e: experts[e], shared=shared)
            got = ys[t][l].cpu().numpy()
            err = rel_l2(got, y_ref)
            print(f"[full-size] {cfg.name}: token {t} layer {l}: rel L2 {err:.3e}", flush=True)
            assert np.isfinite(got).all()
            assert err <= TOL, (t, l, err)
            del experts, shared
    finally:
        del st
        torch.cuda.empty_cache()


@pytest.mark.parametrize("mode,device", [(0, 0), (1, 0), (1, 1)])
def test_full_size_capped_cache(mode, device):
    """DeepSeek-V2-Lite shapes at full size (26 layers, 64 routed experts of
    17.3 MB in a pinned host pool, 24 HBM slots per layer, two shared experts
    in HBM, batch 4), decoded as the bench's capped runs do: the cache's
    copy counts equal the oracle's cache policy, and every output is
    bit-identical to the all-resident run (on-demand loading and ST-MoE
    prefetch; decisions on the host or on the device)."""
    import torch
    from gpuhelp import DEV
    from oracle.stmoe_oracle import decode_reference, decode_storage
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["dsv2lite"]
    print(f"[full-size capped] {cfg.name}: mode {mode}, device decisions {device}", flush=True)
    st = FullStack(cfg, N_TOKENS)
    pool = None
    try:
        _, ys_res, _, _ = _gpu_decode(st, N_TOKENS)
        blob = cfg.blob_bytes
        pool = S.PinnedHost(cfg.L * cfg.E * blob)
        host = pool.tensor()
        for i in range(cfg.L * cfg.E):
            host[i * blob:(i + 1) * blob].copy_(st.blobs[i].view(torch.uint8))
        n_stage = max(0, min(cfg.B * cfg.K, cfg.E) - cfg.C)
        arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.C, blob, n_stage), dtype=torch.uint8, device=DEV)
        demand, side = torch.cuda.Stream(), torch.cuda.Stream()
        warm = W.warm_sets(cfg, st.prof)
        cache = S.ExpertCache(cfg.L, cfg.E, cfg.C, blob, n_stage, arena,
                              [pool.ptr + i * blob for i in range(cfg.L * cfg.E)], demand, side)
        cache.warm(warm)
        cache.set_device_policy(device)
        idx_hist, ys, _, _ = _gpu_decode(st, N_TOKENS, cache=cache, mode=mode)
        demand.synchronize()
        side.synchronize()
        cst = cache.stats()
        cache.close()
        del arena
        for t in range(N_TOKENS):
            assert torch.equal(ys[t], ys_res[t]), t
        ref = decode_reference(cfg.L, cfg.E, cfg.K, cfg.B, lambda t, l: decode_storage(st.x_store[t][l]),
                               lambda l: decode_storage(st.wg[l]), st.prof, N_TOKENS, C=cfg.C, warm=warm,
                               mode=mode)
        assert ref["tie_boundary"] == 0
        n = ref["cache"].n
        print(f"[full-size capped] counts {cst}", flush=True)
        assert cst == dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                           useful=n.useful, wasted=n.wasted)
    finally:
        if pool is not None:
            pool.close()
        del st
        torch.cuda.empty_cache()
