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
        # the seeded inputs have no near-tie, so the predictor state is determined exactly
        assert ties == 0
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


@pytest.mark.parametrize("mode,device,freq", [(0, 0, False), (1, 0, False), (1, 1, False), (0, 1, True),
                                             (1, 0, True)])
def test_full_size_capped_cache(mode, device, freq):
    """DeepSeek-V2-Lite shapes at full size (26 layers, 64 routed experts of
    17.3 MB in a pinned host pool, 24 HBM slots per layer, two shared experts
    in HBM, batch 4), decoded as the bench's capped runs do: the cache's
    copy counts equal the oracle's cache policy, and every output is
    bit-identical to the all-resident run (on-demand loading and ST-MoE
    prefetch; decisions on the host or on the device; least recently used or
    frequency-aware eviction)."""
    import torch
    from gpuhelp import DEV
    from oracle.stmoe_oracle import decode_reference, decode_storage, use_counts, warm_from_profile
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["dsv2lite"]
    print(f"[full-size capped] {cfg.name}: mode {mode}, device decisions {device}, frequency-aware {freq}",
          flush=True)
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
        arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cfg.C, blob, n_stage), dtype=torch.uint8, device=DEV)
        demand, side = torch.cuda.Stream(), torch.cuda.Stream()
        warm = S.warm_sets(st.prof, cfg.E, cfg.C)
        warm_ref = warm_from_profile(st.prof, cfg.L, cfg.E, cfg.C)
        assert np.array_equal(warm, warm_ref)
        cache = S.ExpertCache(cfg.L, cfg.E, cfg.C, blob, n_stage, arena,
                              [pool.ptr + i * blob for i in range(cfg.L * cfg.E)], demand, side)
        cache.warm(warm)
        counts_ref = use_counts(st.prof, cfg.L, cfg.E) if freq else None
        if freq:
            counts = S.use_counts(st.prof, cfg.E)
            assert np.array_equal(counts, counts_ref)
            cache.set_counts(counts)
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
                               lambda l: decode_storage(st.wg[l]), st.prof, N_TOKENS, C=cfg.C, warm=warm_ref,
                               mode=mode, counts=counts_ref)
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


def test_full_depth_qwen235b_shapes():
    """Qwen3-235B-A22B shapes at full depth (94 layers, 128 experts top-8,
    batch 16, hidden 4096, intermediate 1536) for three decode tokens.  The
    stack (454 GB) does not fit in HBM: 768 distinct expert blobs stand in for
    it, expert (l, e) reading blob (l*E + e) mod 768, once from HBM (resident)
    and once from a pinned host pool behind the 45-slot cache.  Selections,
    hit counts and the predictor tables are bit-exact against the oracle; the
    capped run's copy counts equal the oracle's cache policy; its outputs equal
    the resident run's bit for bit; sampled FFN rows match the fp64 oracle on
    the blobs actually read."""
    import torch
    from gpuhelp import DEV, rel_l2, storage_dtype
    from oracle.stmoe_oracle import (MODE_STMOE, decode_reference, decode_storage, moe_ffn,
                                     warm_from_profile)
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen235b"]
    M = 768
    n_tok = 3
    print(f"[full-depth] {cfg.name}: {M} aliased blobs, {n_tok} tokens", flush=True)
    sel = W.planted_trace(cfg, n_tokens=cfg.P + n_tok)
    prof = W.profiling_selections(cfg, sel)
    wg = [W.router_rows(cfg, l) for l in range(cfg.L)]
    wg_dev = [torch.from_numpy(g.view(np.int16)).to(DEV).view(torch.bfloat16) for g in wg]
    x_store = [[W.to_storage(cfg, W.hidden_f64(cfg, sel, cfg.P + t, l)) for l in range(cfg.L)]
               for t in range(n_tok)]
    x_dev = [torch.from_numpy(np.stack(xs).view(np.int16)).to(DEV).view(torch.bfloat16) for xs in x_store]
    blobs = torch.empty((M, cfg.blob_elems), dtype=torch.bfloat16, device=DEV)
    for i in range(M):
        W.expert_blob_torch(cfg, i // cfg.E, i % cfg.E, blobs[i])
    torch.cuda.synchronize()
    which = lambda l, e: (l * cfg.E + e) % M
    pool = arena = None
    try:
        def run(cache=None):
            pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
            pred.profile(prof)
            resident = None if cache else [blobs[which(l, e)].data_ptr() for l in range(cfg.L)
                                           for e in range(cfg.E)]
            ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                                  [g.data_ptr() for g in wg_dev], predictor=pred, cache=cache,
                                  resident_ptrs=resident)
            idx_hist, ys = [], []
            for t in range(n_tok):
                y = torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device=DEV)
                ctx.token(t, x_dev[t], y, mode=MODE_STMOE)
                idx, _ = ctx.last_routing()
                idx_hist.append(idx)
                ys.append(y)
                print(f"[full-depth] token {t} done ({'capped' if cache else 'resident'})", flush=True)
            torch.cuda.synchronize()
            out = (idx_hist, ys, pred.stats(), pred.export())
            ctx.close()
            pred.close()
            return out

        idx_res, ys_res, stats, tables = run()
        blob = cfg.blob_bytes
        pool = S.PinnedHost(M * blob)
        host = pool.tensor()
        for i in range(M):
            host[i * blob:(i + 1) * blob].copy_(blobs[i].view(torch.uint8))
        n_stage = min(cfg.B * cfg.K, cfg.E) - cfg.C
        arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cfg.C, blob, n_stage), dtype=torch.uint8,
                            device=DEV)
        demand, side = torch.cuda.Stream(), torch.cuda.Stream()
        cache = S.ExpertCache(cfg.L, cfg.E, cfg.C, blob, n_stage, arena,
                              [pool.ptr + which(l, e) * blob for l in range(cfg.L) for e in range(cfg.E)],
                              demand, side)
        warm = S.warm_sets(prof, cfg.E, cfg.C)
        warm_ref = warm_from_profile(prof, cfg.L, cfg.E, cfg.C)
        assert np.array_equal(warm, warm_ref)
        cache.warm(warm)
        cache.set_device_policy(1)
        idx_cap, ys_cap, stats_cap, _ = run(cache)
        demand.synchronize()
        side.synchronize()
        cst = cache.stats()
        cache.close()
        print(f"[full-depth] capped counts {cst}", flush=True)
        for t in range(n_tok):
            assert np.array_equal(idx_cap[t], idx_res[t]), t
            assert torch.equal(ys_cap[t], ys_res[t]), t
        assert np.array_equal(stats_cap, stats)
        x_of = lambda t, l: decode_storage(x_store[t][l])
        wg_of = lambda l: decode_storage(wg[l])
        ref = decode_reference(cfg.L, cfg.E, cfg.K, cfg.B, x_of, wg_of, prof, n_tok, C=cfg.C, warm=warm_ref,
                               mode=MODE_STMOE)
        assert ref["tie_boundary"] == 0
        for t in range(n_tok):
            for l in range(cfg.L):
                r = ref["idx"][t * cfg.L + l]
                for b in range(cfg.B):
                    assert sorted(idx_res[t][l][b].tolist()) == sorted(r[b].tolist()), (t, l, b)
        assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
        assert np.array_equal(stats[:, 2], ref["npred"].sum(axis=0))
        _, rci, rcc, rht = ref["predictor"].tables()
        _, ci, cc, ht = tables
        assert np.array_equal(ci, rci) and np.array_equal(cc, rcc) and np.array_equal(ht, rht)
        n = ref["cache"].n
        assert cst == dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                           useful=n.useful, wasted=n.wasted)
        # sampled rows of the FFN output against the fp64 oracle on the blobs read
        for t, l, b in [(0, 0, 0), (1, 47, 9), (n_tok - 1, cfg.L - 1, cfg.B - 1)]:
            r_idx = ref["idx"][t * cfg.L + l][b:b + 1]
            r_w = ref["w"][t * cfg.L + l][b:b + 1]

            def mats(e):
                bb = blobs[which(l, e)].to("cpu").double().numpy()
                n_ = cfg.H * cfg.I
                return (bb[:n_].reshape(cfg.I, cfg.H), bb[n_:2 * n_].reshape(cfg.I, cfg.H),
                        bb[2 * n_:].reshape(cfg.H, cfg.I))

            y_ref = moe_ffn(x_of(t, l)[b:b + 1], r_idx, r_w, mats)
            err = rel_l2(ys_res[t][l][b:b + 1].cpu().numpy(), y_ref)
            print(f"[full-depth] token {t} layer {l} row {b}: rel L2 {err:.3e}", flush=True)
            assert err <= TOL, (t, l, b, err)
    finally:
        if pool is not None:
            pool.close()
        del blobs, arena
        torch.cuda.empty_cache()
