"""End-to-end parity of moe_decode_layer / moe_decode_token against the
oracle's decode loop (Section 4.3.4): routing, predictor statistics, cache
decisions and FFN outputs; prediction never changes the numbers."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


class Stack:
    """Device copies of one synthetic MoE stack."""

    def __init__(self, cfg):
        import torch
        from gpuhelp import DEV, blob_dev, to_dev
        from paper_2606_15453_amd import workload as W
        self.cfg = cfg
        self.sel = W.planted_trace(cfg)
        self.wg = [W.router_rows(cfg, l) for l in range(cfg.L)]
        self.wg_dev = [to_dev(g) for g in self.wg]
        self.blobs = [[blob_dev(cfg, l, e) for e in range(cfg.E)] for l in range(cfg.L)]
        self.shared = [[blob_dev(cfg, l, s, shared=True) for s in range(cfg.n_shared)]
                       for l in range(cfg.L)]
        xs = [[W.to_storage(cfg, W.hidden_f64(cfg, self.sel, cfg.P + t, l)) for l in range(cfg.L)]
              for t in range(cfg.T)]
        self.x_store = xs
        self.x_dev = [to_dev(np.stack(xs[t])) for t in range(cfg.T)]      # [L][B][H] per token
        self.prof = W.profiling_selections(cfg, self.sel)
        from oracle.stmoe_oracle import warm_from_profile
        from paper_2606_15453_amd import stmoe as S
        self.warm = S.warm_sets(self.prof, cfg.E, cfg.C)
        self.warm_ref = warm_from_profile(self.prof, cfg.L, cfg.E, cfg.C)
        assert np.array_equal(self.warm, self.warm_ref)

    def shared_ptrs(self):
        return [s.data_ptr() for l in range(self.cfg.L) for s in self.shared[l]]


def _oracle(st, mode, C=None, ffn_tokens=0, renorm=False, online=True, tables=None, min_score=2,
            max_per_layer=None, staged=0, freq=False):
    from gpuhelp import expert_f64
    from oracle.stmoe_oracle import decode_reference, decode_storage, moe_ffn, use_counts
    cfg = st.cfg

    def ffn_of(l):
        sh = [expert_f64(cfg, l, s, shared=True) for s in range(cfg.n_shared)]
        return lambda x, idx, w: moe_ffn(x, idx, w, lambda e: expert_f64(cfg, l, e), shared=sh)

    return decode_reference(cfg.L, cfg.E, cfg.K, cfg.B, lambda t, l: decode_storage(st.x_store[t][l]),
                            lambda l: decode_storage(st.wg[l]), st.prof, cfg.T, C=C,
                            warm=None if C is None else st.warm_ref, mode=mode, ffn_of=ffn_of,
                            ffn_tokens=ffn_tokens, renorm=renorm, online=online, tables=tables,
                            min_score=min_score, max_per_layer=max_per_layer, staged=staged,
                            counts=use_counts(st.prof, cfg.L, cfg.E) if freq else None)


def _counts(n):
    return dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                useful=n.useful, wasted=n.wasted)


def _cumulative_after_layers(cache, L):
    """The oracle cache's cumulative counts after each decode layer (t, l): its
    acquire and the prefetch issued at the end of that layer."""
    out, c = [], dict(hits=0, demand=0, overflow=0, prefetch=0, useful=0, wasted=0)
    log = list(cache.n.log)
    i = 0
    if log and log[0][0] == "P":                             # the first token's layer-0 prefetch
        c["prefetch"] += len(log[0][3])
        i = 1
    while i < len(log):
        ent = log[i]
        assert ent[0] == "A"
        c["demand"] += len(ent[3])
        c["overflow"] += len(ent[4])
        c["hits"] += ent[5]
        c["useful"] += ent[6]
        c["wasted"] += ent[7]
        i += 1
        if i < len(log) and log[i][0] == "P":
            c["prefetch"] += len(log[i][3])
            i += 1
        out.append(dict(c))
    return out


def _run_gpu(st, mode, capped, renorm=False, online=True, tables=None, after_demand=0, device=0,
             device_until=None, device_pool=False, batch=False, C=None, import_tables=None,
             admission=None, layerwise=False, attn_bytes=0, reports=None, staged=0, head=0, graph=False,
             timing_every=0, freq=None, between=None, copy_wgs=None):
    import torch
    from gpuhelp import DEV, storage_dtype
    from paper_2606_15453_amd import stmoe as S
    cfg = st.cfg
    C = cfg.C if C is None else C
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(st.prof)
    if import_tables is not None:
        pred.import_tables(*import_tables)
    stream = torch.cuda.current_stream()
    cache = None
    keep = []
    if capped:
        host = []
        for l in range(cfg.L):
            for e in range(cfg.E):
                h = st.blobs[l][e] if device_pool else st.blobs[l][e].cpu().pin_memory()
                keep.append(h)
                host.append(h.data_ptr())
        n_stage = max(0, min(cfg.B * cfg.K, cfg.E) - C) + 2 * staged
        arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, C, cfg.blob_bytes, n_stage),
                            dtype=torch.uint8, device=DEV)
        demand, side = torch.cuda.Stream(), torch.cuda.Stream()
        keep += [arena, demand, side]
        cache = S.ExpertCache(cfg.L, cfg.E, C, cfg.blob_bytes, n_stage, arena, host, demand, side)
        cache.warm(st.warm if C == cfg.C else S.warm_sets(st.prof, cfg.E, C))
        cache.set_prefetch_order(after_demand)
        # frequency-aware eviction: counts set before the device takes the state over, or after
        counts = S.use_counts(st.prof, cfg.E) if freq else None
        if freq == "before":
            cache.set_counts(counts)
        if copy_wgs is not None:
            cache.set_copy_workgroups(*copy_wgs)
        cache.set_device_policy(device)
        if freq == "after":
            cache.set_counts(counts)
        if staged:
            cache.set_staged_prefetch(staged, head)
        ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                              [g.data_ptr() for g in st.wg_dev], predictor=pred, cache=cache,
                              shared_ptrs=st.shared_ptrs(), n_shared=cfg.n_shared, renorm=renorm,
                              stream=stream)
    else:
        resident = [st.blobs[l][e].data_ptr() for l in range(cfg.L) for e in range(cfg.E)]
        ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                              [g.data_ptr() for g in st.wg_dev], predictor=pred,
                              resident_ptrs=resident, shared_ptrs=st.shared_ptrs(),
                              n_shared=cfg.n_shared, renorm=renorm, stream=stream)
    ctx.set_online_update(online)
    if batch:
        ctx.set_predictor_batch(True)
    if admission is not None:
        ctx.set_prefetch(*admission)
    if graph:
        ctx.set_graph(True)
    if timing_every:
        ctx.set_timing(timing_every)
    if attn_bytes:
        # decode-attention stand-in: a KV-sized stream on the compute stream before every layer
        kv = torch.zeros(attn_bytes, dtype=torch.uint8, device=DEV)
        kv_out = torch.empty(S.calib_read_out_words(attn_bytes), dtype=torch.int32, device=DEV)
        keep += [kv, kv_out]
    idx_hist, ys = [], []
    for t in range(cfg.T):
        if cache is not None and device_until is not None and t == device_until:
            cache.set_device_policy(0)       # the host policy takes over the device state
        if between is not None:
            between(t, ctx, cache)
        y = torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device=DEV)
        if layerwise:
            for l in range(cfg.L):
                if attn_bytes:
                    S.calib_read(kv, attn_bytes, kv_out, stream=stream)
                rep = ctx.layer(t, l, st.x_dev[t][l], y[l], mode=mode, report=reports is not None)
                if reports is not None:
                    reports.append(rep)
        else:
            ctx.token(t, st.x_dev[t], y, mode=mode)
        idx, _ = ctx.last_routing()
        idx_hist.append(idx)
        ys.append(y.cpu().numpy())
    stats = pred.stats()
    cst = cache.stats() if cache else None
    if tables is not None:
        tables.append(pred.export())
    ctx.close()
    if cache:
        cache.close()
    pred.close()
    return idx_hist, ys, stats, cst


CFGS = [("tiny", dict(T=12)), ("qwen30b", dict(L=4, T=6, P=3, C=10)),
        ("dsv2lite", dict(L=3, T=5, P=2, C=12)), ("qwen30b-b8", dict(L=3, T=4, P=2, C=40))]


@pytest.mark.parametrize("name,over", CFGS)
def test_decode_resident_matches_oracle(name, over):
    from gpuhelp import rel_l2
    from oracle.stmoe_oracle import MODE_STMOE
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    ref = _oracle(st, MODE_STMOE, ffn_tokens=cfg.T)
    assert ref["tie_boundary"] == 0
    idx_hist, ys, stats, _ = _run_gpu(st, 1, capped=False)
    for t in range(cfg.T):
        for l in range(cfg.L):
            r = ref["idx"][t * cfg.L + l]
            for b in range(cfg.B):
                assert sorted(idx_hist[t][l][b].tolist()) == sorted(r[b].tolist())
            err = rel_l2(ys[t][l], ref["y"][(t, l)])
            assert err <= 1e-2, (t, l, err)
    # hit statistics per layer: (hits, |A|, |P|)
    assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
    assert np.array_equal(stats[:, 2], ref["npred"].sum(axis=0))


@pytest.mark.parametrize("over,renorm", [(dict(E=7, K=3, B=2, T=6, P=3), False),
                                         (dict(E=64, K=4, B=4, T=4, P=2, C=16), False),
                                         (dict(B=3, T=6, P=3), True),
                                         (dict(E=7, K=3, B=1, T=6, P=3), False),
                                         (dict(E=64, K=6, B=1, n_shared=2, T=5, P=2, C=12), True),
                                         (dict(E=64, K=16, B=1, T=4, P=2, C=20), False),
                                         (dict(E=65, K=4, B=1, T=4, P=2, C=10), False),
                                         (dict(E=32, K=4, B=1, T=4, P=2, C=10, dtype="bf16"), True),
                                         (dict(E=16, K=16, B=1, T=3, P=2, C=16), True),
                                         (dict(E=2, K=1, B=1, T=4, P=2, C=1), False)])
def test_decode_resident_edge_shapes(over, renorm):
    """The FFN's in-kernel gating at its edges: E not a multiple of 4 (padded
    keys), B*E = 256 (the largest routed in-kernel), renormalised weights; at
    batch 1 the gating in registers of the batch-1 gate/up kernel (E up to 64,
    K up to 16, shared experts, bf16) and above 64 experts the LDS prologue.
    Selections, outputs and hit counts as in the oracle; the capped run (router
    tail kernel, selection passed to the FFN) gives bit-identical outputs."""
    from gpuhelp import rel_l2
    from oracle.stmoe_oracle import MODE_STMOE
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["tiny"].scaled(**over)
    st = Stack(cfg)
    ref = _oracle(st, MODE_STMOE, ffn_tokens=cfg.T, renorm=renorm)
    assert ref["tie_boundary"] == 0
    idx_hist, ys, stats, _ = _run_gpu(st, 1, capped=False, renorm=renorm)
    for t in range(cfg.T):
        for l in range(cfg.L):
            r = ref["idx"][t * cfg.L + l]
            for b in range(cfg.B):
                assert sorted(idx_hist[t][l][b].tolist()) == sorted(r[b].tolist())
            assert rel_l2(ys[t][l], ref["y"][(t, l)]) <= 1e-2
    assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
    assert np.array_equal(stats[:, 2], ref["npred"].sum(axis=0))
    _, ys_cap, _, _ = _run_gpu(st, 1, capped=True, renorm=renorm)
    for t in range(cfg.T):
        assert np.array_equal(ys_cap[t], ys[t]), t


@pytest.mark.parametrize("name,over,mode", [("tiny", dict(T=8), 2), ("tiny", dict(T=8), 3),
                                             ("tiny", dict(L=1, T=6, P=2), 1),
                                             ("qwen30b", dict(L=3, T=4, P=2, C=10), 3)])
def test_decode_resident_ablations(name, over, mode):
    """HT-only, CCT-only and a one-layer model on the resident path, where
    the table update and prediction run beside the FFN: hit counts as in
    the oracle."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    ref = _oracle(st, mode)
    idx_hist, _, stats, _ = _run_gpu(st, mode, capped=False)
    for t in range(cfg.T):
        for l in range(cfg.L):
            r = ref["idx"][t * cfg.L + l]
            for b in range(cfg.B):
                assert sorted(idx_hist[t][l][b].tolist()) == sorted(r[b].tolist())
    assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
    assert np.array_equal(stats[:, 2], ref["npred"].sum(axis=0))


@pytest.mark.parametrize("name,over", CFGS)
@pytest.mark.parametrize("mode,after_demand,device", [(0, 0, 0), (1, 0, 0), (2, 0, 0), (3, 0, 0), (1, 1, 0),
                                                      (0, 0, 1), (1, 0, 1), (3, 0, 1), (1, 1, 1)])
def test_decode_capped_counts_and_invariance(name, over, mode, after_demand, device):
    """At the capped budget the cache makes the oracle's decisions, and the
    outputs are bit-identical to the all-resident run whatever the mode, the
    link order of prefetch copies and where the decisions are taken (host or
    device)."""
    from oracle.stmoe_oracle import decode_reference
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    idx_hist, ys, stats, cst = _run_gpu(st, mode, capped=True, after_demand=after_demand, device=device)
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t])
    ref = _oracle(st, mode, C=cfg.C)
    n = ref["cache"].n
    assert cst == dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                       useful=n.useful, wasted=n.wasted)



@pytest.mark.parametrize("name,over", CFGS)
@pytest.mark.parametrize("mode,device,staged,when", [(0, 0, 0, "before"), (1, 0, 0, "after"), (1, 0, 2, "before"),
                                                     (0, 1, 0, "before"), (1, 1, 0, "after"), (1, 1, 2, "before")])
def test_decode_capped_frequency_aware(name, over, mode, device, staged, when):
    """Frequency-aware eviction (use counts seeded from profiling): the
    oracle's decisions and counts with host or device decisions, prefetch into
    slots or staged, the counts set before or after the device takes over; the
    outputs stay bit-identical to the all-resident run."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys, _, cst = _run_gpu(st, mode, capped=True, device=device, staged=staged, freq=when)
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t])
    ref = _oracle(st, mode, C=cfg.C, staged=staged, freq=True)
    assert cst == _counts(ref["cache"].n)


@pytest.mark.parametrize("name,over", [CFGS[1], CFGS[2]])
def test_decode_frequency_aware_handover_and_graph(name, over):
    """The use counts move with the policy state (device decisions handed back
    to the host mid-run) and live in device memory under graph replay: counts
    as the oracle's, outputs bit-identical to the all-resident run."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    ref = _counts(_oracle(st, 1, C=cfg.C, freq=True)["cache"].n)
    _, ys_a, _, cst_a = _run_gpu(st, 1, capped=True, device=1, device_until=2, freq="before")
    _, ys_b, _, cst_b = _run_gpu(st, 1, capped=True, device=1, graph=True, freq="after")
    for t in range(cfg.T):
        assert np.array_equal(ys_a[t], ys_res[t])
        assert np.array_equal(ys_b[t], ys_res[t])
    assert cst_a == ref and cst_b == ref


@pytest.mark.parametrize("name,over", CFGS)
@pytest.mark.parametrize("mode,online", [(1, True), (2, True), (3, True), (1, False)])
def test_decode_per_token_predictor_launch(name, over, mode, online):
    """One predictor launch per token (every layer's update and prediction in
    layer order, selections in per-parity buffers) gives the per-layer
    launches' selections, outputs, hit statistics and tables, which match the
    oracle (the per-layer tests)."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    t_layer, t_token = [], []
    idx_a, ys_a, stats_a, _ = _run_gpu(st, mode, capped=False, online=online, tables=t_layer)
    idx_b, ys_b, stats_b, _ = _run_gpu(st, mode, capped=False, online=online, tables=t_token, batch=True)
    for t in range(cfg.T):
        assert np.array_equal(idx_a[t], idx_b[t]), t
        assert np.array_equal(ys_a[t], ys_b[t]), t
    assert np.array_equal(stats_a, stats_b)
    for a, b in zip(t_layer[0], t_token[0]):
        assert np.array_equal(a, b)
    ref = _oracle(st, mode, online=online)
    assert np.array_equal(stats_b[:, 0], ref["hits"].sum(axis=0))
    assert np.array_equal(stats_b[:, 2], ref["npred"].sum(axis=0))


def test_per_token_predictor_launch_rejections():
    """Per-token predictor launches need a context without a cache and
    exclude graph replay."""
    import torch
    from gpuhelp import DEV, storage_dtype
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["tiny"].scaled(T=2, P=2)
    st = Stack(cfg)
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(st.prof)
    ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                          [g.data_ptr() for g in st.wg_dev], predictor=pred,
                          resident_ptrs=[st.blobs[l][e].data_ptr() for l in range(cfg.L) for e in range(cfg.E)])
    ctx.set_graph(True)
    with pytest.raises(S.StmoeError):
        ctx.set_predictor_batch(True)
    ctx.set_graph(False)
    ctx.set_predictor_batch(True)
    with pytest.raises(S.StmoeError):
        ctx.set_graph(True)
    ctx.set_predictor_batch(False)
    ctx.close()
    pred.close()


@pytest.mark.parametrize("mode,device", [(0, 0), (1, 0), (1, 1)])
def test_decode_capped_device_memory_pool(mode, device):
    """A backing pool in device memory (copies run device to device): the same
    decisions and counts as the oracle's policy and outputs bit-identical to
    the all-resident run, with host or device decisions."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(L=4, T=6, P=3, C=10)
    st = Stack(cfg)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys, _, cst = _run_gpu(st, mode, capped=True, device=device, device_pool=True)
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t])
    ref = _oracle(st, mode, C=cfg.C)
    n = ref["cache"].n
    assert cst == dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                       useful=n.useful, wasted=n.wasted)


@pytest.mark.parametrize("name,over", [CFGS[1], CFGS[3]])
def test_decode_device_policy_handover(name, over):
    """Device decisions for the first tokens, then the host policy continues
    from the state they left: counts still equal the oracle's and outputs the
    all-resident run's."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys, _, cst = _run_gpu(st, 1, capped=True, device=1, device_until=cfg.T // 2)
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t])
    n = _oracle(st, 1, C=cfg.C)["cache"].n
    assert cst == dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                       useful=n.useful, wasted=n.wasted)


def test_device_policy_rejects_host_calls():
    """While the device decides, the host-side cache calls are refused."""
    import torch
    from gpuhelp import DEV
    from paper_2606_15453_amd import stmoe as S
    L, E, C, blob = 2, 4, 2, 4096
    host = [torch.zeros(blob, dtype=torch.uint8).pin_memory() for _ in range(L * E)]
    arena = torch.empty(S.cache_arena_bytes(L, E, C, blob, 0), dtype=torch.uint8, device=DEV)
    demand, side = torch.cuda.Stream(), torch.cuda.Stream()
    cache = S.ExpertCache(L, E, C, blob, 0, arena, [h.data_ptr() for h in host], demand, side)
    cache.warm(np.array([[0, 1], [2, 3]], dtype=np.int32))
    cache.set_device_policy(1)
    for call in (lambda: cache.acquire(0, [0], 1), lambda: cache.prefetch(0, [0], 1),
                 lambda: cache.warm(np.array([[0, 1], [2, 3]], dtype=np.int32))):
        with pytest.raises(S.StmoeError) as ei:
            call()
        assert ei.value.rc == S.ESTATE
    assert cache.stats() == dict(hits=0, demand=0, overflow=0, prefetch=0, useful=0, wasted=0)
    cache.set_device_policy(0)
    hits, _ = cache.acquire(0, [0, 1], 1)
    assert hits == 2
    cache.close()


def _run_graph(st, mode, timing_every=0, staged=False):
    """Resident run with graph replay and no host sync between tokens.  With
    `staged`, inputs are written straight into the context's staging buffer
    and outputs read from its twin (no copies inside the call)."""
    import torch
    from gpuhelp import DEV, storage_dtype
    from paper_2606_15453_amd import stmoe as S
    cfg = st.cfg
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(st.prof)
    resident = [st.blobs[l][e].data_ptr() for l in range(cfg.L) for e in range(cfg.E)]
    stream = torch.cuda.current_stream()
    ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                          [g.data_ptr() for g in st.wg_dev], predictor=pred, resident_ptrs=resident,
                          shared_ptrs=st.shared_ptrs(), n_shared=cfg.n_shared, stream=stream)
    ctx.set_graph(True)
    if timing_every:
        ctx.set_timing(timing_every)
    ys = [torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device=DEV) for _ in range(cfg.T)]
    xp, yp = ctx.graph_buffers()
    for t in range(cfg.T):
        if staged:
            x = st.x_dev[t].contiguous()
            S.calib_copy(x.data_ptr(), xp, x.numel() * x.element_size(), stream.cuda_stream)
            ctx.token(t, xp, yp, mode=mode)
            S.calib_copy(yp, ys[t].data_ptr(), ys[t].numel() * 4, stream.cuda_stream)
        else:
            ctx.token(t, st.x_dev[t], ys[t], mode=mode)
    torch.cuda.synchronize()
    idx_last, _ = ctx.last_routing()
    out = [y.cpu().numpy() for y in ys]
    stats = pred.stats()
    ctx.close()
    pred.close()
    return idx_last, out, stats


@pytest.mark.parametrize("name,over,timing,staged", [("tiny", dict(T=12), 0, False),
                                                    ("qwen30b", dict(L=4, T=8, P=3), 3, False),
                                                    ("qwen30b-b8", dict(L=3, T=5, P=2), 2, True),
                                                    ("dsv2lite", dict(L=3, T=5, P=2), 0, True)])
def test_decode_graph_replay_matches_eager(name, over, timing, staged):
    """Each token replayed as one HIP graph (event-timed tokens eager, the
    first token eager) gives bit-identical outputs, the same final routing and
    the same predictor hit counts as eager calls, over repeated replays."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    idx_hist, ys_eager, stats_eager, _ = _run_gpu(st, 1, capped=False)
    idx_last, ys_graph, stats_graph = _run_graph(st, 1, timing_every=timing, staged=staged)
    for t in range(cfg.T):
        assert np.array_equal(ys_graph[t], ys_eager[t]), t
    assert np.array_equal(idx_last, idx_hist[-1])
    assert np.array_equal(stats_graph, stats_eager)


@pytest.mark.parametrize("name,over,capped", [("tiny", dict(T=8), False), ("qwen30b", dict(L=3, T=4, P=2, C=10), False),
                                              ("qwen30b", dict(L=3, T=4, P=2, C=10), True)])
def test_decode_online_update_off(name, over, capped):
    """With the online update off the CCTs stay as profiled, HT still tracks
    the selections, and the hit counts follow the oracle run the same way
    (side-stream path without a cache, fused router tail with one)."""
    from oracle.stmoe_oracle import MODE_STMOE, STPredictor
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    ref = _oracle(st, MODE_STMOE, C=cfg.C if capped else None, online=False)
    tables = []
    idx_hist, _, stats, cst = _run_gpu(st, 1, capped=capped, online=False, tables=tables)
    assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
    assert np.array_equal(stats[:, 2], ref["npred"].sum(axis=0))
    prof = STPredictor(cfg.L, cfg.E, cfg.K, cfg.B)
    prof.profile(st.prof)
    _, ci, cc, _ = prof.tables()
    _, gci, gcc, _ = tables[0]
    assert np.array_equal(gci, ci) and np.array_equal(gcc, cc)



def test_ctx_rejects_mismatched_predictor():
    """A predictor made for another shape is refused before any device work."""
    import torch
    from gpuhelp import DEV, storage_dtype
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["tiny"]
    st = Stack(cfg.scaled(T=2, P=2))
    resident = [st.blobs[l][e].data_ptr() for l in range(cfg.L) for e in range(cfg.E)]
    for shape in [(cfg.L, cfg.E * 2, cfg.K, cfg.B), (cfg.L + 1, cfg.E, cfg.K, cfg.B),
                  (cfg.L, cfg.E, cfg.K, cfg.B + 1)]:
        pred = S.Predictor(*shape)
        with pytest.raises(S.StmoeError):
            S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                            [g.data_ptr() for g in st.wg_dev], predictor=pred, resident_ptrs=resident,
                            stream=torch.cuda.current_stream())
        pred.close()


# ---------------------------------------------------------------------------
# The per-layer entry point (moe_decode_layer) with its report, layer by
# layer, with and without a decode-attention stand-in between layers.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,over", [CFGS[0], CFGS[1], CFGS[3]])
@pytest.mark.parametrize("capped,device,mode,attn", [(False, 0, 1, 0), (False, 0, 1, 1 << 24),
                                                     (True, 0, 1, 0), (True, 1, 1, 1 << 24),
                                                     (True, 1, 0, 0), (True, 0, 3, 1 << 24)])
def test_decode_layer_by_layer(name, over, capped, device, mode, attn):
    """moe_decode_layer called once per layer gives the selections and outputs
    of moe_decode_token bit for bit; each layer's report matches the oracle's
    loop: the selection, the layer's hit and prediction counts, the ranked
    prediction for the next layer and the cache counters so far."""
    from oracle.stmoe_oracle import STPredictor, admitted
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    print(f"[layerwise] {cfg.name} capped={capped} device={device} mode={mode} attn={attn}", flush=True)
    idx_tok, ys_tok, stats_tok, cst_tok = _run_gpu(st, mode, capped=capped, device=device)
    reps = []
    idx_lay, ys_lay, stats_lay, cst_lay = _run_gpu(st, mode, capped=capped, device=device, layerwise=True,
                                                   attn_bytes=attn, reports=reps)
    for t in range(cfg.T):
        assert np.array_equal(idx_tok[t], idx_lay[t]), t
        assert np.array_equal(ys_tok[t], ys_lay[t]), t
    assert np.array_equal(stats_tok, stats_lay)
    assert cst_tok == cst_lay
    ref = _oracle(st, mode, C=cfg.C if capped else None)
    assert ref["tie_boundary"] == 0
    cum = _cumulative_after_layers(ref["cache"], cfg.L) if capped else None
    prev = np.zeros((cfg.L, 3), np.int64)
    for t in range(cfg.T):
        for l in range(cfg.L):
            rep = reps[t * cfg.L + l]
            r = ref["idx"][t * cfg.L + l]
            for b in range(cfg.B):
                assert sorted(rep["idx"][b].tolist()) == sorted(r[b].tolist()), (t, l, b)
            ps = np.array(rep["pred_stats"])
            assert ps[0] - prev[l, 0] == ref["hits"][t, l], (t, l)
            assert ps[2] - prev[l, 2] == ref["npred"][t, l], (t, l)
            prev[l] = ps
            if mode:
                assert rep["ranked"] == STPredictor.ranked_union(ref["scores"][t * cfg.L + l]), (t, l)
            else:
                assert rep["n_ranked"] == -1
            if capped:
                assert rep["cache"] == cum[t * cfg.L + l], (t, l)
    if capped:
        assert cst_lay == _counts(ref["cache"].n)


# ---------------------------------------------------------------------------
# Fault injection: correctness never depends on the prediction (Section 4.1:
# prefetching must not change what the model computes).  Wrong tables are
# planted through stmoe_import; capacities at their extremes.
# ---------------------------------------------------------------------------

def _planted_tables(cfg, kind, st):
    """(cct_idx, cct_conf, ht) after profiling, with the planted fault."""
    from oracle.stmoe_oracle import STPredictor
    p = STPredictor(cfg.L, cfg.E, cfg.K, cfg.B)
    p.profile(st.prof)
    _, ci, cc, ht = p.tables()
    if kind in ("zero_conf", "both"):
        cc[:] = 0
    if kind in ("wiped_ht", "both"):
        ht[:] = np.arange(cfg.E - cfg.K, cfg.E)
    return ci, cc, ht


@pytest.mark.parametrize("kind", ["zero_conf", "wiped_ht", "both"])
@pytest.mark.parametrize("cap", ["K", "E"])
@pytest.mark.parametrize("device", [0, 1])
def test_fault_injection_outputs_and_counts(kind, cap, device):
    """Zeroed CCT confidences and/or an HT of wrong experts, at cache
    capacities C = K and C = E: outputs are bit-identical to on-demand loading
    (and to the all-resident run), and the copy counts equal the oracle's
    with the same planted tables."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(L=4, T=6, P=3, C=10) if cap == "K" else W.CONFIGS["tiny"].scaled(T=8)
    C = cfg.K if cap == "K" else cfg.E
    st = Stack(cfg)
    tabs = _planted_tables(cfg, kind, st)
    print(f"[fault] {kind} C={C} device={device}", flush=True)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys_dem, _, cst_dem = _run_gpu(st, 0, capped=True, device=device, C=C)
    _, ys, stats, cst = _run_gpu(st, 1, capped=True, device=device, C=C,
                                 import_tables=(tabs[0].astype(np.uint8), tabs[1].astype(np.uint8), tabs[2]))
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_dem[t]), t
        assert np.array_equal(ys[t], ys_res[t]), t
    from oracle.stmoe_oracle import warm_from_profile
    st.warm_ref = warm_from_profile(st.prof, cfg.L, cfg.E, C)
    ref = _oracle(st, 1, C=C, tables=tabs)
    assert cst == _counts(ref["cache"].n)
    assert np.array_equal(stats[:, 0], ref["hits"].sum(axis=0))
    assert cst_dem == _counts(_oracle(st, 0, C=C)["cache"].n)
    if C == cfg.E:
        assert cst["demand"] == 0 and cst["overflow"] == 0 and cst["prefetch"] == 0


@pytest.mark.parametrize("device", [0, 1])
@pytest.mark.parametrize("min_score,max_per_layer", [(4, None), (2, 1), (4, 8), (7, 3)])
def test_admission_knobs_match_oracle(device, min_score, max_per_layer):
    """The prefetch admission knobs (minimum Eq. 1 score, at most N prefetches
    per layer) take the oracle's admitted prefix: same counts; outputs as the
    all-resident run."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(L=4, T=6, P=3, C=10)
    st = Stack(cfg)
    mpl = max_per_layer if max_per_layer is not None else 1 << 30
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys, _, cst = _run_gpu(st, 1, capped=True, device=device, admission=(min_score, mpl))
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t]), t
    ref = _oracle(st, 1, C=cfg.C, min_score=min_score, max_per_layer=max_per_layer)
    assert cst == _counts(ref["cache"].n)


# ---------------------------------------------------------------------------
# Staged prefetch: predicted experts copied into spare blocks, cancelled when
# the next layer's routing does not select them; residency as on demand.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,over", CFGS)
@pytest.mark.parametrize("mode,n_staged,admission,layerwise,device,head",
                         [(1, 1, None, False, 1, 0), (1, 4, None, False, 1, 0), (3, 2, None, False, 1, 0),
                          (1, 2, (4, 8), False, 1, 0), (1, 3, None, True, 1, 0),
                          (1, 1, None, False, 0, 0), (1, 4, None, False, 0, 4096), (3, 2, None, False, 0, 1 << 16),
                          (1, 2, (4, 8), False, 0, 12288), (1, 3, None, True, 0, 65536)])
def test_decode_capped_staged_prefetch(name, over, mode, n_staged, admission, layerwise, device, head):
    """Staged prefetch (device decisions with cancelled copy kernels; host
    decisions with a head copy and the rest on use): the copy counts equal the
    oracle's staged cache, the hits equal on-demand loading's (residency is
    unchanged by staging), and the outputs are bit-identical to the
    all-resident run, per token and layer by layer with a decode-attention
    stand-in."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[name].scaled(**over)
    st = Stack(cfg)
    print(f"[staged] {cfg.name} mode={mode} n={n_staged} admission={admission} layerwise={layerwise} "
          f"device={device} head={head}", flush=True)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys, _, cst = _run_gpu(st, mode, capped=True, device=device, staged=n_staged, head=head,
                             admission=None if admission is None else admission,
                             layerwise=layerwise, attn_bytes=(1 << 22) if layerwise else 0)
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t]), t
    ms, mpl = (2, None) if admission is None else admission
    ref = _oracle(st, mode, C=cfg.C, staged=n_staged, min_score=ms, max_per_layer=mpl)
    assert cst == _counts(ref["cache"].n)
    dem = _oracle(st, 0, C=cfg.C)["cache"]
    assert cst["hits"] == dem.n.hits
    assert ref["cache"].slot == dem.slot


def test_staged_prefetch_rejections():
    """Staged prefetch needs 2n staging slots; once staged prefetches run,
    decisions cannot move between host and device."""
    import torch
    from gpuhelp import DEV
    from paper_2606_15453_amd import stmoe as S
    L, E, C, blob = 2, 4, 2, 4096
    host = [torch.zeros(blob, dtype=torch.uint8).pin_memory() for _ in range(L * E)]
    arena = torch.empty(S.cache_arena_bytes(L, E, C, blob, 2), dtype=torch.uint8, device=DEV)
    demand, side = torch.cuda.Stream(), torch.cuda.Stream()
    cache = S.ExpertCache(L, E, C, blob, 2, arena, [h.data_ptr() for h in host], demand, side)
    cache.warm(np.array([[0, 1], [2, 3]], dtype=np.int32))
    with pytest.raises(S.StmoeError) as ei:
        cache.set_staged_prefetch(2)                 # host decisions: needs 4 staging slots
    assert ei.value.rc == S.EINVAL
    cache.set_staged_prefetch(1, 1024)
    with pytest.raises(S.StmoeError) as ei:
        cache.set_device_policy(1)                   # host staged prefetch is on
    assert ei.value.rc == S.ESTATE
    cache.set_staged_prefetch(0)
    cache.set_device_policy(1)
    with pytest.raises(S.StmoeError) as ei:
        cache.set_staged_prefetch(2)                 # needs 4 staging slots
    assert ei.value.rc == S.EINVAL
    cache.set_staged_prefetch(1)
    with pytest.raises(S.StmoeError) as ei:
        cache.set_device_policy(0)
    assert ei.value.rc == S.ESTATE
    cache.close()


# ---------------------------------------------------------------------------
# HIP graph replay of the capped decode step with device-side decisions
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode,staged,timing_every", [(0, 0, 0), (1, 0, 0), (1, 0, 3), (1, 2, 0), (3, 0, 4),
                                                      (1, 2, 3)])
def test_graph_replay_capped_device_decisions(mode, staged, timing_every):
    """With device-side cache decisions the whole token (routing, predictor,
    decisions, copy kernels, FFN, prefetch copies) replays as one HIP graph;
    the stamps of the cache policy come from a device token counter that the
    graph advances.  Selections, outputs, predictor statistics and cache
    counts are bit-identical to eager calls and match the oracle, also with
    event-timed (eager) tokens interleaved with replays."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(L=4, T=9, P=3, C=10)
    st = Stack(cfg)
    print(f"[graph] mode={mode} staged={staged} timing_every={timing_every}", flush=True)
    idx_e, ys_e, stats_e, cst_e = _run_gpu(st, mode, capped=True, device=1, staged=staged)
    idx_g, ys_g, stats_g, cst_g = _run_gpu(st, mode, capped=True, device=1, staged=staged, graph=True,
                                           timing_every=timing_every)
    for t in range(cfg.T):
        assert np.array_equal(idx_g[t], idx_e[t]), t
        assert np.array_equal(ys_g[t], ys_e[t]), t
    assert np.array_equal(stats_g, stats_e)
    assert cst_g == cst_e
    ref = _oracle(st, mode, C=cfg.C, staged=staged)
    assert cst_g == _counts(ref["cache"].n)


@pytest.mark.parametrize("copy_wgs,staged", [((1, 1), 0), ((3, 2), 0), ((200, 100), 0), ((2, 1), 2)])
def test_decode_copy_workgroups(copy_wgs, staged):
    """The copy kernels' workgroup counts (device decisions) change the copy
    rate, not the decisions: counts as the oracle's and outputs bit-identical
    to the all-resident run."""
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(L=4, T=6, P=3, C=10)
    st = Stack(cfg)
    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    _, ys, _, cst = _run_gpu(st, 1, capped=True, device=1, staged=staged, copy_wgs=copy_wgs)
    for t in range(cfg.T):
        assert np.array_equal(ys[t], ys_res[t])
    assert cst == _counts(_oracle(st, 1, C=cfg.C, staged=staged)["cache"].n)


def test_graph_replay_follows_setting_changes():
    """Settings changed between replayed tokens (prefetch admission, the online
    update, the staged count, the replacement rule) take effect at the next
    token, as in eager calls: selections, outputs, predictor statistics and
    cache counts equal an eager run with the same changes."""
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen30b"].scaled(L=4, T=10, P=3, C=10)
    st = Stack(cfg)

    def between(t, ctx, cache):
        if t == 2:
            ctx.set_prefetch(4, cfg.K)
        if t == 4:
            ctx.set_online_update(False)
        if t == 6:
            cache.set_staged_prefetch(1, 0)
        if t == 8:
            cache.set_counts(S.use_counts(st.prof, cfg.E))

    _, ys_res, _, _ = _run_gpu(st, 1, capped=False)
    print("[graph settings] eager", flush=True)
    idx_e, ys_e, stats_e, cst_e = _run_gpu(st, 1, capped=True, device=1, staged=2, between=between)
    for t in range(cfg.T):
        assert np.array_equal(ys_e[t], ys_res[t]), t      # staging blocks never alias a slot
    print("[graph settings] replay", flush=True)
    idx_g, ys_g, stats_g, cst_g = _run_gpu(st, 1, capped=True, device=1, staged=2, graph=True, between=between)
    for t in range(cfg.T):
        assert np.array_equal(idx_g[t], idx_e[t]), t
        assert np.array_equal(ys_g[t], ys_e[t]), t
    assert np.array_equal(stats_g, stats_e)
    assert cst_g == cst_e


def test_graph_replay_refuses_host_decisions():
    import torch
    from gpuhelp import DEV, storage_dtype
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["tiny"].scaled(T=2, P=2)
    st = Stack(cfg)
    host = [st.blobs[l][e].cpu().pin_memory() for l in range(cfg.L) for e in range(cfg.E)]
    arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cfg.C, cfg.blob_bytes, 0), dtype=torch.uint8, device=DEV)
    demand, side = torch.cuda.Stream(), torch.cuda.Stream()
    cache = S.ExpertCache(cfg.L, cfg.E, cfg.C, cfg.blob_bytes, 0, arena, [h.data_ptr() for h in host], demand, side)
    cache.warm(st.warm)
    ctx = S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, storage_dtype(cfg),
                          [g.data_ptr() for g in st.wg_dev], cache=cache)
    with pytest.raises(S.StmoeError) as ei:
        ctx.set_graph(True)
    assert ei.value.rc == S.EINVAL
    cache.set_device_policy(1)
    ctx.set_graph(True)
    ctx.close()
    cache.close()
