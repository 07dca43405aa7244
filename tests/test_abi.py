"""The C-ABI library: it loads, exports every declared symbol, rejects invalid
arguments before any device work, and its host-only cache policy makes the
same decisions as the oracle's CacheSim."""
import json
import os
import re

import numpy as np
import pytest

from oracle.stmoe_oracle import CacheSim

S = pytest.importorskip("paper_2606_15453_amd.stmoe")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "stmoe.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", txt)) - {"sizeof"})


def test_every_declared_symbol_is_exported_and_bound():
    names = _declared()
    assert "moe_route_topk" in names and "moe_decode_layer" in names
    for n in names:
        assert hasattr(S._lib, n), n
    assert sorted(S.EXPORTED) == names


def test_invalid_arguments_rejected_without_device_work():
    # K > E, E > 256, H not a multiple of 8, null pointers
    for args in [(16, 4096, 4, 8), (1, 4096, 300, 8), (1, 100, 8, 2), (0, 4096, 8, 2)]:
        B, H, E, K = args
        rc = S._lib.moe_route_topk(16, 16, B, H, E, K, S.BF16, 0, 16, 16, None, 16, 1 << 20, None)
        assert rc == S.EINVAL
    rc = S._lib.moe_route_topk(None, 16, 1, 64, 8, 2, S.BF16, 0, 16, 16, None, 16, 1 << 20, None)
    assert rc == S.EINVAL
    assert "null" in S._lib.stmoe_last_error().decode()
    # workspace too small
    rc = S._lib.moe_route_topk(16, 16, 1, 64, 8, 2, S.BF16, 0, 16, 16, None, 16, 4, None)
    assert rc == S.EINVAL and "workspace" in S._lib.stmoe_last_error().decode()
    rc = S._lib.moe_expert_ffn(16, 16, 16, 1, 2, 100, 64, 8, S.BF16, 16, None, 0, 16, 256, 1 << 20, None)
    assert rc == S.EINVAL
    rc = S._lib.moe_expert_ffn(16, 16, 16, 1, 2, 64, 64, 8, S.BF16, 16, None, 2, 16, 256, 1 << 20, None)
    assert rc == S.EINVAL      # shared experts without pointers
    assert S._lib.stmoe_predict(None, 0, None, 3, None, None, None, None, None, None) == S.EINVAL
    assert S.blob_bytes(4096, 14336, S.BF16) == 3 * 4096 * 14336 * 2
    # read probe: one word per workgroup (256 KiB or 32 KiB regions), unknown patterns refused
    assert S.calib_read_out_words(1 << 30, 1) == 4096
    assert S.calib_read_out_words(1 << 30, 2) == 32768
    assert S.calib_read_out_words((32 << 10) + 16, 2) == 2
    assert S._lib.stmoe_calib_read(256, 1 << 20, 3, 256, None) == S.EINVAL
    assert S._lib.stmoe_calib_read(256 + 8, 1 << 20, 2, 256, None) == S.EINVAL      # misaligned
    assert S._lib.stmoe_calib_copy_grid(256, 512, 1 << 20, 0, None) == S.EINVAL     # workgroups in [1, 1024]
    assert S._lib.stmoe_calib_copy_grid(256, 512, 1 << 20, 1025, None) == S.EINVAL
    # the handoff probe: modes 0..4, chunk2 of 4/8/16/24/32 KiB, aligned buffers
    h = S._lib.stmoe_calib_handoff
    assert h(256, 4096, 4, 512, 4096, 4, 5, 768, 1024, 1280, 4, None) == S.EINVAL      # mode
    assert h(256, 4096, 4, 512, 12288, 4, 1, 768, 1024, 1280, 4, None) == S.EINVAL     # 12 KiB chunk2
    assert h(256, 4096, 4, 512, 4096, 4, 1, 768, 1024, None, 4, None) == S.EINVAL      # no sync words
    assert h(264, 4096, 4, 512, 4096, 4, 0, 768, 1024, 1280, 0, None) == S.EINVAL      # misaligned w1
    assert h(256, 4100, 4, 512, 4096, 4, 0, 768, 1024, 1280, 0, None) == S.EINVAL      # chunk1 % 16
    assert h(256, 4096, 0, 512, 4096, 4, 0, 768, 1024, 1280, 0, None) == S.EINVAL      # no producers
    assert S._lib.expert_cache_set_copy_workgroups(None, 4, 4) == S.EINVAL


def test_pack_expert_is_concatenation():
    rng = np.random.default_rng(0)
    H, I = 16, 8
    g, u, d = (rng.integers(0, 65535, size=s, dtype=np.uint16) for s in ((I, H), (I, H), (H, I)))
    out = np.zeros(3 * H * I, np.uint16)
    S.pack_expert(g, u, d, S.BF16, out)
    assert np.array_equal(out, np.concatenate([g.ravel(), u.ravel(), d.ravel()]))


def test_policy_hand_trace():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "cache_trace.json")))
    p = S.Policy(g["L"], g["E"], g["C"], g["warm"])
    for st in g["steps"]:
        if st["op"] == "A":
            pairs, _ = p.acquire(0, st["set"], st["stamp"])
            assert [list(x) for x in pairs if x[1] >= 0] == st["demand"]
            assert [x[0] for x in pairs if x[1] < 0] == st["overflow"]
        else:
            assert [list(x) for x in p.prefetch(0, st["set"], st["stamp"])] == st["copies"]
    assert p.slots().tolist() == g["final_slots"]
    assert p.stats() == g["counts"]


@pytest.mark.parametrize("freq", [False, True])
@pytest.mark.parametrize("E,C,K,L", [(8, 3, 2, 4), (128, 32, 8, 3), (64, 24, 6, 2), (16, 16, 4, 2)])
def test_policy_matches_oracle_on_random_traces(E, C, K, L, freq):
    rng = np.random.default_rng(E * 100 + C)
    warm = [sorted(rng.choice(E, size=C, replace=False).tolist()) for _ in range(L)]
    counts = rng.integers(0, 6, size=(L, E)) if freq else None
    ref = CacheSim(L, E, C, warm, counts=counts)
    p = S.Policy(L, E, C, warm)
    p.set_counts(counts)
    for t in range(60):
        for l in range(L):
            stamp = t * L + l + 1
            B = int(rng.integers(1, 4))
            U = sorted(set(rng.choice(E, size=min(E, K * B), replace=False).tolist()))
            _, demand, overflow = ref.acquire(l, U, stamp)
            pairs, _ = p.acquire(l, U, stamp)
            assert [x for x in pairs if x[1] >= 0] == [tuple(d) for d in demand]
            assert [x[0] for x in pairs if x[1] < 0] == overflow
            n = int(rng.integers(0, min(E, 2 * K + 3)))
            ranked = rng.permutation(E)[:n].tolist()
            nl = (l + 1) % L
            assert p.prefetch(nl, ranked, stamp) == [tuple(c) for c in ref.prefetch(nl, ranked, stamp)]
    assert p.slots().tolist() == ref.slot
    n = ref.n
    assert p.stats() == dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
                             useful=n.useful, wasted=n.wasted)


@pytest.mark.parametrize("P,B,L,K,E", [(5, 1, 4, 2, 8), (16, 4, 3, 6, 64), (3, 2, 2, 8, 16)])
def test_use_counts_match_oracle(P, B, L, K, E):
    from oracle.stmoe_oracle import use_counts
    rng = np.random.default_rng(P * 7 + E)
    sel = np.stack([np.stack([np.stack([rng.choice(E, K, replace=False) for _ in range(L)])
                              for _ in range(B)]) for _ in range(P)]).astype(np.int32)
    assert np.array_equal(S.use_counts(sel, E), use_counts(sel, L, E))


def test_policy_counts_rejected_and_cleared():
    p = S.Policy(1, 4, 2, [[0, 1]])
    with pytest.raises(S.StmoeError):
        p.set_counts([[0, -1, 0, 0]])
    p.set_counts([[5, 1, 0, 0]])
    assert p.acquire(0, [2], 1)[0] == [(2, 1)]          # expert 1 has fewer uses
    p.set_counts(None)                                    # back to least recently used
    assert p.acquire(0, [3], 2)[0] == [(3, 0)]          # slot 0 (expert 0) was used least recently


def test_policy_rejects_bad_lists():
    p = S.Policy(2, 8, 3)
    with pytest.raises(S.StmoeError):
        p.acquire(0, [1, 1], 1)
    with pytest.raises(S.StmoeError):
        p.prefetch(0, [9], 1)
    with pytest.raises(S.StmoeError):
        p.acquire(5, [1], 1)


@pytest.mark.parametrize("P,B,L,K,E,C", [(5, 1, 4, 2, 8, 3), (16, 4, 3, 6, 64, 24), (3, 2, 2, 8, 16, 20)])
def test_warm_sets_match_oracle(P, B, L, K, E, C):
    """The library's initial residency equals the oracle's (count desc, index asc, -1 padding)."""
    from oracle.stmoe_oracle import warm_from_profile
    rng = np.random.default_rng(P * 1000 + E)
    sel = np.stack([np.stack([np.stack([rng.choice(E, K, replace=False) for _ in range(L)])
                              for _ in range(B)]) for _ in range(P)]).astype(np.int32)
    assert np.array_equal(S.warm_sets(sel, E, C), warm_from_profile(sel, L, E, C))


def test_workspace_queries_and_rejections_without_device_work():
    """Every device buffer comes from the caller: the size queries are host-only,
    and the create calls reject a missing or short workspace before touching the
    device."""
    import ctypes as C_
    n = S._lib.stmoe_workspace_bytes(94, 128, 8, 16)
    assert n > 0 and n % 256 == 0
    assert S._lib.stmoe_workspace_bytes(2, 300, 8, 1) == 0          # E > 256
    h = C_.c_void_p()
    assert S._lib.stmoe_create(4, 8, 2, 1, None, 1 << 20, C_.byref(h)) == S.EINVAL
    assert S._lib.stmoe_create(4, 8, 2, 1, 256, 16, C_.byref(h)) == S.EINVAL
    assert "workspace" in S._lib.stmoe_last_error().decode()
    assert S._lib.stmoe_create(4, 8, 2, 1, 256 + 4, 1 << 30, C_.byref(h)) == S.EINVAL   # misaligned
    assert S.cache_arena_bytes(4, 8, 3, 4096, 1) >= (4 * 3 + 1) * 4096
    assert S.cache_arena_bytes(4, 8, 9, 4096, 1) == 0                                  # C > E
    router = (C_.c_void_p * 4)(*([16] * 4))
    resident = (C_.c_void_p * 32)(*([16] * 32))
    d = S.ModelDesc(4, 8, 2, 1, 256, 512, 0, S.F32, 0, router, None, resident)
    nb = S._lib.moe_ctx_workspace_bytes(C_.byref(d))
    assert nb > 0 and nb % 256 == 0
    assert S._lib.moe_ctx_create(C_.byref(d), None, None, None, None, nb, C_.byref(h)) == S.EINVAL
    assert S._lib.moe_ctx_create(C_.byref(d), None, None, None, 256, nb - 256, C_.byref(h)) == S.EINVAL
    bad = S.ModelDesc(4, 8, 9, 1, 256, 512, 0, S.F32, 0, router, None, resident)        # K > E
    assert S._lib.moe_ctx_workspace_bytes(C_.byref(bad)) == 0
