"""Pins of the oracle's expert-cache policy: a hand-worked trace, invariants
and a lower bound from an exhaustive search of eviction choices."""
import functools
import itertools
import json
import os

import numpy as np
import pytest

from oracle.stmoe_oracle import CacheSim

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_trace():
    with open(os.path.join(GOLD, "cache_trace.json")) as f:
        g = json.load(f)
    c = CacheSim(g["L"], g["E"], g["C"], g["warm"])
    for st in g["steps"]:
        if st["op"] == "A":
            _, demand, overflow = c.acquire(0, st["set"], st["stamp"])
            assert [list(d) for d in demand] == st["demand"]
            assert overflow == st["overflow"]
        else:
            copies = c.prefetch(0, st["set"], st["stamp"])
            assert [list(d) for d in copies] == st["copies"]
    assert c.slot == g["final_slots"]
    n = c.n
    got = dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch,
               useful=n.useful, wasted=n.wasted)
    assert got == g["counts"]


def _random_sets(rng, n, E, K):
    return [sorted(rng.choice(E, size=K, replace=False).tolist()) for _ in range(n)]


@pytest.mark.parametrize("E,C,K", [(8, 3, 2), (16, 4, 5), (6, 6, 2)])
def test_invariants(E, C, K):
    rng = np.random.default_rng(E + C)
    L = 3
    warm = [list(range(C)) for _ in range(L)]
    c = CacheSim(L, E, C, warm)
    tot = 0
    stamp = 0
    for t in range(50):
        for l in range(L):
            stamp += 1
            U = _random_sets(rng, 1, E, K)[0]
            tot += len(U)
            c.acquire(l, U, stamp)
            c.prefetch((l + 1) % L, _random_sets(rng, 1, E, min(E, K + 1))[0], stamp)
            for ll in range(L):
                s = [v for v in c.slot[ll] if v >= 0]
                assert len(s) == len(set(s))
    assert c.n.hits + c.n.demand + c.n.overflow == tot
    outstanding = sum(len(p) for p in c.pending)
    assert c.n.useful + c.n.wasted + outstanding == c.n.prefetch
    if C >= E:
        assert c.n.demand == 0 and c.n.overflow == 0


def test_capacity_covers_all_experts_no_misses():
    E, C = 5, 5
    c = CacheSim(1, E, C, [list(range(E))])
    want = 0
    for s in range(1, 30):
        U = {s % E, (s * 3 + 1) % E}
        want += len(U)
        c.acquire(0, sorted(U), s)
    assert c.n.demand == 0 and c.n.hits == want


def _optimal_misses(seq, C, warm):
    """Fewest slot loads over all eviction choices (exhaustive; tiny inputs)."""
    @functools.lru_cache(maxsize=None)
    def go(i, resident):
        if i == len(seq):
            return 0
        need = [f for f in seq[i] if f not in resident]
        best = None
        keep = frozenset(seq[i])
        evictable = [v for v in resident if v not in keep]
        free = C - len(resident)
        if len(need) > free + len(evictable):
            # more misses than slots: the extra stream without admission
            n_admit = free + len(evictable)
        else:
            n_admit = len(need)
        for adm in itertools.combinations(need, n_admit):
            n_ev = max(0, len(adm) - free)
            for ev in itertools.combinations(evictable, n_ev):
                nr = frozenset((set(resident) - set(ev)) | set(adm))
                v = go(i + 1, nr)
                if best is None or v < best:
                    best = v
        return len(need) + best
    return go(0, frozenset(warm))


def test_on_demand_policy_is_not_better_than_optimum():
    rng = np.random.default_rng(9)
    for trial in range(12):
        E, C, K = 5, 2, 2
        seq = _random_sets(rng, 7, E, K)
        c = CacheSim(1, E, C, [[0, 1]])
        for i, U in enumerate(seq):
            c.acquire(0, U, i + 1)
        opt = _optimal_misses([tuple(s) for s in seq], C, (0, 1))
        assert c.n.demand + c.n.overflow >= opt


def test_hand_worked_staged_trace():
    with open(os.path.join(GOLD, "cache_trace_staged.json")) as f:
        g = json.load(f)
    c = CacheSim(g["L"], g["E"], g["C"], g["warm"], staged=g["staged"])
    for st in g["steps"]:
        if st["op"] == "A":
            c.acquire(0, st["set"], st["stamp"])
        else:
            c.prefetch(0, st["set"], st["stamp"])
        ent = c.n.log[-1]
        got = [ent[0], ent[1], ent[2], [list(x) for x in ent[3]]]
        if ent[0] == "A":
            got += [list(ent[4]), ent[5], ent[6], ent[7]]
        assert got == st["log"]
    assert c.slot == g["final_slots"]
    n = c.n
    assert dict(hits=n.hits, demand=n.demand, overflow=n.overflow, prefetch=n.prefetch, useful=n.useful,
                wasted=n.wasted) == g["counts"]


@pytest.mark.parametrize("E,C,K,S", [(8, 3, 2, 1), (16, 4, 5, 3), (32, 6, 4, 8)])
def test_staged_prefetch_keeps_on_demand_residency(E, C, K, S):
    """With staged prefetch the slots evolve exactly as with on-demand loading
    (same hits), and every miss is either a demand copy, an overflow or a used
    staged copy."""
    rng = np.random.default_rng(E * 7 + S)
    L = 3
    warm = [list(range(C)) for _ in range(L)]
    st = CacheSim(L, E, C, warm, staged=S)
    od = CacheSim(L, E, C, warm)
    tot = 0
    stamp = 0
    for t in range(40):
        for l in range(L):
            stamp += 1
            U = sorted(rng.choice(E, size=K, replace=False).tolist())
            tot += len(U)
            st.acquire(l, U, stamp)
            od.acquire(l, U, stamp)
            assert st.slot == od.slot
            ranked = rng.permutation(E)[:int(rng.integers(0, E))].tolist()
            st.prefetch((l + 1) % L, ranked, stamp)
    assert st.n.hits == od.n.hits
    assert st.n.hits + st.n.demand + st.n.overflow + st.n.useful == tot
    assert st.n.demand + st.n.overflow + st.n.useful == od.n.demand + od.n.overflow
    outstanding = sum(len(x) for x in st.stage)
    assert st.n.useful + st.n.wasted + outstanding == st.n.prefetch


def test_frequency_aware_eviction_hand_trace():
    """counts seed the use counts; a victim has the smallest (uses, last use,
    slot); every acquire adds 1 to each expert it is given.  Worked by hand:
    E = 4, C = 2, slots [0, 1], counts [5, 1, 0, 0]."""
    c = CacheSim(1, 4, 2, [[0, 1]], counts=[[5, 1, 0, 0]])
    # {2}: expert 1 (1 use) goes, not expert 0 (5 uses), although both were last used at 0
    assert c.acquire(0, [2], 1)[1] == [(2, 1)]
    # {3}: expert 2 now has 1 use, expert 0 still 5
    assert c.acquire(0, [3], 2)[1] == [(3, 1)]
    # {0, 2}: 0 hits; 2 replaces 3 (the only slot outside the set)
    assert c.acquire(0, [0, 2], 3)[1] == [(2, 1)]
    # {1}: counts 0:6 1:1 2:2 3:1; slots hold 0 (6) and 2 (2): 2 goes
    assert c.acquire(0, [1], 4)[1] == [(1, 1)]
    # a prefetch of {3} evicts by the same rule (1 has 2 uses, 0 has 6)
    assert c.prefetch(0, [3], 5) == [(3, 1)]
    assert c.acquire(0, [3], 6)[1] == []
    assert c.slot == [[0, 3]]
    assert c.freq == [[6, 2, 2, 2]]
    n = c.n
    assert (n.hits, n.demand, n.overflow, n.prefetch, n.useful, n.wasted) == (2, 4, 0, 1, 1, 0)
    # least recently used on the same first step evicts slot 0 (tie on last use, lower slot)
    lru = CacheSim(1, 4, 2, [[0, 1]])
    assert lru.acquire(0, [2], 1)[1] == [(2, 0)]


def test_frequency_aware_eviction_fills_empty_slots_first():
    c = CacheSim(1, 4, 3, [[0, -1, 1]], counts=[[0, 0, 0, 0]])
    assert c.acquire(0, [2], 1)[1] == [(2, 1)]
    # then the slot of least uses: 0 and 1 have none, 2 has one; tie on last use -> slot 0
    assert c.acquire(0, [3], 2)[1] == [(3, 0)]


def test_use_counts_by_hand():
    from oracle.stmoe_oracle import use_counts
    # three profiling tokens, two rows, one layer, top-1: {1, 1}, {0, 2}, {2, 2}
    sel = np.array([[[[1]], [[1]]], [[[0]], [[2]]], [[[2]], [[2]]]])
    assert use_counts(sel, 1, 4).tolist() == [[1, 1, 2, 0]]


@pytest.mark.parametrize("E,C,K", [(8, 3, 2), (16, 4, 5)])
def test_frequency_aware_invariants(E, C, K):
    rng = np.random.default_rng(E * C)
    L = 2
    c = CacheSim(L, E, C, [list(range(C)) for _ in range(L)], counts=np.zeros((L, E), np.int64))
    tot = 0
    for t in range(40):
        for l in range(L):
            U = _random_sets(rng, 1, E, K)[0]
            tot += len(U)
            c.acquire(l, U, t * L + l + 1)
            s = [v for v in c.slot[l] if v >= 0]
            assert len(s) == len(set(s))
    assert c.n.hits + c.n.demand + c.n.overflow == tot
    # every acquire counted each of its experts once
    assert sum(map(sum, c.freq)) == tot
