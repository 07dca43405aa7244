"""Pins of the oracle's predictor (Algorithms 1-3, Eq. 1) to values fixed by
hand-worked examples, closed forms and special cases."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle.stmoe_oracle import STPredictor, THRESHOLD

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _pairs(p, i):
    idx, conf = p.cct_idx[i], p.cct_conf[i]
    return [[[int(idx[e][s]), int(conf[e][s])] for s in range(p.K)] for e in range(p.E)]


def test_worked_example_replay():
    g = _load("predictor_worked_example.json")
    p = STPredictor(g["L"], g["E"], g["K"], g["B"])
    prof = np.array([[[tok[0], tok[1]]] for tok in g["profiling"]])     # [P][B=1][L][K]
    p.profile(prof)
    assert p.co[0].tolist() == g["co_after_profile"]
    assert _pairs(p, 0) == g["cct_after_profile"]
    assert [p.ht[l][0].tolist() for l in range(2)] == g["ht_after_profile"]
    hits0 = hits1 = npred1 = 0
    for step in g["decode"]:
        sc0 = p.predict(-1, None)
        P0 = STPredictor.prefetch_sets(sc0)[0]
        assert P0 == step["P0"]
        A0 = step["A0"]
        h0 = len(set(A0) & set(P0))
        assert h0 == step["hits0"]
        p.update(0, None, [A0])
        sc1 = p.predict(0, [A0])
        assert sc1[0].tolist() == step["scores1"]
        P1 = STPredictor.prefetch_sets(sc1)[0]
        assert P1 == step["P1"]
        A1 = step["A1"]
        h1 = len(set(A1) & set(P1))
        assert h1 == step["hits1"]
        p.update(1, [A0], [A1])
        assert _pairs(p, 0) == step["cct_after"]
        hits0 += h0
        hits1 += h1
        npred1 += len(P1)
    assert [p.ht[l][0].tolist() for l in range(2)] == g["final_ht"]
    n = len(g["decode"]) * g["K"]
    assert [hits0, n] == g["recall_l0"]
    assert [hits1, n] == g["recall_l1"]
    assert [hits1, npred1] == g["precision_l1"]


def test_literal_algorithm2_gives_same_prefetch_set():
    """Algorithm 2 read literally sets HT members to exactly 2; Eq. 1 adds 2 to
    their CCT score.  Both readings give the same PrefetchSet (text after Alg. 2)."""
    g = _load("predictor_worked_example.json")
    for step in g["decode"]:
        lit = np.array(step["scores1_literal_alg2"])
        eq1 = np.array(step["scores1"])
        assert sorted(np.nonzero(lit >= THRESHOLD)[0].tolist()) == step["P1"]
        assert sorted(np.nonzero(eq1 >= THRESHOLD)[0].tolist()) == step["P1"]


def test_double_replacement():
    d = _load("predictor_worked_example.json")["double_replacement"]
    p = STPredictor(2, d["E"], d["K"], 1)
    p.cct_idx[0][0] = [s[0] for s in d["row"]]
    p.cct_conf[0][0] = [s[1] for s in d["row"]]
    p.update_entry(0, 0, d["F"])
    assert [[int(p.cct_idx[0][0][s]), int(p.cct_conf[0][0][s])] for s in range(d["K"])] == d["after"]


def _random_trace(rng, n, B, L, E, K):
    sel = np.zeros((n, B, L, K), np.int64)
    for t in range(n):
        for b in range(B):
            for l in range(L):
                sel[t, b, l] = rng.choice(E, size=K, replace=False)
    return sel


@pytest.mark.parametrize("E,K,B", [(8, 2, 1), (16, 4, 3), (64, 6, 2)])
def test_invariants_random_trace(E, K, B):
    rng = np.random.default_rng(7)
    L, P = 4, 12
    sel = _random_trace(rng, P + 20, B, L, E, K)
    p = STPredictor(L, E, K, B)
    p.profile(sel[:P])
    co, idx, conf, ht = p.tables()
    # counts sum to the number of observed (e, f) co-activations: P * B * K^2 per pair
    assert (co.sum(axis=(1, 2)) == P * B * K * K).all()
    # each CCT entry keeps the K most co-activated experts
    for i in range(L - 1):
        for e in range(E):
            kept = sorted(co[i, e, idx[i, e]].tolist(), reverse=True)
            assert kept == sorted(co[i, e].tolist(), reverse=True)[:K]
    assert (conf == 2).all()
    for t in range(P, P + 20):
        prev = None
        for l in range(L):
            cur = [sorted(sel[t, b, l].tolist()) for b in range(B)]
            p.update(l, prev, cur)
            assert all(p.ht[l][b].tolist() == cur[b] for b in range(B))
            if l + 1 < L:
                sc = p.predict(l, cur)
                assert sc.max() <= 3 * K + 2
                for b in range(B):
                    ps = set(STPredictor.prefetch_sets(sc)[b])
                    assert set(p.ht[l + 1][b].tolist()) <= ps  # HT members always reach 2
            prev = cur
        _, idx, conf, _ = p.tables()
        assert ((conf >= 0) & (conf <= 3)).all()
        for i in range(L - 1):
            for e in range(E):
                assert len(set(idx[i, e].tolist())) == K          # entries stay distinct


def test_uniform_routing_temporal_overlap_is_k2_over_n():
    """Section 3.2: with independent uniform routing the expected overlap between
    consecutive tokens is K^2/N.  The HT-only predictor's hit count must match."""
    rng = np.random.default_rng(11)
    E, K, L, B, n = 32, 4, 2, 1, 6000
    sel = _random_trace(rng, n + 1, B, L, E, K)
    p = STPredictor(L, E, K, B)
    p.profile(sel[:1])
    hits = []
    for t in range(1, n + 1):
        prev = None
        for l in range(L):
            cur = [sorted(sel[t, 0, l].tolist())]
            sc = p.predict(l - 1, prev, use_cct=False) if l > 0 else p.predict(-1, None)
            hits.append(len(set(cur[0]) & set(STPredictor.prefetch_sets(sc)[0])))
            p.update(l, prev, cur)
            prev = cur
    mean = np.mean(hits)
    expect = K * K / E
    # variance of a hypergeometric overlap, K draws from E with K marked
    var = K * (K / E) * (1 - K / E) * (E - K) / (E - 1)
    assert abs(mean - expect) < 5 * np.sqrt(var / len(hits))


def test_stay_probability_one_gives_full_recall():
    """A trace that never changes is predicted exactly by the HT alone."""
    E, K, L, B = 16, 3, 5, 2
    rng = np.random.default_rng(3)
    base = _random_trace(rng, 1, B, L, E, K)[0]
    sel = np.repeat(base[None], 30, axis=0)
    p = STPredictor(L, E, K, B)
    p.profile(sel[:5])
    for t in range(5, 30):
        prev = None
        for l in range(L):
            cur = [sorted(sel[t, b, l].tolist()) for b in range(B)]
            sc = p.predict(l - 1, prev) if l > 0 else p.predict(-1, None)
            for b in range(B):
                assert set(cur[b]) <= set(STPredictor.prefetch_sets(sc)[b])
            p.update(l, prev, cur)
            prev = cur


def test_deterministic_transitions_k1_full_spatial_recall():
    """K = 1, no temporal reuse, layer l+1 = pi_l(layer l): after profiling has
    seen every expert, the CCT alone predicts every layer >= 1 exactly, and the
    CCT is a per-expert next-expert table whose hits saturate at 3."""
    E, L = 8, 4
    rng = np.random.default_rng(5)
    perms = [rng.permutation(E) for _ in range(L)]

    def chain(e0):
        s = [e0]
        for l in range(1, L):
            s.append(int(perms[l][s[-1]]))
        return s

    prof = np.array([[[[v] for v in chain(e)]] for e in range(E)])          # [P=E][1][L][1]
    p = STPredictor(L, E, 1, 1)
    p.profile(prof)
    for i in range(L - 1):
        assert [p.cct_idx[i][e][0] for e in range(E)] == [int(perms[i + 1][e]) for e in range(E)]
    for t in range(40):
        s = chain(int(rng.integers(E)))
        prev = None
        for l in range(L):
            if l > 0:
                sc = p.predict(l - 1, prev, use_ht=False)
                assert STPredictor.prefetch_sets(sc)[0] == [s[l]]
            p.update(l, prev, [[s[l]]])
            prev = [[s[l]]]
    assert max(p.cct_conf[0][e][0] for e in range(E)) == 3


def test_ranked_union_order():
    sc = np.array([[0, 3, 2, 5, 1], [2, 1, 4, 0, 0]])
    # max per column: [2, 3, 4, 5, 1]; >= 2: f0(2), f1(3), f2(4), f3(5)
    assert STPredictor.ranked_union(sc) == [3, 2, 1, 0]


def test_update_against_exhaustive_reading_small():
    """Every (row, F) pair on a tiny universe: confidences move by exactly +1/-1
    within [0, 3], replaced slots take distinct experts of F not in the old row."""
    E, K = 4, 2
    for row in itertools.permutations(range(E), K):
        for confs in itertools.product(range(4), repeat=K):
            for F in itertools.combinations(range(E), K):
                p = STPredictor(2, E, K, 1)
                p.cct_idx[0][0] = list(row)
                p.cct_conf[0][0] = list(confs)
                p.update_entry(0, 0, F)
                new, nc = p.cct_idx[0][0].tolist(), p.cct_conf[0][0].tolist()
                assert len(set(new)) == K
                for s in range(K):
                    if row[s] in F:
                        assert new[s] == row[s] and nc[s] == min(confs[s] + 1, 3)
                    elif confs[s] > 0:
                        assert new[s] == row[s] and nc[s] == confs[s] - 1
                    else:
                        assert new[s] in F and new[s] not in row and nc[s] == 2
