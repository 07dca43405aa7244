"""Pins of the oracle's gating (Section 2) to invariants and brute force."""
import itertools

import numpy as np
import pytest

from oracle.stmoe_oracle import near_ties, route, softmax_rows, topk_rows


def test_softmax_rows_sum_to_one_and_monotone():
    rng = np.random.default_rng(0)
    z = rng.normal(size=(50, 128)) * 5
    s = softmax_rows(z)
    assert np.all(np.abs(s.sum(axis=1) - 1.0) <= 1e-12)
    for b in range(5):
        o = np.argsort(z[b])
        assert np.all(np.diff(s[b, o]) >= 0)
    # huge logits stay finite (max-subtracted)
    s2 = softmax_rows(np.array([[1000.0, 999.0, -1000.0]]))
    assert np.isfinite(s2).all() and abs(s2[0, 0] / s2[0, 1] - np.e) < 1e-12


@pytest.mark.parametrize("E,K", [(6, 2), (8, 3), (7, 1), (5, 5)])
def test_topk_matches_exhaustive_subset_search(E, K):
    """The selected set maximises the sum of logits over all K-subsets
    (unique when logits are distinct), and is listed in descending order."""
    rng = np.random.default_rng(E * 10 + K)
    for _ in range(40):
        z = rng.normal(size=(1, E))
        best = max(itertools.combinations(range(E), K), key=lambda S: sum(z[0, list(S)]))
        got = topk_rows(z, K)[0]
        assert sorted(got.tolist()) == sorted(best)
        assert all(z[0, got[i]] > z[0, got[i + 1]] for i in range(K - 1))


def test_topk_ties_take_lower_index():
    z = np.array([[1.0, 2.0, 2.0, 0.5, 2.0]])
    assert topk_rows(z, 2)[0].tolist() == [1, 2]
    assert topk_rows(z, 4)[0].tolist() == [1, 2, 4, 0]


def test_near_tie_flags():
    z = np.array([[3.0, 2.99995, 1.0, 0.0],      # order tie inside the top 2
                  [3.0, 1.0, 0.99995, 0.0],      # boundary tie between rank 2 and 3
                  [3.0, 2.0, 1.0, 0.0]])
    b, o = near_ties(z, 2)
    assert b.tolist() == [False, True, False]
    assert o.tolist() == [True, False, False]


def test_route_weights_are_selected_probabilities():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(3, 16))
    wg = rng.normal(size=(10, 16))
    r = route(x, wg, 4)
    z = np.array([[sum(wg[e, h] * x[b, h] for h in range(16)) for e in range(10)] for b in range(3)])
    assert np.allclose(r["z"], z, rtol=0, atol=1e-12)
    for b in range(3):
        ez = np.exp(z[b] - z[b].max())
        for k in range(4):
            assert abs(r["w"][b, k] - ez[r["idx"][b, k]] / ez.sum()) < 1e-15
    rr = route(x, wg, 4, renorm=True)
    assert np.allclose(rr["w"].sum(axis=1), 1.0, atol=1e-15)
    assert np.allclose(rr["w"] * r["w"].sum(axis=1, keepdims=True), r["w"], atol=1e-15)
