"""The link time model behind `bench.py --policy-bound`: a hand-computed
trace, and properties that hold for any trace (no stall without copy time,
offline-optimal replacement never copies more than least-recently-used, a
perfect one-layer staged prefetch never stalls more than on-demand loading,
wrong prefetches into evicted slots never stall less)."""
import random

import pytest

import bench

POLICIES = bench.POLICIES


def test_hand_trace_one_layer_one_slot():
    # one layer, one slot holding expert 0; tokens select 0, 1, 0, 1; a copy
    # takes 1 ms, a layer 0.1 ms (routing 5% of it, then the FFN)
    trace = [[[0]], [[1]], [[0]], [[1]]]
    preds = [[[1]], [[0]], [[1]], [[0]]]
    # on demand: three misses, each waits a whole copy
    assert bench.simulate_policy(trace, preds, 1, 1, [[0]], 1.0, 0.1, 0.0, "demand") == pytest.approx((0.75, 3, 0.0))
    # a perfect staged prefetch starts each copy one layer early: 0.1 ms per
    # copy hidden once the link is busy, 0.075 ms per token
    st, n, w = bench.simulate_policy(trace, preds, 1, 1, [[0]], 1.0, 0.1, 0.0, "perfect_staged")
    assert (st, n, w) == pytest.approx((0.675, 3, 0.0))
    # with one slot nothing can be kept: the optimum copies as often
    assert bench.simulate_policy(trace, preds, 1, 1, [[0]], 1.0, 0.1, 0.0, "optimum") == pytest.approx((0.75, 3, 0.0))


def _random_case(seed, L=3, E=8, C=3, K=2, T=12):
    rng = random.Random(seed)
    trace = [[sorted(rng.sample(range(E), K)) for _ in range(L)] for _ in range(T)]
    preds = [[rng.sample(range(E), rng.randint(0, E)) for _ in range(L)] for _ in range(T)]
    warm = [sorted(rng.sample(range(E), C)) for _ in range(L)]
    return trace, preds, warm, L, C


@pytest.mark.parametrize("seed", range(8))
def test_properties_on_random_traces(seed):
    trace, preds, warm, L, C = _random_case(seed)
    for pol in POLICIES:
        st, _, _ = bench.simulate_policy(trace, preds, L, C, warm, 0.0, 0.05, 0.0, pol, max_staged=C,
                                         counts=[[1] * 8 for _ in range(L)],
                                         cct=([[[e] for e in range(8)]] * (L - 1), [[[1] for e in range(8)]] * (L - 1)))
        assert st == pytest.approx(0.0, abs=1e-9), pol
    demand = bench.simulate_policy(trace, preds, L, C, warm, 0.3, 0.05, 0.0, "demand")
    optimum = bench.simulate_policy(trace, preds, L, C, warm, 0.3, 0.05, 0.0, "optimum")
    assert optimum[1] <= demand[1]
    perfect = bench.simulate_policy(trace, preds, L, C, warm, 0.3, 0.05, 0.0, "perfect_staged", max_staged=C)
    assert perfect[0] <= demand[0] + 1e-9
    # a prediction that names only experts the next layer does not select
    wrong = [[[e for e in range(8) if e not in trace[t + (l + 1) // L][(l + 1) % L]] if t + (l + 1) // L < len(trace)
              else [] for l in range(L)] for t in range(len(trace))]
    evict = bench.simulate_policy(trace, wrong, L, C, warm, 0.3, 0.05, 0.0, "evict")
    assert evict[0] >= demand[0] - 1e-9


def test_everything_resident_copies_nothing():
    trace, preds, _, L, _ = _random_case(3)
    warm = [list(range(8)) for _ in range(L)]
    assert bench.simulate_policy(trace, preds, L, 8, warm, 1.0, 0.05, 0.0, "demand") == pytest.approx((0.0, 0, 0.0))


def test_online_replacement_hand_traces():
    # one layer, slots holding 0 and 1 (both unused so far); tokens select 2, then 0
    trace, none = [[[2]], [[0]]], [[[]], [[]]]
    # least recently used breaks the tie by slot and evicts 0, which the next token needs
    assert bench.simulate_policy(trace, none, 1, 2, [[0, 1]], 1.0, 0.1, 0.0, "demand") == pytest.approx((1.0, 2, 0.0))
    # profiling counts favour 0: least frequently used evicts 1 instead
    assert bench.simulate_policy(trace, none, 1, 2, [[0, 1]], 1.0, 0.1, 0.0, "demand_lfu",
                                 counts=[[10, 0, 5]]) == pytest.approx((0.5, 1, 0.0))
    # two layers; layer 0 always selects expert 0, whose CCT entry names expert 2 for layer 1
    # (confidence 3): layer 1 evicts expert 1 rather than 2, which the next token selects
    trace2 = [[[0], [0]], [[0], [2]]]
    warm2 = [[0, 1], [2, 1]]
    cct = ([[[2], [0], [0]]], [[[3], [0], [0]]])
    none2 = [[[], []], [[], []]]
    lru = bench.simulate_policy(trace2, none2, 2, 2, warm2, 1.0, 0.1, 0.0, "demand")
    cct_run = bench.simulate_policy(trace2, none2, 2, 2, warm2, 1.0, 0.1, 0.0, "demand_cct",
                                    counts=[[1, 1, 1], [1, 1, 1]], cct=cct)
    assert lru[1] == 2 and cct_run[1] == 1
