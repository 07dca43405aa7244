"""Pins of the oracle's expert FFN (Section 2; SwiGLU experts) against an
explicit fp64 triple loop and special cases."""
import math

import numpy as np

from oracle.stmoe_oracle import moe_ffn, silu, swiglu_expert


def _loop_expert(x, wg, wu, wd):
    H, I = len(x), wg.shape[0]
    a = []
    for i in range(I):
        g = 0.0
        u = 0.0
        for h in range(H):
            g += wg[i][h] * x[h]
            u += wu[i][h] * x[h]
        a.append(g / (1.0 + math.exp(-g)) * u)
    y = []
    for h in range(H):
        acc = 0.0
        for i in range(I):
            acc += wd[h][i] * a[i]
        y.append(acc)
    return np.array(y)


def _mats(rng, H, I, E):
    return [(rng.normal(size=(I, H)), rng.normal(size=(I, H)), rng.normal(size=(H, I))) for _ in range(E)]


def test_expert_matches_triple_loop():
    rng = np.random.default_rng(0)
    H, I = 8, 4
    for _ in range(5):
        x = rng.normal(size=H)
        m = _mats(rng, H, I, 1)[0]
        assert np.allclose(swiglu_expert(x, *m), _loop_expert(x, *m), rtol=1e-12, atol=1e-12)


def test_moe_matches_triple_loop_and_special_cases():
    rng = np.random.default_rng(1)
    H, I, E, K, B = 8, 4, 3, 2, 2
    mats = _mats(rng, H, I, E)
    x = rng.normal(size=(B, H))
    idx = np.array([[2, 0], [1, 2]])
    w = rng.random(size=(B, K))
    y = moe_ffn(x, idx, w, lambda e: mats[e])
    for b in range(B):
        ref = sum(w[b, k] * _loop_expert(x[b], *mats[idx[b, k]]) for k in range(K))
        assert np.allclose(y[b], ref, rtol=1e-12, atol=1e-12)
    # x = 0 -> y = 0
    assert np.all(moe_ffn(np.zeros((B, H)), idx, w, lambda e: mats[e]) == 0)
    # linear in the gate weights
    y2 = moe_ffn(x, idx, 2.5 * w, lambda e: mats[e])
    assert np.allclose(y2, 2.5 * y, rtol=1e-12)
    # K = 1 with weight 1 is a single SwiGLU expert
    y1 = moe_ffn(x[:1], np.array([[1]]), np.ones((1, 1)), lambda e: mats[e])
    assert np.allclose(y1[0], _loop_expert(x[0], *mats[1]), rtol=1e-12)
    # shared experts add with weight 1
    ys = moe_ffn(x, idx, w, lambda e: mats[e], shared=[mats[0]])
    for b in range(B):
        assert np.allclose(ys[b] - y[b], _loop_expert(x[b], *mats[0]), rtol=1e-10, atol=1e-12)


def test_silu_values():
    assert silu(0.0) == 0.0
    assert abs(silu(1.0) - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    assert abs(silu(-40.0)) < 1e-15
    assert abs(silu(40.0) - 40.0) < 1e-12
