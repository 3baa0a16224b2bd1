"""Pins for the oracle's grouped-query attention (not GPU)."""
import math

import numpy as np

from oracle import attention


def _brute(q, k, v):
    hq, d = len(q), len(q[0])
    hkv = len(k[0])
    g = hq // hkv
    out = []
    for h in range(hq):
        s = [sum(q[h][i] * k[j][h // g][i] for i in range(d)) / math.sqrt(d) for j in range(len(k))]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        tot = sum(e)
        out.append([sum(e[j] / tot * v[j][h // g][i] for j in range(len(k))) for i in range(d)])
    return np.array(out)


def test_matches_scalar_loops():
    g = np.random.default_rng(0)
    q = g.normal(size=(4, 8))
    k = g.normal(size=(7, 2, 8))
    v = g.normal(size=(7, 2, 8))
    assert np.allclose(attention.attend(q, k, v), _brute(q.tolist(), k.tolist(), v.tolist()),
                       rtol=1e-12, atol=1e-12)


def test_equal_keys_give_mean_of_values():
    g = np.random.default_rng(1)
    k = np.tile(g.normal(size=(1, 2, 16)), (9, 1, 1))
    v = g.normal(size=(9, 2, 16))
    o = attention.attend(g.normal(size=(6, 16)), k, v)
    assert np.allclose(o[0], v[:, 0].mean(0)) and np.allclose(o[5], v[:, 1].mean(0))


def test_dominant_score_selects_value_row():
    d = 16
    k = np.zeros((5, 1, d))
    k[3, 0, 0] = 1.0
    q = np.zeros((2, d))
    q[:, 0] = 200.0 * math.sqrt(d)
    v = np.arange(5 * d, dtype=float).reshape(5, 1, d)
    assert np.allclose(attention.attend(q, k, v), np.stack([v[3, 0]] * 2))


def test_group_mapping_uses_floor_division():
    """Heads 0..G-1 read KV head 0, heads G..2G-1 read KV head 1."""
    k = np.zeros((3, 2, 4))
    v = np.zeros((3, 2, 4))
    v[:, 0] = 1.0
    v[:, 1] = 2.0
    o = attention.attend(np.ones((6, 4)), k, v)
    assert np.allclose(o[:3], 1.0) and np.allclose(o[3:], 2.0)


def test_prefix_plus_tail_equals_concatenation():
    g = np.random.default_rng(2)
    q = g.normal(size=(8, 32))
    kp, vp = g.normal(size=(2, 20, 4, 32))
    kt, vt = g.normal(size=(2, 3, 4, 32))
    a = attention.attend_prefix_tail(q, kp, vp, kt, vt)
    b = _brute(q.tolist(), np.concatenate([kp, kt]).tolist(), np.concatenate([vp, vt]).tolist())
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
