"""Pins of the oracle's synchronization-aware cache-reuse indicator
(Eq. (12)-(15)) against closed forms and a pure-Python loop.  CPU only."""
import math

import numpy as np
import pytest

import oracle

EPS = 1e-6


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_relative_l1_closed_forms():
    y = _rand((2, 7, 5), 0)
    n1 = np.abs(y).sum()
    assert oracle.relative_l1(y, y, EPS) == 0.0
    assert math.isclose(oracle.relative_l1(y, np.zeros_like(y), EPS), n1 / (n1 + EPS),
                        rel_tol=1e-15)
    assert math.isclose(oracle.relative_l1(y, -y, EPS), 2 * n1 / (n1 + EPS), rel_tol=1e-15)
    for c in (0.25, 0.5, 3.0):
        assert math.isclose(oracle.relative_l1(y, (1 - c) * y, EPS), c * n1 / (n1 + EPS),
                            rel_tol=1e-14)
    # all-zero output: only epsilon in the denominator
    z = np.zeros((1, 3, 4))
    assert math.isclose(oracle.relative_l1(z, np.ones_like(z), EPS), 12 / EPS, rel_tol=1e-15)


def test_protected_rows_pure_python_loop():
    B, L, C = 2, 9, 4
    y, yh = _rand((B, L, C), 1), _rand((B, L, C), 2)
    flag = np.zeros((B, L), np.uint8)
    flag[0, [1, 4]] = 1
    flag[1, [0, 8]] = 1
    num = den = 0.0
    for b in range(B):
        for i in range(L):
            if flag[b, i]:
                for c in range(C):
                    num += abs(y[b, i, c] - yh[b, i, c])
                    den += abs(y[b, i, c])
    assert math.isclose(oracle.relative_l1(y, yh, EPS, rows=flag), num / (den + EPS),
                        rel_tol=1e-14)


def test_saliency_drift_closed_forms():
    s = np.random.default_rng(3).random((2, 11))
    assert abs(oracle.saliency_drift(s, s, 0.0)) < 1e-15
    assert abs(oracle.saliency_drift(s, 5.0 * s, 0.0)) < 1e-15   # scale invariant
    a = np.array([[1.0, 0.0, 0.0]])
    b = np.array([[0.0, 2.0, 0.0]])
    assert oracle.saliency_drift(a, b, EPS) == 1.0               # orthogonal maps
    c = np.array([[1.0, 1.0, 0.0]])
    assert math.isclose(oracle.saliency_drift(a, c, 0.0), 1 - 1 / math.sqrt(2), rel_tol=1e-15)


def test_indicator_max_and_threshold():
    B, L, La, C = 1, 8, 3, 4
    yv = np.ones((B, L, C))
    ya = np.ones((B, La, C))
    flag = np.zeros((B, L), np.uint8)
    flag[0, 2] = 1
    s = np.array([[1.0, 0, 0, 0, 0, 0, 0, 0]])
    # only the protected row changes by 100 %: dv = 1/8, dp = 1, ds = 0
    yvh = yv.copy()
    yvh[0, 2] = 0.0
    r = oracle.cache_indicator(yv, yvh, flag, ya, ya, s, s, 0.5, 0.1, 0.2, 0.0)
    assert math.isclose(r["dv"], 1 / 8) and r["da"] == 0.0 and math.isclose(r["dp"], 1.0)
    assert math.isclose(r["sync"], 0.5) and not r["reuse"]        # 0.5 * dp decides
    r = oracle.cache_indicator(yv, yvh, flag, ya, ya, s, s, 0.1, 0.1, 0.2, 0.0)
    assert math.isclose(r["sync"], 1 / 8) and r["reuse"]           # dv decides, below tau
    # saliency drift alone: orthogonal maps -> ds = 1 -> 0.1 < 0.2 reuses
    s2 = np.array([[0.0, 1.0, 0, 0, 0, 0, 0, 0]])
    r = oracle.cache_indicator(yv, yv, flag, ya, ya, s, s2, 0.5, 0.1, 0.2, 0.0)
    assert r["ds"] == 1.0 and math.isclose(r["sync"], 0.1) and r["reuse"]
    # the threshold is strict
    r = oracle.cache_indicator(yv, yv, flag, ya, ya, s, s2, 0.5, 0.2, 0.2, 0.0)
    assert r["sync"] == 0.2 and not r["reuse"]
    # missing audio / saliency / protection contribute 0
    r = oracle.cache_indicator(yv, yv, None, None, None, None, None, 0.5, 0.1, 0.2, EPS)
    assert r["sync"] == 0.0 and r["reuse"]
