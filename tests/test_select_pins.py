"""Pins for the oracle's head selection (§3 'Selecting physical KV heads',
Eq. 2): hand-worked cases (tests/golden/select_heads_worked.json) and
invariances that any correct implementation of s = z(g) + z(o), TopK must
have: positive affine maps of either score, a permutation of the heads, the
choice of population or sample deviation, and the swap of g and o leave the
selected set unchanged (up to the permutation); budgets 0 and N_KV."""
import json
import os

import numpy as np
import pytest

import oracle
from conftest import GOLDEN

CASES = json.load(open(os.path.join(GOLDEN, "select_heads_worked.json")))["cases"]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c["name"])
def test_worked_examples(case):
    g, o = np.array(case["g"]), np.array(case["o"])
    for K, mask in case["masks"].items():
        assert list(oracle.select_heads(g, o, case["Hkv"], int(K))) == mask


def _rand(rng, L=6, Hq=8, Hkv=2):
    return rng.gamma(2.0, size=(L, Hq)), rng.gamma(2.0, size=(L, Hq)), Hkv


@pytest.mark.parametrize("seed", range(20))
def test_affine_invariance(seed):
    rng = np.random.default_rng(seed)
    g, o, Hkv = _rand(rng)
    K = int(rng.integers(1, 12))
    base = oracle.select_heads(g, o, Hkv, K)
    a, b = float(rng.uniform(0.1, 10)), float(rng.uniform(-5, 5))
    assert np.array_equal(oracle.select_heads(a * g + b, o, Hkv, K), base)
    assert np.array_equal(oracle.select_heads(g, a * o + b, Hkv, K), base)
    assert np.array_equal(oracle.select_heads(o, g, Hkv, K), base)


@pytest.mark.parametrize("seed", range(10))
def test_layer_permutation(seed):
    rng = np.random.default_rng(100 + seed)
    g, o, Hkv = _rand(rng)
    K = 4
    perm = rng.permutation(g.shape[0])
    base = oracle.select_heads(g, o, Hkv, K).reshape(g.shape[0], Hkv)
    got = oracle.select_heads(g[perm], o[perm], Hkv, K).reshape(g.shape[0], Hkv)
    assert np.array_equal(got, base[perm])


def test_budgets_and_gqa_grouping():
    rng = np.random.default_rng(7)
    g, o, Hkv = _rand(rng, L=3, Hq=6, Hkv=3)
    assert oracle.select_heads(g, o, Hkv, 0).sum() == 0
    assert oracle.select_heads(g, o, Hkv, 9).sum() == 9
    assert oracle.select_heads(g, o, Hkv, 50).sum() == 9
    # a query head's score counts only toward its own KV group (hq // 2)
    g2 = g.copy()
    g2[1, 4] += 100.0  # layer 1, query head 4 -> KV head 2
    m = oracle.select_heads(g2, o, Hkv, 1).reshape(3, 3)
    assert m[1, 2] == 1 and m.sum() == 1


def test_sample_vs_population_deviation_same_ranking():
    """z with ddof=1 is z with ddof=0 times sqrt((N-1)/N) for both scores."""
    rng = np.random.default_rng(11)
    for _ in range(20):
        g, o, Hkv = _rand(rng)
        gb = g.reshape(g.shape[0], Hkv, -1).mean(-1).ravel()
        ob = o.reshape(o.shape[0], Hkv, -1).mean(-1).ravel()
        s1 = (gb - gb.mean()) / gb.std(ddof=1) + (ob - ob.mean()) / ob.std(ddof=1)
        K = 5
        top = np.argsort(-s1, kind="stable")[:K]
        want = np.zeros(gb.size, np.uint8)
        want[top] = 1
        assert np.array_equal(oracle.select_heads(g, o, Hkv, K), want)
