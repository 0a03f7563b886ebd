"""hg_select_heads (the library's host implementation of §3 Eq. 2) against
the oracle: identical masks on the worked examples and on random score sets
of the paper's model shapes (GQA groups of 1-7 query heads, budgets from the
capped sweep: 1/16, 1/12, 1/8, 1/4), including exact ties and constant
scores; argument errors."""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2609_35800_amd as hg
from conftest import GOLDEN

CASES = json.load(open(os.path.join(GOLDEN, "select_heads_worked.json")))["cases"]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c["name"])
def test_worked_examples(case):
    g, o = np.array(case["g"]), np.array(case["o"])
    for K, mask in case["masks"].items():
        assert list(hg.hg_select_heads(g, o, case["Hkv"], int(K))) == mask


# (L, Hq, Hkv) of GQA models of the sizes the paper evaluates (7B-12B VLMs)
SHAPES = [(28, 28, 4), (32, 32, 8), (32, 32, 32), (48, 40, 8), (28, 16, 8), (80, 64, 8)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("den", [16, 12, 8, 4])
def test_matches_oracle(shape, den):
    L, Hq, Hkv = shape
    rng = np.random.default_rng(L * 1000 + Hq + den)
    for trial in range(3):
        g = rng.gamma(1.5, 1e-3, size=(L, Hq))
        o = rng.gamma(2.0, 1e-2, size=(L, Hq))
        if trial == 1:  # exact ties: duplicate whole layers
            g[1] = g[0]
            o[1] = o[0]
        K = hg.head_budget(L * Hkv, 1, den)
        got = hg.hg_select_heads(g, o, Hkv, K)
        want = oracle.select_heads(g, o, Hkv, K)
        assert got.sum() == K
        assert np.array_equal(got, want)


def test_constant_scores_and_budget_edges():
    g = np.ones((4, 8))
    o = np.full((4, 8), 3.0)
    assert list(hg.hg_select_heads(g, o, 2, 3)) == [1, 1, 1, 0, 0, 0, 0, 0]
    assert hg.hg_select_heads(g, o, 2, 0).sum() == 0
    assert hg.hg_select_heads(g, o, 2, 100).sum() == 8
    # the protected-head counts of the five workloads (1/8 of N_KV), and halves up
    assert [hg.head_budget(n) for n in (8, 112, 1024, 256, 640, 12, 4)] == [1, 14, 128, 32, 80, 2, 1]


def test_head_budget_rounding_and_errors():
    # exact integer rounding, halves up, no floating-point drift at large n
    assert hg.head_budget(20, 1, 8) == 3      # 2.5 -> 3
    assert hg.head_budget(12, 1, 16) == 1     # 0.75 -> 1
    assert hg.head_budget(8, 1, 16) == 1      # 0.5 -> 1
    assert hg.head_budget(7, 1, 16) == 0      # 0.4375 -> 0
    assert hg.head_budget(8192, 1, 1) == 8192 and hg.head_budget(8192, 0, 5) == 0
    assert hg.head_budget(8191, 1, 4) == 2048  # 2047.75
    for n in range(1, 300):
        for num, den in ((1, 16), (1, 12), (1, 8), (1, 4), (3, 8)):
            want = (2 * n * num + den) // (2 * den)
            assert hg.head_budget(n, num, den) == want == int(np.floor(n * num / den + 0.5))
    for bad in ((0, 1, 8), (8, -1, 8), (8, 9, 8), (8, 1, 0)):
        with pytest.raises(hg.HeadGuardError) as e:
            hg.head_budget(*bad)
        assert e.value.status == hg.HG_ERR_SHAPE


def test_errors():
    g = np.ones((2, 4))
    with pytest.raises(hg.HeadGuardError) as e:
        hg.hg_select_heads(g, g, 3, 1)  # 4 query heads do not split into 3 groups
    assert e.value.status == hg.HG_ERR_SHAPE
    with pytest.raises(hg.HeadGuardError) as e:
        hg.hg_select_heads(g, g, 2, -1)
    assert e.value.status == hg.HG_ERR_SHAPE
    bad = g.copy()
    bad[1, 2] = np.nan
    with pytest.raises(hg.HeadGuardError) as e:
        hg.hg_select_heads(bad, g, 2, 1)
    assert e.value.status == hg.HG_ERR_VALUE
