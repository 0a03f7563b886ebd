"""Pins for the oracle's AKVQ-style token retention (§4 Quantization setup: in
each KV head the keys and values of a nominal 2 % of the image tokens, those
with the largest key norms, stay in BF16, with or without head protection).

Each check rests on something other than the oracle itself: hand-computed
counts and fp32 sums, exact integer and rational arithmetic, the textbook
error bound of pairwise summation, and a rank-counting definition of the
top-k selection on brute-force inputs."""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synthkv


def _f32(u16):
    return (np.asarray(u16, np.uint16).astype(np.uint32) << 16).view(np.float32)


def _bf16_of(values):
    """BF16 bit patterns of values that are exactly representable in BF16."""
    f = np.asarray(values, np.float32)
    u = f.view(np.uint32)
    assert np.all(u & 0xFFFF == 0), "not exact in BF16"
    return (u >> 16).astype(np.uint16)


def _exact_sqnorm(row_u16):
    return sum((Fraction(float(x)) ** 2 for x in _f32(row_u16)), Fraction(0))


def _rank_select(scores, k):
    """Token t is kept iff fewer than k tokens precede it in the order
    (larger score first, lower index first among equals)."""
    n = len(scores)
    keep = [t for t in range(n)
            if sum(1 for u in range(n) if scores[u] > scores[t] or (scores[u] == scores[t] and u < t)) < k]
    return np.array(keep, dtype=np.int32)


# ---------------------------------------------------------------- the count

# k = round(n * 2 %), halves rounded up: n/50 worked by hand.
COUNT_2PCT = {0: 0, 1: 0, 24: 0, 25: 1, 26: 1, 49: 1, 74: 1, 75: 2, 100: 2, 124: 2, 125: 3,
              1296: 26, 2880: 58, 3328: 67, 6400: 128}


@pytest.mark.parametrize("n,k", sorted(COUNT_2PCT.items()))
def test_count_two_percent(n, k):
    cfg = oracle.make_config(L=1, B=1, H=1, T=max(n, 1), D=64, img_start=0, img_len=n, bits=2,
                             base=2, keys_only=0, kivi_group=32, retain_permille=20)
    assert oracle.retain_count(cfg) == k


def test_count_other_fractions():
    # 1000 per mille keeps every token, 0 none; 1 per mille of 500 is exactly one half -> 1
    for pm, n, k in ((1000, 37, 37), (0, 37, 0), (1, 500, 1), (1, 499, 0), (125, 8, 1), (500, 3, 2)):
        cfg = oracle.make_config(L=1, B=1, H=1, T=n, D=64, img_start=0, img_len=n, bits=2,
                                 base=2, keys_only=0, kivi_group=32, retain_permille=pm)
        assert oracle.retain_count(cfg) == k, (pm, n)


def test_retention_needs_the_akvq_base():
    mask = np.zeros(2, np.uint8)
    for base in (0, 1):
        cfg = oracle.make_config(L=1, B=1, H=2, T=40, D=64, img_start=0, img_len=40, bits=2,
                                 base=base, keys_only=0, kivi_group=32, retain_permille=20)
        with pytest.raises(ValueError):
            oracle.sizes(cfg, mask)
    for pm in (-1, 1001):
        cfg = oracle.make_config(L=1, B=1, H=2, T=40, D=64, img_start=0, img_len=40, bits=2,
                                 base=2, keys_only=0, kivi_group=32, retain_permille=pm)
        with pytest.raises(ValueError):
            oracle.sizes(cfg, mask)


# ---------------------------------------------------------------- the norm

@pytest.mark.parametrize("D,want", [(64, 2.0 ** 24 + 62), (128, 2.0 ** 24 + 126), (256, 2.0 ** 24 + 254)])
@pytest.mark.parametrize("where", [0, -1, 17])
def test_sqnorm_pairwise_order(D, want, where):
    """One entry 2^12 (square 2^24) among ones.  Worked by hand: the first pair
    2^24 + 1 ties and rounds to even (2^24), every other subtree sums its ones
    exactly, and the running sum stays even: 2^24 + 2 + 4 + ... + D/2 =
    2^24 + D - 2.  (A running left-to-right sum would lose every 1 and give
    2^24; the exact value is 2^24 + D - 1.)"""
    x = np.ones(D, np.float32)
    x[where] = 2.0 ** 12
    got = oracle.key_sqnorm(_bf16_of(x))
    assert got == want


@pytest.mark.parametrize("D", [64, 128, 256])
def test_sqnorm_exact_for_small_integers(D):
    """Integer entries |x| <= 15: every square and partial sum is an integer
    below 2^24, so the fp32 result is the exact sum."""
    rng = np.random.default_rng(D)
    for _ in range(50):
        x = rng.integers(-15, 16, D)
        assert oracle.key_sqnorm(_bf16_of(x)) == float(np.sum(x.astype(np.int64) ** 2))


@pytest.mark.parametrize("D", [64, 128, 256])
def test_sqnorm_within_pairwise_error_bound(D):
    """BF16 squares are exact in fp32 (8-bit significands); pairwise summation
    over log2(D) levels errs by at most gamma_{log2 D} times the exact sum."""
    rng = np.random.default_rng(7 + D)
    levels = int(math.log2(D))
    u = Fraction(1, 2 ** 24)
    gamma = levels * u / (1 - levels * u)
    for _ in range(40):
        x = rng.standard_normal(D) * rng.uniform(0.01, 100)
        row = synthkv.bf16_bits(torch.from_numpy(x.astype(np.float32)).bfloat16())
        exact = _exact_sqnorm(row)
        got = Fraction(oracle.key_sqnorm(row))
        assert abs(got - exact) <= gamma * exact


def test_sqnorm_special_cases():
    D = 64
    assert oracle.key_sqnorm(np.zeros(D, np.uint16)) == 0.0
    assert oracle.key_sqnorm(np.full(D, 0x8000, np.uint16)) == 0.0  # -0 squares to +0
    for v in (3.0, -0.5, 2.0 ** -60):
        x = np.zeros(D, np.float32)
        x[5] = v
        assert oracle.key_sqnorm(_bf16_of(x)) == v * v
    # equal entries: every level doubles exactly
    assert oracle.key_sqnorm(_bf16_of(np.full(D, 1.5, np.float32))) == D * 2.25
    # 2^-70 squares to 2^-140, a subnormal fp32 value, kept exactly (no flush)
    assert oracle.key_sqnorm(_bf16_of(np.full(D, 2.0 ** -70, np.float32))) == D * 2.0 ** -140
    # a single 2^-72 squares to the subnormal 2^-144 and is kept; spread over
    # all D entries (as a rotation would spread it) each square would round to 0
    for D2 in (64, 128):
        x = np.zeros(D2, np.float32)
        x[D2 // 3] = 2.0 ** -72
        assert oracle.key_sqnorm(_bf16_of(x)) == 2.0 ** -144
    # 2^64 squares past the fp32 range
    x = np.zeros(D, np.float32)
    x[0] = 2.0 ** 64
    assert oracle.key_sqnorm(_bf16_of(x)) == math.inf


# ---------------------------------------------------------------- the selection

def test_select_brute_force_with_ties():
    rng = np.random.default_rng(11)
    for n in range(0, 13):
        for _ in range(6):
            scores = rng.integers(0, 4, n).astype(np.float32)  # many ties
            for k in range(0, n + 1):
                got = oracle.retain_select(scores, k)
                assert np.array_equal(got, _rank_select(list(scores), k)), (scores, k)


def test_select_all_orders_of_a_small_set():
    # every permutation of a set with a tie: the lower index wins the tie
    base = [5.0, 3.0, 3.0, 1.0]
    for perm in itertools.permutations(range(4)):
        scores = np.array([base[p] for p in perm], np.float32)
        for k in range(5):
            assert np.array_equal(oracle.retain_select(scores, k), _rank_select(list(scores), k))


def test_select_infinities_tie_to_the_lower_index():
    scores = np.array([1.0, math.inf, 2.0, math.inf, math.inf], np.float32)
    assert list(oracle.retain_select(scores, 2)) == [1, 3]


def test_select_rejects_bad_counts():
    with pytest.raises(ValueError):
        oracle.retain_select(np.zeros(3, np.float32), 4)
    with pytest.raises(ValueError):
        oracle.retain_select(np.zeros(3, np.float32), -1)


def test_selection_matches_exact_norm_ranking():
    """On Gaussian keys the kept set is the top-k by exact norm whenever the
    gap at the boundary exceeds twice the summation error bound."""
    rng = np.random.default_rng(3)
    D, n, k = 64, 300, 6
    gamma = 6 * Fraction(1, 2 ** 24)
    for _ in range(5):
        rows = synthkv.bf16_bits(torch.from_numpy(rng.standard_normal((n, D)).astype(np.float32)).bfloat16())
        exact = [_exact_sqnorm(r) for r in rows]
        order = sorted(range(n), key=lambda t: (-exact[t], t))
        gap = exact[order[k - 1]] - exact[order[k]]
        assert gap > 2 * gamma * exact[order[k - 1]]
        norms = np.array([oracle.key_sqnorm(r) for r in rows], np.float32)
        assert np.array_equal(oracle.retain_select(norms, k), np.sort(order[:k]).astype(np.int32))


# ---------------------------------------------------------------- whole cache

def _workload(**kw):
    w = synthkv.Workload("retain", L=2, B=2, H=3, T=70, D=64, img_start=4, img_len=61, bits=2,
                         base="akvq", keys_only=0, n_protected=2, k_outliers=2,
                         k_outlier_scale=10.0, retain_permille=100)
    return w.with_(**kw)


def _integer_kv(w, seed):
    """Small-integer BF16 caches: exact key norms, many ties."""
    rng = np.random.default_rng(seed)
    shape = (w.L, w.B, w.H, w.T, w.D)
    K = _bf16_of(rng.integers(-6, 7, shape).astype(np.float32))
    V = _bf16_of(rng.integers(-6, 7, shape).astype(np.float32))
    return K.reshape(shape), V.reshape(shape)


def _run(w, K, V, mask):
    cfg = oracle.make_config(**w.config_fields())
    packed = oracle.quantize(cfg, K, V, mask, threads=3)
    Ko = np.full_like(K, 0x7FBF)
    Vo = np.full_like(V, 0x7FBF)
    oracle.dequantize(cfg, mask, packed, Ko, Vo, threads=2)
    return cfg, packed, Ko, Vo


@pytest.mark.parametrize("keys_only", [0, 1])
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_cache_retention(keys_only, bits):
    w = _workload(keys_only=keys_only, bits=bits)
    K, V = _integer_kv(w, 100 + bits)
    mask = np.zeros(w.L * w.H, np.uint8)
    mask[[1, 4]] = 1
    cfg, packed, Ko, Vo = _run(w, K, V, mask)
    n, D, s0 = w.img_len, w.D, w.img_start
    k = round(n * 0.1)  # 6.1 -> 6
    assert oracle.retain_count(cfg) == k == 6
    norms = packed["norm_k"].reshape(w.L, w.B, w.H, n)
    idx = packed["ret_idx"].reshape(w.L, w.B, w.H, k)
    # reference round trip without retention: the same base, fraction 0
    w0 = w.with_(retain_permille=0)
    _, packed0, Ko0, Vo0 = _run(w0, K, V, mask)
    for key in ("codes_k", "meta_k", "side_k", "codes_v", "meta_v", "side_v"):
        assert np.array_equal(packed[key], packed0[key])  # retained tokens are still quantized
    retk = packed["ret_k"].reshape(-1, w.B, k, D)
    retv = packed["ret_v"].reshape(-1, w.B, k, D)
    for l in range(w.L):
        for b in range(w.B):
            for h in range(w.H):
                exact = ((_f32(K[l, b, h, s0:s0 + n]).astype(np.int64)) ** 2).sum(axis=1)
                assert np.array_equal(norms[l, b, h], exact.astype(np.float32))
                want = _rank_select(list(exact), k)
                assert np.array_equal(idx[l, b, h], want)
                keep = np.zeros(n, bool)
                keep[want] = True
                for X, (src, got, ref, ret) in enumerate(((K, Ko, Ko0, retk), (V, Vo, Vo0, retv))):
                    prot, slot = oracle.route(cfg, mask, X, l, h)
                    g = got[l, b, h, s0:s0 + n]
                    if prot:
                        assert np.array_equal(g, src[l, b, h, s0:s0 + n])
                        continue
                    assert np.array_equal(ret[slot, b], src[l, b, h, s0 + want])
                    assert np.array_equal(g[keep], src[l, b, h, s0:s0 + n][keep])
                    assert np.array_equal(g[~keep], ref[l, b, h, s0:s0 + n][~keep])
    for A in (Ko, Vo):  # text rows never written
        assert np.all(A[:, :, :, :s0] == 0x7FBF) and np.all(A[:, :, :, s0 + n:] == 0x7FBF)


def test_sizes_of_the_retention_buffers():
    w = _workload(keys_only=1)
    mask = np.zeros(w.L * w.H, np.uint8)
    mask[[0, 5]] = 1
    sz = oracle.sizes(oracle.make_config(**w.config_fields()), mask)
    # L*B*H = 12 heads-by-batch, n = 61, k = 6; K quantized in 4 heads, V in 6 (keys only)
    assert sz["retain_count"] == 6
    assert sz["norm_k"] == 12 * 61 * 4
    assert sz["ret_idx"] == 12 * 6 * 4
    assert sz["ret_k"] == 4 * 2 * 6 * 64 * 2
    assert sz["ret_v"] == 6 * 2 * 6 * 64 * 2
    off = oracle.sizes(oracle.make_config(**w.with_(retain_permille=0).config_fields()), mask)
    assert off["norm_k"] == off["ret_idx"] == off["ret_k"] == off["ret_v"] == off["retain_count"] == 0


def test_paper_fraction_on_gaussian_keys():
    """2 % of a 96-token span is 2 tokens per head: the two largest key norms
    (exact rational norms, distinct on this draw) are kept bit-identical."""
    w = _workload(img_len=96, T=100, retain_permille=20, L=1, B=2, H=2, n_protected=0)
    K, V = synthkv.gen_kv(w)
    Kb, Vb = synthkv.bf16_bits(K), synthkv.bf16_bits(V)
    mask = np.zeros(w.L * w.H, np.uint8)
    cfg, packed, Ko, Vo = _run(w, Kb, Vb, mask)
    s0, n = w.img_start, w.img_len
    idx = packed["ret_idx"].reshape(w.L, w.B, w.H, 2)
    for b in range(w.B):
        for h in range(w.H):
            exact = [_exact_sqnorm(r) for r in Kb[0, b, h, s0:s0 + n]]
            top = sorted(range(n), key=lambda t: -exact[t])[:2]
            assert list(idx[0, b, h]) == sorted(top)
            for t in top:
                assert np.array_equal(Ko[0, b, h, s0 + t], Kb[0, b, h, s0 + t])
                assert np.array_equal(Vo[0, b, h, s0 + t], Vb[0, b, h, s0 + t])


@pytest.mark.parametrize("n", [0, 4])
def test_degenerate_spans(n):
    """No image tokens, and a span too short to keep any token at 2 %."""
    w = _workload(img_len=n, retain_permille=20)
    K, V = _integer_kv(w, 5)
    mask = np.zeros(w.L * w.H, np.uint8)
    cfg, packed, Ko, Vo = _run(w, K, V, mask)
    assert oracle.retain_count(cfg) == 0
    assert packed["ret_idx"].size == packed["ret_k"].size == packed["ret_v"].size == 0
    assert packed["norm_k"].size == w.L * w.B * w.H * n
    _, packed0, Ko0, Vo0 = _run(w.with_(retain_permille=0), K, V, mask)
    assert np.array_equal(Ko, Ko0) and np.array_equal(Vo, Vo0)
