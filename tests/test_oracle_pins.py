"""Pins for the CPU oracle: each check rests on something other than the
oracle itself -- values worked by hand from the paper's definitions
(tests/golden), brute force over tiny inputs, closed forms, invariants and
independent library routines (torch's BF16 rounding, numpy's fp64 matrix
product).  A plausible slip in the oracle (a dropped term, a wrong sign or
index, a transposed operand, a wrong rounding direction) fails at least one.

HeadGuard, arXiv 2609.35800: per-token min-max (§1; §4 Quantization setup),
KIVI-style and AKVQ-style bases (§2; §4), protection (§3 Applying
protection), storage estimate (§5.4).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from conftest import GOLDEN


# ------------------------------------------------------------- BF16 helpers

def _all_bf16_sorted():
    vals = (np.arange(65536, dtype=np.uint32) << 16).view(np.float32)
    vals = vals[np.isfinite(vals)].astype(np.float64)  # NaN patterns dropped before the cast
    return np.unique(vals)  # sorted, -0 and +0 merge


BF16_TABLE = _all_bf16_sorted()


def bf16_val(h):
    return float(np.array([int(h) << 16], dtype=np.uint32).view(np.float32)[0])


def largest_bf16_le(x):
    return BF16_TABLE[np.searchsorted(BF16_TABLE, x, side="right") - 1]


def smallest_bf16_ge(x):
    return BF16_TABLE[np.searchsorted(BF16_TABLE, x, side="left")]


def _random_f32(rng, n, emin=-140, emax=100):
    sign = rng.choice([-1.0, 1.0], n)
    mant = rng.uniform(1.0, 2.0, n)
    exp = rng.integers(emin, emax, n)
    return (sign * mant * np.exp2(exp.astype(np.float64))).astype(np.float32)


def test_bf16_rne_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([_random_f32(rng, 20000),
                        # exact halfway cases: low half 0x8000 with odd/even high part
                        (np.array([0x3F808000, 0x3F818000, 0xBF808000, 0xBF818000,
                                   0x00008000, 0x00018000], dtype=np.uint32)
                         .view(np.float32))])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle.bf16_rne(v) for v in x], dtype=np.uint16)
    assert np.array_equal(got, ref)


def test_bf16_directed_rounding_brute_force():
    rng = np.random.default_rng(2)
    x = np.concatenate([_random_f32(rng, 20000), np.float32([1.0, -1.0, 0.5, -3.0, 1e-40, -1e-40])])
    for v in x:
        v64 = float(v)
        rd, ru = bf16_val(oracle.bf16_rd(v)), bf16_val(oracle.bf16_ru(v))
        assert rd == largest_bf16_le(v64), v
        assert ru == smallest_bf16_ge(v64), v
        if v64 == bf16_val(oracle.bf16_rne(v)):
            assert rd == ru == v64


# ------------------------------------------------- P1: worked examples

def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden("minmax_hand_examples.json")["cases"],
                         ids=lambda c: c["name"])
def test_minmax_hand_examples(case):
    q, meta = oracle.quantize_group(np.float32(case["values"]), case["bits"])
    assert list(q) == case["codes"]
    assert meta == int(case["meta"], 16)
    assert bf16_val(meta & 0xFFFF) == case["S"]
    assert bf16_val(meta >> 16) == case["m"]
    recon = [oracle.level(meta, int(c)) for c in q]
    assert recon == case["recon_fp32"]
    assert [bf16_val(oracle.bf16_rne(r)) for r in recon] == case["recon_bf16"]


# --------------------------------------------- P2: brute-force nearest level

def _check_group(v, bits, q, meta):
    levels = (1 << bits) - 1
    S = bf16_val(meta & 0xFFFF)
    m = bf16_val(meta >> 16)
    assert (meta >> 16) != 0x8000 and (meta & 0xFFFF) != 0x8000  # canonical zeros
    # m is the largest BF16 not above the minimum
    assert m == largest_bf16_le(float(v.min()))
    # s is the fp32 quotient; S the smallest BF16 not below it, floored at 2^-126
    s32 = (np.float32(v.max()) - np.float32(m)) / np.float32(levels)
    if s32 == 0:
        assert S == 0.0 and np.all(q == 0)
        return
    assert S == max(smallest_bf16_ge(float(s32)), 2.0 ** -126)
    # the grid covers the range
    assert m <= v.min() and m + levels * S >= v.max()
    assert np.all(q <= levels)
    # every code is a nearest level (ties within rounding of t exempt)
    grid = m + S * np.arange(levels + 1, dtype=np.float64)
    for x, c in zip(v.astype(np.float64), q):
        d = np.abs(x - grid)
        assert d[c] <= d.min() + 2.0 ** -18 * S, (x, c, d)


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_quantize_group_brute_force(bits):
    rng = np.random.default_rng(100 + bits)
    for trial in range(400):
        m = int(rng.integers(1, 9))
        scale = 2.0 ** float(rng.integers(-20, 20))
        v = (rng.standard_normal(m) * scale).astype(np.float32)
        v = torch.from_numpy(v).to(torch.bfloat16).float().numpy()  # BF16 inputs
        if trial % 7 == 0:
            v[:] = v[0]  # constant group
        q, meta = oracle.quantize_group(v, bits)
        _check_group(v, bits, q, meta)


def test_quantize_group_fp32_inputs_and_tiny_ranges():
    """fp32 (rotated) inputs, tiny and subnormal ranges, signed zeros."""
    rng = np.random.default_rng(7)
    cases = [np.float32([0.0, -0.0, 0.0]), np.float32([-0.0, -0.0]),
             np.float32([1e-39, 2e-39, 3e-39]), np.float32([1e-45, 0.0]),
             np.float32([2.0 ** -125, 2.0 ** -125 + 2.0 ** -132]),
             np.float32([-1e-38, 1e-38])]
    for _ in range(300):
        cases.append((rng.standard_normal(int(rng.integers(1, 9))) *
                      2.0 ** float(rng.integers(-30, 30))).astype(np.float32))
    for v in cases:
        for bits in (2, 3, 4):
            q, meta = oracle.quantize_group(v, bits)
            _check_group(v, bits, q, meta)


# ---------------------------------------------------------- P3 invariants

@pytest.mark.parametrize("bits", [2, 3, 4])
def test_reconstruction_error_bound(bits):
    rng = np.random.default_rng(11)
    for _ in range(300):
        v = torch.from_numpy(rng.standard_normal(128).astype(np.float32) *
                             np.float32(2.0 ** rng.integers(-8, 8))).to(torch.bfloat16).float().numpy()
        q, meta = oracle.quantize_group(v, bits)
        S = bf16_val(meta & 0xFFFF)
        span = max(abs(float(v.min())), abs(float(v.max())))
        tol = S / 2 + 4 * np.spacing(np.float32(span))
        for x, c in zip(v, q):
            r = oracle.level(meta, int(c))
            assert abs(float(x) - r) <= tol
            rb = bf16_val(oracle.bf16_rne(r))
            assert abs(float(x) - rb) <= tol + abs(rb) * 2.0 ** -8


# ----------------------------------------------------- P4 Hadamard rotation

def _hadamard(D):
    i = np.arange(D)
    pc = np.vectorize(lambda a: bin(a).count("1"))(i[:, None] & i[None, :])
    return np.where(pc % 2 == 0, 1.0, -1.0)


@pytest.mark.parametrize("case", _golden("fwht_worked.json")["cases"], ids=str)
def test_fwht_worked_examples(case):
    assert list(oracle.fwht_raw(case["x"])) == case["raw"]
    if case["norm"] is not None:
        assert list(oracle.fwht_norm(case["x"])) == case["norm"]


@pytest.mark.parametrize("D", [2, 4, 8, 16, 32, 64, 128, 256])
def test_fwht_matches_explicit_matrix(D):
    rng = np.random.default_rng(D)
    Hm = _hadamard(D)
    c = 1.0 / math.sqrt(D)
    assert oracle.fwht_scale(D) == float(np.float32(c))
    for _ in range(50):
        x = (rng.standard_normal(D) * np.exp2(rng.integers(-6, 6, D))).astype(np.float32)
        exact = (Hm @ x.astype(np.float64)) * c
        got = oracle.fwht_norm(x).astype(np.float64)
        bound = 1.01 * (math.log2(D) + 1) * 2.0 ** -24 * c * np.abs(x).astype(np.float64).sum() + 1e-45
        assert np.all(np.abs(got - exact) <= bound)


@pytest.mark.parametrize("D", [4, 16, 64, 128, 256])
def test_fwht_integer_identities(D):
    rng = np.random.default_rng(3 * D)
    x = rng.integers(-1000, 1000, D).astype(np.float32)
    once = oracle.fwht_raw(x)
    assert np.array_equal(once.astype(np.float64), _hadamard(D) @ x.astype(np.float64))
    assert np.array_equal(oracle.fwht_raw(once), x * D)  # H H = D I, exact
    ones = oracle.fwht_norm(np.ones(D, dtype=np.float32))
    assert ones[0] == np.float32(np.float32(D) * np.float32(1.0 / math.sqrt(D)))
    assert np.all(ones[1:] == 0)


@pytest.mark.parametrize("D", [64, 128, 256])
def test_fwht_orthonormal_round_trip(D):
    rng = np.random.default_rng(5)
    for _ in range(50):
        x = rng.standard_normal(D).astype(np.float32)
        back = oracle.fwht_norm(oracle.fwht_norm(x))
        assert np.max(np.abs(back - x)) <= 1e-5 * max(1.0, float(np.abs(x).max())) * math.log2(D)


# ------------------------------------------------------------- routing

def _cfg(**kw):
    base = dict(L=1, B=1, H=4, T=8, D=8, img_start=0, img_len=8, bits=2, base=0,
                keys_only=0, kivi_group=4)
    base.update(kw)
    return oracle.make_config(**base)


@pytest.mark.parametrize("keys_only", [0, 1])
@pytest.mark.parametrize("LH", [(1, 1), (1, 4), (2, 2), (4, 1)])
def test_route_all_masks(keys_only, LH):
    L, H = LH
    c = _cfg(L=L, H=H, keys_only=keys_only)
    for bits in range(1 << (L * H)):
        mask = np.array([(bits >> i) & 1 for i in range(L * H)], dtype=np.uint8)
        for X in (0, 1):
            seen = {True: [], False: []}
            for l in range(L):
                for h in range(H):
                    prot, slot = oracle.route(c, mask, X, l, h)
                    kept = bool(mask[l * H + h]) and (X == 0 or not keys_only)
                    assert prot == kept
                    seen[prot].append(slot)
            for k in (True, False):  # ranks in row-major order: 0, 1, 2, ...
                assert seen[k] == list(range(len(seen[k])))


# ------------------------------------------------------- P7 storage model

def test_storage_model_matches_paper():
    g = _golden("storage_model.json")
    D, bits = g["D"], g["bits"]
    LH = 64  # 8 of 64 heads protected = the paper's 1/8
    mask = np.zeros(LH, dtype=np.uint8)
    mask[:: int(1 / g["protected_fraction"])] = 1
    res = {}
    for name, m, ko in (("uniform", np.zeros(LH, np.uint8), 0), ("kv", mask, 0), ("k_only", mask, 1)):
        c = _cfg(L=8, H=8, D=D, bits=bits, T=16, img_len=16, keys_only=ko)
        s = oracle.sizes(c, m)
        total = sum(s[k] for k in ("codes_k", "meta_k", "side_k", "codes_v", "meta_v", "side_v"))
        res[name] = total * 8 / (2 * 8 * 8 * 16 * D)
    assert res["uniform"] == 2.25 and res["kv"] == 3.96875 and res["k_only"] == 3.109375
    for k, printed in g["printed_bits_per_element"].items():
        assert round(res[k], g["printed_decimals"]) == printed
    assert round(100 * (1 - res["k_only"] / res["kv"])) == g["printed_k_only_saving_percent"]
    # K-only halves the extra storage of K+V
    assert (res["k_only"] - res["uniform"]) * 2 == res["kv"] - res["uniform"]


def test_sizes_layout_closed_form():
    c = _cfg(L=3, B=2, H=5, T=40, D=16, img_start=3, img_len=29, bits=3, base=1, kivi_group=8)
    mask = np.zeros(15, np.uint8)
    mask[[1, 7, 8]] = 1
    s = oracle.sizes(c, mask)
    assert s["n_protected"] == 3 and s["n_unprot_k"] == 12 and s["n_unprot_v"] == 12
    assert s["codes_k"] == 12 * 2 * 29 * 6 and s["codes_v"] == 12 * 2 * 29 * 6
    assert s["meta_k"] == 12 * 2 * 4 * 16 * 4  # ceil(29/8) = 4 groups x 16 channels
    assert s["meta_v"] == 12 * 2 * 29 * 4
    assert s["side_k"] == s["side_v"] == 3 * 2 * 29 * 16 * 2
