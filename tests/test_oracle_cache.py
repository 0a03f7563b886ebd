"""Whole-cache pins for the CPU oracle: protection routing (§3 Applying
protection), the KIVI-style per-channel key groups and per-token values (§2;
§4), AKVQ-style rotation (§2; §4), text KV untouched (§3), and the invariants
every base must satisfy.  Each check rests on an independent fact: bit
identity of protected/text rows, transposition equivalence with the per-token
routine (itself pinned by brute force), error bounds from the stored scale,
Parseval for the orthonormal rotation."""
import math

import numpy as np
import pytest
import torch

import oracle
import synthkv


def _bits(t):
    return synthkv.bf16_bits(t)


def _f32(u16):
    return (u16.astype(np.uint32) << 16).view(np.float32)


def small_workload(base="minmax", **kw):
    w = synthkv.Workload("small", L=2, B=2, H=3, T=50, D=16, img_start=5, img_len=37,
                         bits=2, base=base, keys_only=0, n_protected=2,
                         k_outliers=2, k_outlier_scale=10.0, kivi_group=8)
    return w.with_(**kw)


def run_oracle(w, mask=None, threads=2):
    K, V = synthkv.gen_kv(w)
    Kb, Vb = _bits(K), _bits(V)
    if mask is None:
        mask = synthkv.protect_mask(w)
    cfg = oracle.make_config(**w.config_fields())
    packed = oracle.quantize(cfg, Kb, Vb, mask, threads=threads)
    Ko = np.full_like(Kb, 0x7FBF)  # sentinel (a NaN pattern the method never writes)
    Vo = np.full_like(Vb, 0x7FBF)
    oracle.dequantize(cfg, mask, packed, Ko, Vo, threads=threads)
    return cfg, mask, Kb, Vb, packed, Ko, Vo


def img(a, w):
    return a[:, :, :, w.img_start:w.img_start + w.img_len, :]


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
@pytest.mark.parametrize("keys_only", [0, 1])
def test_text_untouched_and_protected_identical(base, keys_only):
    w = small_workload(base, keys_only=keys_only)
    cfg, mask, Kb, Vb, packed, Ko, Vo = run_oracle(w)
    # text rows are never written
    for A in (Ko, Vo):
        assert np.all(A[:, :, :, :w.img_start] == 0x7FBF)
        assert np.all(A[:, :, :, w.img_start + w.img_len:] == 0x7FBF)
        assert not np.any(img(A, w) == 0x7FBF)
    m2 = mask.reshape(w.L, w.H).astype(bool)
    for l in range(w.L):
        for h in range(w.H):
            kk = np.array_equal(img(Ko, w)[l, :, h], img(Kb, w)[l, :, h])
            vv = np.array_equal(img(Vo, w)[l, :, h], img(Vb, w)[l, :, h])
            if m2[l, h]:
                assert kk
                assert vv == (not keys_only) or vv  # V identical only if protected
                if not keys_only:
                    assert vv
            else:
                assert not kk and not vv  # 2-bit quantization changes N(0,1) data


def test_mask_special_cases():
    w = small_workload("minmax")
    LH = w.L * w.H
    # all protected, K+V: the lossless BF16 reference
    cfg, mask, Kb, Vb, packed, Ko, Vo = run_oracle(w, np.ones(LH, np.uint8))
    assert np.array_equal(img(Ko, w), img(Kb, w)) and np.array_equal(img(Vo, w), img(Vb, w))
    assert packed["codes_k"].size == packed["codes_v"].size == 0
    # all protected, K-only: keys exact, values quantized
    w1 = w.with_(keys_only=1)
    cfg, mask, Kb, Vb, packed, Ko, Vo = run_oracle(w1, np.ones(LH, np.uint8))
    assert np.array_equal(img(Ko, w), img(Kb, w))
    assert packed["side_v"].size == 0 and packed["codes_v"].size > 0
    # nothing protected: the pure base, same codes as slice-by-slice
    cfg, mask, Kb, Vb, packed, Ko, Vo = run_oracle(w, np.zeros(LH, np.uint8))
    assert packed["side_k"].size == packed["side_v"].size == 0
    row = w.D * w.bits // 8
    codes_k = packed["codes_k"].reshape(LH, w.B, w.img_len, row)
    for l in range(w.L):
        for b in range(w.B):
            for h in range(w.H):
                c, _ = oracle.quantize_slice(cfg, 0, img(Kb, w)[l, b, h])
                assert np.array_equal(codes_k[l * w.H + h, b], c)


def test_threads_do_not_change_results():
    w = small_workload("akvq")
    a = run_oracle(w, threads=1)
    b = run_oracle(w, threads=5)
    for k in a[4]:
        assert np.array_equal(a[4][k], b[4][k])
    assert np.array_equal(a[5], b[5]) and np.array_equal(a[6], b[6])


def _unpack(codes_row, bits, D):
    bitsarr = np.unpackbits(codes_row, bitorder="little")
    return np.array([int(sum(int(bitsarr[bits * i + k]) << k for k in range(bits)))
                     for i in range(D)])


def test_kivi_keys_equal_transposed_per_token():
    """P5: KIVI-style key codes of a G x D tile are the per-token routine
    applied to each channel's G values; last group ragged."""
    w = small_workload("kivi", img_len=37, kivi_group=8, bits=3)
    cfg = oracle.make_config(**w.config_fields())
    K, _ = synthkv.gen_kv(w)
    rows = img(_bits(K), w)[1, 0, 2]  # one slice [n, D]
    codes, meta = oracle.quantize_slice(cfg, 0, rows)
    x = _f32(rows)
    G = w.kivi_group
    for g0 in range(0, w.img_len, G):
        tile = x[g0:g0 + G]  # last group: 5 tokens
        for d in range(w.D):
            q, mw = oracle.quantize_group(tile[:, d].copy(), w.bits)
            assert meta[g0 // G, d] == mw
            for t in range(tile.shape[0]):
                assert _unpack(codes[g0 + t], w.bits, w.D)[d] == q[t]


def test_values_are_per_token_in_every_base():
    for base in ("minmax", "kivi", "akvq"):
        w = small_workload(base)
        cfg = oracle.make_config(**w.config_fields())
        _, V = synthkv.gen_kv(w)
        rows = img(_bits(V), w)[0, 1, 1]
        codes, meta = oracle.quantize_slice(cfg, 1, rows)
        x = _f32(rows)
        for t in range(w.img_len):
            q, mw = oracle.quantize_group(x[t].copy(), w.bits)
            assert meta[t] == mw
            assert np.array_equal(_unpack(codes[t], w.bits, w.D), q)


def test_packing_lsb_first():
    """Codes occupy bits [b*i, b*i+b) of each token row, least significant first."""
    w = small_workload("minmax", bits=3, D=16)
    cfg = oracle.make_config(**w.config_fields())
    rows = np.zeros((w.img_len, w.D), np.uint16)
    vals = np.arange(8, dtype=np.float32)  # 0..7 -> codes 0..7 exactly
    rows[:] = torch.from_numpy(np.tile(vals, 2)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    codes, meta = oracle.quantize_slice(cfg, 1, rows)
    expect = 0
    for i, q in enumerate(list(range(8)) * 2):
        expect |= q << (3 * i)
    assert int.from_bytes(codes[0].tobytes(), "little") == expect


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_minmax_error_bound_and_constant_tokens(bits):
    w = small_workload("minmax", bits=bits)
    K, V = synthkv.gen_kv(w)
    K[0, 0, 0, w.img_start + 3, :] = 2.5  # a constant token
    Kb, Vb = _bits(K), _bits(V)
    mask = np.zeros(w.L * w.H, np.uint8)
    cfg = oracle.make_config(**w.config_fields())
    packed = oracle.quantize(cfg, Kb, Vb, mask)
    Ko, Vo = Kb.copy(), Vb.copy()
    oracle.dequantize(cfg, mask, packed, Ko, Vo)
    assert np.array_equal(Ko[0, 0, 0, w.img_start + 3], Kb[0, 0, 0, w.img_start + 3])
    meta = packed["meta_k"].reshape(w.L * w.H, w.B, w.img_len)
    x, xh = _f32(img(Kb, w)), _f32(img(Ko, w))
    for l in range(w.L):
        for b in range(w.B):
            for h in range(w.H):
                S = _f32((meta[l * w.H + h, b] & 0xFFFF).astype(np.uint16))
                err = np.abs(x[l, b, h] - xh[l, b, h]).max(axis=1)
                bf_half_ulp = np.abs(xh[l, b, h]).max(axis=1) * 2.0 ** -8
                assert np.all(err <= S / 2 + bf_half_ulp + 1e-30)


def test_akvq_parseval_bound():
    w = small_workload("akvq", D=64, img_len=20)
    K, V = synthkv.gen_kv(w)
    Kb, Vb = _bits(K), _bits(V)
    mask = np.zeros(w.L * w.H, np.uint8)
    cfg = oracle.make_config(**w.config_fields())
    packed = oracle.quantize(cfg, Kb, Vb, mask)
    Ko, Vo = Kb.copy(), Vb.copy()
    oracle.dequantize(cfg, mask, packed, Ko, Vo)
    meta = packed["meta_k"].reshape(w.L * w.H, w.B, w.img_len)
    x, xh = _f32(img(Kb, w)).astype(np.float64), _f32(img(Ko, w)).astype(np.float64)
    for l in range(w.L):
        for b in range(w.B):
            for h in range(w.H):
                S = _f32((meta[l * w.H + h, b] & 0xFFFF).astype(np.uint16)).astype(np.float64)
                err = np.linalg.norm(x[l, b, h] - xh[l, b, h], axis=1)
                norm = np.linalg.norm(xh[l, b, h], axis=1)
                assert np.all(err <= math.sqrt(w.D) * S / 2 * 1.001 + norm * 2.0 ** -8 + 1e-6)
    # in the rotated domain each element is within S/2 of its level
    rows = img(Kb, w)[0, 0, 0]
    codes, m = oracle.quantize_slice(cfg, 0, rows)
    for t in range(w.img_len):
        y = oracle.fwht_norm(_f32(rows[t]))
        q = _unpack(codes[t], w.bits, w.D)
        S = _f32(np.uint16([m[t] & 0xFFFF]))[0]
        lv = np.array([oracle.level(int(m[t]), int(c)) for c in q])
        assert np.all(np.abs(y - lv) <= S / 2 * (1 + 1e-6) + 1e-30)


def test_empty_span():
    w = small_workload("minmax", img_len=0)
    cfg, mask, Kb, Vb, packed, Ko, Vo = run_oracle(w)
    assert all(v.size == 0 for v in packed.values())
    assert np.all(Ko == 0x7FBF)


# ------------------------------------------------- KIVI-style keys, whole sequence

def test_kivi_whole_sequence_keys():
    """kivi_group = 0 (§4: KIVI-style key ranges recomputed over the supplied
    sequence, text included; text KV stays BF16): per channel, the metadata is
    the per-token routine over the channel's T values; image codes are that
    group's codes at the image positions."""
    w = small_workload("kivi", kivi_group=0, bits=2, img_start=5, img_len=37, T=50)
    cfg = oracle.make_config(**w.config_fields())
    K, _ = synthkv.gen_kv(w)
    sl = _bits(K)[1, 0, 2]  # whole slice [T, D]
    codes, meta = oracle.quantize_slice_seq(cfg, 0, sl)
    assert meta.shape == (1, w.D)
    x = _f32(sl)
    for d in range(w.D):
        q, mw = oracle.quantize_group(x[:, d].copy(), w.bits)
        assert meta[0, d] == mw
        for t in range(w.img_len):
            assert _unpack(codes[t], w.bits, w.D)[d] == q[w.img_start + t]
    # a text outlier widens the range and so changes the image tokens' metadata
    sl2 = sl.copy()
    sl2[0, 3] = 0x4700  # 32768.0 in a text row
    _, meta2 = oracle.quantize_slice_seq(cfg, 0, sl2)
    assert meta2[0, 3] != meta[0, 3] and np.array_equal(np.delete(meta2, 3), np.delete(meta, 3))
    # the image-rows entry point cannot see the text and refuses this mode
    with pytest.raises(ValueError):
        oracle.quantize_slice(cfg, 0, sl[w.img_start:w.img_start + w.img_len])


def test_kivi_whole_sequence_cache_round_trip():
    w = small_workload("kivi", kivi_group=0, bits=3)
    cfg, mask, Kb, Vb, packed, Ko, Vo = run_oracle(w)
    sizes = oracle.sizes(cfg, mask)
    assert sizes["meta_k"] == sizes["n_unprot_k"] * w.B * w.D * 4
    assert np.all(Ko[:, :, :, :w.img_start] == 0x7FBF)  # text untouched
    meta = packed["meta_k"].reshape(-1, w.B, 1, w.D)
    x, xh = _f32(img(Kb, w)), _f32(img(Ko, w))
    m2 = mask.reshape(w.L, w.H).astype(bool)
    u = 0
    for l in range(w.L):
        for h in range(w.H):
            if m2[l, h]:
                continue
            for b in range(w.B):
                S = _f32((meta[u, b, 0] & 0xFFFF).astype(np.uint16))
                err = np.abs(x[l, b, h] - xh[l, b, h])
                assert np.all(err <= S / 2 + np.abs(xh[l, b, h]) * 2.0 ** -8 + 1e-30)
            u += 1
