"""GPU parity: the HIP library against the CPU oracle on the same seeded BF16
bytes.  Packed codes, metadata and the BF16 side store must be bit-exact;
dequantized BF16 within 1 BF16 ulp (expected: 0).  Text rows must stay
untouched and canary bytes after every output buffer intact.

Small shapes are compared element by element and span several workgroup
tiles (128 tokens; 64 in dequantize) with ragged tails; every base, head_dim, bit width and
protection mode is covered, with special values (constant tokens, signed
zeros, tiny/subnormal ranges, exact ties, large magnitudes) and degenerate
masks and spans."""
import numpy as np
import pytest
import torch

import synthkv
from hgtest import compare_full, f32_of_bf16

pytestmark = pytest.mark.gpu


def _assert_exact(rep, tag):
    bad = {k: v for k, v in rep.items() if k.endswith("_mismatch") and v}
    assert rep["canaries"], f"{tag}: canary bytes overwritten"
    assert rep.get("exchange_timeouts", 0) == 0, f"{tag}: exchange waits ran out of polls"
    assert not bad, f"{tag}: packed mismatches {bad}"
    assert rep["K_ulp"] <= 1 and rep["V_ulp"] <= 1, f"{tag}: dequant ulp {rep}"
    # the reconstruction rule is exact on both sides: report any ulp drift
    assert rep["K_exact"] and rep["V_exact"], f"{tag}: dequant not bit-exact {rep}"


def small(base, D=128, bits=2, keys_only=0, img_len=300, img_start=7, text=13, L=2, B=2, H=3,
          n_protected=2, seed=0):
    return synthkv.Workload(f"{base}-D{D}-b{bits}-ko{keys_only}-n{img_len}", L=L, B=B, H=H,
                            T=img_start + img_len + text, D=D, img_start=img_start,
                            img_len=img_len, bits=bits, base=base, keys_only=keys_only,
                            n_protected=n_protected, k_outliers=4, k_outlier_scale=10.0,
                            kivi_group=32, seed=seed)


CASES = [small(b, D, bits, ko)
         for b in ("minmax", "kivi", "akvq") for D in (64, 128, 256) for bits in (2, 3, 4)
         for ko in (0, 1)]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_small_parity(w):
    K, V = synthkv.gen_kv(w)
    rep = compare_full(w, K, V, synthkv.protect_mask(w))
    _assert_exact(rep, w.name)


def test_tiny_workload():
    w = synthkv.WORKLOADS["tiny"]
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), "tiny")


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
# (16, 17, 48, 63 and 65 end at or just past the 16-token wavefront tiles and
# 64-token workgroup tiles of the dequantize kernels)
@pytest.mark.parametrize("img_len", [1, 5, 16, 17, 31, 32, 33, 48, 63, 65, 127, 128, 129, 257])
def test_ragged_spans(base, img_len):
    w = small(base, img_len=img_len, img_start=3, text=2, L=1, B=2, H=2, n_protected=1)
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
@pytest.mark.parametrize("img_len", [1, 7, 8, 9, 31, 33, 41])
def test_ragged_spans_head_dim_256(base, img_len):
    """Head_dim 256 loads whole rows into an LDS stage 8 tokens (one pass) at
    a time; spans ending inside a pass or a 32-token tile."""
    w = small(base, D=256, img_len=img_len, img_start=3, text=2, L=1, B=2, H=2, n_protected=1)
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
@pytest.mark.parametrize("which", ["none", "all"])
@pytest.mark.parametrize("keys_only", [0, 1])
def test_degenerate_masks(base, which, keys_only):
    w = small(base, keys_only=keys_only, img_len=100)
    K, V = synthkv.gen_kv(w)
    mask = np.full(w.L * w.H, 1 if which == "all" else 0, np.uint8)
    rep = compare_full(w, K, V, mask)
    _assert_exact(rep, f"{base}-{which}")


@pytest.mark.parametrize("base,keys_only,retain,kivi_group",
                         [("minmax", 0, 0, 32), ("kivi", 1, 0, 32), ("kivi", 0, 0, 0), ("akvq", 0, 100, 32)])
def test_maximum_head_count(base, keys_only, retain, kivi_group):
    """L*H at the routing limit (8192 heads): the mask bitmap and its prefix
    counts span every word; protected heads sit in the first and last words.
    With whole-sequence KIVI keys the resident kernel finds each work item's
    head by its rank among the quantized heads across all 256 words."""
    import paper_2609_35800_amd as hg
    w = synthkv.Workload(f"maxheads-{base}-{kivi_group}", L=128, B=1, H=64, T=40, D=64, img_start=3,
                         img_len=33, bits=3, base=base, keys_only=keys_only, n_protected=0,
                         k_outliers=2, k_outlier_scale=10.0, kivi_group=kivi_group, retain_permille=retain)
    assert w.L * w.H == hg.HG_MAX_HEADS
    rng = np.random.default_rng(8192)
    mask = (rng.random(w.L * w.H) < 0.125).astype(np.uint8)
    mask[[0, 31, 32, 8191]] = 1
    mask[8190] = 0
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, mask), w.name)


@pytest.mark.parametrize("base,kivi_group,retain", [("minmax", 32, 0), ("kivi", 32, 0), ("kivi", 0, 0),
                                                     ("akvq", 32, 20)])
def test_long_span(base, kivi_group, retain):
    """A 70001-token image span (547 workgroup tiles per slice, ragged tail;
    the retention selection reads its norms from global memory)."""
    w = synthkv.Workload(f"long-{base}-{kivi_group}-{retain}", L=1, B=1, H=2, T=70011, D=64, img_start=6,
                         img_len=70001, bits=2, base=base, keys_only=0, n_protected=0, k_outliers=2,
                         k_outlier_scale=10.0, kivi_group=kivi_group, retain_permille=retain)
    K, V = synthkv.gen_kv(w)
    mask = np.array([0, 1], np.uint8)
    _assert_exact(compare_full(w, K, V, mask), w.name)


def _special_values(w, K, V):
    """Plant constant tokens, signed zeros, tiny ranges, ties and large values."""
    s = w.img_start
    bf = torch.bfloat16
    for X in (K, V):
        X[0, 0, 0, s + 0] = 1.5                                  # constant token
        X[0, 0, 0, s + 1] = 0.0                                  # all +0
        X[0, 0, 0, s + 2] = -0.0                                 # all -0
        X[0, 0, 0, s + 3, ::2] = -0.0                            # mixed zeros
        X[0, 0, 0, s + 4] = torch.linspace(1e-38, 3e-38, w.D).to(bf)   # tiny range
        X[0, 0, 0, s + 5] = torch.linspace(-2e-39, 2e-39, w.D).to(bf)  # subnormal span
        X[0, 0, 0, s + 6] = (torch.arange(w.D) % 8).to(bf) * 0.5      # exact ties
        X[0, 0, 0, s + 7] = torch.linspace(-7e28, 5e28, w.D).to(bf)    # large (< 2^96)
        X[0, 0, 0, s + 8] = 0.0
        X[0, 0, 0, s + 8, 5] = 1e-40                             # one denormal
        # the same token in a KIVI group: per-channel constants
        X[0, 1, 1, s + 32:s + 64] = X[0, 1, 1, s + 32:s + 33]
    return K, V


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_special_values(base, bits):
    w = small(base, bits=bits, img_len=96, n_protected=0)
    K, V = synthkv.gen_kv(w)
    K, V = _special_values(w, K, V)
    rep = compare_full(w, K, V, np.zeros(w.L * w.H, np.uint8))
    _assert_exact(rep, f"special-{base}-{bits}")


def test_empty_span_is_a_noop():
    import paper_2609_35800_amd as hg
    w = small("minmax", img_len=0, img_start=4, text=8)
    K, V = synthkv.gen_kv(w)
    rep = compare_full(w, K, V, synthkv.protect_mask(w))
    _assert_exact(rep, "empty")
    cfg = hg.make_config(**w.config_fields())
    assert all(v == 0 for k, v in hg.hg_packed_sizes(cfg, synthkv.protect_mask(w)).items()
               if k in hg.BUFFERS)


def test_side_stream_and_determinism():
    """Same bytes on a non-default stream and on a second run."""
    from hgtest import gpu_run
    w = small("akvq", img_len=200)
    K, V = synthkv.gen_kv(w)
    mask = synthkv.protect_mask(w)
    s = torch.cuda.Stream()
    a = gpu_run(w, K, V, mask, stream=s)
    b = gpu_run(w, K, V, mask)
    for n in a[0]:
        assert np.array_equal(a[0][n], b[0][n])
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[2], b[2])


def test_pointer_errors_are_caught_before_launch():
    """Host memory and misaligned device pointers are rejected with a status;
    no kernel runs and the outputs keep their canaries."""
    import paper_2609_35800_amd as hg
    from hgtest import alloc_with_canary, canaries_intact
    w = small("minmax", img_len=64)
    K, V = synthkv.gen_kv(w)
    mask = synthkv.protect_mask(w)
    cfg = hg.make_config(**w.config_fields())
    packed, raw = alloc_with_canary(hg.hg_packed_sizes(cfg, mask))
    Kg, Vg = K.cuda(), V.cuda()
    with pytest.raises(hg.HeadGuardError) as e:
        hg.hg_quantize(cfg, K, Vg, mask, packed)  # K in host memory
    assert e.value.status == hg.HG_ERR_POINTER
    flat = torch.empty(Kg.numel() + 8, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(hg.HeadGuardError) as e:
        hg.hg_quantize(cfg, flat[1:].data_ptr(), Vg, mask, packed)  # 2-byte offset
    assert e.value.status == hg.HG_ERR_ALIGN
    torch.cuda.synchronize()
    assert canaries_intact(raw)
    assert all(bool((packed[n] == 0xA5).all()) for n in packed if packed[n].numel())
