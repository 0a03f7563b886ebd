"""GPU parity of the AKVQ-style token retention (§4 Quantization setup: per KV
head the keys and values of a nominal 2 % of the image tokens with the
largest key norms stay in BF16, with or without head protection) against the
CPU oracle on the same seeded BF16 bytes.

Every output is compared element by element: the squared key norms (fp32 bit
patterns), the retained token lists, the retained rows, the packed codes and
metadata, and the reconstruction with the retained rows written back.  Small
shapes span several 256-token selection chunks with ragged tails; inputs with
many equal norms exercise the tie rule; the one-pass simulated quantization is
checked in place and out of place; every slice of the full InternVL3-8B-shaped
cache at the paper's 2 % is checked, for quantize then dequantize and for the
one-pass form."""
import numpy as np
import pytest
import torch

import synthkv
import wholecache
from hgtest import compare_full
from test_gpu_fakequant import check as check_fake
from test_gpu_parity import _assert_exact, _special_values, small

pytestmark = pytest.mark.gpu


def retain_case(D=128, bits=2, keys_only=0, permille=20, img_len=600, **kw):
    w = small("akvq", D=D, bits=bits, keys_only=keys_only, img_len=img_len, **kw)
    return w.with_(retain_permille=permille, name=w.name + f"-r{permille}")


CASES = [retain_case(D, bits, ko, pm) for D in (64, 128, 256) for bits in (2, 3, 4) for ko in (0, 1)
         for pm in (20, 100)]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_small_parity(w):
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("img_len", [1, 24, 25, 49, 75, 255, 256, 257, 513])
@pytest.mark.parametrize("permille", [20, 333, 1000])
def test_ragged_spans_and_fractions(img_len, permille):
    w = retain_case(img_len=img_len, img_start=3, text=2, L=1, B=2, H=2, n_protected=1,
                    permille=permille)
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("img_len", [12288, 12289, 13000])
def test_long_spans(img_len):
    """Spans at and past the length whose norms the selection stages in LDS;
    longer ones are selected from global memory."""
    w = retain_case(img_len=img_len, img_start=5, text=3, L=1, B=1, H=2, n_protected=0,
                    permille=20)
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, np.zeros(w.L * w.H, np.uint8)), w.name)


def _integer_kv(w, lo, hi, seed):
    g = torch.Generator().manual_seed(seed)
    shape = (w.L, w.B, w.H, w.T, w.D)
    K = torch.randint(lo, hi, shape, generator=g).to(torch.bfloat16)
    V = torch.randint(lo, hi, shape, generator=g).to(torch.bfloat16)
    return K, V


@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("spread", [1, 3])
def test_ties_go_to_the_lower_token(D, spread):
    """Entries in {-spread..spread}: key norms are small integers, so most
    tokens tie with others and the selection boundary falls inside a tie."""
    w = retain_case(D=D, img_len=700, permille=50, n_protected=1)
    K, V = _integer_kv(w, -spread, spread + 1, 17 + D + spread)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), f"ties-{D}-{spread}")


def test_identical_keys():
    """Every key equal: all norms tie and the first k tokens are kept."""
    w = retain_case(img_len=300, permille=100, n_protected=0)
    K, V = synthkv.gen_kv(w)
    K[:] = K[:, :, :, :1].clone()
    rep = compare_full(w, K, V, np.zeros(w.L * w.H, np.uint8))
    _assert_exact(rep, "identical")


def test_identical_keys_many_workgroups_per_cu():
    """All norms equal in every one of 2048 heads (several selection
    workgroups per compute unit): no selection pass runs, and the scan's
    shared totals must not overwrite the key bounds before every wavefront
    has read them."""
    w = retain_case(img_len=200, permille=100, n_protected=0, L=8, B=16, H=16, text=5, img_start=3)
    K, V = synthkv.gen_kv(w)
    K[:] = K[:, :, :, :1].clone()
    _assert_exact(compare_full(w, K, V, np.zeros(w.L * w.H, np.uint8)), "identical-many")


def test_special_values():
    """Large keys square to +inf (ties among infinities), subnormal and zero
    squares, signed zeros."""
    w = retain_case(img_len=96, permille=100, n_protected=0)
    K, V = synthkv.gen_kv(w)
    K, V = _special_values(w, K, V)
    s = w.img_start
    K[0, 0, 0, s + 9, 3] = 2.0 ** 70     # squares past fp32: +inf norm
    K[0, 0, 0, s + 10, 7] = -2.0 ** 80   # another +inf, later token
    K[0, 0, 1, s + 11] = 2.0 ** -72      # subnormal squares
    _assert_exact(compare_full(w, K, V, np.zeros(w.L * w.H, np.uint8)), "special")


@pytest.mark.parametrize("which", ["none", "all"])
@pytest.mark.parametrize("keys_only", [0, 1])
def test_degenerate_masks(which, keys_only):
    w = retain_case(img_len=300, keys_only=keys_only, permille=50)
    K, V = synthkv.gen_kv(w)
    mask = np.full(w.L * w.H, 1 if which == "all" else 0, np.uint8)
    _assert_exact(compare_full(w, K, V, mask), f"mask-{which}-{keys_only}")


def test_empty_span():
    w = retain_case(img_len=0, img_start=4, text=8)
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), "empty")


# ---------------------------------------------------------------- one pass

FAKE_CASES = [retain_case(D, bits, ko, pm, img_len=400) for D in (64, 128, 256) for bits in (2, 4)
              for ko in (0, 1) for pm in (20, 250)]


@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("w", FAKE_CASES, ids=lambda w: w.name)
def test_fake_quantize(w, inplace):
    K, V = synthkv.gen_kv(w)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace)


@pytest.mark.parametrize("k_in_place", [True, False])
def test_fake_quantize_one_tensor_in_place(k_in_place):
    """One output is its input and the other is not: the retained rows of
    the in-place tensor must be saved before they are overwritten."""
    import paper_2609_35800_amd as hg
    from test_gpu_fakequant import SENTINEL, oracle_roundtrip
    w = retain_case(img_len=300, permille=50)
    K, V = synthkv.gen_kv(w)
    mask = synthkv.protect_mask(w)
    cfg = hg.make_config(**w.config_fields())
    Kg, Vg = K.cuda().contiguous(), V.cuda().contiguous()
    fresh = lambda t: torch.full(t.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    Ko = Kg if k_in_place else fresh(Kg)
    Vo = fresh(Vg) if k_in_place else Vg
    hg.hg_fake_quantize(cfg, Kg, Vg, mask, Ko, Vo, hg.alloc_fake_workspace(cfg, mask))
    torch.cuda.synchronize()
    Kb, Vb = synthkv.bf16_bits(K), synthkv.bf16_bits(V)
    oK, oV = oracle_roundtrip(w, Kb, Vb, mask, Kb if k_in_place else np.full_like(Kb, SENTINEL),
                              np.full_like(Vb, SENTINEL) if k_in_place else Vb)
    assert np.array_equal(synthkv.bf16_bits(Ko), oK)
    assert np.array_equal(synthkv.bf16_bits(Vo), oV)


def test_fake_quantize_ties_in_place():
    w = retain_case(img_len=500, permille=60)
    K, V = _integer_kv(w, -2, 3, 5)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace=True)


# ---------------------------------------------------------------- full size

def test_full_size_internvl_two_percent():
    """The InternVL3-8B-shaped cache at the paper's 2 %: every slice's norms,
    token list, retained rows, codes, metadata and reconstruction against the
    oracle."""
    w = synthkv.WORKLOADS["internvl-8b"].with_(retain_permille=20)
    import paper_2609_35800_amd as hg
    sizes = hg.hg_packed_sizes(hg.make_config(**w.config_fields()), synthkv.protect_mask(w))
    assert sizes["retain_count"] == 67  # round(0.02 * 3328)
    wholecache.assert_whole(wholecache.quantize_dequantize(w), w)


@pytest.mark.parametrize("inplace", [False, True])
def test_full_size_internvl_two_percent_one_pass(inplace):
    w = synthkv.WORKLOADS["internvl-8b"].with_(retain_permille=20)
    wholecache.assert_whole(wholecache.fake_quantize(w, inplace=inplace), w)
