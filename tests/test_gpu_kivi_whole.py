"""GPU parity of KIVI-style keys with one range per channel over the whole
supplied sequence, text included (kivi_group = 0; §4 Quantization setup),
against the oracle: codes, metadata, side store and reconstruction
bit-exact for quantize / dequantize and for the one-pass simulated
quantization; every slice of the full LLaVA-NeXT-7B-shaped cache.

Slices of up to 3072 rows go through the resident kernel (each workgroup
holds a 64-channel part of a slice on chip and refills its row slots with
its next slice while coding); longer slices through the two-pass kernel.
Both are covered, including several slices per workgroup stream and the
boundary at 3072 / 3073 rows."""
import numpy as np
import pytest
import torch

import synthkv
import wholecache
from hgtest import compare_full
from test_gpu_fakequant import check as check_fake
from test_gpu_parity import _assert_exact, small

pytestmark = pytest.mark.gpu

CASES = [small("kivi", D, bits, ko).with_(kivi_group=0, name=f"kiviseq-D{D}-b{bits}-ko{ko}")
         for D in (64, 128, 256) for bits in (2, 3, 4) for ko in (0, 1)]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_small(w):
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("w", CASES[:6], ids=lambda w: w.name)
@pytest.mark.parametrize("inplace", [False, True])
def test_fake(w, inplace):
    K, V = synthkv.gen_kv(w)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace)


@pytest.mark.parametrize("img_len,img_start,text", [(1, 0, 0), (5, 3, 40), (130, 0, 7), (64, 64, 0)])
def test_spans(img_len, img_start, text):
    w = small("kivi", img_len=img_len, img_start=img_start, text=text, L=1, B=2, H=2,
              n_protected=1).with_(kivi_group=0)
    K, V = synthkv.gen_kv(w)
    K[0, 0, 0, 0, 3] = 3000.0  # a large value in the first row (text when img_start > 0)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), f"span{img_len}")


def test_full_size_llava():
    """The LLaVA-NeXT-7B-shaped cache with one key range per channel over the
    whole sequence: every slice against the oracle."""
    w = synthkv.WORKLOADS["llava-next-7b"].with_(kivi_group=0)
    wholecache.assert_whole(wholecache.quantize_dequantize(w), w)


@pytest.mark.parametrize("inplace", [False, True])
def test_full_size_llava_one_pass(inplace):
    w = synthkv.WORKLOADS["llava-next-7b"].with_(kivi_group=0)
    wholecache.assert_whole(wholecache.fake_quantize(w, inplace=inplace), w)


# Enough (head, row) items that every workgroup stream of the resident kernel
# takes several slices (streams: 256 / 128 / 64 at head_dim 64 / 128 / 256),
# so each slot's refill with the next slice is exercised.
STREAM_CASES = [small("kivi", D, bits, ko, img_len=150, img_start=20, text=30, L=2, B=20, H=8,
                      n_protected=2).with_(kivi_group=0, name=f"kiviseq-streams-D{D}-b{bits}-ko{ko}")
                for D in (64, 128, 256) for bits in (2, 3) for ko in (0, 1)]


@pytest.mark.parametrize("w", STREAM_CASES, ids=lambda w: w.name)
def test_resident_streams(w):
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("w", STREAM_CASES[2:4], ids=lambda w: w.name)
@pytest.mark.parametrize("inplace", [False, True])
def test_resident_streams_fake(w, inplace):
    K, V = synthkv.gen_kv(w)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace)


# Slices at the resident capacity (3072 rows: every row slot filled), one row
# past it (the two-pass kernel), and longer; image spans at the start, in the
# middle and at the end of the slice.
BOUNDARY = [(3072, 3000, 40), (3073, 3000, 40), (3072, 3072, 0), (3072, 100, 2972),
            (3200, 3100, 0), (4000, 1000, 1500)]


@pytest.mark.parametrize("D", [128, 256])
@pytest.mark.parametrize("T,img_len,img_start", BOUNDARY, ids=lambda v: str(v))
def test_capacity_boundary(D, T, img_len, img_start):
    w = small("kivi", D, 3, 0, img_len=img_len, img_start=img_start, text=T - img_len - img_start,
              L=1, B=2, H=2, n_protected=1).with_(kivi_group=0)
    assert w.T == T
    K, V = synthkv.gen_kv(w)
    K[0, :, :, T - 1, 5] = -4000.0  # an extreme in the last row of every slice
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), f"T{T}-n{img_len}-s{img_start}")


@pytest.mark.parametrize("T,img_len,img_start", BOUNDARY[:2], ids=lambda v: str(v))
@pytest.mark.parametrize("inplace", [False, True])
def test_capacity_boundary_fake(T, img_len, img_start, inplace):
    w = small("kivi", 128, 2, 1, img_len=img_len, img_start=img_start, text=T - img_len - img_start,
              L=1, B=2, H=2, n_protected=1).with_(kivi_group=0)
    K, V = synthkv.gen_kv(w)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace)


@pytest.mark.parametrize("which", ["none", "all", "last"])
@pytest.mark.parametrize("keys_only", [0, 1])
def test_degenerate_masks(which, keys_only):
    """No key head protected, every one (no work item for the key kernel),
    and only the last head quantized (the rank search lands in the last word)."""
    w = small("kivi", 128, 2, keys_only, img_len=90, img_start=5, text=9, L=3, B=2, H=12,
              n_protected=0).with_(kivi_group=0)
    K, V = synthkv.gen_kv(w)
    mask = np.full(w.L * w.H, 1 if which != "none" else 0, np.uint8)
    if which == "last":
        mask[-1] = 0
    _assert_exact(compare_full(w, K, V, mask), f"mask-{which}-ko{keys_only}")
