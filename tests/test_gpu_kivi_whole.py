"""GPU parity of KIVI-style keys with one range per channel over the whole
supplied sequence, text included (kivi_group = 0; §4 Quantization setup),
against the oracle: codes, metadata, side store and reconstruction
bit-exact for quantize / dequantize and for the one-pass simulated
quantization; every slice of the full LLaVA-NeXT-7B-shaped cache.

Slices of up to 32 workgroups' capacity (24 slots of 8192/D rows: 3072,
1536 and 768 rows at head_dim 64, 128 and 256) go through the partitioned
resident kernel: P workgroups each hold a run of a slice's rows on chip and
combine their partial ranges through the call's workspace (past 8, P is
rounded up to 16 or 32); longer slices go through the split kernels (a
range launch over chunks of every slice merging per-channel ranges into the
workspace, then a code launch), and a slice one workgroup holds, on a device
too small for a group, through the two-pass kernel (no workspace).
Covered: one to eight, 16 and 32 workgroups per slice and the capacity
boundaries, several slices per group (with the grid shrunk through the
HG_TEST_CUS hook), identical bytes for different grid sizes, and no exchange
wait running out of polls."""
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


def test_long_single_slice():
    """One key slice of 2^21 + 5 tokens at head_dim 128 (512 MiB, text rows at
    both ends): far past 32 workgroups' capacity, so the split kernels range
    and code it in 1025 and 1024 chunks; every byte against the oracle."""
    T = (1 << 21) + 5
    w = synthkv.Workload("kiviseq-long-slice", L=1, B=1, H=1, T=T, D=128, img_start=1000, img_len=T - 1777,
                         bits=2, base="kivi", keys_only=0, n_protected=0, k_outliers=4, k_outlier_scale=10.0,
                         kivi_group=0, seed=21)
    assert T > 8 * capacity(128)
    wholecache.assert_whole(wholecache.quantize_dequantize(w), w)


@pytest.mark.parametrize("fake", [False, True])
def test_two_pass_without_workspace(fake, monkeypatch):
    """Slices one workgroup holds need no workspace; on a device with fewer
    than 8 compute units (the grid hook) there is no group of 8 to run them, so
    the two-pass kernel takes them."""
    monkeypatch.setenv("HG_TEST_CUS", "4")
    w = small("kivi", 128, 3, 0, img_len=1000, img_start=9, text=20, L=2, B=3, H=2,
              n_protected=1).with_(kivi_group=0, name="kiviseq-two-pass")
    assert w.T <= capacity(128)
    K, V = synthkv.gen_kv(w)
    mask = synthkv.protect_mask(w)
    if fake:
        check_fake(w, K, V, mask, False)
    else:
        _assert_exact(compare_full(w, K, V, mask), w.name)


def test_split_batches(monkeypatch):
    """More quantized key slices than the workspace holds range words for
    (2048), through the split kernels (forced by the grid hook: 4 compute
    units cannot hold a group of 8): the slices are taken in two batches, the
    second batch's words cleared by a kernel of their own."""
    monkeypatch.setenv("HG_TEST_CUS", "4")
    w = small("kivi", 64, 2, 1, img_len=50, img_start=3000, text=23, L=8, B=3, H=128,
              n_protected=24).with_(kivi_group=0, name="kiviseq-split-batches")
    assert w.T > capacity(64) and (w.L * w.H - w.n_protected) * w.B > 2048
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


def capacity(D):
    """Rows one workgroup of the partitioned kernel holds."""
    return 24 * 8192 // D


# Enough (head, row) items that every group takes several slices once the
# grid is shrunk to 32 compute units' worth (32 workgroups: 32, 16 and 8
# groups of 1, 2 and 4 workgroups), so each slot's refill with the next
# slice and the alternation of the exchange buffers are exercised.
STREAM_CASES = [small("kivi", D, bits, ko, img_len=T - 50, img_start=20, text=30, L=2, B=6, H=8,
                      n_protected=2).with_(kivi_group=0, name=f"kiviseq-streams-D{D}-T{T}-b{bits}-ko{ko}")
                for D in (64, 128, 256) for T in (200, capacity(D) + 300, 3 * capacity(D) + 7)
                for bits in (2, 3) for ko in (0, 1)]


@pytest.mark.parametrize("w", STREAM_CASES, ids=lambda w: w.name)
def test_resident_streams(w, monkeypatch):
    monkeypatch.setenv("HG_TEST_CUS", "32")
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), w.name)


@pytest.mark.parametrize("w", STREAM_CASES[2:4] + STREAM_CASES[8:10], ids=lambda w: w.name)
@pytest.mark.parametrize("inplace", [False, True])
def test_resident_streams_fake(w, inplace, monkeypatch):
    monkeypatch.setenv("HG_TEST_CUS", "32")
    K, V = synthkv.gen_kv(w)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace)


@pytest.mark.parametrize("cus", ["", "256", "64", "24", "16", "8", "1"])
def test_grid_size_does_not_change_the_bytes(cus, monkeypatch):
    """The same cache (two workgroups per slice) under persistent grids sized
    for 256 down to 1 compute units (fewer than 16 are too few workgroups for
    a multiple of 8 groups: the split kernels take over), and once more with
    the full grid: every run equals the oracle."""
    w = small("kivi", 128, 2, 0, img_len=3000, img_start=5, text=3, L=2, B=6, H=5,
              n_protected=2).with_(kivi_group=0)
    monkeypatch.setenv("HG_TEST_CUS", cus)
    K, V = synthkv.gen_kv(w)
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), f"cus{cus or 'all'}")


# Slices at each workgroup count's capacity and one row past it (one to eight
# workgroups per slice, then 16 and 32; past 32 workgroups' capacity, the
# split kernels), spans at the start, in the middle and at the end of the
# slice (the middle only for the longest slices).
def _boundary_cases():
    out = []
    for D in (64, 128, 256):
        c = capacity(D)
        for T in (c, c + 1, 2 * c + 1, 3 * c - 5, 8 * c, 8 * c + 1):
            for img_start, img_len in ((0, T), (T // 3, T // 2), (T - 40, 40)):
                out.append((D, T, img_len, img_start))
        for T in (16 * c, 16 * c + 1, 32 * c, 32 * c + 1):
            out.append((D, T, T // 2, T // 3))
    return out


@pytest.mark.parametrize("D,T,img_len,img_start", _boundary_cases(), ids=lambda v: str(v))
def test_capacity_boundary(D, T, img_len, img_start):
    w = small("kivi", D, 3, 0, img_len=img_len, img_start=img_start, text=T - img_len - img_start,
              L=1, B=2, H=2, n_protected=1).with_(kivi_group=0)
    assert w.T == T
    K, V = synthkv.gen_kv(w)
    K[0, :, :, T - 1, 5] = -4000.0  # an extreme in the last row of every slice
    K[0, :, :, 0, 9] = 5000.0       # and in the first
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w)), f"D{D}-T{T}-n{img_len}-s{img_start}")


@pytest.mark.parametrize("T", [1536, 1537, 3008, 12288, 12289, 24577, 49152, 49153])
@pytest.mark.parametrize("inplace", [False, True])
def test_capacity_boundary_fake(T, inplace):
    w = small("kivi", 128, 2, 1, img_len=T - 60, img_start=20, text=40,
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


def _stale_words(ws):
    """Every 64-bit word of an exchange workspace set to what a partner would
    fold in if the words were not cleared before the key kernel: a small
    sequence tag (1 to 8, the first slices' tags) above the BF16 bits of the
    range [-1000, 1000]."""
    n = ws.numel() // 8
    tags = (np.arange(n, dtype=np.uint64) % np.uint64(8)) + np.uint64(1)
    words = (tags << np.uint64(32)) | (np.uint64(0x447A) << np.uint64(16)) | np.uint64(0xC47A)
    ws[: n * 8].copy_(torch.from_numpy(words.view(np.uint8)).to(ws.device))


# Two workgroups per slice (head_dim 128), 2-bit, keys and values quantized.
STALE_CASE = next(w for w in STREAM_CASES
                  if w.D == 128 and w.T == capacity(128) + 300 and w.bits == 2 and not w.keys_only)


# Resident kernel with several slices per group (32 and 256 compute units'
# grids) and the split kernels (8), every call on a workspace holding
# stale tagged words: the call must clear them before the key kernel reads.
@pytest.mark.parametrize("cus", ["32", "", "8"])
def test_stale_exchange_words(cus, monkeypatch):
    monkeypatch.setenv("HG_TEST_CUS", cus)
    w = STALE_CASE
    K, V = synthkv.gen_kv(w)
    prefill = lambda pk: _stale_words(pk["workspace"])  # noqa: E731
    _assert_exact(compare_full(w, K, V, synthkv.protect_mask(w), prefill=prefill), f"stale-cus{cus or 'all'}")


@pytest.mark.parametrize("inplace", [False, True])
def test_stale_exchange_words_fake(inplace, monkeypatch):
    monkeypatch.setenv("HG_TEST_CUS", "32")
    w = STALE_CASE
    K, V = synthkv.gen_kv(w)
    check_fake(w, K, V, synthkv.protect_mask(w), inplace, prefill_ws=_stale_words)
