"""GPU parity at the full sizes of the five workloads, in the launch
configuration the bench times: the whole cache is quantized and dequantized
on the GPU, then a seeded sample of (tensor, layer, batch row, head) slices is
recomputed by the CPU oracle slice by slice (codes, metadata and
reconstruction bit-exact), and properties that hold at any size are checked
over everything on the device: protected rows bit-identical in the side store
and after dequantization, text rows untouched, canaries intact, every scale a
non-negative BF16 and the per-group error within half a step."""
import numpy as np
import pytest
import torch

import oracle
import synthkv
from hgtest import alloc_with_canary, canaries_intact, bf16_ulp_diff

pytestmark = pytest.mark.gpu

SENTINEL = 0x7FBF
N_SAMPLES = 12  # sampled slices per tensor


def _run_full(w, mask):
    import paper_2609_35800_amd as hg
    K, V = synthkv.gen_kv(w, device="cuda")
    cfg = hg.make_config(**w.config_fields())
    sizes = hg.hg_packed_sizes(cfg, mask)
    packed, raw = alloc_with_canary(sizes)
    Ko = torch.full(K.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    Vo = torch.full(V.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    hg.hg_quantize(cfg, K, V, mask, packed)
    hg.hg_dequantize(cfg, mask, packed, Ko, Vo)
    torch.cuda.synchronize()
    return K, V, Ko, Vo, packed, raw, sizes


def _slot_views(w, packed, X):
    name = "kv"[X]
    row = w.D * w.bits // 8
    codes = packed["codes_" + name].view(-1, w.B, w.img_len, row)
    meta = packed["meta_" + name].view(torch.int32)
    if w.base == "kivi" and X == 0:
        meta = meta.view(-1, w.B, -(-w.img_len // w.kivi_group), w.D)
    else:
        meta = meta.view(-1, w.B, w.img_len)
    side = packed["side_" + name].view(torch.int16)
    side = side.view(-1, w.B, w.img_len, w.D) if side.numel() else None
    return codes, meta, side


def _check_workload(w):
    mask = synthkv.protect_mask(w)
    K, V, Ko, Vo, packed, raw, sizes = _run_full(w, mask)
    ocfg = oracle.make_config(**w.config_fields())
    s0, n = w.img_start, w.img_len
    assert canaries_intact(raw)
    rng = np.random.default_rng([w.seed, 99])
    mask2 = mask.reshape(w.L, w.H).astype(bool)
    for X, (src, rec) in enumerate(((K, Ko), (V, Vo))):
        codes, meta, side = _slot_views(w, packed, X)
        src_i = src.view(torch.int16)
        rec_i = rec.view(torch.int16)
        # text rows untouched, everywhere
        assert bool((rec_i[:, :, :, :s0] == SENTINEL).all())
        assert bool((rec_i[:, :, :, s0 + n:] == SENTINEL).all())
        # kept heads: side store and reconstruction bit-identical, everywhere
        kept = mask2 & (X == 0 or not w.keys_only)
        p = 0
        for l in range(w.L):
            for h in range(w.H):
                if kept[l, h]:
                    img = src_i[l, :, h, s0:s0 + n]
                    assert torch.equal(side[p], img), (X, l, h)
                    assert torch.equal(rec_i[l, :, h, s0:s0 + n], img), (X, l, h)
                    p += 1
        # scales are non-negative BF16 values; KIVI / min-max error bound on device
        m32 = meta.reshape(-1)
        assert bool(((m32 & 0x8000) == 0).all()), "negative scale"
        # sampled slices against the oracle, slice by slice
        picks = [(int(rng.integers(w.L)), int(rng.integers(w.B)), int(rng.integers(w.H)))
                 for _ in range(N_SAMPLES)]
        for l, b, h in picks:
            prot, slot = oracle.route(ocfg, mask, X, l, h)
            rows = synthkv.bf16_bits(src[l, b, h, s0:s0 + n])
            if prot:
                assert np.array_equal(side[slot, b].cpu().numpy().view(np.uint16), rows)
                continue
            oc, om = oracle.quantize_slice(ocfg, X, rows)
            gc = codes[slot, b].cpu().numpy()
            gm = meta[slot, b].cpu().numpy().view(np.uint32)
            assert np.array_equal(gc, oc), (X, l, b, h, int(np.count_nonzero(gc != oc)))
            assert np.array_equal(gm, om), (X, l, b, h)
            orec = oracle.dequantize_slice(ocfg, X, oc, om)
            grec = synthkv.bf16_bits(rec[l, b, h, s0:s0 + n])
            assert bf16_ulp_diff(grec, orec) <= 1
            assert np.array_equal(grec, orec), (X, l, b, h)


@pytest.mark.parametrize("name", ["tiny", "qwen2.5-vl-7b", "llava-next-7b", "internvl-8b", "gemma-3-12b",
                                  "llava-1.5-7b", "72b-long-tp8"])
def test_workload(name):
    _check_workload(synthkv.WORKLOADS[name])
    torch.cuda.empty_cache()


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_72b_long_bit_sweep(bits):
    _check_workload(synthkv.WORKLOADS["72b-long"].with_(bits=bits))
    torch.cuda.empty_cache()
