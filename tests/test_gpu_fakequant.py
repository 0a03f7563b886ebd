"""GPU parity of the one-pass simulated quantization (hg_fake_quantize, §4
Quantization setup) against its definition, the oracle's dequantize of its
quantize: image rows bit-exact, protected rows bit-identical, text rows
untouched, in place and out of place, on small and ragged caches (the full
sizes are compared slice by slice in test_gpu_workloads.py)."""
import numpy as np
import pytest
import torch

import oracle
import synthkv
from hgtest import bf16_ulp_diff, exchange_timeouts
from test_gpu_parity import _special_values, small

pytestmark = pytest.mark.gpu
SENTINEL = 0x7FBF


def oracle_roundtrip(w, Kb, Vb, mask, init_K, init_V):
    cfg = oracle.make_config(**w.config_fields())
    packed = oracle.quantize(cfg, Kb, Vb, mask, threads=8)
    Ko, Vo = init_K.copy(), init_V.copy()
    oracle.dequantize(cfg, mask, packed, Ko, Vo, threads=8)
    return Ko, Vo


def run_fake(w, K, V, mask, inplace, prefill_ws=None):
    import paper_2609_35800_amd as hg
    cfg = hg.make_config(**w.config_fields())
    Kg, Vg = K.cuda().contiguous(), V.cuda().contiguous()
    ws = hg.alloc_fake_workspace(cfg, mask)
    if prefill_ws is not None and ws is not None:
        prefill_ws(ws)
    if inplace:
        hg.hg_fake_quantize(cfg, Kg, Vg, mask, Kg, Vg, ws)
        Ko, Vo = Kg, Vg
    else:
        Ko = torch.full(Kg.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        Vo = torch.full(Vg.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        hg.hg_fake_quantize(cfg, Kg, Vg, mask, Ko, Vo, ws)
    torch.cuda.synchronize()
    if w.base == "kivi" and w.kivi_group == 0:
        assert exchange_timeouts(ws) == 0, "exchange waits ran out of polls"
    return synthkv.bf16_bits(Ko), synthkv.bf16_bits(Vo)


def check(w, K, V, mask, inplace, prefill_ws=None):
    Kb, Vb = synthkv.bf16_bits(K), synthkv.bf16_bits(V)
    gK, gV = run_fake(w, K, V, mask, inplace, prefill_ws)
    initK = Kb if inplace else np.full_like(Kb, SENTINEL)
    initV = Vb if inplace else np.full_like(Vb, SENTINEL)
    oK, oV = oracle_roundtrip(w, Kb, Vb, mask, initK, initV)
    assert bf16_ulp_diff(gK, oK) <= 1 and bf16_ulp_diff(gV, oV) <= 1
    assert np.array_equal(gK, oK), (w.name, int(np.count_nonzero(gK != oK)))
    assert np.array_equal(gV, oV), (w.name, int(np.count_nonzero(gV != oV)))


CASES = [small(b, D, bits, ko) for b in ("minmax", "kivi", "akvq") for D in (64, 128, 256)
         for bits in (2, 3, 4) for ko in (0, 1)]


@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_small(w, inplace):
    K, V = synthkv.gen_kv(w)
    check(w, K, V, synthkv.protect_mask(w), inplace)


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
@pytest.mark.parametrize("img_len", [1, 16, 17, 31, 33, 63, 65, 129, 257])  # 16- and 64-token tiles too
def test_ragged(base, img_len):
    w = small(base, img_len=img_len, img_start=3, text=2, L=1, B=2, H=2, n_protected=1)
    K, V = synthkv.gen_kv(w)
    check(w, K, V, synthkv.protect_mask(w), inplace=False)


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
@pytest.mark.parametrize("img_len", [1, 7, 9, 33])
@pytest.mark.parametrize("inplace", [False, True])
def test_ragged_head_dim_256(base, img_len, inplace):
    """Head_dim 256: whole-row loads staged through LDS, spans ending inside a
    pass; in place, each wavefront's loads precede its stores."""
    w = small(base, D=256, img_len=img_len, img_start=3, text=2, L=1, B=2, H=2, n_protected=1)
    K, V = synthkv.gen_kv(w)
    check(w, K, V, synthkv.protect_mask(w), inplace=inplace)


@pytest.mark.parametrize("base", ["minmax", "kivi", "akvq"])
def test_special_values(base):
    w = small(base, bits=2, img_len=96, n_protected=0)
    K, V = synthkv.gen_kv(w)
    K, V = _special_values(w, K, V)
    check(w, K, V, np.zeros(w.L * w.H, np.uint8), inplace=True)
