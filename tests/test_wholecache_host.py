"""The whole-cache comparison used by the full-size GPU tests, checked on the
CPU with the oracle standing in for the GPU: the per-layer byte ranges of a
whole-cache oracle run equal one-layer oracle runs for every buffer, every
slice is counted once, and a single planted byte difference fails exactly the
slices that own it."""
import numpy as np
import pytest

import oracle
import synthkv
import wholecache
from test_gpu_parity import small

CASES = [small("minmax", D=64, L=3, B=2, H=4, img_len=70, n_protected=3),
         small("kivi", D=64, keys_only=1, L=3, B=2, H=4, img_len=70, n_protected=3),
         small("kivi", D=64, L=3, B=2, H=4, img_len=70, n_protected=3).with_(kivi_group=0, name="kw"),
         small("akvq", D=64, L=3, B=2, H=4, img_len=70, n_protected=3).with_(retain_permille=100, name="ar")]


def _whole(w, mask):
    K, V = synthkv.gen_kv(w)
    Kb, Vb = synthkv.bf16_bits(K), synthkv.bf16_bits(V)
    cfg = oracle.make_config(**w.config_fields())
    pk = oracle.quantize(cfg, Kb, Vb, mask, threads=4)
    Ko, Vo = np.full_like(Kb, wholecache.SENTINEL), np.full_like(Vb, wholecache.SENTINEL)
    oracle.dequantize(cfg, mask, pk, Ko, Vo, threads=4)
    return Kb, Vb, {n: v.view(np.uint8).reshape(-1) for n, v in pk.items()}, Ko, Vo


def _run(w, mask, Kb, Vb, pk, Ko, Vo):
    ocfg, rows, lsizes, offs = wholecache.layer_layout(w, mask)
    rep = wholecache.Report(expected=2 * w.L * w.B * w.H)
    for l in range(w.L):
        opk = oracle.quantize(ocfg, Kb[l:l + 1], Vb[l:l + 1], rows[l], threads=2)
        oK, oV = np.full_like(Kb[l:l + 1], wholecache.SENTINEL), np.full_like(Vb[l:l + 1], wholecache.SENTINEL)
        oracle.dequantize(ocfg, rows[l], opk, oK, oV, threads=2)
        gpu = {n: pk[n][offs[l][n]:offs[l][n] + lsizes[l][n]] for n in pk}
        obytes = {n: v.view(np.uint8).reshape(-1) for n, v in opk.items()}
        wholecache.check_layer(w, ocfg, rows[l], gpu, obytes, (Ko[l], Vo[l]), (oK[0], oV[0]), rep, l,
                               packed=True)
        rep.layers += 1
    return rep


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_layer_ranges_equal_one_layer_runs(w):
    mask = synthkv.protect_mask(w)
    rep = _run(w, mask, *_whole(w, mask))
    assert rep.ok() and rep.slices == 2 * w.L * w.B * w.H, rep.failures


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
@pytest.mark.parametrize("buf", ["codes_k", "meta_v", "side_k", "rec_v", "ret_idx"])
def test_a_planted_difference_fails_one_slice(w, buf):
    mask = synthkv.protect_mask(w)
    Kb, Vb, pk, Ko, Vo = _whole(w, mask)
    if buf == "rec_v":
        Vo[1, 1, 2, w.img_start + 5, 3] ^= 1
    else:
        if pk[buf].size == 0:
            pytest.skip(f"{buf} is empty in this case")
        pk[buf][pk[buf].size // 2] ^= 0x10
    rep = _run(w, mask, Kb, Vb, pk, Ko, Vo)
    bad = 2 if buf == "ret_idx" else 1  # a head's token list belongs to its K and V slices
    assert rep.slices == 2 * w.L * w.B * w.H - bad and len(rep.failures) == bad, rep.failures
