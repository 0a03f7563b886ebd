"""Whole-cache parity at full size: every (tensor, layer, batch row, head)
slice of a cache the GPU quantized is compared with the CPU oracle, element
by element, streamed one layer at a time so host memory stays bounded.

The oracle runs layer l as a cache of one layer with that layer's row of the
mask.  Packed buffers are ordered by slot, slots rank heads in row-major
(layer, head) order, and the retention buffers are [L][B][H]-major, so the
GPU's outputs for layer l are one contiguous byte range of each buffer, at
the sum of the one-layer sizes of the layers before it (the test checks that
those sums add up to the whole cache's sizes).

A slice passes when everything it owns matches: its codes and metadata (or
its BF16 side-store rows, when its head keeps the tensor), its retained-token
list, norms and rows (token retention), and its reconstructed rows, text rows
included (they must still hold the sentinel the outputs were filled with, or
the input, in place).  Each check returns the number of passing slices, which
the tests require to be 2*L*B*H."""
from __future__ import annotations

import os
from dataclasses import dataclass, field
from typing import Dict, List

import numpy as np
import torch

import oracle
import synthkv
from hgtest import PAD, alloc_with_canary, canaries_intact, exchange_timeouts

SENTINEL = 0x7FBF
# oracle threads: the host's cores, at most 16
THREADS = max(1, min(os.cpu_count() or 1, 16))


@dataclass
class Report:
    slices: int = 0          # slices that passed
    expected: int = 0        # 2 * L * B * H
    layers: int = 0
    failures: List[str] = field(default_factory=list)
    canaries: bool = True

    def ok(self) -> bool:
        return not self.failures and self.slices == self.expected and self.canaries


def layer_layout(w: synthkv.Workload, mask: np.ndarray):
    """One-layer oracle config, and per layer its mask row, sizes and the byte
    offsets of its part of every packed buffer."""
    sub = w.with_(L=1)
    ocfg = oracle.make_config(**sub.config_fields())
    rows, sizes, offs = [], [], []
    run: Dict[str, int] = {}
    for l in range(w.L):
        m = np.ascontiguousarray(mask[l * w.H:(l + 1) * w.H])
        sz = oracle.sizes(ocfg, m)
        rows.append(m)
        sizes.append(sz)
        offs.append({n: run.get(n, 0) for n in sz})
        for n in sz:
            run[n] = run.get(n, 0) + sz[n]
    whole = oracle.sizes(oracle.make_config(**w.config_fields()), mask)
    for n in ("codes_k", "meta_k", "side_k", "codes_v", "meta_v", "side_v",
              "norm_k", "ret_idx", "ret_k", "ret_v"):
        assert run[n] == whole[n], (n, run[n], whole[n])
    return ocfg, rows, sizes, offs


def _by_item(a: np.ndarray, lead) -> np.ndarray:
    """[*lead, rest] view of a flat buffer."""
    n = int(np.prod(lead))
    return a.reshape(*lead, a.size // n if n else 0)


def _slices_equal(g: np.ndarray, o: np.ndarray, lead) -> np.ndarray:
    """Per-item equality over the leading dims of two flat buffers."""
    assert g.shape == o.shape and g.dtype == o.dtype, (g.shape, o.shape, g.dtype, o.dtype)
    return (_by_item(g, lead) == _by_item(o, lead)).all(axis=-1)


def check_layer(w, ocfg, m, gpu: Dict[str, np.ndarray], opk: Dict[str, np.ndarray],
                g_rec, o_rec, rep: Report, l: int, packed: bool) -> None:
    """Counts the passing slices of layer l.  gpu / opk: the layer's packed
    buffers as byte arrays (GPU / oracle); g_rec / o_rec: the layer's
    reconstructed K and V as uint16 [B, H, T, D]."""
    B, H = w.B, w.H
    retain = w.retain_permille > 0
    if retain and packed:
        eq_norm = _slices_equal(gpu["norm_k"], opk["norm_k"], (B, H))
        eq_idx = _slices_equal(gpu["ret_idx"], opk["ret_idx"], (B, H))
    for X in (0, 1):
        x = "kv"[X]
        eq_rec = _slices_equal(g_rec[X].reshape(-1), o_rec[X].reshape(-1), (B, H))
        kept = [bool(m[h]) and (X == 0 or not w.keys_only) for h in range(H)]
        n_p, n_u = sum(kept), H - sum(kept)
        if packed:
            eq_codes = _slices_equal(gpu["codes_" + x], opk["codes_" + x], (n_u, B))
            eq_meta = _slices_equal(gpu["meta_" + x], opk["meta_" + x], (n_u, B))
            eq_side = _slices_equal(gpu["side_" + x], opk["side_" + x], (n_p, B))
            if retain:
                eq_ret = _slices_equal(gpu["ret_" + x], opk["ret_" + x], (n_u, B))
        p = u = 0
        for h in range(H):
            for b in range(B):
                ok = bool(eq_rec[b, h])
                if packed:
                    if kept[h]:
                        ok &= bool(eq_side[p, b])
                    else:
                        ok &= bool(eq_codes[u, b] and eq_meta[u, b])
                        if retain:
                            ok &= bool(eq_ret[u, b])
                    if retain:
                        ok &= bool(eq_norm[b, h] and eq_idx[b, h])
                if ok:
                    rep.slices += 1
                elif len(rep.failures) < 8:
                    what = "side" if (packed and kept[h]) else "codes/meta/rec"
                    rep.failures.append(f"{'KV'[X]} l={l} b={b} h={h}: {what} differs")
            if kept[h]:
                p += 1
            else:
                u += 1


def _host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint8).reshape(-1)


def quantize_dequantize(w: synthkv.Workload, mask=None) -> Report:
    """hg_quantize then hg_dequantize of the whole cache on the GPU (outputs
    surrounded by canary bytes, reconstruction buffers pre-filled with a
    sentinel), then every slice against the oracle, layer by layer."""
    import paper_2609_35800_amd as hg
    mask = synthkv.protect_mask(w) if mask is None else mask
    ocfg, rows, lsizes, offs = layer_layout(w, mask)
    K, V = synthkv.gen_kv(w, device="cuda")
    cfg = hg.make_config(**w.config_fields())
    packed, raw = alloc_with_canary(hg.hg_packed_sizes(cfg, mask))
    Ko = torch.full(K.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    Vo = torch.full(V.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    hg.hg_quantize(cfg, K, V, mask, packed)
    hg.hg_dequantize(cfg, mask, packed, Ko, Vo)
    torch.cuda.synchronize()
    rep = Report(expected=2 * w.L * w.B * w.H)
    for l in range(w.L):
        Kb, Vb = synthkv.bf16_bits(K[l:l + 1]), synthkv.bf16_bits(V[l:l + 1])
        opk = oracle.quantize(ocfg, Kb, Vb, rows[l], threads=THREADS)
        oK, oV = np.full_like(Kb, SENTINEL), np.full_like(Vb, SENTINEL)
        oracle.dequantize(ocfg, rows[l], opk, oK, oV, threads=THREADS)
        gpu = {n: _host(packed[n][offs[l][n]:offs[l][n] + lsizes[l][n]]) for n in hg.BUFFERS}
        obytes = {n: v.view(np.uint8).reshape(-1) for n, v in opk.items()}
        g_rec = (synthkv.bf16_bits(Ko[l]), synthkv.bf16_bits(Vo[l]))
        check_layer(w, ocfg, rows[l], gpu, obytes, g_rec, (oK[0], oV[0]), rep, l, packed=True)
        rep.layers += 1
    rep.canaries = canaries_intact(raw)
    if exchange_timeouts(packed.get("workspace")):
        rep.failures.append("KIVI exchange waits ran out of polls")
    del K, V, Ko, Vo, packed, raw
    torch.cuda.empty_cache()
    return rep


def fake_quantize(w: synthkv.Workload, inplace: bool, mask=None) -> Report:
    """hg_fake_quantize of the whole cache on the GPU (out of place into
    sentinel-filled outputs, or in place), then every slice's reconstruction
    against the oracle's dequantize of its quantize, layer by layer (in place,
    each layer's input is regenerated from its seed)."""
    import paper_2609_35800_amd as hg
    mask = synthkv.protect_mask(w) if mask is None else mask
    ocfg, rows, _, _ = layer_layout(w, mask)
    K, V = synthkv.gen_kv(w, device="cuda")
    cfg = hg.make_config(**w.config_fields())
    ws = hg.alloc_fake_workspace(cfg, mask)
    if inplace:
        Ko, Vo = K, V
    else:
        Ko = torch.full(K.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        Vo = torch.full(V.shape, SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, ws)
    torch.cuda.synchronize()
    rep_timeouts = exchange_timeouts(ws) if (w.base == "kivi" and w.kivi_group == 0) else 0
    del ws
    chans = synthkv.outlier_channels(w)
    rep = Report(expected=2 * w.L * w.B * w.H)
    if rep_timeouts:
        rep.failures.append("KIVI exchange waits ran out of polls")
    for l in range(w.L):
        if inplace:
            Kb = synthkv.bf16_bits(synthkv.gen_layer(w, 0, l, "cuda", chans))[None]
            Vb = synthkv.bf16_bits(synthkv.gen_layer(w, 1, l, "cuda", chans))[None]
        else:
            Kb, Vb = synthkv.bf16_bits(K[l:l + 1]), synthkv.bf16_bits(V[l:l + 1])
        opk = oracle.quantize(ocfg, Kb, Vb, rows[l], threads=THREADS)
        oK = Kb.copy() if inplace else np.full_like(Kb, SENTINEL)
        oV = Vb.copy() if inplace else np.full_like(Vb, SENTINEL)
        oracle.dequantize(ocfg, rows[l], opk, oK, oV, threads=THREADS)
        g_rec = (synthkv.bf16_bits(Ko[l]), synthkv.bf16_bits(Vo[l]))
        check_layer(w, ocfg, rows[l], {}, {}, g_rec, (oK[0], oV[0]), rep, l, packed=False)
        rep.layers += 1
    del K, V, Ko, Vo
    torch.cuda.empty_cache()
    return rep


def assert_whole(rep: Report, w: synthkv.Workload) -> None:
    assert not rep.failures, (w.name, rep.failures)
    assert rep.canaries, (w.name, "canary bytes after an output buffer were overwritten")
    assert rep.layers == w.L
    assert rep.slices == rep.expected == 2 * w.L * w.B * w.H, (w.name, rep.slices, rep.expected)
    print(f"{w.name}: {rep.slices} of {rep.expected} slices bit-exact against the oracle", flush=True)


__all__ = ["quantize_dequantize", "fake_quantize", "assert_whole", "layer_layout", "check_layer",
           "Report", "SENTINEL", "PAD"]
