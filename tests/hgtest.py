"""Shared helpers for the GPU parity tests: run the HIP library and the CPU
oracle on the same seeded BF16 bytes and compare their outputs."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synthkv

CANARY = 0xA5
PAD = 256  # canary bytes after every output buffer


def f32_of_bf16(u16: np.ndarray) -> np.ndarray:
    return (u16.astype(np.uint32) << 16).view(np.float32)


def bf16_ulp_diff(a: np.ndarray, b: np.ndarray) -> int:
    """Max distance in BF16 units in the last place (sign-magnitude aware)."""
    def key(u):
        u = u.astype(np.int32)
        return np.where(u & 0x8000, -(u & 0x7FFF), u & 0x7FFF)
    if a.size == 0:
        return 0
    return int(np.abs(key(a) - key(b)).max())


def alloc_with_canary(sizes, device="cuda"):
    """Packed buffers with PAD canary bytes after each; returns (views, raw)."""
    import paper_2609_35800_amd as hg
    views, raw = {}, {}
    for n in hg.PACKED:
        t = torch.full((sizes[n] + PAD,), CANARY, dtype=torch.uint8, device=device)
        raw[n] = t
        views[n] = t[: sizes[n]]
    return views, raw


def canaries_intact(raw) -> bool:
    return all(bool((t[-PAD:] == CANARY).all()) for t in raw.values())


def gpu_run(w: synthkv.Workload, K: torch.Tensor, V: torch.Tensor, mask: np.ndarray,
            stream=None, sentinel: int = 0x7FBF, prefill=None):
    """Quantize + dequantize on the GPU; returns host copies of everything.
    prefill(packed), if given, writes the output buffers before the call."""
    import paper_2609_35800_amd as hg
    cfg = hg.make_config(**w.config_fields())
    sizes = hg.hg_packed_sizes(cfg, mask)
    packed, raw = alloc_with_canary(sizes)
    if prefill is not None:
        prefill(packed)
    Kg, Vg = K.cuda().contiguous(), V.cuda().contiguous()
    Ko = torch.full(Kg.shape, sentinel, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    Vo = torch.full(Vg.shape, sentinel, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    if stream is not None:  # inputs were written on the current stream
        stream.wait_stream(torch.cuda.current_stream())
    hg.hg_quantize(cfg, Kg, Vg, mask, packed, stream=stream)
    hg.hg_dequantize(cfg, mask, packed, Ko, Vo, stream=stream)
    torch.cuda.synchronize()
    out = {n: packed[n].cpu().numpy() for n in hg.BUFFERS}
    out["_exchange_timeouts"] = exchange_timeouts(packed.get("workspace"))
    return out, synthkv.bf16_bits(Ko), synthkv.bf16_bits(Vo), canaries_intact(raw)


def exchange_timeouts(ws) -> int:
    """Waits that ran out of polls, counted in a KIVI exchange workspace's
    first 8 bytes (0 when the call used no workspace)."""
    if ws is None or ws.numel() < 8:
        return 0
    return int(ws[:8].cpu().numpy().view(np.uint64)[0])


def oracle_run(w: synthkv.Workload, Kb: np.ndarray, Vb: np.ndarray, mask: np.ndarray,
               sentinel: int = 0x7FBF, threads: int = 8):
    cfg = oracle.make_config(**w.config_fields())
    packed = oracle.quantize(cfg, Kb, Vb, mask, threads=threads)
    Ko = np.full_like(Kb, sentinel)
    Vo = np.full_like(Vb, sentinel)
    oracle.dequantize(cfg, mask, packed, Ko, Vo, threads=threads)
    as_bytes = {k: v.view(np.uint8) for k, v in packed.items()}
    return as_bytes, Ko, Vo


def compare_full(w, K, V, mask, stream=None, prefill=None):
    """Element-by-element parity of every output; returns a report dict."""
    Kb, Vb = synthkv.bf16_bits(K), synthkv.bf16_bits(V)
    g_pk, g_K, g_V, canary_ok = gpu_run(w, K, V, mask, stream=stream, prefill=prefill)
    o_pk, o_K, o_V = oracle_run(w, Kb, Vb, mask)
    rep = {"canaries": canary_ok, "exchange_timeouts": g_pk.pop("_exchange_timeouts")}
    for n in o_pk:
        assert g_pk[n].size == o_pk[n].size, n
        rep[n + "_mismatch"] = int(np.count_nonzero(g_pk[n] != o_pk[n]))
    rep["K_ulp"] = bf16_ulp_diff(g_K, o_K)
    rep["V_ulp"] = bf16_ulp_diff(g_V, o_V)
    rep["K_exact"] = bool(np.array_equal(g_K, o_K))
    rep["V_exact"] = bool(np.array_equal(g_V, o_V))
    return rep
