"""The entry points inside a captured HIP graph: hg_quantize followed by
hg_dequantize (and, separately, the one-pass hg_fake_quantize, out of place
and in place) is captured once (the calls only launch kernels on the given
stream: no allocation, no synchronisation, no memset) and replayed several
times, with the outputs cleared by eager work in between; every replay must
write exactly the bytes of the eager calls.  Covers the per-token, KIVI
(grouped and whole-sequence, with one, 2 and 16 workgroups per slice) and
AKVQ-with-retention paths."""
import numpy as np
import pytest
import torch

import synthkv
from test_gpu_parity import small

pytestmark = pytest.mark.gpu

CASES = [small("minmax", img_len=300), small("kivi", keys_only=1, img_len=300),
         small("kivi", img_len=300).with_(kivi_group=0, name="kivi-whole"),
         # whole-sequence keys held by 2 and by 16 workgroups per slice (the
         # exchange words cleared inside the graph on every replay)
         small("kivi", img_len=3000, H=2).with_(kivi_group=0, name="kivi-whole-2-partners"),
         small("kivi", img_len=12500, L=1, H=2, n_protected=1).with_(kivi_group=0, name="kivi-whole-16-partners"),
         small("akvq", img_len=300).with_(retain_permille=50, name="akvq-retain")]


def _snapshot(packed, Ko, Vo):
    return {**{n: t.clone() for n, t in packed.items()}, "K": Ko.clone(), "V": Vo.clone()}


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_capture_and_replay(w):
    import paper_2609_35800_amd as hg
    mask = synthkv.protect_mask(w)
    cfg = hg.make_config(**w.config_fields())
    K, V = synthkv.gen_kv(w, device="cuda")
    packed = hg.alloc_packed(cfg, mask)
    Ko, Vo = torch.zeros_like(K), torch.zeros_like(V)

    def clear():
        for t in packed.values():
            t.fill_(0xA5)
        Ko.fill_(0.0)
        Vo.fill_(0.0)

    clear()
    hg.hg_quantize(cfg, K, V, mask, packed)
    hg.hg_dequantize(cfg, mask, packed, Ko, Vo)
    torch.cuda.synchronize()
    want = _snapshot(packed, Ko, Vo)

    clear()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        hg.hg_quantize(cfg, K, V, mask, packed)
        hg.hg_dequantize(cfg, mask, packed, Ko, Vo)
    torch.cuda.synchronize()
    for _ in range(3):
        clear()  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(packed, Ko, Vo)
        for name in want:
            assert torch.equal(got[name].view(torch.uint8), want[name].view(torch.uint8)), name
    del graph


@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_capture_one_pass(w, inplace):
    """hg_fake_quantize only launches kernels too, with token retention
    included (its workspace is the caller's buffer): out of place, and in
    place with the inputs restored by eager work before every replay."""
    import paper_2609_35800_amd as hg
    mask = synthkv.protect_mask(w)
    cfg = hg.make_config(**w.config_fields())
    K0, V0 = synthkv.gen_kv(w, device="cuda")
    K, V = K0.clone(), V0.clone()
    Ko, Vo = (K, V) if inplace else (torch.zeros_like(K), torch.zeros_like(V))
    ws = hg.alloc_fake_workspace(cfg, mask)
    # retention's lists, or the exchange area of several workgroups per slice
    assert (ws is not None) == (w.retain_permille > 0 or "partners" in w.name)

    def reset():
        K.copy_(K0)
        V.copy_(V0)
        if not inplace:
            Ko.fill_(0.0)
            Vo.fill_(0.0)
        if ws is not None:
            ws.fill_(0xA5)  # the workspace's contents on entry do not matter

    reset()
    hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, ws)
    torch.cuda.synchronize()
    want_k, want_v = Ko.clone(), Vo.clone()
    reset()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, ws)
    for _ in range(3):
        reset()  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(Ko.view(torch.int16), want_k.view(torch.int16))
        assert torch.equal(Vo.view(torch.int16), want_v.view(torch.int16))
    del graph
