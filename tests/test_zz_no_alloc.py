"""hg_fake_quantize_noalloc (the one-pass call for callers that cannot
allocate device memory; its workspace is the library's own device array)
against hg_fake_quantize with a caller workspace: the same bytes, on two calls
in a row, the second on a smaller cache, in place and out of place, with and
without token retention, and with whole-sequence KIVI keys (whose workgroups
exchange partial ranges through the workspace, or, for long slices, merge
chunk ranges into it).  A cache whose workspace
would exceed the array is refused before any device work."""
import ctypes as C

import numpy as np
import pytest
import torch

import synthkv
from test_gpu_parity import small

pytestmark = pytest.mark.gpu


def _big(permille):
    # the InternVL3-8B-shaped cache: in place, its workspace at 2 % (norms,
    # token lists, saved rows) is about 85 MiB of the 96 MiB array
    return synthkv.WORKLOADS["internvl-8b"].with_(retain_permille=permille)


def _small(permille):
    w = small("akvq", D=64, bits=3, img_len=301, img_start=5, text=11, L=2, B=2, H=4, n_protected=1)
    return w.with_(retain_permille=permille, name=f"small-r{permille}")


def _one_pass(hg, w, mask, inplace, noalloc):
    cfg = hg.make_config(**w.config_fields())
    K, V = synthkv.gen_kv(w, device="cuda")
    if inplace:
        Ko, Vo = K, V
    else:
        Ko = torch.full(K.shape, 0x7FBF, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        Vo = Ko.clone()
    if noalloc:
        lib = hg.library()
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        rc = lib.hg_fake_quantize_noalloc(C.byref(cfg), K.data_ptr(), V.data_ptr(), m.ctypes.data_as(C.c_void_p),
                                          Ko.data_ptr(), Vo.data_ptr(),
                                          torch.cuda.current_stream().cuda_stream)
        assert rc == hg.HG_OK, hg.hg_last_error()
    else:
        hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, hg.alloc_fake_workspace(cfg, mask))
    torch.cuda.synchronize()
    return Ko.view(torch.int16).clone(), Vo.view(torch.int16).clone()


def _kivi_whole(kind):
    # the workgroups holding a slice exchange their partial ranges through the
    # workspace (2 MiB at head_dim 128): 2 workgroups per slice on the
    # LLaVA-NeXT-shaped cache, 16 on the smaller one; slices past 32
    # workgroups' rows merge chunk ranges into the same area
    if kind == "big":
        return synthkv.WORKLOADS["llava-next-7b"].with_(kivi_group=0, L=8)
    if kind == "long":
        w = small("kivi", D=128, bits=2, img_len=60000, img_start=5, text=11, L=2, B=2, H=2, n_protected=1)
        return w.with_(kivi_group=0, name="long-kivi-whole")
    w = small("kivi", D=128, bits=2, img_len=12500, img_start=5, text=11, L=1, B=2, H=2, n_protected=1)
    return w.with_(kivi_group=0, name="small-kivi-whole")


@pytest.mark.parametrize("first", ["big", "long"])
@pytest.mark.parametrize("inplace", [False, True])
def test_whole_sequence_kivi_keys_on_two_calls(inplace, first):
    import paper_2609_35800_amd as hg
    for w in (_kivi_whole(first), _kivi_whole("small")):
        mask = synthkv.protect_mask(w)
        need = hg.hg_packed_sizes(hg.make_config(**w.config_fields()), mask)["fake_workspace"]
        assert 0 < need <= hg.HG_NOALLOC_SCRATCH_BYTES
        gK, gV = _one_pass(hg, w, mask, inplace, noalloc=True)
        wK, wV = _one_pass(hg, w, mask, inplace, noalloc=False)
        assert torch.equal(gK, wK), w.name
        assert torch.equal(gV, wV), w.name


@pytest.mark.parametrize("permille", [20, 0])
@pytest.mark.parametrize("inplace", [False, True])
def test_matches_the_workspace_entry_point_on_two_calls(permille, inplace):
    import paper_2609_35800_amd as hg
    for w in (_big(permille), _small(permille)):  # the second call is on a smaller cache
        mask = synthkv.protect_mask(w)
        if permille:
            need = hg.hg_packed_sizes(hg.make_config(**w.config_fields()), mask)["fake_workspace"]
            assert 0 < need <= hg.HG_NOALLOC_SCRATCH_BYTES
        gK, gV = _one_pass(hg, w, mask, inplace, noalloc=True)
        wK, wV = _one_pass(hg, w, mask, inplace, noalloc=False)
        assert torch.equal(gK, wK), w.name
        assert torch.equal(gV, wV), w.name


def test_too_large_a_workspace_is_refused():
    import paper_2609_35800_amd as hg
    # in place, 2048 heads x 40000 tokens of norms alone exceed the array
    w = small("akvq", D=64, img_len=40000, img_start=0, text=0, L=8, B=16, H=16, n_protected=0)
    w = w.with_(retain_permille=20)
    cfg = hg.make_config(**w.config_fields())
    mask = np.zeros(w.L * w.H, np.uint8)
    assert hg.hg_packed_sizes(cfg, mask)["fake_workspace"] > hg.HG_NOALLOC_SCRATCH_BYTES
    lib = hg.library()
    base = 1 << 36  # never dereferenced: the size check comes first
    rc = lib.hg_fake_quantize_noalloc(C.byref(cfg), base, base + (1 << 34), mask.ctypes.data_as(C.c_void_p),
                                      base, base + (1 << 34), None)
    assert rc == hg.HG_ERR_SHAPE and "array holds" in hg.hg_last_error()
