"""Launch failures on a working device, forced from the host through the
library's test hook (HG_FAIL_LAUNCH=i makes launch step i of every call
report hipErrorLaunchFailure without enqueuing it): the call returns
HG_ERR_HIP with the HIP error in hg_last_error; a failure at the first step
leaves every output byte untouched; a failure at a later step returns the
same status; and once the hook is cleared the same buffers give the oracle's
bytes (the device and the library are unaffected).  Every kernel that does
run exits normally."""
import numpy as np
import pytest
import torch

import synthkv
from hgtest import compare_full
from test_gpu_parity import _assert_exact, small

pytestmark = pytest.mark.gpu

FILL = 0xA5


def _setup(w):
    import paper_2609_35800_amd as hg
    mask = synthkv.protect_mask(w)
    cfg = hg.make_config(**w.config_fields())
    K, V = synthkv.gen_kv(w, device="cuda")
    packed = {n: torch.full((sz,), FILL, dtype=torch.uint8, device="cuda")
              for n, sz in hg.hg_packed_sizes(cfg, mask).items() if n in hg.PACKED}
    Ko = torch.full(K.shape, 0x7FBF, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    Vo = Ko.clone()
    return hg, mask, cfg, K, V, packed, Ko, Vo


def _untouched(packed, Ko, Vo):
    torch.cuda.synchronize()
    return (all(bool((t == FILL).all()) for t in packed.values())
            and bool((Ko.view(torch.int16) == 0x7FBF).all()) and bool((Vo.view(torch.int16) == 0x7FBF).all()))


CASES = [small("minmax"), small("kivi", keys_only=1).with_(kivi_group=0, name="kivi-whole"),
         small("akvq", img_len=300).with_(retain_permille=50, name="akvq-retain")]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_first_launch_failure_touches_nothing(w, monkeypatch):
    hg, mask, cfg, K, V, packed, Ko, Vo = _setup(w)
    monkeypatch.setenv("HG_FAIL_LAUNCH", "0")
    for call in (lambda: hg.hg_quantize(cfg, K, V, mask, packed),
                 lambda: hg.hg_dequantize(cfg, mask, packed, Ko, Vo),
                 lambda: hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, hg.alloc_fake_workspace(cfg, mask))):
        with pytest.raises(hg.HeadGuardError) as e:
            call()
        assert e.value.status == hg.HG_ERR_HIP
        assert "launch" in hg.hg_last_error()
    assert _untouched(packed, Ko, Vo)
    # cleared: the same call on the same buffers works and matches the oracle
    monkeypatch.delenv("HG_FAIL_LAUNCH")
    Kc, Vc = K.cpu(), V.cpu()
    _assert_exact(compare_full(w, Kc, Vc, mask), w.name)


@pytest.mark.parametrize("w", CASES[1:], ids=lambda w: w.name)
def test_later_launch_failure_is_reported(w, monkeypatch):
    """Calls of two or more launches (whole-sequence KIVI keys after the
    values; the retention selection after the quantizer) fail at step 1 with
    the same status; the first step's kernel ran and exited normally."""
    hg, mask, cfg, K, V, packed, Ko, Vo = _setup(w)
    monkeypatch.setenv("HG_FAIL_LAUNCH", "1")
    with pytest.raises(hg.HeadGuardError) as e:
        hg.hg_quantize(cfg, K, V, mask, packed)
    assert e.value.status == hg.HG_ERR_HIP and "launch" in hg.hg_last_error()
    torch.cuda.synchronize()
    monkeypatch.setenv("HG_FAIL_LAUNCH", "")
    hg.hg_quantize(cfg, K, V, mask, packed)
    torch.cuda.synchronize()
