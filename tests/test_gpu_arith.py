"""Exhaustive GPU checks of the arithmetic shortcuts the kernels take, run with
the kernels' own device helpers (tests/probes/hg_probes.hip):
  - the hardware fp32 -> BF16 conversion used by dequantize equals round to
    nearest even on the bit pattern for every finite fp32 value;
  - the fma-corrected division by 2^b - 1 used for the scale equals the IEEE
    quotient for every non-negative finite fp32 dividend (b = 2, 3, 4);
  - the refined hardware reciprocal equals the IEEE 1/S for every BF16 scale
    S in [2^-126, 2^101] (the range inputs below 2^100 can produce)."""
import ctypes as C
import os

import pytest
import torch

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "probes", "libhg_probes.so")


@pytest.fixture(scope="module")
def probes():
    if not os.path.exists(LIB):
        from probes import build
        build.build()
    lib = C.CDLL(LIB)
    lib.hgp_bf16_convert.argtypes = [C.c_void_p, C.c_void_p]
    lib.hgp_div_levels.argtypes = [C.c_int, C.c_void_p, C.c_void_p]
    lib.hgp_rcp_scale.argtypes = [C.c_void_p, C.c_void_p]
    return lib


def _run(fn, *args):
    cnt = torch.zeros(3, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    assert fn(*args, C.c_void_p(cnt.data_ptr()), C.c_void_p(stream)) == 0
    torch.cuda.synchronize()
    return [int(v) for v in cnt.cpu()]


def test_bf16_hardware_conversion_is_rne(probes):
    checked, bad, _ = _run(probes.hgp_bf16_convert)
    assert checked == (1 << 32) - (1 << 24)  # every pattern but Inf/NaN
    assert bad == 0


@pytest.mark.parametrize("levels", [3, 7, 15])
def test_division_by_levels_is_correctly_rounded(probes, levels):
    checked, bad, _ = _run(probes.hgp_div_levels, levels)
    assert checked == 0x7F800000
    assert bad == 0


def test_scale_reciprocal_is_correctly_rounded(probes):
    checked, bad, outside = _run(probes.hgp_rcp_scale)
    # positive normal BF16 up to 2^101: exponent fields 1..227 (128 mantissas
    # each) and 2^101 itself
    assert checked == 227 * 128 + 1
    assert bad == 0
    print(f"mismatches above 2^101 (outside the precondition): {outside}")
