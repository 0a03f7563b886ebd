"""GPU parity at the full sizes of the five workloads (and three more cache
shapes), in the launch configuration the bench times: the whole cache is
quantized and dequantized on the GPU, then every (tensor, layer, batch row,
head) slice is recomputed by the CPU oracle — codes, metadata, BF16 side
store, retention outputs and reconstruction, text rows included — and must be
bit-exact; canary bytes after every packed buffer must be intact.  The
72B-shaped cache is swept over 2, 3 and 4 bits.  Each test asserts that it
compared 2*L*B*H slices."""
import pytest

import synthkv
import wholecache

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "qwen2.5-vl-7b", "llava-next-7b", "internvl-8b", "gemma-3-12b",
                                  "llava-1.5-7b", "72b-long-tp8"])
def test_workload(name):
    w = synthkv.WORKLOADS[name]
    wholecache.assert_whole(wholecache.quantize_dequantize(w), w)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_72b_long_bit_sweep(bits):
    w = synthkv.WORKLOADS["72b-long"].with_(bits=bits)
    wholecache.assert_whole(wholecache.quantize_dequantize(w), w)


@pytest.mark.parametrize("name", ["qwen2.5-vl-7b", "llava-next-7b", "internvl-8b", "72b-long"])
def test_one_pass_out_of_place(name):
    """The one-pass simulated quantization against the oracle's dequantize of
    its quantize, whole cache."""
    w = synthkv.WORKLOADS[name]
    wholecache.assert_whole(wholecache.fake_quantize(w, inplace=False), w)


@pytest.mark.parametrize("name", ["qwen2.5-vl-7b", "internvl-8b"])
def test_one_pass_in_place(name):
    w = synthkv.WORKLOADS[name]
    wholecache.assert_whole(wholecache.fake_quantize(w, inplace=True), w)
