"""GPU parity at the full sizes of the five workloads (and four more cache
shapes, one a 128K-token context), in the launch configuration the bench times: the whole cache is
quantized and dequantized on the GPU, then every (tensor, layer, batch row,
head) slice is recomputed by the CPU oracle — codes, metadata, BF16 side
store, retention outputs and reconstruction, text rows included — and must be
bit-exact; canary bytes after every packed buffer must be intact.  The
72B-shaped cache is swept over 2, 3 and 4 bits, and a LLaVA-NeXT-shaped cache
is grown past 4 GiB per tensor.  Each test asserts that it compared 2*L*B*H
slices."""
import pytest

import synthkv
import wholecache

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "qwen2.5-vl-7b", "llava-next-7b", "internvl-8b", "gemma-3-12b",
                                  "llava-1.5-7b", "72b-long-tp8", "qwen2.5-vl-7b-128k"])
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


# LLaVA-NeXT-shaped heads over 36 layers of 4096 tokens (4000 of them image):
# 2.4e9 BF16 elements, 4.5 GiB, per tensor, past 2^31 elements and 2^32 bytes,
# so every offset into K, V and their reconstruction must be formed in 64 bits.
PAST_4GIB = synthkv.WORKLOADS["llava-next-7b"].with_(name="llava-next-past-4gib", L=36, T=4096, img_len=4000)


@pytest.mark.parametrize("kivi_group", [32, 0])
def test_tensors_past_4_gib(kivi_group):
    w = PAST_4GIB.with_(kivi_group=kivi_group)
    assert w.L * w.B * w.H * w.T * w.D > 2 ** 31
    wholecache.assert_whole(wholecache.quantize_dequantize(w), w)


def test_one_pass_past_4_gib():
    wholecache.assert_whole(wholecache.fake_quantize(PAST_4GIB, inplace=False), PAST_4GIB)
