"""GPU parity on seeded random configurations that draw every option at once
(§3 Applying protection, §4 Quantization setup): shape, head_dim, bit width,
base, K-only or K+V protection, the KIVI-style key group (32 tokens or the
whole sequence, long enough for several workgroups per slice), AKVQ-style
token retention, the image span (empty, at the start, at the end, the whole
sequence or inside it) and the protected heads.  Quantize and dequantize must
equal the oracle bit for bit; the one-pass mode (in place or out of place,
alternating) must equal the oracle's dequantize of its quantize."""
import numpy as np
import pytest

import synthkv
from hgtest import compare_full
from test_gpu_fakequant import check
from test_gpu_parity import _assert_exact

pytestmark = pytest.mark.gpu

N_CASES = 96


def draw(i: int) -> synthkv.Workload:
    rng = np.random.default_rng([20261202, i])
    D = int(rng.choice([64, 128, 256]))
    base = str(rng.choice(["minmax", "kivi", "akvq"]))
    whole = base == "kivi" and rng.random() < 0.6
    if whole:  # long sequences, few slices: the oracle stays fast
        L, B, H = 1, int(rng.integers(1, 3)), int(rng.integers(1, 4))
        # one workgroup holds 24 slots of 512 / D rows per wavefront, 16
        # wavefronts: up to 1.2x, 2.5x or 9x that (several partners per
        # slice, and past eight, 16 workgroups per slice)
        rows = 24 * 16 * (512 // D)
        T = int(rng.integers(1, int(rows * float(rng.choice([1.2, 2.5, 9.0])))))
    else:
        L, B, H = (int(x) for x in rng.integers(1, [4, 4, 6]))
        T = int(rng.integers(1, 700))
    kind = str(rng.choice(["empty", "start", "end", "whole", "inside"]))
    if kind == "empty":
        img_start, img_len = int(rng.integers(0, T + 1)), 0
    elif kind == "start":
        img_start, img_len = 0, int(rng.integers(1, T + 1))
    elif kind == "end":
        img_start = int(rng.integers(0, T))
        img_len = T - img_start
    elif kind == "whole":
        img_start, img_len = 0, T
    else:
        img_start = int(rng.integers(0, T))
        img_len = int(rng.integers(0, T - img_start + 1))
    bits = int(rng.choice([2, 3, 4]))
    keys_only = int(rng.integers(0, 2))
    n_protected = int(rng.integers(0, L * H + 1))
    retain = int(rng.choice([20, 137, 1000])) if base == "akvq" and rng.random() < 0.5 else 0
    name = (f"r{i}-{base}-D{D}-b{bits}-L{L}B{B}H{H}T{T}-s{img_start}+{img_len}-ko{keys_only}"
            f"-p{n_protected}" + ("-whole" if whole else "") + (f"-ret{retain}" if retain else ""))
    return synthkv.Workload(name, L=L, B=B, H=H, T=T, D=D, img_start=img_start, img_len=img_len,
                            bits=bits, base=base, keys_only=keys_only, n_protected=n_protected,
                            k_outliers=4, k_outlier_scale=10.0, kivi_group=0 if whole else 32,
                            seed=i, retain_permille=retain)


CASES = [draw(i) for i in range(N_CASES)]


@pytest.mark.parametrize("i", range(N_CASES), ids=lambda i: CASES[i].name)
def test_random_config(i):
    w = CASES[i]
    K, V = synthkv.gen_kv(w)
    mask = synthkv.protect_mask(w)
    _assert_exact(compare_full(w, K, V, mask), w.name)
    check(w, K, V, mask, inplace=bool(i % 2))
