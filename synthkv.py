"""Seeded synthetic KV caches and protection masks.

Input generation only: this module holds none of the quantizer's arithmetic.
It feeds the same BF16 bytes to the HIP library and to the CPU oracle, so a
parity result never depends on how the numbers were drawn.

Workloads stand in for the image-token KV caches of the VLMs the paper
evaluates (§4 "Models and tasks"); no model weights or datasets are used.
Recipe (one per named workload):
  * K, V: BF16 tensors [L][B][H][T][D]; every entry is an fp32 draw from
    N(0, 1) rounded to BF16 (round to nearest even);
  * keys carry `k_outliers` outlier channels per (layer, head), a fixed set
    drawn once per (l, h) and shared by every batch row and token (text
    included); those channels are multiplied by `k_outlier_scale` before the
    BF16 rounding.  Values have no outliers;
  * the image span is one contiguous run of `img_len` tokens starting at
    `img_start` = floor(text/2): half of the text tokens precede the image;
  * the protection mask marks the first `n_protected` entries of a seeded
    permutation of the L*H (layer, KV-head) indices, i.e. round(L*H/8) as in
    the paper's main budget (§3, head budget).
Streams: torch.Generator seeded per (seed, tensor, layer) draws the Gaussian
values (on the device the tensors live on); numpy default_rng([seed, 2]) draws
the outlier channel sets, row-major over (l, h), and then the mask
permutation.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np
import torch

BASES = {"minmax": 0, "kivi": 1, "akvq": 2}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    L: int
    B: int
    H: int
    T: int
    D: int
    img_start: int
    img_len: int
    bits: int
    base: str
    keys_only: int
    n_protected: int
    k_outliers: int
    k_outlier_scale: float
    kivi_group: int = 32
    seed: int = 0
    retain_permille: int = 0  # AKVQ-style token retention; 20 = the paper's 2 %

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def image_tokens(self) -> int:
        """Image tokens per call: every batch row carries the span."""
        return self.B * self.img_len

    def config_fields(self) -> Dict[str, int]:
        """The fields both sides' config structs take, as plain ints."""
        return dict(L=self.L, B=self.B, H=self.H, T=self.T, D=self.D,
                    img_start=self.img_start, img_len=self.img_len,
                    bits=self.bits, base=BASES[self.base],
                    keys_only=self.keys_only, kivi_group=self.kivi_group,
                    retain_permille=self.retain_permille)


# The five workloads: a tiny case, then caches shaped like the paper's 7B-72B
# VLMs (Qwen2.5-VL-7B, LLaVA-NeXT-7B, InternVL3-8B, a 72B model) with image
# spans of 1296-6400 tokens; LLaVA-1.5-7B- and Gemma-3-12B-shaped caches
# (576-token spans; head_dim 256); and
# one GPU's share of the 72B cache under an eight-way split by KV head; and a
# Qwen2.5-VL-7B-shaped 128K-token context with whole-sequence KIVI keys.
WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", L=2, B=1, H=4, T=288, D=64, img_start=16, img_len=256,
                     bits=2, base="minmax", keys_only=1, n_protected=1,
                     k_outliers=4, k_outlier_scale=10.0),
    "qwen2.5-vl-7b": Workload("qwen2.5-vl-7b", L=28, B=8, H=4, T=1360, D=128,
                              img_start=32, img_len=1296, bits=2, base="minmax",
                              keys_only=0, n_protected=14, k_outliers=4,
                              k_outlier_scale=10.0),
    "llava-next-7b": Workload("llava-next-7b", L=32, B=4, H=32, T=3008, D=128,
                              img_start=64, img_len=2880, bits=2, base="kivi",
                              keys_only=1, n_protected=128, k_outliers=4,
                              k_outlier_scale=10.0, kivi_group=32),
    "internvl-8b": Workload("internvl-8b", L=32, B=8, H=8, T=3456, D=128,
                            img_start=64, img_len=3328, bits=2, base="akvq",
                            keys_only=0, n_protected=32, k_outliers=8,
                            k_outlier_scale=20.0),
    "72b-long": Workload("72b-long", L=80, B=2, H=8, T=6656, D=128, img_start=128,
                         img_len=6400, bits=2, base="minmax", keys_only=0,
                         n_protected=80, k_outliers=8, k_outlier_scale=20.0),
    # LLaVA-1.5-7B-shaped: 32 KV heads (no grouping), one 576-token image
    "llava-1.5-7b": Workload("llava-1.5-7b", L=32, B=16, H=32, T=640, D=128, img_start=32,
                             img_len=576, bits=2, base="minmax", keys_only=0, n_protected=128,
                             k_outliers=4, k_outlier_scale=10.0),
    # Gemma-3-12B-shaped: head_dim 256, one 256-token image per prompt
    "gemma-3-12b": Workload("gemma-3-12b", L=48, B=32, H=8, T=320, D=256, img_start=32,
                            img_len=256, bits=2, base="minmax", keys_only=0, n_protected=48,
                            k_outliers=8, k_outlier_scale=20.0),
    # one GPU's share of the 72B cache split by KV head over eight GPUs
    "72b-long-tp8": Workload("72b-long-tp8", L=80, B=2, H=1, T=6656, D=128, img_start=128,
                             img_len=6400, bits=2, base="minmax", keys_only=0,
                             n_protected=10, k_outliers=8, k_outlier_scale=20.0),
    # Qwen2.5-VL-7B-shaped heads over a 128K-token context (a long video),
    # KIVI-style keys over the whole sequence: slices longer than 32
    # workgroups hold
    "qwen2.5-vl-7b-128k": Workload("qwen2.5-vl-7b-128k", L=28, B=1, H=4, T=131072, D=128,
                                   img_start=536, img_len=130000, bits=2, base="kivi",
                                   keys_only=1, n_protected=14, k_outliers=4,
                                   k_outlier_scale=10.0, kivi_group=0),
}


def outlier_channels(w: Workload) -> np.ndarray:
    """[L, H, k_outliers] channel indices of the outlier key channels."""
    rng = np.random.default_rng([w.seed, 2])
    out = np.zeros((w.L, w.H, max(w.k_outliers, 0)), dtype=np.int64)
    for l in range(w.L):
        for h in range(w.H):
            if w.k_outliers:
                out[l, h] = rng.choice(w.D, w.k_outliers, replace=False)
    return out


def protect_mask(w: Workload) -> np.ndarray:
    """uint8 [L*H], row-major (l, h); n_protected ones."""
    rng = np.random.default_rng([w.seed, 2])
    for _ in range(w.L * w.H):  # skip the outlier draws so the streams match
        if w.k_outliers:
            rng.choice(w.D, w.k_outliers, replace=False)
    perm = rng.permutation(w.L * w.H)
    mask = np.zeros(w.L * w.H, dtype=np.uint8)
    mask[perm[: w.n_protected]] = 1
    return mask


def _layer_seed(seed: int, X: int, l: int) -> int:
    return (seed * 1_000_003 + X * 65_537 + l * 7919 + 12345) & 0x7FFF_FFFF_FFFF


def gen_layer(w: Workload, X: int, l: int, device: str = "cpu",
              chans: Optional[np.ndarray] = None) -> torch.Tensor:
    """BF16 [B, H, T, D] for tensor X (0 = K, 1 = V) of layer l."""
    g = torch.Generator(device=device)
    g.manual_seed(_layer_seed(w.seed, X, l))
    x = torch.randn((w.B, w.H, w.T, w.D), generator=g, device=device,
                    dtype=torch.float32)
    if X == 0 and w.k_outliers:
        if chans is None:
            chans = outlier_channels(w)
        scale = torch.ones((w.H, w.D), dtype=torch.float32)
        for h in range(w.H):
            scale[h, torch.from_numpy(chans[l, h])] = float(w.k_outlier_scale)
        x *= scale.to(device).view(1, w.H, 1, w.D)
    return x.to(torch.bfloat16)


def gen_kv(w: Workload, device: str = "cpu"):
    """(K, V) BF16 tensors [L, B, H, T, D] on `device`."""
    chans = outlier_channels(w)
    K = torch.empty((w.L, w.B, w.H, w.T, w.D), dtype=torch.bfloat16, device=device)
    V = torch.empty_like(K)
    for l in range(w.L):
        K[l] = gen_layer(w, 0, l, device, chans)
        V[l] = gen_layer(w, 1, l, device, chans)
    return K, V


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Host uint16 view of a BF16 tensor's bit patterns."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
