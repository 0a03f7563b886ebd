"""HeadGuard head-masked low-bit image-KV quantizer on MI355X (gfx950).

A thin ctypes binding over libheadguard.so (include/headguard.h): the entry
points keep their C names and only marshal arguments; every step of the
quantizer runs in the library's HIP kernels.  torch is used for device memory
and streams.  There is no fallback: if the library is missing or fails to load
the import raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# HG_LIBRARY may name another build of the same ABI; default: the in-tree build.
LIB_PATH = os.environ.get("HG_LIBRARY") or os.path.join(_HERE, "libheadguard.so")

HG_BASE_MINMAX, HG_BASE_KIVI, HG_BASE_AKVQ = 0, 1, 2
BASES = {"minmax": HG_BASE_MINMAX, "kivi": HG_BASE_KIVI, "akvq": HG_BASE_AKVQ}
STATUS = ("HG_OK", "HG_ERR_NULL", "HG_ERR_SHAPE", "HG_ERR_SPAN", "HG_ERR_BITS", "HG_ERR_BASE",
          "HG_ERR_HEADDIM", "HG_ERR_ALIGN", "HG_ERR_MASK", "HG_ERR_NO_DEVICE", "HG_ERR_HIP",
          "HG_ERR_POINTER", "HG_ERR_VALUE")
for _i, _n in enumerate(STATUS):
    globals()[_n] = _i
HG_MAX_HEADS = 8192  # largest L*H the routing holds (headguard.h)
BUFFERS = ("codes_k", "meta_k", "side_k", "codes_v", "meta_v", "side_v",
           "norm_k", "ret_idx", "ret_k", "ret_v")  # the packed outputs
PACKED = BUFFERS + ("workspace",)  # the fields of hg_packed


class hg_config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in
                ("L", "B", "H", "T", "D", "img_start", "img_len", "bits", "base",
                 "keys_only", "kivi_group", "retain_permille")]


class hg_sizes(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in BUFFERS] + [("workspace", C.c_uint64),
                                                     ("fake_workspace", C.c_uint64)] + [
        ("n_protected", C.c_int32), ("n_unprot_k", C.c_int32), ("n_unprot_v", C.c_int32),
        ("retain_count", C.c_int32)]


class hg_packed(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in PACKED]


class HeadGuardError(RuntimeError):
    def __init__(self, status: int, detail: str):
        name = STATUS[status] if 0 <= status < len(STATUS) else f"status {status}"
        super().__init__(f"{name}: {detail}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python paper_2609_35800_amd/build.py`")
    lib = C.CDLL(LIB_PATH)
    P = C.c_void_p
    lib.hg_packed_sizes.argtypes = [C.POINTER(hg_config), P, C.POINTER(hg_sizes)]
    lib.hg_quantize.argtypes = [C.POINTER(hg_config), P, P, P, C.POINTER(hg_packed), P]
    lib.hg_dequantize.argtypes = [C.POINTER(hg_config), P, C.POINTER(hg_packed), P, P, P]
    lib.hg_select_heads.argtypes = [P, P, C.c_int32, C.c_int32, C.c_int32, C.c_int32, P]
    lib.hg_fake_quantize.argtypes = [C.POINTER(hg_config), P, P, P, P, P, P, C.c_uint64, P]
    lib.hg_head_budget.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_int32)]
    lib.hg_fake_quantize_noalloc.argtypes = [C.POINTER(hg_config), P, P, P, P, P, P]
    for f in ("hg_packed_sizes", "hg_quantize", "hg_dequantize", "hg_select_heads",
              "hg_fake_quantize", "hg_head_budget", "hg_fake_quantize_noalloc"):
        getattr(lib, f).restype = C.c_int
    lib.hg_status_string.argtypes = [C.c_int]
    lib.hg_status_string.restype = C.c_char_p
    lib.hg_last_error.argtypes = []
    lib.hg_last_error.restype = C.c_char_p
    return lib


_lib = _load()


def library() -> C.CDLL:
    return _lib


# ------------------------------------------------------------ raw C entry points

def hg_status_string(status: int) -> str:
    return _lib.hg_status_string(int(status)).decode()


def hg_last_error() -> str:
    return _lib.hg_last_error().decode()


def _check(status: int) -> None:
    if status != 0:
        raise HeadGuardError(status, hg_last_error())


def _mask_arg(mask) -> np.ndarray:
    m = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8).reshape(-1))
    return m


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr() if t.numel() > 0 else None


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_config(L, B, H, T, D, img_start, img_len, bits, base, keys_only, kivi_group=32,
                retain_permille=0) -> hg_config:
    if isinstance(base, str):
        base = BASES[base]
    return hg_config(L=L, B=B, H=H, T=T, D=D, img_start=img_start, img_len=img_len, bits=bits,
                     base=base, keys_only=keys_only, kivi_group=kivi_group,
                     retain_permille=retain_permille)


def hg_packed_sizes(cfg: hg_config, protect_mask) -> Dict[str, int]:
    m = _mask_arg(protect_mask)
    out = hg_sizes()
    _check(_lib.hg_packed_sizes(C.byref(cfg), m.ctypes.data_as(C.c_void_p), C.byref(out)))
    return {n: getattr(out, n) for n, _ in hg_sizes._fields_}


def _packed_struct(packed: Dict[str, torch.Tensor]) -> hg_packed:
    return hg_packed(**{n: _ptr(packed.get(n)) for n in PACKED})


def hg_quantize(cfg: hg_config, K: torch.Tensor, V: torch.Tensor, protect_mask,
                packed: Dict[str, torch.Tensor], stream=None) -> None:
    """Enqueue quantize+pack of the image KV of K, V into `packed` buffers."""
    m = _mask_arg(protect_mask)
    pk = _packed_struct(packed)
    _check(_lib.hg_quantize(C.byref(cfg), _ptr(K), _ptr(V), m.ctypes.data_as(C.c_void_p),
                            C.byref(pk), _stream(stream)))


def hg_dequantize(cfg: hg_config, protect_mask, packed: Dict[str, torch.Tensor],
                  K_out: torch.Tensor, V_out: torch.Tensor, stream=None) -> None:
    """Enqueue reconstruction of the image rows of K_out, V_out."""
    m = _mask_arg(protect_mask)
    pk = _packed_struct(packed)
    _check(_lib.hg_dequantize(C.byref(cfg), m.ctypes.data_as(C.c_void_p), C.byref(pk),
                              _ptr(K_out), _ptr(V_out), _stream(stream)))


def hg_fake_quantize(cfg: hg_config, K: torch.Tensor, V: torch.Tensor, protect_mask,
                     K_out: torch.Tensor, V_out: torch.Tensor, workspace: Optional[torch.Tensor] = None,
                     stream=None) -> None:
    """Enqueue the one-pass quantize-and-reconstruct of the image rows of K, V
    into K_out, V_out (which may be K, V themselves).  `workspace`: a device
    buffer of at least hg_packed_sizes(...)["fake_workspace"] bytes, needed
    with token retention and with whole-sequence KIVI keys longer than one
    workgroup holds (see alloc_fake_workspace)."""
    m = _mask_arg(protect_mask)
    ws = _ptr(workspace)
    nbytes = workspace.numel() * workspace.element_size() if ws is not None else 0
    _check(_lib.hg_fake_quantize(C.byref(cfg), _ptr(K), _ptr(V), m.ctypes.data_as(C.c_void_p),
                                 _ptr(K_out), _ptr(V_out), ws, nbytes, _stream(stream)))


def hg_fake_quantize_noalloc(cfg: hg_config, K: torch.Tensor, V: torch.Tensor, protect_mask,
                             K_out: torch.Tensor, V_out: torch.Tensor, stream=None) -> None:
    """hg_fake_quantize with its workspace (retention lists, or the
    whole-sequence key exchange area) taken from the library's own device
    array (HG_NOALLOC_SCRATCH_BYTES per GPU): nothing is allocated;
    overlapping calls on one GPU race on that array."""
    m = _mask_arg(protect_mask)
    _check(_lib.hg_fake_quantize_noalloc(C.byref(cfg), _ptr(K), _ptr(V), m.ctypes.data_as(C.c_void_p),
                                         _ptr(K_out), _ptr(V_out), _stream(stream)))


HG_NOALLOC_SCRATCH_BYTES = 96 << 20  # headguard.h


# ------------------------------------------------------------ allocation helper

def alloc_packed(cfg: hg_config, protect_mask, device="cuda") -> Dict[str, torch.Tensor]:
    """Device buffers of the sizes hg_packed_sizes reports (uint8 tensors),
    the quantize call's workspace included."""
    sz = hg_packed_sizes(cfg, protect_mask)
    return {n: torch.empty(sz[n], dtype=torch.uint8, device=device) for n in PACKED}


def alloc_fake_workspace(cfg: hg_config, protect_mask, device="cuda") -> Optional[torch.Tensor]:
    """The one-pass call's workspace (uint8 tensor), or None when it needs none."""
    n = hg_packed_sizes(cfg, protect_mask)["fake_workspace"]
    return torch.empty(n, dtype=torch.uint8, device=device) if n else None


# ------------------------------------------------------------ head selection

def hg_select_heads(g, o, Hkv: int, K: int) -> np.ndarray:
    """Protection mask uint8 [L*Hkv] from per-query-head scores g, o [L][Hq]."""
    g = np.ascontiguousarray(g, dtype=np.float64)
    o = np.ascontiguousarray(o, dtype=np.float64)
    if g.shape != o.shape or g.ndim != 2:
        raise ValueError("g and o must both be [L, Hq]")
    L, Hq = g.shape
    mask = np.zeros(L * Hkv, dtype=np.uint8)
    _check(_lib.hg_select_heads(g.ctypes.data_as(C.c_void_p), o.ctypes.data_as(C.c_void_p),
                                L, Hq, Hkv, int(K), mask.ctypes.data_as(C.c_void_p)))
    return mask


def head_budget(n_kv: int, num: int = 1, den: int = 8) -> int:
    """hg_head_budget: K = round(n_kv * num / den), halves rounded up."""
    out = C.c_int32()
    _check(_lib.hg_head_budget(int(n_kv), int(num), int(den), C.byref(out)))
    return out.value
