"""HeadGuard CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain scalar C implementation of the head-masked image-KV quantizer
(hg_oracle.c), loaded through ctypes.  Only tests, the smoke entry and the
bench's CPU-baseline leg may import this package; the library under test never
does.  The oracle shares no code with the HIP path.

All arrays are numpy host arrays: BF16 caches as uint16 bit patterns
[L][B][H][T][D], the mask as uint8 [L*H].
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hg_oracle.c")
_LIB = os.environ.get("HG_ORACLE_LIB") or os.path.join(_HERE, "libhg_oracle.so")
CFLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
          "-pthread", "-Wall", "-Wextra"]


def build() -> str:
    """Compile the oracle with gcc (always; the caller decides when)."""
    tmp = _LIB + ".tmp"
    subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


class Config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in
                ("L", "B", "H", "T", "D", "img_start", "img_len", "bits", "base",
                 "keys_only", "kivi_group", "retain_permille")]


class Sizes(C.Structure):
    _fields_ = [("codes_k", C.c_uint64), ("meta_k", C.c_uint64), ("side_k", C.c_uint64),
                ("codes_v", C.c_uint64), ("meta_v", C.c_uint64), ("side_v", C.c_uint64),
                ("norm_k", C.c_uint64), ("ret_idx", C.c_uint64), ("ret_k", C.c_uint64),
                ("ret_v", C.c_uint64),
                ("n_protected", C.c_int32), ("n_unprot_k", C.c_int32),
                ("n_unprot_v", C.c_int32), ("retain_count", C.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = C.CDLL(_LIB)
        P = C.c_void_p
        L.hgo_bf16_to_f32.argtypes = [C.c_uint16]; L.hgo_bf16_to_f32.restype = C.c_float
        for f in ("hgo_bf16_rne", "hgo_bf16_rd", "hgo_bf16_ru"):
            getattr(L, f).argtypes = [C.c_float]
            getattr(L, f).restype = C.c_uint16
        L.hgo_quantize_group.argtypes = [P, C.c_int, C.c_int, C.c_int, P, C.c_int]
        L.hgo_quantize_group.restype = C.c_uint32
        L.hgo_level.argtypes = [C.c_uint32, C.c_uint]; L.hgo_level.restype = C.c_float
        L.hgo_fwht_norm.argtypes = [P, C.c_int]; L.hgo_fwht_norm.restype = None
        L.hgo_fwht_raw.argtypes = [P, C.c_int]; L.hgo_fwht_raw.restype = None
        L.hgo_fwht_scale.argtypes = [C.c_int]; L.hgo_fwht_scale.restype = C.c_float
        L.hgo_route.argtypes = [C.POINTER(Config), P, C.c_int, C.c_int, C.c_int,
                                C.POINTER(C.c_int), C.POINTER(C.c_int)]
        L.hgo_sizes.argtypes = [C.POINTER(Config), P, C.POINTER(Sizes)]
        L.hgo_quantize_slice.argtypes = [C.POINTER(Config), C.c_int, P, P, P]
        L.hgo_quantize_slice_seq.argtypes = [C.POINTER(Config), C.c_int, P, P, P]
        L.hgo_dequantize_slice.argtypes = [C.POINTER(Config), C.c_int, P, P, P]
        L.hgo_quantize.argtypes = [C.POINTER(Config), P, P, P, P, P, P, P, P, P, C.c_int]
        L.hgo_dequantize.argtypes = [C.POINTER(Config), P, P, P, P, P, P, P, P, P, C.c_int]
        L.hgo_select_heads.argtypes = [P, P, C.c_int, C.c_int, C.c_int, C.c_int, P]
        L.hgo_retain_count.argtypes = [C.POINTER(Config)]
        L.hgo_key_sqnorm.argtypes = [P, C.c_int]; L.hgo_key_sqnorm.restype = C.c_float
        L.hgo_retain_select.argtypes = [P, C.c_int, C.c_int, P]
        L.hgo_retain.argtypes = [C.POINTER(Config), P, P, P, P, P, P, P, C.c_int]
        L.hgo_restore_retained.argtypes = [C.POINTER(Config), P, P, P, P, P, P]
        for f in ("hgo_route", "hgo_sizes", "hgo_quantize_slice", "hgo_quantize_slice_seq",
                  "hgo_dequantize_slice",
                  "hgo_quantize", "hgo_dequantize", "hgo_select_heads", "hgo_retain_count",
                  "hgo_retain_select", "hgo_retain", "hgo_restore_retained"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.c_void_p)


def make_config(**f) -> Config:
    return Config(**{k: int(v) for k, v in f.items()})


RETAIN_BUFFERS = ("norm_k", "ret_idx", "ret_k", "ret_v")


# ---------------------------------------------------------------- small pieces

def bf16_to_f32(h: int) -> float:
    return lib().hgo_bf16_to_f32(int(h))


def bf16_rne(x: float) -> int:
    return lib().hgo_bf16_rne(float(x))


def bf16_rd(x: float) -> int:
    return lib().hgo_bf16_rd(float(x))


def bf16_ru(x: float) -> int:
    return lib().hgo_bf16_ru(float(x))


def quantize_group(v, bits: int):
    """Codes (uint8) and the metadata word of one group of fp32 values."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    q = np.zeros(v.size, dtype=np.uint8)
    meta = lib().hgo_quantize_group(_ptr(v), v.size, 1, bits, _ptr(q), 1)
    return q, int(meta)


def level(meta: int, q: int) -> float:
    return float(np.float32(lib().hgo_level(int(meta), int(q))))


def fwht_norm(a) -> np.ndarray:
    a = np.array(a, dtype=np.float32, copy=True)
    lib().hgo_fwht_norm(_ptr(a), a.size)
    return a


def fwht_raw(a) -> np.ndarray:
    a = np.array(a, dtype=np.float32, copy=True)
    lib().hgo_fwht_raw(_ptr(a), a.size)
    return a


def fwht_scale(D: int) -> float:
    return float(np.float32(lib().hgo_fwht_scale(D)))


# ---------------------------------------------------------------- the cache

def route(cfg: Config, mask: np.ndarray, X: int, l: int, h: int):
    """(is_protected, slot) of tensor X (0 = K, 1 = V) at (l, h)."""
    p, s = C.c_int(), C.c_int()
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    rc = lib().hgo_route(C.byref(cfg), _ptr(mask), X, l, h, C.byref(p), C.byref(s))
    if rc:
        raise ValueError("hgo_route: bad arguments")
    return bool(p.value), s.value


def sizes(cfg: Config, mask: np.ndarray) -> Dict[str, int]:
    out = Sizes()
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    if lib().hgo_sizes(C.byref(cfg), _ptr(mask), C.byref(out)):
        raise ValueError("hgo_sizes: bad config")
    return {n: getattr(out, n) for n, _ in Sizes._fields_}


def _slice_outputs(cfg: Config, X: int):
    n, D = cfg.img_len, cfg.D
    codes = np.zeros((n, D * cfg.bits // 8), dtype=np.uint8)
    if cfg.base == 1 and X == 0:
        ng = (1 if n > 0 else 0) if cfg.kivi_group == 0 else -(-n // cfg.kivi_group)
        meta = np.zeros((ng, D), dtype=np.uint32)
    else:
        meta = np.zeros(n, dtype=np.uint32)
    return codes, meta


def quantize_slice(cfg: Config, X: int, rows: np.ndarray):
    """Codes (uint8 [n, D*bits/8]) and meta (uint32) of one unprotected slice,
    from its n image rows."""
    rows = np.ascontiguousarray(rows, dtype=np.uint16)
    codes, meta = _slice_outputs(cfg, X)
    if lib().hgo_quantize_slice(C.byref(cfg), X, _ptr(rows), _ptr(codes), _ptr(meta)):
        raise ValueError("hgo_quantize_slice failed")
    return codes, meta


def quantize_slice_seq(cfg: Config, X: int, slice_rows: np.ndarray):
    """The same from the whole slice [T, D] (text rows included)."""
    slice_rows = np.ascontiguousarray(slice_rows, dtype=np.uint16)
    codes, meta = _slice_outputs(cfg, X)
    if lib().hgo_quantize_slice_seq(C.byref(cfg), X, _ptr(slice_rows), _ptr(codes), _ptr(meta)):
        raise ValueError("hgo_quantize_slice_seq failed")
    return codes, meta


def dequantize_slice(cfg: Config, X: int, codes: np.ndarray, meta: np.ndarray) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    meta = np.ascontiguousarray(meta, dtype=np.uint32)
    out = np.zeros((cfg.img_len, cfg.D), dtype=np.uint16)
    if lib().hgo_dequantize_slice(C.byref(cfg), X, _ptr(codes), _ptr(meta), _ptr(out)):
        raise ValueError("hgo_dequantize_slice failed")
    return out


def quantize(cfg: Config, K: np.ndarray, V: np.ndarray, mask: np.ndarray, threads: int = 1):
    """Whole-cache quantize; returns a dict of flat numpy output buffers."""
    K = np.ascontiguousarray(K, dtype=np.uint16)
    V = np.ascontiguousarray(V, dtype=np.uint16)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    sz = sizes(cfg, mask)
    out = {
        "codes_k": np.zeros(sz["codes_k"], dtype=np.uint8),
        "meta_k": np.zeros(sz["meta_k"] // 4, dtype=np.uint32),
        "side_k": np.zeros(sz["side_k"] // 2, dtype=np.uint16),
        "codes_v": np.zeros(sz["codes_v"], dtype=np.uint8),
        "meta_v": np.zeros(sz["meta_v"] // 4, dtype=np.uint32),
        "side_v": np.zeros(sz["side_v"] // 2, dtype=np.uint16),
    }
    rc = lib().hgo_quantize(C.byref(cfg), _ptr(K), _ptr(V), _ptr(mask),
                            _ptr(out["codes_k"]), _ptr(out["meta_k"]), _ptr(out["side_k"]),
                            _ptr(out["codes_v"]), _ptr(out["meta_v"]), _ptr(out["side_v"]),
                            int(threads))
    if rc:
        raise ValueError("hgo_quantize failed")
    out["norm_k"] = np.zeros(sz["norm_k"] // 4, dtype=np.float32)
    out["ret_idx"] = np.zeros(sz["ret_idx"] // 4, dtype=np.int32)
    out["ret_k"] = np.zeros(sz["ret_k"] // 2, dtype=np.uint16)
    out["ret_v"] = np.zeros(sz["ret_v"] // 2, dtype=np.uint16)
    if cfg.retain_permille > 0:
        rc = lib().hgo_retain(C.byref(cfg), _ptr(K), _ptr(V), _ptr(mask), _ptr(out["norm_k"]),
                              _ptr(out["ret_idx"]), _ptr(out["ret_k"]), _ptr(out["ret_v"]),
                              int(threads))
        if rc:
            raise ValueError("hgo_retain failed")
    return out


def dequantize(cfg: Config, mask: np.ndarray, packed: Dict[str, np.ndarray],
               K_out: np.ndarray, V_out: np.ndarray, threads: int = 1) -> None:
    """Writes the image rows of K_out / V_out in place (text rows untouched)."""
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    assert K_out.flags["C_CONTIGUOUS"] and V_out.flags["C_CONTIGUOUS"]
    p = {k: np.ascontiguousarray(v) for k, v in packed.items()}
    rc = lib().hgo_dequantize(C.byref(cfg), _ptr(mask),
                              _ptr(p["codes_k"]), _ptr(p["meta_k"]), _ptr(p["side_k"]),
                              _ptr(p["codes_v"]), _ptr(p["meta_v"]), _ptr(p["side_v"]),
                              _ptr(K_out), _ptr(V_out), int(threads))
    if rc:
        raise ValueError("hgo_dequantize failed")
    if cfg.retain_permille > 0:
        rc = lib().hgo_restore_retained(C.byref(cfg), _ptr(mask), _ptr(p["ret_idx"]),
                                        _ptr(p["ret_k"]), _ptr(p["ret_v"]), _ptr(K_out), _ptr(V_out))
        if rc:
            raise ValueError("hgo_restore_retained failed")


def retain_count(cfg: Config) -> int:
    return int(lib().hgo_retain_count(C.byref(cfg)))


def key_sqnorm(key) -> float:
    """fp32 squared norm of one BF16 key (uint16 bit patterns)."""
    key = np.ascontiguousarray(key, dtype=np.uint16)
    return float(np.float32(lib().hgo_key_sqnorm(_ptr(key), key.size)))


def retain_select(sqnorm, k: int) -> np.ndarray:
    """Indices (ascending) of the k largest values, lower index first among equals."""
    sqnorm = np.ascontiguousarray(sqnorm, dtype=np.float32)
    idx = np.zeros(k, dtype=np.int32)
    if lib().hgo_retain_select(_ptr(sqnorm), sqnorm.size, int(k), _ptr(idx)):
        raise ValueError("hgo_retain_select: bad arguments")
    return idx


def select_heads(g: np.ndarray, o: np.ndarray, Hkv: int, K: int) -> np.ndarray:
    """Protection mask uint8 [L*Hkv] from per-query-head scores g, o [L][Hq]."""
    g = np.ascontiguousarray(g, dtype=np.float64)
    o = np.ascontiguousarray(o, dtype=np.float64)
    L, Hq = g.shape
    mask = np.zeros(L * Hkv, dtype=np.uint8)
    if lib().hgo_select_heads(_ptr(g), _ptr(o), L, Hq, Hkv, int(K), _ptr(mask)):
        raise ValueError("hgo_select_heads: bad arguments")
    return mask
