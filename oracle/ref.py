"""ctypes binding of the CPU oracle in ``uzip_ref.c``.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The GPU library never imports this
module and this module never imports the GPU library.

Arrays are passed as numpy bit patterns: ``uint16`` for bf16/fp16 and
``uint32`` for fp32; streams are ``uint8`` arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "uzip_ref.c")
LIB_PATH = os.path.join(_HERE, "_build", "libuzip_ref.so")

# FP8 formats are coded in pairs: one element = a 16-bit unit of two values
DTYPES = {"bf16": 0, "fp16": 1, "fp32": 2, "e4m3fn": 3, "e5m2": 4}
ELEM_BYTES = {"bf16": 2, "fp16": 2, "fp32": 4, "e4m3fn": 2, "e5m2": 2}
BITS_DTYPE = {"bf16": np.uint16, "fp16": np.uint16, "fp32": np.uint32, "e4m3fn": np.uint16, "e5m2": np.uint16}

REF_EINVAL, REF_ENOSPC, REF_ECORRUPT = -1, -2, -3
# stream-wide table modes (sections 3.3.1 and 3.4)
TABLE_MODES = {"per_block": 0, "sampled": 1, "external": 2}


def build() -> str:
    """Compile the oracle with gcc (plain C, strict IEEE float semantics)."""
    os.makedirs(os.path.dirname(LIB_PATH), exist_ok=True)
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-fexcess-precision=standard", "-Wall", "-Wextra",
           SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB_PATH)
        vp, u8p = ctypes.c_void_p, ctypes.c_void_p
        u32, u64, i64 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int64
        L.ref_split_word.argtypes = [ctypes.c_int, u32, ctypes.POINTER(u32), ctypes.POINTER(u32)]
        L.ref_merge_word.argtypes = [ctypes.c_int, u32, u32]
        L.ref_merge_word.restype = u32
        L.ref_build_table.argtypes = [vp, u32, vp, vp]
        L.ref_rans_encode.argtypes = [u8p, u32, vp, vp, vp, vp, u64]
        L.ref_rans_encode.restype = i64
        L.ref_rans_decode.argtypes = [vp, vp, u64, vp, vp, u32, u8p]
        L.ref_rans_decode.restype = i64
        L.ref_max_compressed_size.argtypes = [ctypes.c_int, u64, u32]
        L.ref_max_compressed_size.restype = u64
        L.ref_block_section.argtypes = [vp, u64, ctypes.c_int, u32, u64, u8p, u64,
                                        ctypes.POINTER(ctypes.c_int)]
        L.ref_block_section.restype = i64
        L.ref_compress.argtypes = [vp, u64, ctypes.c_int, u32, u8p, u64]
        L.ref_compress.restype = i64
        L.ref_decompress.argtypes = [u8p, u64, ctypes.c_int, u64, vp]
        L.ref_decompress.restype = ctypes.c_int
        L.ref_build_table_all.argtypes = [vp, u64, vp]
        L.ref_sampled_table.argtypes = [vp, u64, ctypes.c_int, vp]
        L.ref_max_compressed_size_mode.argtypes = [ctypes.c_int, u64, u32, ctypes.c_int]
        L.ref_max_compressed_size_mode.restype = u64
        L.ref_compress_table.argtypes = [vp, u64, ctypes.c_int, u32, ctypes.c_int, vp, u8p, u64]
        L.ref_compress_table.restype = i64
        L.ref_decompress_table.argtypes = [u8p, u64, ctypes.c_int, u64, vp, vp]
        L.ref_decompress_table.restype = ctypes.c_int
        L.ref_reduce.argtypes = [vp, vp, ctypes.c_int, vp, ctypes.c_int, u64, u32, vp, u8p, u64]
        L.ref_reduce.restype = i64
        L.ref_half_to_float.argtypes = [u32]
        L.ref_half_to_float.restype = ctypes.c_float
        L.ref_float_to_half.argtypes = [ctypes.c_float]
        L.ref_float_to_half.restype = u32
        L.ref_bf16_to_float.argtypes = [u32]
        L.ref_bf16_to_float.restype = ctypes.c_float
        L.ref_float_to_bf16.argtypes = [ctypes.c_float]
        L.ref_float_to_bf16.restype = u32
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _bits(x: np.ndarray, dtype: str) -> np.ndarray:
    want = BITS_DTYPE[dtype]
    x = np.ascontiguousarray(x)
    if x.dtype != want:
        x = x.view(want)
    return x


def split_word(dtype: str, w: int) -> tuple[int, int]:
    s, r = ctypes.c_uint32(), ctypes.c_uint32()
    lib().ref_split_word(DTYPES[dtype], w, ctypes.byref(s), ctypes.byref(r))
    return s.value, r.value


def merge_word(dtype: str, sym: int, raw: int) -> int:
    return lib().ref_merge_word(DTYPES[dtype], sym, raw)


def build_table(count, n_b: int):
    c = np.ascontiguousarray(count, dtype=np.uint32)
    assert c.shape == (256,)
    f = np.zeros(256, np.uint32)
    cum = np.zeros(256, np.uint32)
    lib().ref_build_table(_ptr(c), n_b, _ptr(f), _ptr(cum))
    return f, cum


def rans_encode(sym: np.ndarray, freq, cum, max_words: int | None = None):
    sym = np.ascontiguousarray(sym, dtype=np.uint8)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    c = np.ascontiguousarray(cum, dtype=np.uint32)
    cap = len(sym) + 64 if max_words is None else max_words
    words = np.zeros(max(cap, 1), np.uint16)
    state = np.zeros(64, np.uint32)
    w = lib().ref_rans_encode(_ptr(sym), len(sym), _ptr(f), _ptr(c), _ptr(state), _ptr(words), cap)
    if w < 0:
        return None
    return state, words[:w].copy()


def rans_decode(state, words, freq, cum, n_b: int):
    st = np.ascontiguousarray(state, dtype=np.uint32)
    wd = np.ascontiguousarray(words, dtype=np.uint16)
    if wd.size == 0:
        wd = np.zeros(1, np.uint16)
        nw = 0
    else:
        nw = len(wd)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    c = np.ascontiguousarray(cum, dtype=np.uint32)
    out = np.zeros(max(n_b, 1), np.uint8)
    used = lib().ref_rans_decode(_ptr(st), _ptr(wd), nw, _ptr(f), _ptr(c), n_b, _ptr(out))
    if used < 0:
        return None
    return out[:n_b], used


def max_compressed_size(dtype: str, n: int, block_bytes: int) -> int:
    return lib().ref_max_compressed_size(DTYPES[dtype], n, block_bytes)


def compress(x: np.ndarray, dtype: str, block_bytes: int) -> np.ndarray:
    """Whole-stream compress of the bit patterns in ``x``."""
    xb = _bits(x, dtype).ravel()
    n = xb.size
    cap = max_compressed_size(dtype, n, block_bytes)
    out = np.zeros(cap, np.uint8)
    total = lib().ref_compress(_ptr(xb) if n else None, n, DTYPES[dtype], block_bytes, _ptr(out), cap)
    if total < 0:
        raise ValueError(f"ref_compress failed: {total}")
    return out[:total]


def decompress(stream: np.ndarray, dtype: str, n: int):
    """Returns the decoded bit patterns, or None if the stream is corrupt."""
    s = np.ascontiguousarray(stream, dtype=np.uint8)
    out = np.zeros(max(n, 1), BITS_DTYPE[dtype])
    rc = lib().ref_decompress(_ptr(s), s.size, DTYPES[dtype], n, _ptr(out))
    if rc != 0:
        return None
    return out[:n]


def build_table_all(count, n_s: int) -> np.ndarray:
    """All-symbol table freq[256] of a histogram over n_s symbols."""
    c = np.ascontiguousarray(count, dtype=np.uint32)
    assert c.shape == (256,)
    f = np.zeros(256, np.uint32)
    lib().ref_build_table_all(_ptr(c), n_s, _ptr(f))
    return f


def sampled_table(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stream-wide table from the first 256 KiB of ``x`` (uint32[256])."""
    xb = _bits(x, dtype).ravel()
    f = np.zeros(256, np.uint32)
    lib().ref_sampled_table(_ptr(xb) if xb.size else None, xb.size, DTYPES[dtype], _ptr(f))
    return f


def max_compressed_size_mode(dtype: str, n: int, block_bytes: int, mode: str) -> int:
    return lib().ref_max_compressed_size_mode(DTYPES[dtype], n, block_bytes, TABLE_MODES[mode])


def compress_table(x: np.ndarray, dtype: str, block_bytes: int, mode: str, table=None) -> np.ndarray:
    """Compress with a table mode; ``table`` (256 frequencies) for "external"."""
    xb = _bits(x, dtype).ravel()
    n = xb.size
    cap = max_compressed_size_mode(dtype, n, block_bytes, mode)
    out = np.zeros(cap, np.uint8)
    t = None if table is None else np.ascontiguousarray(table, dtype=np.uint16)
    total = lib().ref_compress_table(_ptr(xb) if n else None, n, DTYPES[dtype], block_bytes,
                                     TABLE_MODES[mode], _ptr(t) if t is not None else None, _ptr(out), cap)
    if total < 0:
        raise ValueError(f"ref_compress_table failed: {total}")
    return out[:total]


def decompress_table(stream: np.ndarray, dtype: str, n: int, table=None):
    """Decodes any table mode; None if the stream (or table) is rejected."""
    s = np.ascontiguousarray(stream, dtype=np.uint8)
    out = np.zeros(max(n, 1), BITS_DTYPE[dtype])
    t = None if table is None else np.ascontiguousarray(table, dtype=np.uint16)
    rc = lib().ref_decompress_table(_ptr(s), s.size, DTYPES[dtype], n, _ptr(t) if t is not None else None,
                                    _ptr(out))
    if rc != 0:
        return None
    return out[:n]


def block_section(x: np.ndarray, dtype: str, block_bytes: int, b: int):
    """One block's section bytes and its STORED flag."""
    xb = _bits(x, dtype).ravel()
    be = block_bytes // ELEM_BYTES[dtype]
    cap = be + 64
    sec = np.zeros(cap, np.uint8)
    stored = ctypes.c_int()
    ln = lib().ref_block_section(_ptr(xb), xb.size, DTYPES[dtype], block_bytes, b, _ptr(sec),
                                 cap, ctypes.byref(stored))
    if ln < 0:
        raise ValueError(f"ref_block_section failed: {ln}")
    return sec[:ln], bool(stored.value)


def reduce(streams, dtype: str, n: int, block_bytes: int, local=None):
    """Fused reduce of ``streams``; returns (output stream, reduced tensor)."""
    arrs = [np.ascontiguousarray(s, dtype=np.uint8) for s in streams]
    ptrs = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    sizes = (ctypes.c_uint64 * len(arrs))(*[a.size for a in arrs])
    y = np.zeros(max(n, 1), BITS_DTYPE[dtype])
    cap = max_compressed_size(dtype, n, block_bytes)
    out = np.zeros(cap, np.uint8)
    loc = None
    if local is not None:
        loc = _bits(local, dtype).ravel()
    total = lib().ref_reduce(ptrs, sizes, len(arrs), _ptr(loc) if loc is not None else None,
                             DTYPES[dtype], n, block_bytes, _ptr(y), _ptr(out), cap)
    if total < 0:
        raise ValueError(f"ref_reduce failed: {total}")
    return out[:total], y[:n]


def compress_chunked(x: np.ndarray, dtype: str, block_bytes: int, chunk_bytes: int, mode: str = "per_block",
                     table=None):
    """Each chunk of ``chunk_bytes`` of input is an independent stream (with
    a table mode: a sampled table per chunk, or the given table for all)."""
    xb = _bits(x, dtype).ravel()
    ce = chunk_bytes // ELEM_BYTES[dtype]
    if mode == "per_block":
        return [compress(xb[c:c + ce], dtype, block_bytes) for c in range(0, xb.size, ce)]
    return [compress_table(xb[c:c + ce], dtype, block_bytes, mode, table) for c in range(0, xb.size, ce)]


def half_to_float(h: int) -> float:
    return lib().ref_half_to_float(h)


def float_to_half(f: float) -> int:
    return lib().ref_float_to_half(f)


def bf16_to_float(b: int) -> float:
    return lib().ref_bf16_to_float(b)


def float_to_bf16(f: float) -> int:
    return lib().ref_float_to_bf16(f)
