"""Python binding of libuzip (gfx950 block-wise lossless float codec).

The C functions keep their names (``uzip_compress``, ``uzip_decompress``,
``uzip_reduce_fused``, ``uzip_compress_chunked``, ...); this module only
marshals arguments.  torch provides device memory and the current stream;
every step of the codec runs in the HIP kernels of ``csrc/uzip.hip``.
There is no CPU fallback: importing this module fails if the library has
not been built.

Convenience wrappers (``compress``, ``decompress``, ``reduce_fused``,
``compress_chunked``) allocate outputs and workspaces with torch and call
the C ABI on ``torch.cuda.current_stream()``.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .build import LIB_PATH

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python paper_2604_17172_amd/build.py` "
        "(or __graft_entry__.build()); there is no fallback implementation")

_lib = ctypes.CDLL(LIB_PATH)

BF16, FP16, FP32, E4M3FN, E5M2 = 0, 1, 2, 3, 4
OP_COMPRESS, OP_DECOMPRESS, OP_REDUCE, OP_CHUNKED, OP_COMPRESS_TABLE, OP_CHUNKED_TABLE = 0, 1, 2, 3, 4, 5
TABLE_PER_BLOCK, TABLE_SAMPLED, TABLE_EXTERNAL = 0, 1, 2
TABLE_BYTES = 512
WS_NO_OUT_RAW = 1 << 16
OK, EINVAL, ENOSPC, ECORRUPT, EHIP, EUNSUPPORTED, ETIMEOUT = 0, -1, -2, -3, -4, -5, -6

_c = ctypes
_vp, _u32, _u64, _sz, _int = _c.c_void_p, _c.c_uint32, _c.c_uint64, _c.c_size_t, _c.c_int

_lib.uzip_max_compressed_size.argtypes = [_int, _u64, _u32]
_lib.uzip_max_compressed_size.restype = _sz
_lib.uzip_workspace_size.argtypes = [_int, _int, _u64, _u32, _u64]
_lib.uzip_workspace_size.restype = _sz
_lib.uzip_compress.argtypes = [_vp, _u64, _int, _u32, _vp, _sz, _vp, _vp, _sz, _vp]
_lib.uzip_compress.restype = _int
_lib.uzip_decompress.argtypes = [_vp, _sz, _int, _u64, _vp, _sz, _vp, _vp, _sz, _vp]
_lib.uzip_decompress.restype = _int
_lib.uzip_reduce_fused.argtypes = [_c.POINTER(_vp), _c.POINTER(_sz), _int, _vp, _int, _u64, _u32, _vp, _sz,
                                   _vp, _vp, _vp, _vp, _sz, _vp]
_lib.uzip_reduce_fused.restype = _int
_lib.uzip_compress_chunked.argtypes = [_vp, _u64, _int, _u32, _u64, _vp, _sz, _vp, _vp, _u32, _vp, _sz, _vp]
_lib.uzip_compress_chunked.restype = _int
_lib.uzip_build_table.argtypes = [_vp, _u64, _int, _vp, _vp]
_lib.uzip_build_table.restype = _int
_lib.uzip_compress_table.argtypes = [_vp, _u64, _int, _u32, _int, _vp, _vp, _sz, _vp, _vp, _sz, _vp]
_lib.uzip_compress_table.restype = _int
_lib.uzip_compress_chunked_table.argtypes = [_vp, _u64, _int, _u32, _u64, _int, _vp, _vp, _sz, _vp, _vp, _u32, _vp,
                                             _sz, _vp]
_lib.uzip_compress_chunked_table.restype = _int
_lib.uzip_decompress_table.argtypes = [_vp, _sz, _int, _u64, _vp, _vp, _sz, _vp, _vp, _sz, _vp]
_lib.uzip_decompress_table.restype = _int
_lib.uzip_status_str.argtypes = [_int]
_lib.uzip_status_str.restype = _c.c_char_p
_lib.uzip_inject_scan_stall.argtypes = [_u32, _u32]
_lib.uzip_inject_scan_stall.restype = _int
_lib.uzip_compress_noalloc.argtypes = [_vp, _u64, _int, _u32, _vp, _sz, _vp, _vp]
_lib.uzip_compress_noalloc.restype = _int
_lib.uzip_decompress_chunked.argtypes = [_vp, _sz, _u64, _u64, _int, _u64, _u32, _u64, _vp, _sz, _vp, _vp]
_lib.uzip_decompress_chunked.restype = _int
_lib.uzip_decompress_chunked_table.argtypes = [_vp, _sz, _u64, _u64, _int, _u64, _u32, _u64, _vp, _vp, _sz, _vp,
                                               _vp]
_lib.uzip_decompress_chunked_table.restype = _int

EXPORTED = ["uzip_max_compressed_size", "uzip_workspace_size", "uzip_compress", "uzip_decompress",
            "uzip_reduce_fused", "uzip_compress_chunked", "uzip_status_str", "uzip_build_table",
            "uzip_compress_table", "uzip_decompress_table", "uzip_compress_chunked_table",
            "uzip_inject_scan_stall", "uzip_compress_noalloc", "uzip_decompress_chunked",
            "uzip_decompress_chunked_table"]


class UzipError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {uzip_status_str(status)} ({status})")
        self.status = status


# ---------------------------------------------------------------- raw C ABI
def uzip_max_compressed_size(dtype: int, n_elems: int, block_bytes: int) -> int:
    return _lib.uzip_max_compressed_size(dtype, n_elems, block_bytes)


def uzip_workspace_size(op: int, dtype: int, n_elems: int, block_bytes: int, aux: int = 0) -> int:
    return _lib.uzip_workspace_size(op, dtype, n_elems, block_bytes, aux)


def uzip_compress(d_in, n_elems, dtype, block_bytes, d_out, out_cap, d_out_size, d_ws, ws_bytes, stream) -> int:
    return _lib.uzip_compress(d_in, n_elems, dtype, block_bytes, d_out, out_cap, d_out_size, d_ws, ws_bytes, stream)


def uzip_compress_noalloc(d_in, n_elems, dtype, block_bytes, d_out, out_cap, d_out_size, stream) -> int:
    return _lib.uzip_compress_noalloc(d_in, n_elems, dtype, block_bytes, d_out, out_cap, d_out_size, stream)


def uzip_decompress(d_in, in_bytes, dtype, n_elems, d_out, out_cap, d_status, d_ws, ws_bytes, stream) -> int:
    return _lib.uzip_decompress(d_in, in_bytes, dtype, n_elems, d_out, out_cap, d_status, d_ws, ws_bytes, stream)


def uzip_reduce_fused(d_in, in_bytes, n_in, d_local_raw, dtype, n_elems, block_bytes, d_out, out_cap,
                      d_out_size, d_out_raw, d_status, d_ws, ws_bytes, stream) -> int:
    ptrs = (_vp * n_in)(*d_in)
    sizes = (_sz * n_in)(*in_bytes)
    return _lib.uzip_reduce_fused(ptrs, sizes, n_in, d_local_raw, dtype, n_elems, block_bytes, d_out, out_cap,
                                  d_out_size, d_out_raw, d_status, d_ws, ws_bytes, stream)


def uzip_compress_chunked(d_in, n_elems, dtype, block_bytes, chunk_bytes, d_out, slot_bytes, chunk_sizes,
                          flags, epoch, d_ws, ws_bytes, stream) -> int:
    return _lib.uzip_compress_chunked(d_in, n_elems, dtype, block_bytes, chunk_bytes, d_out, slot_bytes,
                                      chunk_sizes, flags, epoch, d_ws, ws_bytes, stream)


def uzip_build_table(d_in, n_elems, dtype, d_table, stream) -> int:
    return _lib.uzip_build_table(d_in, n_elems, dtype, d_table, stream)


def uzip_compress_table(d_in, n_elems, dtype, block_bytes, mode, d_table, d_out, out_cap, d_out_size, d_ws,
                        ws_bytes, stream) -> int:
    return _lib.uzip_compress_table(d_in, n_elems, dtype, block_bytes, mode, d_table, d_out, out_cap, d_out_size,
                                    d_ws, ws_bytes, stream)


def uzip_compress_chunked_table(d_in, n_elems, dtype, block_bytes, chunk_bytes, mode, d_table, d_out, slot_bytes,
                                chunk_sizes, flags, epoch, d_ws, ws_bytes, stream) -> int:
    return _lib.uzip_compress_chunked_table(d_in, n_elems, dtype, block_bytes, chunk_bytes, mode, d_table, d_out,
                                            slot_bytes, chunk_sizes, flags, epoch, d_ws, ws_bytes, stream)


def uzip_decompress_table(d_in, in_bytes, dtype, n_elems, d_table, d_out, out_cap, d_status, d_ws, ws_bytes,
                          stream) -> int:
    return _lib.uzip_decompress_table(d_in, in_bytes, dtype, n_elems, d_table, d_out, out_cap, d_status, d_ws,
                                      ws_bytes, stream)


def uzip_decompress_chunked(d_in, slot_bytes, first_chunk, n_chunks, dtype, n_elems, block_bytes, chunk_bytes,
                            d_out, out_cap, d_status, stream) -> int:
    return _lib.uzip_decompress_chunked(d_in, slot_bytes, first_chunk, n_chunks, dtype, n_elems, block_bytes,
                                        chunk_bytes, d_out, out_cap, d_status, stream)


def uzip_decompress_chunked_table(d_in, slot_bytes, first_chunk, n_chunks, dtype, n_elems, block_bytes,
                                  chunk_bytes, d_table, d_out, out_cap, d_status, stream) -> int:
    return _lib.uzip_decompress_chunked_table(d_in, slot_bytes, first_chunk, n_chunks, dtype, n_elems, block_bytes,
                                              chunk_bytes, d_table, d_out, out_cap, d_status, stream)


def uzip_status_str(status: int) -> str:
    return _lib.uzip_status_str(status).decode()


def uzip_inject_scan_stall(spin_limit: int, held_block: int) -> int:
    return _lib.uzip_inject_scan_stall(spin_limit, held_block)


# ---------------------------------------------------------------- torch helpers
# FP8 formats are coded in pairs: one element is a 16-bit unit of two values
_TORCH_DTYPE = {torch.bfloat16: BF16, torch.float16: FP16, torch.float32: FP32,
                torch.float8_e4m3fn: E4M3FN, torch.float8_e5m2: E5M2}
_NAME_DTYPE = {"bf16": BF16, "fp16": FP16, "fp32": FP32, "e4m3fn": E4M3FN, "e5m2": E5M2}
_ELEM = {BF16: 2, FP16: 2, FP32: 4, E4M3FN: 2, E5M2: 2}
_BITS = {BF16: torch.int16, FP16: torch.int16, FP32: torch.int32, E4M3FN: torch.int16, E5M2: torch.int16}


def dtype_code(dt) -> int:
    if isinstance(dt, int):
        return dt
    if isinstance(dt, str):
        return _NAME_DTYPE[dt]
    return _TORCH_DTYPE[dt]


def _stream(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _check(rc: int, what: str) -> None:
    if rc != OK:
        raise UzipError(rc, what)


def _n_elems(x: torch.Tensor, dt: int) -> int:
    """Elements of x in units of the codec's element (FP8: value pairs)."""
    nbytes = x.numel() * x.element_size()
    if nbytes % _ELEM[dt]:
        raise ValueError(f"{nbytes} bytes is not a whole number of {_ELEM[dt]}-byte elements "
                         "(FP8 tensors are coded in pairs and need an even length)")
    return nbytes // _ELEM[dt]


def _dev_empty(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def check_sizes(sizes: torch.Tensor, what: str) -> None:
    """Wait for the stream's work and raise if an encoder call marked a
    stream invalid (its size reads 0: the bounded wait of the single-pass
    scan ran out)."""
    torch.cuda.current_stream(sizes.device).synchronize()
    if bool((sizes == 0).any()):
        raise UzipError(ETIMEOUT, what)


def compress(x: torch.Tensor, block_bytes: int = 65536, dtype=None, out: torch.Tensor | None = None,
             ws: torch.Tensor | None = None, stream=None, check: bool = False, size: torch.Tensor | None = None):
    """Compress a contiguous CUDA tensor (bf16/fp16/fp32/float8, or an
    int16/int32 bit view with ``dtype`` given; float8 tensors are coded as
    pairs of values).  Returns (stream buffer, device u64 size; ``size``, a
    device int64[1], is reused when given).  With ``check`` the call waits
    for the GPU and raises UzipError(ETIMEOUT) if the stream was marked
    invalid (size 0)."""
    assert x.is_cuda and x.is_contiguous()
    dt = dtype_code(dtype if dtype is not None else x.dtype)
    n = _n_elems(x, dt)
    cap = uzip_max_compressed_size(dt, n, block_bytes)
    if cap == 0:
        _check(EINVAL, "uzip_compress")
    if out is None:
        out = _dev_empty(cap, x.device)
    wsb = uzip_workspace_size(OP_COMPRESS, dt, n, block_bytes)
    if ws is None:
        ws = _dev_empty(wsb, x.device)
    if size is None:
        size = torch.zeros(1, dtype=torch.int64, device=x.device)
    _check(uzip_compress(x.data_ptr() if n else None, n, dt, block_bytes, out.data_ptr(), out.numel(),
                         size.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream)), "uzip_compress")
    if check:
        check_sizes(size, "uzip_compress")
    return out, size


def decompress(s: torch.Tensor, dtype, n_elems: int, out: torch.Tensor | None = None,
               in_bytes: int | None = None, ws: torch.Tensor | None = None, stream=None,
               status: torch.Tensor | None = None):
    """Decompress a stream of n_elems elements (FP8: pairs).  Returns
    (bit-pattern tensor, int16 per FP8 pair; device u32 status).  A
    ``status`` given (device int32[1]) is reused as it is: the decoder only
    writes it on an error, so the caller zeroes it."""
    dt = dtype_code(dtype)
    if out is None:
        out = torch.empty(max(n_elems, 1), dtype=_BITS[dt], device=s.device)[:n_elems]
    if status is None:
        status = torch.zeros(1, dtype=torch.int32, device=s.device)
    nbytes = s.numel() * s.element_size() if in_bytes is None else in_bytes
    wsb = uzip_workspace_size(OP_DECOMPRESS, dt, n_elems, 65536, 0)
    if ws is None:
        ws = _dev_empty(wsb, s.device)
    _check(uzip_decompress(s.data_ptr(), nbytes, dt, n_elems, out.data_ptr() if n_elems else None,
                           n_elems * _ELEM[dt], status.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream)),
           "uzip_decompress")
    return out, status


def reduce_fused(streams, dtype, n_elems: int, block_bytes: int = 65536, local: torch.Tensor | None = None,
                 want_raw: bool = True, in_bytes=None, out: torch.Tensor | None = None,
                 ws: torch.Tensor | None = None, stream=None, check: bool = False):
    """Fused decompress -> fp32 reduce -> recompress.  Returns
    (stream buffer, device u64 size, reduced tensor or None, device status).
    With ``check`` the call waits for the GPU and raises UzipError with the
    device status (ECORRUPT, ETIMEOUT) if it is not OK."""
    dt = dtype_code(dtype)
    dev = streams[0].device
    cap = uzip_max_compressed_size(dt, n_elems, block_bytes)
    if out is None:
        out = _dev_empty(cap, dev)
    raw = torch.empty(max(n_elems, 1), dtype=_BITS[dt], device=dev)[:n_elems] if want_raw else None
    aux = len(streams) | (0 if want_raw else WS_NO_OUT_RAW)
    wsb = uzip_workspace_size(OP_REDUCE, dt, n_elems, block_bytes, aux)
    if ws is None:
        ws = _dev_empty(wsb, dev)
    size = torch.zeros(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    sizes = in_bytes if in_bytes is not None else [t.numel() * t.element_size() for t in streams]
    _check(uzip_reduce_fused([t.data_ptr() for t in streams], sizes, len(streams),
                             local.data_ptr() if local is not None else None, dt, n_elems, block_bytes,
                             out.data_ptr(), out.numel(), size.data_ptr(),
                             raw.data_ptr() if raw is not None and n_elems else None, status.data_ptr(),
                             ws.data_ptr(), ws.numel(), _stream(stream)), "uzip_reduce_fused")
    if check:
        torch.cuda.current_stream(dev).synchronize()
        _check(int(status.item()), "uzip_reduce_fused")
    return out, size, raw, status


def compress_chunked(x: torch.Tensor, block_bytes: int, chunk_bytes: int, dtype=None, epoch: int = 1,
                     flags: torch.Tensor | None = None, out: torch.Tensor | None = None,
                     ws: torch.Tensor | None = None, stream=None, check: bool = False):
    """Split-send producer.  Returns (buffer of n_chunks slots, slot_bytes,
    device u64 chunk sizes, flags [2 n_chunks] u32).  ``check`` as for
    ``compress`` (any chunk of size 0)."""
    assert x.is_cuda and x.is_contiguous()
    dt = dtype_code(dtype if dtype is not None else x.dtype)
    n = _n_elems(x, dt)
    e = _ELEM[dt]
    ce = chunk_bytes // e
    chunks = (n + ce - 1) // ce
    slot = uzip_max_compressed_size(dt, min(n, ce), block_bytes)
    slot = (slot + 255) // 256 * 256
    if out is None:
        out = _dev_empty(slot * max(chunks, 1), x.device)
    wsb = uzip_workspace_size(OP_CHUNKED, dt, n, block_bytes, chunk_bytes)
    if ws is None:
        ws = _dev_empty(wsb, x.device)
    sizes = torch.zeros(max(chunks, 1), dtype=torch.int64, device=x.device)
    if flags is None:
        flags = torch.zeros(2 * max(chunks, 1), dtype=torch.int32, device=x.device)
    _check(uzip_compress_chunked(x.data_ptr() if n else None, n, dt, block_bytes, chunk_bytes, out.data_ptr(),
                                 slot, sizes.data_ptr(), flags.data_ptr(), epoch, ws.data_ptr(), ws.numel(),
                                 _stream(stream)), "uzip_compress_chunked")
    if check and chunks:
        check_sizes(sizes[:chunks], "uzip_compress_chunked")
    return out, slot, sizes, flags


def decompress_chunked(buf: torch.Tensor, slot_bytes: int, dtype, n_elems: int, block_bytes: int,
                       chunk_bytes: int, first: int = 0, count: int | None = None, out: torch.Tensor | None = None,
                       table: torch.Tensor | None = None, shared: bool = False, stream=None):
    """Decode chunk streams first .. first + count - 1 of a split-send
    producer's slots (``shared``: streams with a stream-wide table, ``table``
    for EXTERNAL ones) into ``out``, the whole tensor's bit-pattern buffer.
    Returns (out, device u32 status)."""
    dt = dtype_code(dtype)
    ce = chunk_bytes // _ELEM[dt]
    chunks = (n_elems + ce - 1) // ce
    if count is None:
        count = chunks - first
    if out is None:
        out = torch.empty(max(n_elems, 1), dtype=_BITS[dt], device=buf.device)[:n_elems]
    status = torch.zeros(1, dtype=torch.int32, device=buf.device)
    cap = out.numel() * out.element_size()
    if shared or table is not None:
        rc = uzip_decompress_chunked_table(buf.data_ptr(), slot_bytes, first, count, dt, n_elems, block_bytes,
                                           chunk_bytes, table.data_ptr() if table is not None else None,
                                           out.data_ptr() if n_elems else None, cap, status.data_ptr(),
                                           _stream(stream))
        _check(rc, "uzip_decompress_chunked_table")
    else:
        rc = uzip_decompress_chunked(buf.data_ptr(), slot_bytes, first, count, dt, n_elems, block_bytes,
                                     chunk_bytes, out.data_ptr() if n_elems else None, cap, status.data_ptr(),
                                     _stream(stream))
        _check(rc, "uzip_decompress_chunked")
    return out, status


_MODE = {"per_block": TABLE_PER_BLOCK, "sampled": TABLE_SAMPLED, "external": TABLE_EXTERNAL}


def build_table(x: torch.Tensor, dtype=None, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The stream-wide table of ``x`` (from its first 256 KiB): int16[256]
    holding the u16 frequencies."""
    assert x.is_cuda and x.is_contiguous()
    dt = dtype_code(dtype if dtype is not None else x.dtype)
    n = _n_elems(x, dt)
    if out is None:
        out = torch.empty(256, dtype=torch.int16, device=x.device)
    _check(uzip_build_table(x.data_ptr() if n else None, n, dt, out.data_ptr(), _stream(stream)), "uzip_build_table")
    return out


def compress_table(x: torch.Tensor, block_bytes: int, mode="sampled", table: torch.Tensor | None = None, dtype=None,
                   out: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None):
    """Compress with a table mode ("per_block", "sampled", "external" with
    ``table``).  Returns (stream buffer, device u64 size)."""
    assert x.is_cuda and x.is_contiguous()
    dt = dtype_code(dtype if dtype is not None else x.dtype)
    md = _MODE[mode] if isinstance(mode, str) else mode
    n = _n_elems(x, dt)
    cap = uzip_max_compressed_size(dt, n, block_bytes)
    if cap == 0:
        _check(EINVAL, "uzip_compress_table")
    cap += TABLE_BYTES
    if out is None:
        out = _dev_empty(cap, x.device)
    wsb = uzip_workspace_size(OP_COMPRESS_TABLE, dt, n, block_bytes)
    if ws is None:
        ws = _dev_empty(wsb, x.device)
    size = torch.zeros(1, dtype=torch.int64, device=x.device)
    _check(uzip_compress_table(x.data_ptr() if n else None, n, dt, block_bytes, md,
                               table.data_ptr() if table is not None else None, out.data_ptr(), out.numel(),
                               size.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream)), "uzip_compress_table")
    return out, size


def decompress_table(s: torch.Tensor, dtype, n_elems: int, table: torch.Tensor | None = None,
                     out: torch.Tensor | None = None, in_bytes: int | None = None, ws: torch.Tensor | None = None,
                     stream=None):
    """Decompress a stream with a stream-wide table.  Returns (bit-pattern
    tensor, device u32 status)."""
    dt = dtype_code(dtype)
    if out is None:
        out = torch.empty(max(n_elems, 1), dtype=_BITS[dt], device=s.device)[:n_elems]
    status = torch.zeros(1, dtype=torch.int32, device=s.device)
    nbytes = s.numel() * s.element_size() if in_bytes is None else in_bytes
    if ws is None:
        ws = _dev_empty(uzip_workspace_size(OP_DECOMPRESS, dt, n_elems, 65536, 0), s.device)
    _check(uzip_decompress_table(s.data_ptr(), nbytes, dt, n_elems, table.data_ptr() if table is not None else None,
                                 out.data_ptr() if n_elems else None, n_elems * _ELEM[dt], status.data_ptr(),
                                 ws.data_ptr(), ws.numel(), _stream(stream)), "uzip_decompress_table")
    return out, status


def compress_chunked_table(x: torch.Tensor, block_bytes: int, chunk_bytes: int, mode="sampled",
                           table: torch.Tensor | None = None, dtype=None, epoch: int = 1,
                           flags: torch.Tensor | None = None, out: torch.Tensor | None = None,
                           ws: torch.Tensor | None = None, stream=None):
    """Split-send producer with a table mode.  Returns (buffer of n_chunks
    slots, slot_bytes, device u64 chunk sizes, flags)."""
    assert x.is_cuda and x.is_contiguous()
    dt = dtype_code(dtype if dtype is not None else x.dtype)
    md = _MODE[mode] if isinstance(mode, str) else mode
    n = _n_elems(x, dt)
    ce = chunk_bytes // _ELEM[dt]
    chunks = (n + ce - 1) // ce
    slot = uzip_max_compressed_size(dt, min(n, ce), block_bytes) + TABLE_BYTES
    slot = (slot + 255) // 256 * 256
    if out is None:
        out = _dev_empty(slot * max(chunks, 1), x.device)
    if ws is None:
        ws = _dev_empty(uzip_workspace_size(OP_CHUNKED_TABLE, dt, n, block_bytes, chunk_bytes), x.device)
    sizes = torch.zeros(max(chunks, 1), dtype=torch.int64, device=x.device)
    if flags is None:
        flags = torch.zeros(2 * max(chunks, 1), dtype=torch.int32, device=x.device)
    _check(uzip_compress_chunked_table(x.data_ptr() if n else None, n, dt, block_bytes, chunk_bytes, md,
                                       table.data_ptr() if table is not None else None, out.data_ptr(), slot,
                                       sizes.data_ptr(), flags.data_ptr(), epoch, ws.data_ptr(), ws.numel(),
                                       _stream(stream)), "uzip_compress_chunked_table")
    return out, slot, sizes, flags
