"""The C-ABI library loads, exports what include/uzip.h declares, and its
host-side logic (sizes, argument checks) is right.  No GPU is touched: every
call here returns before the library makes any HIP call."""
import os
import re

import numpy as np
import pytest

from oracle import ref

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "uzip.h")).read()
    return sorted(set(re.findall(r"\b(uzip_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    import paper_2604_17172_amd as uz
    names = _declared()
    assert set(names) == set(uz.EXPORTED)
    for name in names:
        assert hasattr(uz._lib, name), name


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32", "e4m3fn", "e5m2"])
@pytest.mark.parametrize("bb", [4096, 65536, 262144, 1 << 20, 1 << 22])
def test_max_size_matches_oracle(dtype, bb):
    import paper_2604_17172_amd as uz
    for n in (0, 1, 511, 4097, 1 << 20, (1 << 20) + 7, 1 << 29):
        assert uz.uzip_max_compressed_size(uz.dtype_code(dtype), n, bb) == ref.max_compressed_size(dtype, n, bb)


def test_invalid_arguments_rejected_on_host():
    import paper_2604_17172_amd as uz
    assert uz.uzip_max_compressed_size(7, 100, 65536) == 0
    assert uz.uzip_max_compressed_size(0, 100, 65535) == 0
    assert uz.uzip_max_compressed_size(0, 100, 2048) == 0
    assert uz.uzip_max_compressed_size(0, 100, 1 << 23) == 0      # above 4 MiB
    assert uz.uzip_max_compressed_size(0, 100, 3 << 20) == 0      # not a power of two
    assert uz.uzip_max_compressed_size(0, 100, 1 << 22) > 0
    assert uz.uzip_compress(None, 10, 7, 65536, None, 0, None, None, 0, None) == uz.EINVAL
    assert uz.uzip_compress(None, 10, 0, 65535, None, 0, None, None, 0, None) == uz.EINVAL
    # misaligned pointers
    assert uz.uzip_compress(16, 10, 0, 65536, 24, 1 << 20, None, 32, 1 << 20, None) == uz.EINVAL
    # output too small
    assert uz.uzip_compress(16, 1000, 0, 65536, 32, 100, None, 48, 1 << 20, None) == uz.ENOSPC
    assert uz.uzip_decompress(16, 100, 9, 10, 32, 100, None, None, 0, None) == uz.EINVAL
    assert uz.uzip_decompress(16, 100, 0, 1000, 32, 100, None, None, 0, None) == uz.ENOSPC
    # the decoder keeps no state in a workspace: 256 reserved bytes, NULL accepted
    assert uz.uzip_workspace_size(uz.OP_DECOMPRESS, 0, 1 << 29, 65536, 0) == 256
    assert uz.uzip_reduce_fused([16] * 17, [64] * 17, 17, None, 0, 10, 65536, 32, 1 << 20, None, None,
                                None, 48, 1 << 20, None) == uz.EINVAL
    assert uz.uzip_reduce_fused([], [], 0, None, 0, 10, 65536, 32, 1 << 20, None, None,
                                None, 48, 1 << 20, None) == uz.EINVAL
    # chunk size not a multiple of the block size
    assert uz.uzip_compress_chunked(16, 1000, 0, 65536, 65536 + 4096, 32, 1 << 20, 48, 64, 1, 80,
                                    1 << 20, None) == uz.EINVAL
    assert uz.uzip_workspace_size(uz.OP_CHUNKED, 0, 1000, 65536, 3000) == 0
    assert uz.uzip_workspace_size(uz.OP_REDUCE, 0, 1000, 65536, 0) == 0
    assert uz.uzip_workspace_size(uz.OP_REDUCE, 0, 1000, 65536, 17) == 0
    # FP8 pairs are coded but not reduced
    for dt in (uz.E4M3FN, uz.E5M2):
        assert uz.uzip_max_compressed_size(dt, 100, 65536) == uz.uzip_max_compressed_size(uz.BF16, 100, 65536)
        assert uz.uzip_workspace_size(uz.OP_REDUCE, dt, 1000, 65536, 2) == 0
        assert uz.uzip_reduce_fused([16, 32], [64, 64], 2, None, dt, 10, 65536, 48, 1 << 20, None, None,
                                    None, 64, 1 << 20, None) == uz.EINVAL
    assert uz.uzip_max_compressed_size(5, 100, 65536) == 0
    # batched chunk decode: a range past the tensor's chunks, a chunk size
    # that is not a multiple of the block size, a misaligned slot size, an
    # output that does not reach the last chosen chunk; an empty range is a
    # no-op that touches nothing
    n, bb, cb = 3 * (1 << 19) + 5, 65536, 1 << 20              # 4 chunks
    args = dict(dtype=0, n_elems=n, block_bytes=bb, chunk_bytes=cb)

    def dc(first, count, slot=1 << 20, cap=2 * n, cbytes=cb, **kw):
        a = {**args, "chunk_bytes": cbytes, **kw}
        return uz.uzip_decompress_chunked(16, slot, first, count, a["dtype"], a["n_elems"], a["block_bytes"],
                                          a["chunk_bytes"], 32, cap, None, None)
    assert dc(3, 2) == uz.EINVAL and dc(5, 0) == uz.EINVAL
    assert dc(0, 1, cbytes=cb + 4096) == uz.EINVAL
    assert dc(0, 1, slot=(1 << 20) + 8) == uz.EINVAL
    assert dc(0, 2, cap=2 * (1 << 20) - 2) == uz.ENOSPC
    assert dc(0, 4, cap=2 * n - 2) == uz.ENOSPC
    assert dc(2, 0) == uz.OK and dc(4, 0) == uz.OK
    assert dc(0, 1, dtype=9) == uz.EINVAL
    assert uz.uzip_decompress_chunked_table(16, 1 << 20, 0, 1, 0, n, bb, cb, 24, 32, 2 * n, None,
                                            None) == uz.EINVAL   # misaligned table


def test_element_count_bound():
    """Element counts above 2^48 are refused before anything is enqueued
    (sizes computed from them would come near 64-bit overflow)."""
    import paper_2604_17172_amd as uz
    big = (1 << 48) + 1
    assert uz.uzip_max_compressed_size(0, 1 << 48, 65536) > 0
    assert uz.uzip_max_compressed_size(0, big, 65536) == 0
    assert uz.uzip_max_compressed_size(0, (1 << 64) - 1, 65536) == 0
    assert uz.uzip_workspace_size(uz.OP_COMPRESS, 0, big, 65536, 0) == 0
    assert uz.uzip_workspace_size(uz.OP_DECOMPRESS, 0, big, 65536, 0) == 0
    assert uz.uzip_compress(16, big, 0, 65536, 32, 1 << 62, 48, 64, 1 << 20, None) == uz.EINVAL
    assert uz.uzip_compress_noalloc(16, big, 0, 65536, 32, 1 << 62, 48, None) == uz.EINVAL
    assert uz.uzip_compress_chunked(16, big, 0, 65536, 1 << 20, 32, 1 << 22, 48, 64, 1, 80, 1 << 20,
                                    None) == uz.EINVAL
    assert uz.uzip_compress_table(16, big, 0, 65536, uz.TABLE_SAMPLED, None, 32, 1 << 62, 48, 64, 1 << 20,
                                  None) == uz.EINVAL
    assert uz.uzip_build_table(16, big, 0, 32, None) == uz.EINVAL
    assert uz.uzip_decompress(16, 1 << 40, 0, big, 32, 1 << 62, None, None, 0, None) == uz.EINVAL
    assert uz.uzip_decompress_chunked(16, 1 << 22, 0, 1, 0, big, 65536, 1 << 20, 32, 1 << 62, None,
                                      None) == uz.EINVAL
    assert uz.uzip_reduce_fused([16], [1 << 40], 1, None, 0, big, 65536, 32, 1 << 62, None, None, None, 48,
                                1 << 20, None) == uz.EINVAL


def test_workspace_sizes_are_bounded():
    """The workspace is a status word per block, plus a fixed pool of
    per-workgroup overflow slots for the words of a block that can leave the
    LDS staging window (at most 2048 slots whatever the tensor size; a slot
    holds a block's worst-case word count less the window's 7424 words),
    plus the reduced tensor when the fused reduce has no caller buffer for
    it.  Section 4.1 reports a compressor footprint of about 164 MB (0.1% of
    an H200's memory)."""
    import paper_2604_17172_amd as uz
    n = 1 << 29
    nb = n // 32768
    ws = uz.uzip_workspace_size(uz.OP_COMPRESS, 0, n, 65536)
    assert 0 < ws <= 8 * nb + 40e6            # 1 GiB bf16, 64 KiB blocks: 39.5 MB
    # the slot pool does not grow with the tensor
    ws2 = uz.uzip_workspace_size(uz.OP_COMPRESS, 0, 2 * n, 65536)
    assert ws2 - ws <= 8 * nb + 512
    wsc = uz.uzip_workspace_size(uz.OP_CHUNKED, 0, n, 65536, 4 << 20)
    assert 0 < wsc <= ws + 16 * (n // (2 << 20)) + 1024
    # blocks whose words fit the window need no slots at all
    assert uz.uzip_workspace_size(uz.OP_COMPRESS, 0, n, 16384) <= 8 * (n // 8192) + 4096
    # 256 KiB blocks: fp32 (65536 elements) 1 GiB, 106.6 MB
    wl = uz.uzip_workspace_size(uz.OP_COMPRESS, 2, 1 << 28, 262144)
    assert wl <= 8 * ((1 << 28) // 65536) + 107e6 and wl < 164e6
    assert uz.uzip_workspace_size(uz.OP_COMPRESS, 2, 1 << 29, 262144) - wl <= 8 * ((1 << 28) // 65536) + 512
    # 16-bit elements in 256 KiB blocks (131072 elements, up to 65536 words a
    # block): 2048 slots of 117.5 KB, 241 MB -- 0.08% of the MI355X's 288 GB
    for dt in (uz.BF16, uz.FP16, uz.E4M3FN):
        wh = uz.uzip_workspace_size(uz.OP_COMPRESS, dt, 1 << 28, 262144)
        assert wh <= 8 * ((1 << 28) // 131072) + 241e6 + 4096
        assert uz.uzip_workspace_size(uz.OP_COMPRESS, dt, 1 << 30, 262144) - wh <= 8 * 3 * 2048 + 512
    wr = uz.uzip_workspace_size(uz.OP_REDUCE, 0, 1 << 23, 65536, 8 | uz.WS_NO_OUT_RAW)
    assert wr >= 2 * (1 << 23)


def test_status_strings():
    import paper_2604_17172_amd as uz
    assert uz.uzip_status_str(0) == "ok"
    assert "corrupt" in uz.uzip_status_str(uz.ECORRUPT)
    assert "invalid" in uz.uzip_status_str(uz.ETIMEOUT)
    # fault injection only stores settings on the host; restore the defaults
    assert uz.uzip_inject_scan_stall(0, 0xFFFFFFFF) == uz.OK
    assert uz.uzip_status_str(123) == "unknown status"


def test_table_api_host_checks():
    import paper_2604_17172_amd as uz
    n, bb = 1 << 20, 65536
    base = uz.uzip_workspace_size(uz.OP_COMPRESS, uz.BF16, n, bb)
    # the compressor's own workspace, the table, and 16 x 256 sample counts
    # (the sample is split over 16 workgroups)
    assert uz.uzip_workspace_size(uz.OP_COMPRESS_TABLE, uz.BF16, n, bb) == base + uz.TABLE_BYTES + 16 * 256 * 4
    # bad mode, missing or misaligned table, too small an output
    assert uz.uzip_compress_table(16, 100, 0, bb, 3, None, 32, 1 << 20, None, 48, 1 << 20, None) == uz.EINVAL
    assert uz.uzip_compress_table(16, 100, 0, bb, uz.TABLE_EXTERNAL, None, 32, 1 << 20, None, 48, 1 << 20,
                                  None) == uz.EINVAL
    assert uz.uzip_compress_table(16, 100, 0, bb, uz.TABLE_EXTERNAL, 24, 32, 1 << 20, None, 48, 1 << 20,
                                  None) == uz.EINVAL
    cap = uz.uzip_max_compressed_size(uz.BF16, 1000, bb)
    assert uz.uzip_compress_table(16, 1000, 0, bb, uz.TABLE_SAMPLED, None, 32, cap, None, 48, 1 << 20,
                                  None) == uz.ENOSPC
    assert uz.uzip_compress_table(16, 1000, 7, bb, uz.TABLE_SAMPLED, None, 32, cap + 512, None, 48, 1 << 20,
                                  None) == uz.EINVAL
    assert uz.uzip_build_table(16, 100, 0, 24, None) == uz.EINVAL
    assert uz.uzip_build_table(16, 100, 9, 32, None) == uz.EINVAL
    assert uz.uzip_decompress_table(16, 100, 0, 10, 24, 32, 100, None, 48, 256, None) == uz.EINVAL
