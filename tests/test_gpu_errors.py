"""GPU: the encoder's failure path and the decoder's null workspace.

The single-pass scan that places each block's section bounds its wait for
earlier blocks; a wait that runs out marks the stream invalid (size and
magic 0, the split-send producer's DONE flag raised over the zero size, the
fused reduce's status UZIP_ETIMEOUT).  The condition is forced from the
host with uzip_inject_scan_stall: one block never publishes its size and
the wait is bounded at 1000 polls (about a millisecond), so every later block of its stream
gives up quickly and every kernel ends normally.  After the defaults are
restored, the same workspaces give streams equal to the oracle's.
"""
import struct
import sys

import numpy as np
import pytest
import torch

from oracle import ref
import workloads as W

pytestmark = pytest.mark.gpu

NONE = 0xFFFFFFFF


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def uz():
    import paper_2604_17172_amd as m
    return m


@pytest.fixture
def stall(uz):
    def set_(spin, held):
        assert uz.uzip_inject_scan_stall(spin, held) == uz.OK
    yield set_
    uz.uzip_inject_scan_stall(0, NONE)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_compress_marks_a_stalled_stream_invalid(uz, stall):
    x = W.normal_bf16(40 * 32768 + 1000, seed=50)
    xt = dev(x.view(np.int16))
    out = torch.empty(uz.uzip_max_compressed_size(uz.BF16, x.size, 65536), dtype=torch.uint8, device="cuda")
    ws = torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, uz.BF16, x.size, 65536), dtype=torch.uint8,
                     device="cuda")
    say(f"[errors] compress n={x.size}, block 5 held, 1000 polls")
    stall(1000, 5)
    _, size = uz.compress(xt, 65536, dtype="bf16", out=out, ws=ws)
    torch.cuda.synchronize()
    assert int(size.item()) == 0
    assert struct.unpack_from("<I", out[:4].cpu().numpy().tobytes())[0] == 0
    with pytest.raises(uz.UzipError) as e:
        uz.compress(xt, 65536, dtype="bf16", out=out, ws=ws, check=True)
    assert e.value.status == uz.ETIMEOUT
    # the last block held: nothing waits for it, the stream is valid
    stall(1000, 40)
    _, size = uz.compress(xt, 65536, dtype="bf16", out=out, ws=ws, check=True)
    want = ref.compress(x, "bf16", 65536)
    assert np.array_equal(out[: int(size.item())].cpu().numpy(), want)
    # defaults restored: the same workspace gives the oracle's stream
    stall(0, NONE)
    _, size = uz.compress(xt, 65536, dtype="bf16", out=out, ws=ws, check=True)
    assert np.array_equal(out[: int(size.item())].cpu().numpy(), want)


# 7 chunks: every workgroup takes any chunk's blocks; 81 chunks and 321
# blocks: on a chip of 8 XCDs each chunk is coded on one XCD
@pytest.mark.parametrize("full_chunks", [6, 80])
def test_chunked_producer_marks_only_the_stalled_chunk(uz, stall, full_chunks):
    bb, cb = 16384, 65536               # four blocks per chunk
    x = W.normal_bf16(full_chunks * 32768 + 5000, seed=51)
    xt = dev(x.view(np.int16))
    chunks = -(-x.size // (cb // 2))
    flags = torch.zeros(2 * chunks, dtype=torch.int32).pin_memory()
    say(f"[errors] chunked n={x.size} chunks={chunks}, global block 9 (chunk 2) held")
    stall(1000, 9)
    out, slot, sizes, _ = uz.compress_chunked(xt, bb, cb, dtype="bf16", epoch=7, flags=flags)
    torch.cuda.synchronize()
    assert bool((flags == 7).all()), "every DONE and RAW_READY flag is raised"
    sz = sizes.cpu().numpy()
    host = out.cpu().numpy()
    want = ref.compress_chunked(x, "bf16", bb, cb)
    for c in range(chunks):
        if c == 2:
            assert sz[c] == 0
            assert struct.unpack_from("<I", host[c * slot:c * slot + 4].tobytes())[0] == 0
        else:
            assert np.array_equal(host[c * slot:c * slot + sz[c]], want[c]), c
    stall(0, NONE)
    out, slot, sizes, _ = uz.compress_chunked(xt, bb, cb, dtype="bf16", epoch=8, flags=flags, check=True)
    host = out.cpu().numpy()
    for c in range(chunks):
        assert np.array_equal(host[c * slot:c * slot + int(sizes[c].item())], want[c]), c


def test_reduce_reports_a_stalled_coding_pass(uz, stall):
    xs = W.reduce_slices(n_in=3, tokens=64, hidden=8192, seed=52)   # 16 blocks
    n = xs[0].size
    streams = [ref.compress(v, "bf16", 65536) for v in xs]
    d = [dev(s) for s in streams]
    say(f"[errors] reduce n={n} x3, block 3 held")
    stall(1000, 3)
    _, size, _, status = uz.reduce_fused(d, "bf16", n, 65536)
    torch.cuda.synchronize()
    assert int(status.item()) == uz.ETIMEOUT and int(size.item()) == 0
    with pytest.raises(uz.UzipError) as e:
        uz.reduce_fused(d, "bf16", n, 65536, check=True)
    assert e.value.status == uz.ETIMEOUT
    stall(0, NONE)
    out, size, raw, status = uz.reduce_fused(d, "bf16", n, 65536, check=True)
    want_s, want_y = ref.reduce(streams, "bf16", n, 65536)
    assert np.array_equal(out[: int(size.item())].cpu().numpy(), want_s)


def test_decompress_without_workspace(uz):
    x = W.normal_bf16(100_000, seed=53)
    s = dev(ref.compress(x, "bf16", 65536))
    y = torch.empty(x.size, dtype=torch.int16, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    rc = uz.uzip_decompress(s.data_ptr(), s.numel(), uz.BF16, x.size, y.data_ptr(), 2 * x.size,
                            status.data_ptr(), None, 0, torch.cuda.current_stream().cuda_stream)
    assert rc == uz.OK
    torch.cuda.synchronize()
    assert int(status.item()) == 0 and np.array_equal(y.cpu().numpy().view(np.uint16), x)
