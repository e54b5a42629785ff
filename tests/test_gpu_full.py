"""GPU parity at the full sizes of the five measured configurations.

Every stream the GPU writes is compared byte for byte with the CPU oracle's
stream for the same seeded input (whole streams: the oracle compresses a
GiB in seconds), and every stream is decoded on the GPU back to the input.
The launch configuration is the one bench.py times (the same entry points
and block/chunk sizes).
"""
import sys
import time

import numpy as np
import pytest
import torch

from oracle import ref
import workloads as W

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

# FP8 formats are coded as 16-bit pairs of values
EB = {"bf16": 2, "fp16": 2, "fp32": 4, "e4m3fn": 2, "e5m2": 2}
NP_BITS = {"bf16": np.int16, "fp16": np.int16, "fp32": np.int32, "e4m3fn": np.int16, "e5m2": np.int16}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def uz():
    import paper_2604_17172_amd as m
    return m


def to_dev(x, dtype):
    return torch.from_numpy(np.ascontiguousarray(x).view(NP_BITS[dtype])).cuda()


def first_diff(a, b):
    n = min(a.size, b.size)
    d = np.nonzero(a[:n] != b[:n])[0]
    return int(d[0]) if d.size else n


def check_whole(uz, x, dtype, bb, label):
    say(f"[full] {label}: dtype={dtype} n={x.size} block={bb}")
    t0 = time.time()
    want = ref.compress(x, dtype, bb)
    say(f"[full] {label}: oracle {time.time() - t0:.1f}s, ratio {want.size / (EB[dtype] * x.size):.4f}")
    xt = to_dev(x, dtype)
    out, size = uz.compress(xt, bb, dtype=dtype)
    torch.cuda.synchronize()
    got = out[:int(size.item())].cpu().numpy()
    assert got.size == want.size and np.array_equal(got, want), \
        f"{label}: stream differs (sizes {got.size}/{want.size}, first diff at {first_diff(got, want)})"
    y, status = uz.decompress(out, dtype, x.size)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(y, xt), f"{label}: round trip not lossless"


def check_chunked(uz, x, dtype, bb, cb, label):
    say(f"[full] {label}: chunked dtype={dtype} n={x.size} block={bb} chunk={cb}")
    xt = to_dev(x, dtype)
    flags = torch.zeros(2 * ((x.size * EB[dtype] + cb - 1) // cb), dtype=torch.int32).pin_memory()
    out, slot, sizes, _ = uz.compress_chunked(xt, bb, cb, dtype=dtype, epoch=11, flags=flags)
    torch.cuda.synchronize()
    assert bool((flags == 11).all())
    buf = out.cpu().numpy()
    sz = sizes.cpu().numpy()
    ce = cb // EB[dtype]
    t0 = time.time()
    for c in range(sz.size):
        w = ref.compress(x[c * ce:(c + 1) * ce], dtype, bb)
        assert sz[c] == w.size, f"{label}: chunk {c} size {sz[c]} != {w.size}"
        assert np.array_equal(buf[c * slot:c * slot + w.size], w), f"{label}: chunk {c} differs"
    say(f"[full] {label}: {sz.size} chunks equal to the oracle ({time.time() - t0:.1f}s)")
    # every chunk decodes back to its slice, one call per chunk
    y = torch.empty_like(xt)
    for c in range(sz.size):
        n_c = min(ce, x.size - c * ce)
        yc, st = uz.decompress(out[c * slot:(c + 1) * slot], dtype, n_c, out=y[c * ce:c * ce + n_c])
        assert int(st.item()) == 0
    torch.cuda.synchronize()
    assert torch.equal(y, xt)
    # and all chunks in one launch
    y.zero_()
    _, st = uz.decompress_chunked(out, slot, dtype, x.size, bb, cb, out=y)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and torch.equal(y, xt)


def test_normal_bf16_4MiB(uz):
    check_whole(uz, W.normal_bf16(), "bf16", 65536, "normal_bf16_4MiB")


def test_weight_sync_1GiB_whole_stream(uz):
    check_whole(uz, W.weight_sync(), "bf16", 65536, "weight_sync_bf16_1GiB")


def test_weight_sync_1GiB_split_send_producer(uz):
    check_chunked(uz, W.weight_sync(), "bf16", 65536, 4 << 20, "weight_sync_bf16_1GiB")


def test_grad_fp32_1GiB(uz):
    check_whole(uz, W.grad_fp32(), "fp32", 262144, "grad_fp32_1GiB")


def test_grad_fp16_512MiB(uz):
    check_whole(uz, W.grad_fp16(), "fp16", 262144, "grad_fp16_512MiB")


def test_kv_cache_2GiB_chunked(uz):
    check_chunked(uz, W.kv_cache(), "bf16", 65536, 1 << 20, "kv_cache_bf16_2GiB")


@pytest.mark.parametrize("fmt", ["e4m3fn", "e5m2"])
def test_fp8_pairs_1GiB_whole_stream(uz, fmt):
    """1 GiB of FP8 N(0, 1) values (2^29 pairs), 64 KiB blocks: the
    benchmark's FP8 workload."""
    check_whole(uz, W.normal_fp8_pairs(1 << 29, fmt), fmt, 65536, f"normal_{fmt}_pairs_1GiB")


def test_weight_sync_1GiB_sampled_table(uz):
    """The whole 1 GiB buffer with one table sampled from its first 256 KiB."""
    x = W.weight_sync()
    say(f"[full] weight_sync sampled table: n={x.size}")
    t0 = time.time()
    want = ref.compress_table(x, "bf16", 65536, "sampled")
    say(f"[full] oracle {time.time() - t0:.1f}s, ratio {want.size / (2 * x.size):.4f}")
    xt = to_dev(x, "bf16")
    out, size = uz.compress_table(xt, 65536, "sampled", dtype="bf16")
    torch.cuda.synchronize()
    got = out[:int(size.item())].cpu().numpy()
    assert got.size == want.size and np.array_equal(got, want), f"first diff at {first_diff(got, want)}"
    y, st = uz.decompress_table(out, "bf16", x.size)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and torch.equal(y, xt)


def test_weight_sync_1GiB_chunked_sampled_tables(uz):
    """Split-send producer, 4 MiB chunks, each with the table sampled from
    its own first 256 KiB."""
    x = W.weight_sync()
    cb, bb = 4 << 20, 65536
    say(f"[full] weight_sync chunked sampled tables: n={x.size}")
    xt = to_dev(x, "bf16")
    flags = torch.zeros(2 * ((x.size * 2 + cb - 1) // cb), dtype=torch.int32).pin_memory()
    out, slot, sizes, _ = uz.compress_chunked_table(xt, bb, cb, "sampled", dtype="bf16", epoch=5, flags=flags)
    torch.cuda.synchronize()
    assert bool((flags == 5).all())
    buf = out.cpu().numpy()
    sz = sizes.cpu().numpy()
    ce = cb // 2
    t0 = time.time()
    for c in range(sz.size):
        w = ref.compress_table(x[c * ce:(c + 1) * ce], "bf16", bb, "sampled")
        assert sz[c] == w.size and np.array_equal(buf[c * slot:c * slot + w.size], w), f"chunk {c}"
    say(f"[full] {sz.size} chunks equal to the oracle ({time.time() - t0:.1f}s), ratio {sz.sum() / (2 * x.size):.4f}")
    y = torch.empty_like(xt)
    for c in range(sz.size):
        yc, st = uz.decompress_table(out[c * slot:(c + 1) * slot], "bf16", ce, out=y[c * ce:(c + 1) * ce])
        assert int(st.item()) == 0
    torch.cuda.synchronize()
    assert torch.equal(y, xt)


def test_reduce_8x16MiB(uz):
    xs = W.reduce_slices()
    n = xs[0].size
    say(f"[full] reduce_8x_bf16_16MiB: n={n}")
    t0 = time.time()
    streams = [ref.compress(v, "bf16", 65536) for v in xs]
    want_s, want_y = ref.reduce(streams, "bf16", n, 65536)
    say(f"[full] reduce oracle {time.time() - t0:.1f}s")
    dstreams = [torch.from_numpy(s).cuda() for s in streams]
    out, size, raw, status = uz.reduce_fused(dstreams, "bf16", n, 65536)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out[:int(size.item())].cpu().numpy()
    assert np.array_equal(got, want_s), f"reduce stream differs at {first_diff(got, want_s)}"
    assert np.array_equal(raw.cpu().numpy().view(np.uint16), want_y)
    # the GPU's own compressed shares give the same result
    gstreams = []
    for v in xs:
        o, sz = uz.compress(to_dev(v, "bf16"), 65536, dtype="bf16")
        gstreams.append(o[:int(sz.item())].clone())
    out2, size2, _, st2 = uz.reduce_fused(gstreams, "bf16", n, 65536, want_raw=False)
    torch.cuda.synchronize()
    assert int(st2.item()) == 0 and np.array_equal(out2[:int(size2.item())].cpu().numpy(), want_s)


def test_split_send_ordering_seen_from_the_host(uz):
    """Split-send (section 3.2.3, Property 2 of section 3.2.1): a chunk's
    uncompressed part is final, and usable, as soon as its RAW_READY flag is
    up, before its stream is done.  The producer writes the chunk streams,
    their sizes and the flags straight into pinned host memory while this
    thread polls the flags.  At the first sight of RAW_READY[c] the chunk's
    raw plane is read and compared with the oracle's; at the first sight of
    DONE[c] the whole stream and its size.  DONE flags are read before
    RAW_READY flags in every poll, so a DONE without its RAW_READY would be
    seen.  512 MiB of the weight-sync buffer, 4 MiB chunks, 64 KiB blocks."""
    from concurrent.futures import ThreadPoolExecutor
    bb, cb = 65536, 4 << 20
    x = W.weight_sync(256 << 20)
    n = x.size
    ce = cb // 2
    chunks = -(-n // ce)
    t0 = time.time()
    with ThreadPoolExecutor(16) as ex:
        want = list(ex.map(lambda c: ref.compress(x[c * ce:(c + 1) * ce], "bf16", bb), range(chunks)))
    say(f"[full] split-send ordering: {chunks} chunks, oracle {time.time() - t0:.1f}s")
    slot = (uz.uzip_max_compressed_size(uz.BF16, ce, bb) + 255) // 256 * 256
    out = torch.zeros(slot * chunks, dtype=torch.uint8).pin_memory()
    sizes = torch.zeros(chunks, dtype=torch.int64).pin_memory()
    flags = torch.zeros(2 * chunks, dtype=torch.int32).pin_memory()
    ws = torch.empty(uz.uzip_workspace_size(uz.OP_CHUNKED, uz.BF16, n, bb, cb), dtype=torch.uint8, device="cuda")
    xt = to_dev(x, "bf16")
    ob, sb, fl = out.numpy(), sizes.numpy(), flags.numpy()
    raw_off = 32 + (4 * (ce // 32768) + 15) // 16 * 16       # every chunk here is full
    epoch = 5
    torch.cuda.synchronize()
    rc = uz.uzip_compress_chunked(xt.data_ptr(), n, uz.BF16, bb, cb, out.data_ptr(), slot, sizes.data_ptr(),
                                  flags.data_ptr(), epoch, ws.data_ptr(), ws.numel(),
                                  torch.cuda.current_stream().cuda_stream)
    assert rc == uz.OK
    raw_seen = np.zeros(chunks, bool)
    done_seen = np.zeros(chunks, bool)
    lead = 0           # chunks whose RAW_READY was seen while DONE was still down
    deadline = time.time() + 60
    while not done_seen.all():
        assert time.time() < deadline, "flags never all raised"
        done = fl[1::2].copy() == epoch
        raw = fl[0::2].copy() == epoch
        assert not (done & ~raw).any(), f"DONE before RAW_READY for chunks {np.flatnonzero(done & ~raw)}"
        for c in np.flatnonzero(raw & ~raw_seen):
            raw_seen[c] = True
            lead += int(not done[c])
            got = ob[c * slot + raw_off:c * slot + raw_off + ce]
            assert np.array_equal(got, want[c][raw_off:raw_off + ce]), f"raw plane of chunk {c} not final"
        for c in np.flatnonzero(done & ~done_seen):
            done_seen[c] = True
            sz = int(sb[c])
            assert sz == want[c].size, f"chunk {c} size {sz} != {want[c].size}"
            assert np.array_equal(ob[c * slot:c * slot + sz], want[c]), f"chunk {c} stream not final at DONE"
    torch.cuda.synchronize()
    say(f"[full] split-send ordering: RAW_READY seen before DONE for {lead} of {chunks} chunks")
    assert lead >= 1


def test_split_send_chunks_read_by_the_copy_engine_at_done(uz):
    """Split-send into device memory (section 3.2.3): a consumer outside the
    GPU's caches -- a NIC, here the copy engine -- may read a chunk's stream
    as soon as its DONE flag is up.  The producer writes the streams to
    device memory and the sizes and flags to pinned host memory; this thread
    polls the flags and, at the first sight of DONE[c], copies the chunk's
    slot to the host on a second stream.  One block of chunk 700 is held
    from the host (uzip_inject_scan_stall, a wait of 100000 polls, about
    0.1 s), so the producer is still running while the other chunks are
    copied; that chunk ends marked invalid, and so may a chunk whose block
    was taken by a wave held up in that wait.  Every copy of a chunk not
    marked invalid is compared with the oracle's stream.  1 GiB of the
    weight-sync buffer, 1 MiB chunks (1024 chunks), 64 KiB blocks."""
    from concurrent.futures import ThreadPoolExecutor
    bb, cb = 65536, 1 << 20
    x = W.weight_sync()
    n = x.size
    ce = cb // 2
    chunks = -(-n // ce)
    held_chunk = 700
    held = held_chunk * (cb // bb) + 3
    t0 = time.time()
    with ThreadPoolExecutor(16) as ex:
        want = list(ex.map(lambda c: ref.compress(x[c * ce:(c + 1) * ce], "bf16", bb), range(chunks)))
    say(f"[full] copy at DONE: {chunks} chunks, oracle {time.time() - t0:.1f}s, block {held} held")
    slot = (uz.uzip_max_compressed_size(uz.BF16, ce, bb) + 255) // 256 * 256
    out = torch.zeros(slot * chunks, dtype=torch.uint8, device="cuda")
    host = torch.zeros(slot * chunks, dtype=torch.uint8).pin_memory()
    sizes = torch.zeros(chunks, dtype=torch.int64).pin_memory()
    flags = torch.zeros(2 * chunks, dtype=torch.int32).pin_memory()
    ws = torch.empty(uz.uzip_workspace_size(uz.OP_CHUNKED, uz.BF16, n, bb, cb), dtype=torch.uint8, device="cuda")
    xt = to_dev(x, "bf16")
    fl = flags.numpy()
    side = torch.cuda.Stream()
    epoch = 9
    torch.cuda.synchronize()
    assert uz.uzip_inject_scan_stall(100000, held) == uz.OK
    try:
        rc = uz.uzip_compress_chunked(xt.data_ptr(), n, uz.BF16, bb, cb, out.data_ptr(), slot, sizes.data_ptr(),
                                      flags.data_ptr(), epoch, ws.data_ptr(), ws.numel(),
                                      torch.cuda.current_stream().cuda_stream)
        assert rc == uz.OK
        copied = np.zeros(chunks, bool)
        pending = []
        lead = 0       # copies seen complete while some DONE flag was still down
        deadline = time.time() + 60
        with torch.cuda.stream(side):
            while not copied.all():
                assert time.time() < deadline, "flags never all raised"
                finished = 0
                while pending and pending[0].query():
                    pending.pop(0)
                    finished += 1
                done = fl[1::2].copy() == epoch     # read after the queries
                if not done.all():
                    lead += finished
                for c in np.flatnonzero(done & ~copied):
                    copied[c] = True
                    host[c * slot:(c + 1) * slot].copy_(out[c * slot:(c + 1) * slot], non_blocking=True)
                    ev = torch.cuda.Event()
                    ev.record(side)
                    pending.append(ev)
        torch.cuda.synchronize()
    finally:
        uz.uzip_inject_scan_stall(0, 0xFFFFFFFF)
    hb, sb = host.numpy(), sizes.numpy()
    assert int(sb[held_chunk]) == 0
    invalid = []
    for c in range(chunks):
        if int(sb[c]) == 0:
            # marked invalid: size 0 and magic 0, in the copy taken at DONE
            assert not hb[c * slot:c * slot + 4].any(), f"chunk {c}: size 0 but magic set"
            invalid.append(c)
            continue
        assert int(sb[c]) == want[c].size, f"chunk {c} size {int(sb[c])} != {want[c].size}"
        assert np.array_equal(hb[c * slot:c * slot + want[c].size], want[c]), f"chunk {c} not in memory at DONE"
    say(f"[full] copy at DONE: {lead} of {chunks} copies complete while the producer ran; "
        f"chunks marked invalid: {invalid}")
    assert len(invalid) <= 64 and lead >= chunks // 2


def test_reduce_full_tensor_reading(uz):
    """The other reading of the activation slices (section 3.4, the fused
    reduce of one rank): each of the 8 inputs is the whole [8192 x 8192]
    bf16 tensor (128 MiB, 2048 blocks), reduced and recompressed in one
    call; stream and reduced tensor against the oracle."""
    from concurrent.futures import ThreadPoolExecutor
    xs = W.reduce_slices(tokens=8192)
    n = xs[0].size
    say(f"[full] reduce, full-tensor reading: 8 x n={n}")
    t0 = time.time()
    with ThreadPoolExecutor(8) as ex:
        streams = list(ex.map(lambda v: ref.compress(v, "bf16", 65536), xs))
    want_s, want_y = ref.reduce(streams, "bf16", n, 65536)
    say(f"[full] reduce full-tensor oracle {time.time() - t0:.1f}s")
    dstreams = [torch.from_numpy(s).cuda() for s in streams]
    del xs
    out, size, raw, status = uz.reduce_fused(dstreams, "bf16", n, 65536)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    got = out[:int(size.item())].cpu().numpy()
    assert np.array_equal(got, want_s), f"reduce stream differs at {first_diff(got, want_s)}"
    assert np.array_equal(raw.cpu().numpy().view(np.uint16), want_y)
