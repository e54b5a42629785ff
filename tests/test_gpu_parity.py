"""GPU parity: the HIP library against the CPU oracle, byte for byte.

Sizes here are ones the oracle finishes in seconds while spanning many
codec blocks, several chunks and ragged tails.  Every call goes through the
C ABI (via the ctypes binding).  Integer codec work must be bit-exact; the
fused reduce is a fixed-order binary32 sum, so its output is bit-exact too.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import ref
import workloads as W

pytestmark = pytest.mark.gpu

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


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_dev_bits(x, dtype):
    return dev(x.view(NP_BITS[dtype]))


def host_bits(t, dtype):
    return t.cpu().numpy().view(np.uint16 if EB[dtype] == 2 else np.uint32)


def gpu_compress(uz, x, dtype, bb):
    xt = to_dev_bits(x, dtype)
    out, size = uz.compress(xt, bb, dtype=dtype)
    torch.cuda.synchronize()
    n = int(size.item())
    return out, out[:n].cpu().numpy()


def special_words(dtype, n, seed):
    rng = np.random.default_rng(seed)
    bits = 8 * EB[dtype]
    specials = {"bf16": [0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC0, 0x7F81, 0xFFFF, 0x0001, 0x807F],
                "fp16": [0x0000, 0x8000, 0x7C00, 0xFC00, 0x7E00, 0x7C01, 0xFFFF, 0x0001, 0x83FF],
                "fp32": [0, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 0x7F800001, 0xFFFFFFFF, 1,
                         0x807FFFFF],
                # pairs: NaN/NaN, -0/+0, max/min subnormal, +-inf (e5m2), NaN beside a normal
                "e4m3fn": [0x7F7F, 0x0080, 0xFE7E, 0x0180, 0xFF38, 0x7F01, 0xFFFF, 0x0000, 0x8808],
                "e5m2": [0x7F7F, 0x0080, 0xFC7C, 0x7B03, 0x7CFC, 0x7E3C, 0xFFFF, 0x0000, 0x8484]}[dtype]
    if dtype in ("e4m3fn", "e5m2"):
        x = W.normal_fp8_pairs(n, dtype, seed=seed)
    elif dtype == "bf16":
        x = W.normal_bf16(n, seed=seed)
    elif dtype == "fp16":
        x = W.grad_fp16(n, seed=seed)
    else:
        x = W.grad_fp32(n, seed=seed)
    if n:
        pos = rng.integers(0, n, max(1, n // 20))
        x[pos] = rng.choice(specials, pos.size)
        noise = rng.integers(0, n, max(1, n // 100))
        x[noise] = rng.integers(0, 1 << bits, noise.size, dtype=np.uint64).astype(x.dtype)
    return x


def check_roundtrip(uz, x, dtype, bb, label):
    say(f"[parity] {label}: dtype={dtype} n={x.size} block={bb}")
    want = ref.compress(x, dtype, bb)
    out, got = gpu_compress(uz, x, dtype, bb)
    assert got.size == want.size, f"{label}: size {got.size} != oracle {want.size}"
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{label}: {bad.size} bytes differ, first at {bad[0]}")
    y, status = uz.decompress(out, dtype, x.size)
    torch.cuda.synchronize()
    assert int(status.item()) == 0, label
    assert np.array_equal(host_bits(y, dtype), x), f"{label}: decode not lossless"
    # the GPU decoder on the oracle's stream
    y2, status2 = uz.decompress(dev(want), dtype, x.size)
    torch.cuda.synchronize()
    assert int(status2.item()) == 0 and np.array_equal(host_bits(y2, dtype), x), label


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
@pytest.mark.parametrize("n", [1, 511, 512, 513, 8191, 70_001])
def test_edge_sizes(uz, dtype, n):
    x = special_words(dtype, n, seed=n)
    for bb in (4096, 65536):
        check_roundtrip(uz, x, dtype, bb, f"edge n={n}")


def test_normal_bf16_4MiB_blocks_64k(uz):
    """The 4 MiB N(0, 0.02) bf16 configuration with 64 KiB blocks."""
    x = W.normal_bf16()
    check_roundtrip(uz, x, "bf16", 65536, "normal_bf16_4MiB")


@pytest.mark.parametrize("dtype,bb", [("fp32", 262144), ("fp16", 262144), ("bf16", 262144), ("fp32", 4096)])
def test_grad_and_large_blocks(uz, dtype, bb):
    n = 3 * (bb // EB[dtype]) + 12345
    x = {"fp32": W.grad_fp32, "fp16": W.grad_fp16, "bf16": W.normal_bf16}[dtype](n, seed=3)
    check_roundtrip(uz, x, dtype, bb, f"grad {dtype}")


# 1 MiB and 4 MiB blocks (up to 2^21 symbols a block): the large-block
# encoder's window slides into much bigger overflow slots
@pytest.mark.parametrize("dtype,bb", [("bf16", 1 << 22), ("fp16", 1 << 22), ("fp32", 1 << 22),
                                      ("bf16", 1 << 20), ("fp32", 1 << 20), ("e4m3fn", 1 << 22)])
def test_largest_blocks(uz, dtype, bb):
    n = 3 * (bb // EB[dtype]) + 12345
    x = {"fp32": lambda: W.grad_fp32(n, seed=4), "fp16": lambda: W.grad_fp16(n, seed=4),
         "bf16": lambda: W.normal_bf16(n, seed=4),
         "e4m3fn": lambda: W.normal_fp8_pairs(n, "e4m3fn", sigma=1.0, seed=4)}[dtype]()
    check_roundtrip(uz, x, dtype, bb, f"{bb >> 20} MiB blocks {dtype}")


def test_largest_block_closed_form(uz):
    """A 4 MiB bf16 block of one symbol with one outlier: counts 2^21 - 1
    and 1, table (2047, 1) -- c (M - k) at its largest."""
    x = np.full(1 << 21, 0x3F80, np.uint16)
    x[12345] = 0x4000
    check_roundtrip(uz, x, "bf16", 1 << 22, "4 MiB block, one outlier")


def test_concurrent_calls_on_two_streams(uz):
    """Two compress calls in flight at once on two streams, each with its
    own workspace (calls are re-entrant; a wave only waits on blocks of its
    own call, whose tickets running waves hold), then two decompress calls
    the same way: both equal the oracle's streams and decode back."""
    say("[parity] two streams at once")
    cases = [(W.normal_bf16(1 << 22, seed=61), "bf16", 65536), (W.grad_fp32(1 << 21, seed=62), "fp32", 262144)]
    xts, outs, wss, sizes = [], [], [], []
    for x, d, bb in cases:
        dt = uz.dtype_code(d)
        xts.append(to_dev_bits(x, d))
        outs.append(torch.empty(uz.uzip_max_compressed_size(dt, x.size, bb), dtype=torch.uint8, device="cuda"))
        wss.append(torch.empty(uz.uzip_workspace_size(uz.OP_COMPRESS, dt, x.size, bb), dtype=torch.uint8,
                               device="cuda"))
        sizes.append(torch.zeros(1, dtype=torch.int64, device="cuda"))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for k, (x, d, bb) in enumerate(cases):
        uz.compress(xts[k], bb, dtype=d, out=outs[k], ws=wss[k], size=sizes[k], stream=streams[k])
    torch.cuda.synchronize()
    ys, sts = [], []
    for k, (x, d, bb) in enumerate(cases):
        want = ref.compress(x, d, bb)
        got = outs[k][:int(sizes[k].item())].cpu().numpy()
        assert np.array_equal(got, want), d
        ys.append(torch.empty_like(xts[k]))
        sts.append(torch.zeros(1, dtype=torch.int32, device="cuda"))
    dws = [torch.empty(uz.uzip_workspace_size(uz.OP_DECOMPRESS, uz.dtype_code(d), x.size, bb), dtype=torch.uint8,
                       device="cuda") for x, d, bb in cases]
    torch.cuda.synchronize()
    for k, (x, d, bb) in enumerate(cases):
        uz.decompress(outs[k], d, x.size, out=ys[k], ws=dws[k], status=sts[k], stream=streams[k])
    torch.cuda.synchronize()
    for k, (x, d, bb) in enumerate(cases):
        assert int(sts[k].item()) == 0
        assert np.array_equal(host_bits(ys[k], d), x), d


def test_weight_sync_prefix(uz):
    x = W.weight_sync(1 << 23)   # embedding + first layers: N(0,1), N(0,0.02), N(1,0.05) regions
    check_roundtrip(uz, x, "bf16", 65536, "weight_sync prefix")
    x = W.weight_sync(136_134_656 + 2_000_000)[-6_000_000:]   # across the embedding/layer boundary
    check_roundtrip(uz, np.ascontiguousarray(x), "bf16", 65536, "weight_sync boundary")


def test_kv_cache_small(uz):
    x = W.kv_cache(layers=2, tokens=512)
    check_roundtrip(uz, x, "bf16", 65536, "kv_cache small")


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
def test_all_stored_random_bits(uz, dtype):
    x = W.random_bits(200_003, 8 * EB[dtype], seed=9)
    check_roundtrip(uz, x, dtype, 65536, "random bits")


@pytest.mark.parametrize("dtype,bb", [("bf16", 16384), ("e4m3fn", 16384), ("fp32", 65536)])
def test_stored_and_coded_blocks_interleaved(uz, dtype, bb):
    """Runs of incompressible blocks between coded ones in one stream: a
    block's section is written after the next block's first pass, from the
    staging area for a coded block and re-read from the input for a STORED
    one, and the look-back fills in the inclusive prefixes of both kinds."""
    per = bb // EB[dtype]
    n_blocks = 600
    n = n_blocks * per - 123
    x = special_words(dtype, n, seed=31)
    noise = W.random_bits(n, 8 * EB[dtype], seed=32).astype(x.dtype)
    rng = np.random.default_rng(33)
    for b in range(n_blocks):
        if rng.random() < 0.3:  # about 30% of the blocks: random bits, so STORED
            x[b * per:(b + 1) * per] = noise[b * per:(b + 1) * per]
    check_roundtrip(uz, x, dtype, bb, "stored and coded blocks interleaved")


def test_single_symbol_blocks(uz):
    x = np.full(3 * 32768 + 5, 0x3F80, np.uint16)
    x[40000:40010] = 0x4000
    check_roundtrip(uz, x, "bf16", 65536, "constant blocks")


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
def test_stored_coded_boundary(uz, dtype):
    """A one-symbol block codes to 290 bytes: STORED at 289 and 290
    elements, CODED at 291 (the strict inequality of the STORED rule)."""
    one = {"bf16": 0x3F80, "fp16": 0x3C00, "fp32": 0x3F800000}[dtype]
    for n in (289, 290, 291):
        x = np.full(n, one, np.uint32 if dtype == "fp32" else np.uint16)
        check_roundtrip(uz, x, dtype, 65536, f"boundary n={n}")


def test_uniform_bf16(uz):
    x = W.uniform_bf16(1 << 21, seed=11)
    check_roundtrip(uz, x, "bf16", 65536, "uniform bf16")


def test_empty_tensor(uz):
    say("[parity] empty")
    x = np.zeros(0, np.uint16)
    out, size = uz.compress(torch.zeros(0, dtype=torch.int16, device="cuda"), 65536, dtype="bf16")
    torch.cuda.synchronize()
    assert int(size.item()) == 32
    assert np.array_equal(out[:32].cpu().numpy(), ref.compress(x, "bf16", 65536))
    y, status = uz.decompress(out, "bf16", 0)
    torch.cuda.synchronize()
    assert int(status.item()) == 0 and y.numel() == 0


# ---------------------------------------------------------- FP8 pairs (section 4.1)
@pytest.mark.parametrize("dtype", ["e4m3fn", "e5m2"])
@pytest.mark.parametrize("n", [1, 511, 513, 8191, 70_001])
def test_fp8_edge_sizes(uz, dtype, n):
    x = special_words(dtype, n, seed=n + 7)
    for bb in (4096, 65536):
        check_roundtrip(uz, x, dtype, bb, f"fp8 edge n={n}")


@pytest.mark.parametrize("dtype", ["e4m3fn", "e5m2"])
@pytest.mark.parametrize("sigma,bb", [(1.0, 65536), (0.02, 65536), (1.0, 262144), (0.3, 4096)])
def test_fp8_normal_pairs(uz, dtype, sigma, bb):
    """4 MiB of FP8 N(0, sigma^2) values (2 Mi pairs), several block sizes."""
    x = W.normal_fp8_pairs(1 << 21, dtype, sigma=sigma, seed=21)
    check_roundtrip(uz, x, dtype, bb, f"fp8 normal sigma={sigma}")


@pytest.mark.parametrize("dtype", ["e4m3fn", "e5m2"])
def test_fp8_random_bits_stored(uz, dtype):
    x = W.random_bits(200_003, 16, seed=19)
    check_roundtrip(uz, x, dtype, 65536, "fp8 random bits")


@pytest.mark.parametrize("dtype", ["e4m3fn", "e5m2"])
def test_fp8_tensor_input_counts_pairs(uz, dtype):
    """A float8 tensor is taken as pairs: the same stream as its int16 view."""
    say(f"[parity] fp8 tensor input {dtype}")
    x = W.normal_fp8_pairs(100_001, dtype, seed=4)
    f8 = dev(x.view(np.uint8)).view(W.FP8_TORCH[dtype])
    out, size = uz.compress(f8, 65536)
    torch.cuda.synchronize()
    got = out[:int(size.item())].cpu().numpy()
    assert np.array_equal(got, ref.compress(x, dtype, 65536))
    with pytest.raises(ValueError):
        uz.compress(f8[:-1].clone(), 65536)


# (4096, 16384): 66 chunks and 264 blocks, the XCD-local producer
@pytest.mark.parametrize("bb,cb,n", [(65536, 1 << 20, 3 * (1 << 19) + 999), (4096, 16384, 66 * 8192 - 7)])
@pytest.mark.parametrize("dtype", ["e4m3fn", "e5m2"])
def test_fp8_chunked_producer(uz, dtype, bb, cb, n):
    say(f"[parity] fp8 chunked dtype={dtype} n={n} block={bb} chunk={cb}")
    x = special_words(dtype, n, seed=41)
    out, slot, sizes, flags = uz.compress_chunked(to_dev_bits(x, dtype), bb, cb, dtype=dtype, epoch=5)
    torch.cuda.synchronize()
    assert np.all(flags.cpu().numpy() == 5)
    sz = sizes.cpu().numpy()
    buf = out.cpu().numpy()
    for c, w in enumerate(ref.compress_chunked(x, dtype, bb, cb)):
        assert sz[c] == w.size and np.array_equal(buf[c * slot:c * slot + w.size], w), f"chunk {c}"


def test_fp8_stream_dtype_must_match(uz):
    """An e4m3fn stream decoded as e5m2 (or bf16) is reported corrupt."""
    say("[parity] fp8 dtype mismatch")
    x = W.normal_fp8_pairs(10_000, "e4m3fn", seed=2)
    out, _ = gpu_compress(uz, x, "e4m3fn", 65536)
    for other in ("e5m2", "bf16"):
        _, st = uz.decompress(out, other, x.size)
        torch.cuda.synchronize()
        assert int(st.item()) == uz.ECORRUPT


# ---------------------------------------------------------- split-send producer
# The last five run the XCD-local producer on a chip of 8 XCDs (at least 64
# chunks, or a multiple of 8, and 256 blocks): each chunk coded on one XCD,
# flags raised after a write-back of that XCD's L2.
@pytest.mark.parametrize("dtype,bb,cb,n", [("bf16", 65536, 1 << 20, 3 * (1 << 19) + 77_777),
                                           ("fp32", 262144, 1 << 20, 2 * (1 << 18) + 1),
                                           ("fp16", 4096, 16384, 100_000),
                                           ("bf16", 4096, 16384, 64 * 8192 + 777),
                                           ("fp16", 4096, 16384, 70 * 8192 + 1234),
                                           ("fp32", 16384, 65536, 66 * 16384 + 5),
                                           ("bf16", 4096, 131072, 8 * 65536),
                                           ("fp16", 4096, 65536, 24 * 32768 - 100),
                                           ("bf16", 1 << 22, 1 << 22, 3 * (1 << 21) + 99),
                                           ("fp32", 1 << 20, 1 << 22, 2 * (1 << 20) + 5)])
def test_chunked_producer_matches_per_chunk_oracle(uz, dtype, bb, cb, n):
    say(f"[parity] chunked dtype={dtype} n={n} block={bb} chunk={cb}")
    x = special_words(dtype, n, seed=31)
    xt = to_dev_bits(x, dtype)
    out, slot, sizes, flags = uz.compress_chunked(xt, bb, cb, dtype=dtype, epoch=7)
    torch.cuda.synchronize()
    want = ref.compress_chunked(x, dtype, bb, cb)
    sz = sizes.cpu().numpy()
    fl = flags.cpu().numpy()
    assert np.all(fl == 7)
    buf = out.cpu().numpy()
    ce = cb // EB[dtype]
    for c, w in enumerate(want):
        assert sz[c] == w.size
        assert np.array_equal(buf[c * slot:c * slot + w.size], w), f"chunk {c}"
        y, st = uz.decompress(out[c * slot:(c + 1) * slot], dtype, min(ce, n - c * ce))
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        assert np.array_equal(host_bits(y, dtype), x[c * ce:(c + 1) * ce])


def test_chunked_flags_host_mapped(uz):
    """Flags in pinned host memory: the device publishes them with
    system-scope release stores; the host sees the final values."""
    say("[parity] chunked host-mapped flags")
    x = W.normal_bf16(5 * (1 << 19), seed=5)
    xt = to_dev_bits(x, "bf16")
    flags = torch.zeros(2 * 5, dtype=torch.int32).pin_memory()
    out, slot, sizes, fl = uz.compress_chunked(xt, 65536, 1 << 20, dtype="bf16", epoch=3, flags=flags)
    torch.cuda.synchronize()
    assert np.all(flags.numpy() == 3)
    want = ref.compress_chunked(x, "bf16", 65536, 1 << 20)
    buf = out.cpu().numpy()
    for c, w in enumerate(want):
        assert np.array_equal(buf[c * slot:c * slot + w.size], w)


# ---------------------------------------------------------- fused reduce
@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
@pytest.mark.parametrize("n_in", [1, 2, 8])
def test_reduce_matches_oracle(uz, dtype, n_in):
    n = 150_001
    bb = 65536 if dtype != "fp32" else 262144
    say(f"[parity] reduce dtype={dtype} n_in={n_in} n={n}")
    xs = [special_words(dtype, n, seed=200 + i) for i in range(n_in)]
    streams = [ref.compress(v, dtype, bb) for v in xs]
    local = special_words(dtype, n, seed=77)
    for use_local in (False, True):
        for want_raw in (True, False):
            dstreams = [dev(s) for s in streams]
            out, size, raw, status = uz.reduce_fused(dstreams, dtype, n, bb,
                                                     local=to_dev_bits(local, dtype) if use_local else None,
                                                     want_raw=want_raw)
            torch.cuda.synchronize()
            want_s, want_y = ref.reduce(streams, dtype, n, bb, local=local if use_local else None)
            assert int(status.item()) == 0
            got = out[:int(size.item())].cpu().numpy()
            assert np.array_equal(got, want_s), (use_local, want_raw)
            if want_raw:
                assert np.array_equal(host_bits(raw, dtype), want_y)


@pytest.mark.parametrize("dtype,bb", [("bf16", 1 << 20), ("fp32", 1 << 22)])
def test_reduce_largest_blocks(uz, dtype, bb):
    """Blocks of 1 MiB and 4 MiB: the decode-reduce kernel and the separate
    coding pass (such a block's words do not fit the fused kernel's LDS)."""
    n = 2 * (bb // EB[dtype]) + 999
    say(f"[parity] reduce dtype={dtype} n={n} block={bb}")
    xs = [special_words(dtype, n, seed=300 + i) for i in range(3)]
    streams = [ref.compress(v, dtype, bb) for v in xs]
    out, size, raw, status = uz.reduce_fused([dev(v) for v in streams], dtype, n, bb, want_raw=True)
    torch.cuda.synchronize()
    want_s, want_y = ref.reduce(streams, dtype, n, bb)
    assert int(status.item()) == 0
    assert np.array_equal(out[:int(size.item())].cpu().numpy(), want_s)
    assert np.array_equal(host_bits(raw, dtype), want_y)


@pytest.mark.parametrize("dtype,bb", [("bf16", 16384), ("bf16", 4096), ("fp16", 8192), ("fp32", 16384)])
def test_reduce_small_blocks(uz, dtype, bb):
    """Blocks down to the 4 KiB minimum: many more blocks per share than
    64 KiB blocks give, and a ragged last block."""
    n = 200_003
    n_in = 5
    say(f"[parity] reduce small blocks dtype={dtype} block={bb} n_in={n_in} n={n}")
    xs = [special_words(dtype, n, seed=400 + i) for i in range(n_in)]
    streams = [ref.compress(v, dtype, bb) for v in xs]
    local = special_words(dtype, n, seed=499)
    out, size, raw, status = uz.reduce_fused([dev(t) for t in streams], dtype, n, bb, local=to_dev_bits(local, dtype))
    torch.cuda.synchronize()
    want_s, want_y = ref.reduce(streams, dtype, n, bb, local=local)
    assert int(status.item()) == 0
    assert np.array_equal(out[:int(size.item())].cpu().numpy(), want_s)
    assert np.array_equal(host_bits(raw, dtype), want_y)


def test_reduce_sixteen_inputs_with_stored_blocks(uz):
    n = 70_000
    say("[parity] reduce n_in=16")
    xs = [special_words("bf16", n, seed=300 + i) for i in range(15)] + [W.random_bits(n, 16, seed=5)]
    streams = [ref.compress(v, "bf16", 65536) for v in xs]
    out, size, raw, status = uz.reduce_fused([dev(s) for s in streams], "bf16", n, 65536)
    torch.cuda.synchronize()
    want_s, want_y = ref.reduce(streams, "bf16", n, 65536)
    assert int(status.item()) == 0
    assert np.array_equal(out[:int(size.item())].cpu().numpy(), want_s)
    assert np.array_equal(host_bits(raw, "bf16"), want_y)


def test_reduce_two_uneven_input_groups(uz):
    """Eleven inputs: decoded in a group of eight and a group of three; the
    fp32 partial sums carry over between the groups in input order."""
    n = 90_001
    say("[parity] reduce n_in=11")
    xs = [special_words("fp16", n, seed=400 + i) for i in range(11)]
    streams = [ref.compress(v, "fp16", 65536) for v in xs]
    local = special_words("fp16", n, seed=78)
    out, size, raw, status = uz.reduce_fused([dev(s) for s in streams], "fp16", n, 65536,
                                             local=to_dev_bits(local, "fp16"))
    torch.cuda.synchronize()
    want_s, want_y = ref.reduce(streams, "fp16", n, 65536, local=local)
    assert int(status.item()) == 0
    assert np.array_equal(out[:int(size.item())].cpu().numpy(), want_s)
    assert np.array_equal(host_bits(raw, "fp16"), want_y)


def test_reduce_eight_slices_share(uz):
    """Eight bf16 shares [tokens x 8192] with per-token scales (64 tokens)."""
    xs = W.reduce_slices(n_in=8, tokens=64, hidden=8192, seed=5)
    n = xs[0].size
    say("[parity] reduce 8 slices")
    streams = [ref.compress(v, "bf16", 65536) for v in xs]
    out, size, raw, status = uz.reduce_fused([dev(s) for s in streams], "bf16", n, 65536)
    torch.cuda.synchronize()
    want_s, want_y = ref.reduce(streams, "bf16", n, 65536)
    assert int(status.item()) == 0
    assert np.array_equal(out[:int(size.item())].cpu().numpy(), want_s)
    assert np.array_equal(host_bits(raw, "bf16"), want_y)


# ---------------------------------------------------------- corrupt streams
def test_corrupt_streams_reported(uz):
    """Header, directory and truncation damage is reported through the
    device status word; the decoder's reads stay inside the stream."""
    say("[parity] corrupt streams")
    x = W.normal_bf16(100_000, seed=8)
    good = ref.compress(x, "bf16", 4096)
    cases = []
    for off in (0, 4, 5, 6, 7, 8, 12, 16, 24, 32, 36):
        bad = good.copy()
        bad[off] ^= 0x5A
        cases.append((f"byte {off}", bad, good.size))
    cases.append(("truncated", good, good.size - 16))
    cases.append(("tiny", good, 8))
    for label, s, nbytes in cases:
        y, status = uz.decompress(dev(s), "bf16", 100_000, in_bytes=nbytes)
        torch.cuda.synchronize()
        assert int(status.item()) == uz.ECORRUPT, label
    # payload damage: never out of bounds; mostly detected
    rng = np.random.default_rng(3)
    detected = 0
    for _ in range(40):
        bad = good.copy()
        pos = int(rng.integers(100, good.size))
        bad[pos] ^= 1 << int(rng.integers(0, 8))
        y, status = uz.decompress(dev(bad), "bf16", 100_000)
        torch.cuda.synchronize()
        detected += int(status.item()) != 0 or not np.array_equal(host_bits(y, "bf16"), x)
    assert detected >= 30


def test_reduce_rejects_mismatched_inputs(uz):
    say("[parity] reduce mismatch")
    a = W.normal_bf16(50_000, seed=1)
    s1 = ref.compress(a, "bf16", 65536)
    s2 = ref.compress(a[:40_000], "bf16", 65536)
    out, size, raw, status = uz.reduce_fused([dev(s1), dev(s2)], "bf16", 50_000, 65536)
    torch.cuda.synchronize()
    assert int(status.item()) == uz.ECORRUPT


@pytest.mark.parametrize("dtype,spread", [("bf16", 64), ("bf16", 200), ("fp16", 30)])
def test_high_entropy_blocks_spill_staging(uz, dtype, spread):
    """Exponents spread over many values: a 64 KiB block codes to more words
    than the encoder's LDS staging window holds (it spills to the
    workgroup's overflow slot) while the block still stays CODED (spread 64)
    or turns STORED part way (spread 200)."""
    rng = np.random.default_rng(spread)
    n = 5 * 32768 + 999
    if dtype == "bf16":
        e = rng.integers(127 - spread // 2, 127 + spread // 2, n)
        x = ((e << 7) | rng.integers(0, 128, n) | (rng.integers(0, 2, n) << 15)).astype(np.uint16)
    else:
        e = rng.integers(1, spread + 1, n)
        x = ((e << 10) | rng.integers(0, 1024, n) | (rng.integers(0, 2, n) << 15)).astype(np.uint16)
    check_roundtrip(uz, x, dtype, 65536, f"spread {spread}")


# --------------------------------------------- tables whose largest counts tie
# Blocks whose maximal exponent counts tie and whose table remainder is
# nonzero (the remainder goes to the smallest tied symbol; the closed forms
# are in test_oracle_ties.py): the GPU's table must match the oracle's.
TIE_BLOCKS = [{120: 12000, 121: 12000, 122: 8768},
              {100: 2768, 125: 10000, 130: 10000, 140: 10000},
              {60: 16384, 61: 16384},
              {7: 6000, 8: 6000, 9: 6000, 10: 6000, 11: 6000, 12: 2768}]


def test_tied_block_tables_bf16(uz):
    x = np.concatenate([W.exponent_multiset(c, "bf16", seed=40 + i) for i, c in enumerate(TIE_BLOCKS)])
    x = np.concatenate([x, W.normal_bf16(20_000, seed=44)])
    check_roundtrip(uz, x, "bf16", 65536, "tied maxima, 64 KiB blocks")
    check_roundtrip(uz, x, "bf16", 16384, "tied maxima, 16 KiB blocks")


def test_tied_block_table_fp32(uz):
    x = np.concatenate([W.exponent_multiset({3: 224, 126: 400, 127: 400}, "fp32", seed=45 + i) for i in range(9)])
    check_roundtrip(uz, x, "fp32", 4096, "tied maxima, fp32 4 KiB blocks")


def test_tied_stream_wide_table(uz):
    x = W.exponent_multiset({120: 50000, 121: 50000, 122: 31072}, "bf16", seed=33)
    x = np.concatenate([x, W.normal_bf16(70_000, seed=46)])
    say(f"[parity] sampled table with tied maxima: n={x.size}")
    want = ref.compress_table(x, "bf16", 65536, "sampled")
    out, size = uz.compress_table(to_dev_bits(x, "bf16"), 65536, "sampled", dtype="bf16")
    torch.cuda.synchronize()
    got = out[: int(size.item())].cpu().numpy()
    assert np.array_equal(got, want)
    tab = uz.build_table(to_dev_bits(x, "bf16"), dtype="bf16")
    torch.cuda.synchronize()
    assert np.array_equal(tab.cpu().numpy().view(np.uint16).astype(np.uint32), ref.sampled_table(x, "bf16"))
