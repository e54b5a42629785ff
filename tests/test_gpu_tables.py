"""GPU parity of the stream-wide table modes (sections 3.3.1 and 3.4): the
table the GPU samples, and every stream the GPU writes with it, equal the
oracle's byte for byte; the GPU decoder takes both the GPU's and the
oracle's streams back to the input.  Through the C ABI (ctypes binding)."""
import sys

import numpy as np
import pytest
import torch

from oracle import ref
import workloads as W

pytestmark = pytest.mark.gpu

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


def host_bits(t, dtype):
    return t.cpu().numpy().view(np.uint16 if EB[dtype] == 2 else np.uint32)


def data(dtype, n, seed):
    if dtype in ("e4m3fn", "e5m2"):
        x = W.normal_fp8_pairs(max(n, 1), dtype, seed=seed)
    elif dtype == "bf16":
        x = W.weight_sync(max(n, 1))[::-1].copy() if seed % 2 else W.normal_bf16(max(n, 1), seed=seed)
    elif dtype == "fp16":
        x = W.grad_fp16(max(n, 1), seed=seed)
    else:
        x = W.grad_fp32(max(n, 1), seed=seed)
    return np.ascontiguousarray(x[:n])


def check(uz, x, dtype, bb, mode, label, table=None):
    say(f"[tables] {label}: dtype={dtype} n={x.size} block={bb} mode={mode}")
    want = ref.compress_table(x, dtype, bb, mode, table)
    t_dev = dev(table.astype(np.uint16).view(np.int16)) if table is not None else None
    out, size = uz.compress_table(dev(x.view(NP_BITS[dtype])), bb, mode, t_dev, dtype=dtype)
    torch.cuda.synchronize()
    got = out[:int(size.item())].cpu().numpy()
    assert got.size == want.size, f"{label}: size {got.size} != oracle {want.size}"
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{label}: {bad.size} bytes differ, first at {bad[0]}")
    for s in (out, dev(want)):
        y, st = uz.decompress_table(s, dtype, x.size, t_dev)
        torch.cuda.synchronize()
        assert int(st.item()) == 0, label
        assert np.array_equal(host_bits(y, dtype), x), f"{label}: decode not lossless"


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32", "e4m3fn", "e5m2"])
def test_sampled_table_matches_oracle(uz, dtype):
    for n in (1, 777, 262144 // EB[dtype], 300_000):
        x = data(dtype, n, seed=n)
        t = uz.build_table(dev(x.view(NP_BITS[dtype])), dtype=dtype)
        torch.cuda.synchronize()
        assert np.array_equal(t.cpu().numpy().view(np.uint16), ref.sampled_table(x, dtype)), (dtype, n)


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32", "e4m3fn", "e5m2"])
@pytest.mark.parametrize("n", [1, 511, 513, 8191, 70_001])
def test_edge_sizes(uz, dtype, n):
    x = data(dtype, n, seed=n + 3)
    for bb in (4096, 65536):
        check(uz, x, dtype, bb, "sampled", f"edge n={n}")


@pytest.mark.parametrize("dtype,bb", [("bf16", 65536), ("bf16", 262144), ("fp32", 262144), ("fp16", 262144),
                                      ("e4m3fn", 65536), ("fp32", 65536), ("bf16", 1 << 22)])
def test_multi_block_streams(uz, dtype, bb):
    n = 5 * (bb // EB[dtype]) + 4321
    check(uz, data(dtype, n, seed=7), dtype, bb, "sampled", "multi-block")


def test_weight_sync_prefix_sampled(uz):
    check(uz, W.weight_sync(1 << 23), "bf16", 65536, "sampled", "weight_sync prefix")


def test_external_table_reused_across_calls(uz):
    """Section 3.4: one table, built from the first call's tensor, codes
    later tensors of the same kind and stays out of their streams."""
    x0 = W.normal_bf16(1 << 20, seed=1)
    t = uz.build_table(dev(x0.view(np.int16)), dtype="bf16")
    torch.cuda.synchronize()
    tab = t.cpu().numpy().view(np.uint16)
    assert np.array_equal(tab, ref.sampled_table(x0, "bf16"))
    for seed in (2, 3):
        check(uz, W.normal_bf16(3 * 32768 + 99, seed=seed), "bf16", 65536, "external", f"reuse {seed}", tab)
    check(uz, W.normal_fp8_pairs(200_000, "e5m2", seed=4), "e5m2", 65536, "external", "fp8 external",
          ref.sampled_table(W.normal_fp8_pairs(200_000, "e5m2", seed=5), "e5m2"))


def test_symbols_outside_the_sample(uz):
    for dtype in ("bf16", "fp32"):
        bits = 8 * EB[dtype]
        ns = 262144 // EB[dtype]
        head = np.full(ns, 0x3F80 if bits == 16 else 0x3F800000, W.random_bits(1, bits).dtype)
        x = np.concatenate([head, W.random_bits(100_003, bits, seed=9), W.random_bits(50_000, bits, seed=1) & 0x80FF])
        check(uz, x, dtype, 65536, "sampled", "outside the sample")


def test_invalid_external_table_codes_nothing(uz):
    say("[tables] invalid external table")
    x = W.normal_bf16(50_000, seed=3)
    bad = ref.sampled_table(x, "bf16").astype(np.uint16)
    bad[5] = 0
    out, size = uz.compress_table(dev(x.view(np.int16)), 65536, "external", dev(bad.view(np.int16)), dtype="bf16")
    torch.cuda.synchronize()
    assert int(size.item()) == 0


def test_modes_are_not_mixed_up(uz):
    say("[tables] mode checks")
    x = W.normal_bf16(70_000, seed=6)
    xt = dev(x.view(np.int16))
    s_plain, _ = uz.compress(xt, 65536, dtype="bf16")
    s_samp, _ = uz.compress_table(xt, 65536, "sampled", dtype="bf16")
    t = uz.build_table(xt, dtype="bf16")
    s_ext, _ = uz.compress_table(xt, 65536, "external", t, dtype="bf16")
    torch.cuda.synchronize()
    for s, fn in ((s_samp, lambda s: uz.decompress(s, "bf16", x.size)),
                  (s_plain, lambda s: uz.decompress_table(s, "bf16", x.size)),
                  (s_ext, lambda s: uz.decompress_table(s, "bf16", x.size))):
        _, st = fn(s)
        torch.cuda.synchronize()
        assert int(st.item()) == uz.ECORRUPT


def test_empty_tensor(uz):
    say("[tables] empty")
    x = np.zeros(0, np.uint16)
    for mode in ("sampled", "external"):
        t = dev(ref.sampled_table(x, "bf16").astype(np.uint16).view(np.int16))
        out, size = uz.compress_table(torch.zeros(0, dtype=torch.int16, device="cuda"), 65536, mode, t, dtype="bf16")
        torch.cuda.synchronize()
        want = ref.compress_table(x, "bf16", 65536, mode, t.cpu().numpy().view(np.uint16))
        assert int(size.item()) == 32 and np.array_equal(out[:32].cpu().numpy(), want)
        y, st = uz.decompress_table(out, "bf16", 0, t)
        torch.cuda.synchronize()
        assert int(st.item()) == 0 and y.numel() == 0


def check_chunked(uz, x, dtype, bb, cb, mode, label, table=None):
    say(f"[tables] {label}: chunked dtype={dtype} n={x.size} block={bb} chunk={cb} mode={mode}")
    t_dev = dev(table.astype(np.uint16).view(np.int16)) if table is not None else None
    xt = dev(x.view(NP_BITS[dtype]))
    out, slot, sizes, flags = uz.compress_chunked_table(xt, bb, cb, mode, t_dev, dtype=dtype, epoch=9)
    torch.cuda.synchronize()
    assert bool((flags == 9).all())
    buf = out.cpu().numpy()
    sz = sizes.cpu().numpy()
    ce = cb // EB[dtype]
    for c, w in enumerate(ref.compress_chunked(x, dtype, bb, cb, mode, table)):
        assert sz[c] == w.size, f"{label}: chunk {c} size {sz[c]} != {w.size}"
        assert np.array_equal(buf[c * slot:c * slot + w.size], w), f"{label}: chunk {c} differs"
        y, st = uz.decompress_table(out[c * slot:(c + 1) * slot], dtype, min(ce, x.size - c * ce), t_dev)
        torch.cuda.synchronize()
        assert int(st.item()) == 0 and np.array_equal(host_bits(y, dtype), x[c * ce:(c + 1) * ce]), label


def test_chunked_sampled_table_per_chunk(uz):
    """Each chunk samples its own first 256 KiB: across the boundary between
    the N(0, 1) embedding and the N(0, 0.02) layers of the weight buffer."""
    x = np.ascontiguousarray(W.weight_sync(136_134_656 + 3_000_000)[-6_000_000:])
    check_chunked(uz, x, "bf16", 65536, 1 << 20, "sampled", "boundary")
    check_chunked(uz, W.grad_fp32(3 * (1 << 18) + 5, seed=2), "fp32", 262144, 1 << 20, "sampled", "fp32")
    check_chunked(uz, W.normal_fp8_pairs(700_001, "e4m3fn", seed=3), "e4m3fn", 4096, 16384, "sampled", "fp8 small")


def test_chunked_external_table(uz):
    x = W.normal_bf16(5 * (1 << 19) + 17, seed=4)
    check_chunked(uz, x, "bf16", 65536, 1 << 20, "external", "external", ref.sampled_table(x, "bf16"))


@pytest.mark.parametrize("n_chunks,chunk_bytes", [(3, 1 << 20), (600, 1 << 18)])
def test_chunked_invalid_external_table(uz, n_chunks, chunk_bytes):
    """An EXTERNAL table whose frequencies do not sum to M codes nothing:
    every chunk is marked invalid (magic and size 0) and both its flags are
    raised, also when the call has more blocks (2400) than the encoder has
    workgroups.  Sizes and slots start as 0xFF bytes, so a chunk left
    untouched would show."""
    ce = chunk_bytes // 2
    say(f"[tables] chunked invalid table: {n_chunks} chunks of {chunk_bytes} bytes")
    x = W.normal_bf16(n_chunks * ce, seed=5)
    bad = ref.sampled_table(x, "bf16").astype(np.uint16)
    bad[0] += 1
    slot = (uz.uzip_max_compressed_size(uz.BF16, ce, 65536) + uz.TABLE_BYTES + 255) // 256 * 256
    out = torch.full((slot * n_chunks,), 0xFF, dtype=torch.uint8, device="cuda")
    sizes = torch.full((n_chunks,), -1, dtype=torch.int64, device="cuda")
    flags = torch.zeros(2 * n_chunks, dtype=torch.int32, device="cuda")
    ws = torch.empty(uz.uzip_workspace_size(uz.OP_CHUNKED_TABLE, uz.BF16, x.size, 65536, chunk_bytes),
                     dtype=torch.uint8, device="cuda")
    xt, t = dev(x.view(np.int16)), dev(bad.view(np.int16))
    rc = uz.uzip_compress_chunked_table(xt.data_ptr(), x.size, uz.BF16, 65536, chunk_bytes, uz.TABLE_EXTERNAL,
                                        t.data_ptr(), out.data_ptr(), slot, sizes.data_ptr(), flags.data_ptr(), 4,
                                        ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert rc == uz.OK
    torch.cuda.synchronize()
    assert bool((sizes == 0).all()) and bool((flags == 4).all())
    magic = out.view(n_chunks, slot)[:, :8].cpu().numpy()
    assert not magic.any()
