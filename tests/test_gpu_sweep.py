"""GPU parity over a seeded sweep of shapes: element type, length, block
and chunk size, value distribution and table mode drawn from a fixed seed,
each case compared byte for byte with the oracle and decoded back through
every decode entry point that applies (whole stream, chunk streams in one
launch, a stream-wide table).  Sizes stay where the oracle takes well under
a second per case; the cases span single partial blocks, ragged tails,
several chunks, STORED and CODED blocks side by side."""
import sys

import numpy as np
import pytest
import torch

from oracle import ref
import workloads as W

pytestmark = pytest.mark.gpu

EB = {"bf16": 2, "fp16": 2, "fp32": 4, "e4m3fn": 2, "e5m2": 2}
NP_BITS = {"bf16": np.int16, "fp16": np.int16, "fp32": np.int32, "e4m3fn": np.int16, "e5m2": np.int16}
DTYPES = ["bf16", "fp16", "fp32", "e4m3fn", "e5m2"]


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


def case(seed):
    """(dtype, n, block_bytes, chunk_bytes, kind, data) of sweep case `seed`."""
    rng = np.random.default_rng(1000 + seed)
    dtype = DTYPES[seed % len(DTYPES)]
    # 4 KiB .. 256 KiB; seeds from 30 on: 512 KiB .. 4 MiB
    bb = int(2 ** (rng.integers(12, 19) if seed < 30 else rng.integers(19, 23)))
    chunk = bb * int(2 ** rng.integers(0, 4))           # 1 .. 8 blocks a chunk
    n = int(np.exp(rng.uniform(0, np.log(3_000_000))))  # 1 .. 3 M elements, log-uniform
    kind = ("normal", "wide", "bits", "mixed")[int(rng.integers(0, 4))]
    bits = 8 * EB[dtype]
    if dtype in ("e4m3fn", "e5m2"):
        x = W.normal_fp8_pairs(n, dtype, sigma=float(rng.choice([0.05, 1.0, 40.0])), seed=seed)
    elif kind == "bits":
        x = W.random_bits(n, bits, seed=seed)
    elif dtype == "bf16":
        x = W.normal_bf16(n, sigma=0.02 if kind == "normal" else 3.0, seed=seed)
    elif dtype == "fp16":
        x = W.grad_fp16(n, seed=seed)
    else:
        x = W.grad_fp32(n, seed=seed)
    x = np.ascontiguousarray(x[:n])
    if kind == "mixed" and n > 64:
        # stretches of random bits (STORED blocks) between coded ones
        r = W.random_bits(n, bits, seed=seed + 1)
        lo = int(rng.integers(0, n // 2))
        x[lo:lo + n // 3] = r[lo:lo + n // 3].astype(x.dtype)
    return dtype, n, bb, chunk, kind, x


@pytest.mark.parametrize("seed", range(40))
def test_sweep_matches_oracle(uz, seed):
    dtype, n, bb, chunk, kind, x = case(seed)
    say(f"[sweep] seed={seed} dtype={dtype} n={n} block={bb} chunk={chunk} kind={kind}")
    xt = dev(x.view(NP_BITS[dtype]))
    # whole stream
    want = ref.compress(x, dtype, bb)
    out, size = uz.compress(xt, bb, dtype=dtype, check=True)
    got = out[:int(size.item())].cpu().numpy()
    assert got.size == want.size and np.array_equal(got, want), f"seed {seed}: stream differs"
    y, st = uz.decompress(dev(want), dtype, n)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and np.array_equal(host_bits(y, dtype), x)
    # split-send producer, then all its chunk streams in one launch
    cout, slot, sizes, flags = uz.compress_chunked(xt, bb, chunk, dtype=dtype, epoch=seed + 1, check=True)
    sz = sizes.cpu().numpy()
    buf = cout.cpu().numpy()
    for c, w in enumerate(ref.compress_chunked(x, dtype, bb, chunk)):
        assert sz[c] == w.size and np.array_equal(buf[c * slot:c * slot + w.size], w), f"seed {seed}: chunk {c}"
    yc, stc = uz.decompress_chunked(cout, slot, dtype, n, bb, chunk)
    torch.cuda.synchronize()
    assert int(stc.item()) == 0 and np.array_equal(host_bits(yc, dtype), x)
    # one sampled table for the stream
    wt = ref.compress_table(x, dtype, bb, "sampled")
    tout, tsize = uz.compress_table(xt, bb, "sampled", dtype=dtype)
    gt = tout[:int(tsize.item())].cpu().numpy()
    assert gt.size == wt.size and np.array_equal(gt, wt), f"seed {seed}: sampled-table stream differs"
    yt, stt = uz.decompress_table(tout, dtype, n)
    torch.cuda.synchronize()
    assert int(stt.item()) == 0 and np.array_equal(host_bits(yt, dtype), x)


def reduce_case(seed):
    rng = np.random.default_rng(5000 + seed)
    dtype = ("bf16", "fp16", "fp32")[seed % 3]
    n_in = int(rng.integers(1, 17))
    bb = int(2 ** (rng.integers(12, 19) if seed < 15 else rng.integers(19, 23)))   # from seed 15: 512 KiB .. 4 MiB
    n = int(np.exp(rng.uniform(0, np.log(400_000))))
    gen = {"bf16": lambda k: W.normal_bf16(n, sigma=float(rng.choice([0.02, 1.0])), seed=k),
           "fp16": lambda k: W.grad_fp16(n, seed=k), "fp32": lambda k: W.grad_fp32(n, seed=k)}[dtype]
    xs = [np.ascontiguousarray(gen(100 * seed + i)[:n]) for i in range(n_in)]
    local = np.ascontiguousarray(gen(100 * seed + 99)[:n]) if rng.integers(0, 2) else None
    return dtype, n_in, n, bb, xs, local


@pytest.mark.parametrize("seed", range(20))
def test_reduce_sweep_matches_oracle(uz, seed):
    dtype, n_in, n, bb, xs, local = reduce_case(seed)
    say(f"[sweep] reduce seed={seed} dtype={dtype} n_in={n_in} n={n} block={bb} local={local is not None}")
    streams = [ref.compress(v, dtype, bb) for v in xs]
    want_s, want_y = ref.reduce(streams, dtype, n, bb, local=local)
    out, size, raw, status = uz.reduce_fused([dev(s) for s in streams], dtype, n, bb,
                                             local=dev(local.view(NP_BITS[dtype])) if local is not None else None,
                                             check=True)
    got = out[:int(size.item())].cpu().numpy()
    assert got.size == want_s.size and np.array_equal(got, want_s), f"seed {seed}: output stream differs"
    assert np.array_equal(host_bits(raw, dtype), np.asarray(want_y).view(host_bits(raw, dtype).dtype)[:n])
