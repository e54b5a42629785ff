"""GPU: uzip_compress_noalloc (the encoder on the library's static device
scratch, for callers that cannot allocate) gives the bytes uzip_compress
gives with a caller workspace, on consecutive calls that reuse the scratch
-- the second smaller than the first and with a block size whose overflow
slots fill the scratch -- and refuses, before any launch, sizes beyond the
scratch's limit."""
import sys

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def uz():
    import paper_2604_17172_amd as m
    return m


def _noalloc(uz, xt, n, code, bb):
    cap = uz.uzip_max_compressed_size(code, n, bb)
    out = torch.empty(cap, dtype=torch.uint8, device="cuda")
    size = torch.zeros(1, dtype=torch.int64, device="cuda")
    rc = uz.uzip_compress_noalloc(xt.data_ptr(), n, code, bb, out.data_ptr(), cap, size.data_ptr(),
                                  torch.cuda.current_stream().cuda_stream)
    assert rc == uz.OK, uz.uzip_status_str(rc)
    return out, size


def test_noalloc_matches_compress_on_consecutive_calls(uz):
    cases = [
        # 48 MiB of the 1 GiB weight-sync buffer, bf16, 64 KiB blocks (768 blocks)
        (W.weight_sync(24 << 20), "bf16", uz.BF16, 65536, np.int16),
        # smaller: fp16 gradients in 256 KiB blocks, whose slots are 117.5 KB
        # each, so the scratch holds fewer slots than the grid would take
        (W.grad_fp16(3 << 20), "fp16", uz.FP16, 262144, np.int16),
        # smaller still, fp32 with a ragged tail
        (W.grad_fp32(300_001), "fp32", uz.FP32, 65536, np.int32),
        # 4 MiB blocks (2 MiB slots) and a partial last block
        (W.normal_bf16((5 << 20) + 999, seed=3), "bf16", uz.BF16, 1 << 22, np.int16),
    ]
    for x, name, code, bb, bits in cases:
        say(f"[noalloc] {name} n={x.size} block={bb}")
        xt = torch.from_numpy(x.view(bits)).cuda()
        want, wsize = uz.compress(xt, bb, dtype=name)
        got, gsize = _noalloc(uz, xt, x.size, code, bb)
        torch.cuda.synchronize()
        n_want, n_got = int(wsize.item()), int(gsize.item())
        assert n_got == n_want > 32
        assert torch.equal(got[:n_got], want[:n_want])
        y, st = uz.decompress(got, name, x.size)
        torch.cuda.synchronize()
        assert int(st.item()) == 0 and np.array_equal(y.cpu().numpy().view(x.dtype), x)


def test_noalloc_limits(uz):
    # more blocks than the scratch's 4,194,304 status words: refused on the host
    n = (4194304 + 1) * 2048
    rc = uz.uzip_compress_noalloc(256, n, uz.BF16, 4096, 512, 1 << 62, None, None)
    assert rc == uz.ENOSPC
    assert uz.uzip_compress_noalloc(256, 1000, uz.BF16, 4096, 520, 1 << 20, None, None) == uz.EINVAL
    # an empty tensor still gives the 32-byte header
    out = torch.empty(64, dtype=torch.uint8, device="cuda")
    size = torch.zeros(1, dtype=torch.int64, device="cuda")
    assert uz.uzip_compress_noalloc(None, 0, uz.BF16, 65536, out.data_ptr(), 64, size.data_ptr(),
                                    torch.cuda.current_stream().cuda_stream) == uz.OK
    torch.cuda.synchronize()
    assert int(size.item()) == 32
