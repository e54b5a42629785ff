"""Pins of the tables' remainder rule, and a wide C-vs-Python cross-check.

The table reading (section 3.3.1 leaves normalisation open) gives the
remainder M - sum(f) to the most frequent symbol and, when several symbols
share the largest count, to the smallest of them.  The closed forms below
are worked out by hand from that rule on blocks whose largest counts tie
and whose remainder is nonzero, so sending the remainder to the largest
tied symbol, to the smallest present symbol or dropping it fails them.

The cross-check runs the C oracle and the independent Python model
(oracle/model.py) on more than ten thousand small streams -- a third of
them built with tied maxima -- and on every block of the 4 MiB bf16
workload; it pins the C code against slips in writing the reading down.
"""
import os
import struct
from concurrent.futures import ProcessPoolExecutor

import numpy as np
import pytest

from oracle import model, ref
import workloads as W

EB = {"bf16": 2, "fp16": 2, "fp32": 4, "e4m3fn": 2, "e5m2": 2}


def pad16(v):
    return -(-v // 16) * 16


def sections(stream: np.ndarray, dtype: str, n: int, table_bytes: int = 0):
    """(stored flag, section bytes) of every block of a stream."""
    b = stream.tobytes()
    nb = struct.unpack_from("<I", b, 12)[0]
    raw_off = 32 + pad16(4 * nb) + table_bytes
    coded = raw_off + pad16((EB[dtype] - 1) * n)
    out, start = [], 0
    for i in range(nb):
        d = struct.unpack_from("<I", b, 32 + 4 * i)[0]
        end = 16 * (d & 0x7FFFFFFF)
        out.append((bool(d >> 31), b[coded + start:coded + end]))
        start = end
    return out


def coded_table(sec: bytes) -> dict:
    """{symbol: f} stored in a CODED section (bitmap after the 64 states)."""
    present = [s for s in range(256) if sec[256 + s // 8] >> (s % 8) & 1]
    return dict(zip(present, struct.unpack_from(f"<{len(present)}H", sec, 288)))


# ------------------------------------------------------ per-block tables
# 64 KiB bf16 block (32768 symbols), k = 3, M - k = 2045:
#   f(12000) = 1 + floor(12000 * 2045 / 32768) = 1 + 748 = 749
#   f(8768)  = 1 + floor(8768 * 2045 / 32768)  = 1 + 547 = 548
#   remainder 2048 - (749 + 749 + 548) = 2 -> the smaller tied exponent, 120
TIE2 = ({120: 12000, 121: 12000, 122: 8768}, {120: 751, 121: 749, 122: 548})
# k = 4, M - k = 2044:  f(10000) = 1 + 623 = 624,  f(2768) = 1 + 172 = 173;
# remainder 2048 - (3 * 624 + 173) = 3 -> 125, the smallest of the three
# tied exponents (100 is smaller but less frequent)
TIE3 = ({100: 2768, 125: 10000, 130: 10000, 140: 10000}, {100: 173, 125: 627, 130: 624, 140: 624})
# fp32, 4 KiB block (1024 symbols), k = 3, M - k = 2045:
#   f(400) = 1 + floor(400 * 2045 / 1024) = 1 + 798 = 799
#   f(224) = 1 + floor(224 * 2045 / 1024) = 1 + 447 = 448
#   remainder 2048 - (799 + 799 + 448) = 2 -> 126
TIE_FP32 = ({3: 224, 126: 400, 127: 400}, {3: 448, 126: 801, 127: 799})


@pytest.mark.parametrize("case", [TIE2, TIE3], ids=["two_tied", "three_tied"])
def test_block_table_tie_goes_to_the_smallest_symbol(case):
    counts, want = case
    x = W.exponent_multiset(counts, "bf16", seed=31)
    assert x.size == 32768
    s = ref.compress(x, "bf16", 65536)
    [(stored, sec)] = sections(s, "bf16", x.size)
    assert not stored
    assert coded_table(sec) == want
    assert np.array_equal(ref.decompress(s, "bf16", x.size), x)
    # the table routine itself on the same counts
    c = np.zeros(256, np.uint32)
    for e, v in counts.items():
        c[e] = v
    f, _ = ref.build_table(c, 32768)
    assert {int(e): int(f[e]) for e in np.flatnonzero(f)} == want


def test_block_table_tie_fp32():
    counts, want = TIE_FP32
    x = W.exponent_multiset(counts, "fp32", seed=32)
    s = ref.compress(x, "fp32", 4096)
    [(stored, sec)] = sections(s, "fp32", x.size)
    assert not stored and coded_table(sec) == want


# ------------------------------------------------------ stream-wide tables
# SAMPLED: the sample is the first 256 KiB (131072 bf16 symbols), every
# symbol kept (M - 256 = 1792):
#   f(50000) = 1 + floor(50000 * 1792 / 131072) = 1 + 683 = 684
#   f(31072) = 1 + floor(31072 * 1792 / 131072) = 1 + 424 = 425
#   253 unseen symbols: 1 each
#   remainder 2048 - (2 * 684 + 425 + 253) = 2 -> 120
SAMPLE_TIE = {120: 50000, 121: 50000, 122: 31072}


def test_stream_wide_table_tie_goes_to_the_smallest_symbol():
    x = W.exponent_multiset(SAMPLE_TIE, "bf16", seed=33)
    s = ref.compress_table(x, "bf16", 65536, "sampled")
    nb = struct.unpack_from("<I", s.tobytes(), 12)[0]
    f = np.frombuffer(s.tobytes(), np.uint16, 256, 32 + pad16(4 * nb))
    want = np.ones(256, np.int64)
    want[120], want[121], want[122] = 686, 684, 425
    assert np.array_equal(f.astype(np.int64), want)
    assert np.array_equal(ref.decompress_table(s, "bf16", x.size), x)


# ------------------------------------------------------ C oracle vs Python model
def _tied_stream(rng: np.random.Generator, dtype: str, n: int) -> np.ndarray:
    """n values whose exponents have two or more tied maximal counts."""
    k = int(rng.integers(2, 9))
    exps = rng.choice(np.arange(1, 255), k, replace=False)
    ties = int(rng.integers(2, k + 1))
    top = max(n // (ties + 1), 1)
    counts = {int(e): top for e in exps[:ties]}
    rest = n - top * ties
    for e in exps[ties:]:
        if rest <= 0:
            break
        c = int(rng.integers(1, max(top, 2)))
        c = min(c, rest, top - 1) if top > 1 else 0
        if c > 0:
            counts[int(e)] = c
            rest -= c
    if rest > 0:   # fill with further tied maxima, never a larger count
        for e in range(1, 255):
            if rest <= 0:
                break
            if e not in counts:
                c = min(rest, top)
                counts[e] = c
                rest -= c
    return W.exponent_multiset(counts, dtype, seed=int(rng.integers(1 << 30)))[:n]


def _one(seed: int):
    rng = np.random.default_rng([seed, 7])
    kind = seed % 3
    if kind == 0:
        dtype = ("bf16", "fp32")[seed % 2]
        n = int(rng.integers(300, 1100))
        x = _tied_stream(rng, dtype, n)
        bb = 4096 if rng.random() < 0.7 else 8192
    else:
        dtype = ["bf16", "fp16", "fp32", "e4m3fn", "e5m2"][seed % 5]
        n = int(rng.integers(0, 1200))
        bits = 8 * EB[dtype]
        if kind == 1:
            x = W.random_bits(n, bits, seed=seed)
        else:   # narrow exponent range: mostly CODED blocks
            v = rng.standard_normal(n).astype(np.float32) * np.float32(rng.uniform(1e-3, 10))
            if dtype == "bf16":
                x = W.to_bf16_bits(v)
            elif dtype == "fp16":
                x = W.to_fp16_bits(v)
            elif dtype == "fp32":
                x = v.view(np.uint32)
            else:
                x = W.random_bits(n, 16, seed=seed) & np.uint16(0xB7B7)
        bb = 4096
    a = ref.compress(x, dtype, bb).tobytes()
    b = model.compress([int(v) for v in x], dtype, bb)
    coded = sum(1 for st, _ in sections(np.frombuffer(a, np.uint8), dtype, x.size) if not st) if a == b else -1
    return seed, a == b, coded


def test_c_oracle_matches_python_model_ten_thousand_streams():
    workers = min(8, os.cpu_count() or 1)
    with ProcessPoolExecutor(workers) as ex:
        res = list(ex.map(_one, range(10_000), chunksize=64))
    bad = [s for s, ok, _ in res if not ok]
    assert not bad, f"streams differ for seeds {bad[:10]}"
    assert sum(c for _, _, c in res) > 4000   # plenty of CODED blocks among them


def _model_block(args):
    syms, = args
    sec, stored = model.section(list(syms))
    return sec, stored


def test_c_oracle_matches_python_model_normal_bf16_4MiB():
    """Every block of the 4 MiB bf16 workload (N(0, 0.02), 64 KiB blocks):
    the model's sections and raw plane against the C oracle's stream."""
    x = W.normal_bf16()
    s = ref.compress(x, "bf16", 65536)
    secs = sections(s, "bf16", x.size)
    assert len(secs) == 64
    planes = [model.to_planes("bf16", int(v)) for v in x]
    sym = np.array([p[0] for p in planes], np.uint8)
    raw = np.array([p[1] for p in planes], np.uint8)
    nb = 64
    raw_off = 32 + pad16(4 * nb)
    assert np.array_equal(s[raw_off:raw_off + x.size], raw)
    workers = min(8, os.cpu_count() or 1)
    with ProcessPoolExecutor(workers) as ex:
        got = list(ex.map(_model_block, [(sym[b * 32768:(b + 1) * 32768].tolist(),) for b in range(nb)]))
    for b, ((stored, sec), (msec, mstored)) in enumerate(zip(secs, got)):
        assert stored == mstored and sec == msec, b
