"""Pins of the CPU oracle against what the paper and mathematics fix.

Every test here runs on the CPU.  None of them re-derives the oracle's
formulas: they check it against independent facts -- IEEE field semantics
(numpy's frexp/float16/float32 and torch's bfloat16), losslessness
(section 1 and the conclusion: no numerical change), the split fractions of
Property 2 (section 3.2.1), the ratio the paper prints for bf16 U[-1, 1]
(section 5.2.1), ANS as an entropy coder (its size against the information
content of the block under its own table, and the Gibbs inequality), closed
forms for degenerate blocks, brute force on tiny inputs, exact arithmetic
identities of the fused reduce (section 3.4) and an independently written
Python model of the same stream format.
"""
import itertools
import math
import struct

import numpy as np
import pytest
import torch

from oracle import model, ref
import workloads as W

EB = {"bf16": 2, "fp16": 2, "fp32": 4, "e4m3fn": 2, "e5m2": 2}
L_STATE = 1 << 15
M = 2048


def header(stream):
    magic, ver, code, pb, flg, be, nb, n, total = struct.unpack_from("<IBBBBIIQQ", stream.tobytes(), 0)
    return dict(magic=magic, ver=ver, code=code, pb=pb, flags=flg, be=be, nb=nb, n=n, total=total)


def pad16(v):
    return -(-v // 16) * 16


# ---------------------------------------------------------------- Step 1 split
def _field_from_value_bf16(w):
    """IEEE fields of a bf16 word from the VALUE it denotes (numpy)."""
    v = np.array([w << 16], np.uint32).view(np.float32)[0]
    sign = int(np.signbit(v))
    if np.isnan(v) or np.isinf(v):
        return 255, sign, None
    a = abs(float(v))
    if a == 0.0:
        return 0, sign, 0
    m, e = math.frexp(a)           # a = m 2^e, m in [0.5, 1)
    if e - 1 >= -126:              # normal: (1 + f/128) 2^(E-127)
        E = e - 1 + 127
        frac = round((a / 2.0 ** (e - 1) - 1.0) * 128)
        return E, sign, frac
    return 0, sign, round(a / 2.0 ** -126 * 128)   # subnormal: f/128 2^-126


def test_split_bf16_exhaustive():
    for w in range(1 << 16):
        s, r = ref.split_word("bf16", w)
        E, sign, frac = _field_from_value_bf16(w)
        assert s == E, w
        assert r & 1 == sign, w
        if frac is not None:
            assert r >> 1 == frac, w
        assert ref.merge_word("bf16", s, r) == w


def test_split_fp16_exhaustive():
    vals = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
    for w in range(1 << 16):
        v = vals[w]
        s, r = ref.split_word("fp16", w)
        sign = int(np.signbit(v))
        assert r & 1 == sign
        if np.isfinite(v):
            a = abs(float(v))
            if a == 0.0:
                E, frac = 0, 0
            else:
                m, e = math.frexp(a)
                if e - 1 >= -14:
                    E, frac = e - 1 + 15, round((a / 2.0 ** (e - 1) - 1.0) * 1024)
                else:
                    E, frac = 0, round(a / 2.0 ** -14 * 1024)
            # symbol = 5-bit exponent and the top 3 fraction bits
            assert s == (E << 3) | (frac >> 7), w
            assert r >> 1 == frac & 127, w
        else:
            assert s >> 3 == 31
        assert ref.merge_word("fp16", s, r) == w


def test_split_fp32_fields_and_bijection():
    rng = np.random.default_rng(0)
    words = list(rng.integers(0, 1 << 32, 20000, dtype=np.uint64))
    for e in range(256):
        for mant in (0, 1, 0x3FFFFF, 0x400000, 0x7FFFFF):
            for sgn in (0, 1):
                words.append((sgn << 31) | (e << 23) | mant)
    for w in words:
        w = int(w)
        s, r = ref.split_word("fp32", w)
        v = np.array([w], np.uint32).view(np.float32)[0]
        if np.isfinite(v) and v != 0:
            a = abs(float(v))
            m, e2 = math.frexp(a)
            E = e2 - 1 + 127 if e2 - 1 >= -126 else 0
            assert s == E
        assert r & 1 == int(np.signbit(v))
        assert ref.merge_word("fp32", s, r) == w


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
def test_raw_plane_fraction_property2(dtype):
    """Property 2 (section 3.2.1): the uncompressed part is about half of a
    bf16 tensor and three quarters of an fp32 tensor -- exactly (E-1)/E."""
    n = 100_003
    x = W.random_bits(n, 8 * EB[dtype], seed=5)
    s = ref.compress(x, dtype, 65536)
    h = header(s)
    raw_off = 32 + pad16(4 * h["nb"])
    coded_off = raw_off + pad16((EB[dtype] - 1) * n)
    raw_bytes = (EB[dtype] - 1) * n
    assert raw_bytes / (EB[dtype] * n) == (EB[dtype] - 1) / EB[dtype]
    # the raw plane holds exactly the low E-1 bytes of each rotated value
    plane = s[raw_off:raw_off + raw_bytes].reshape(n, EB[dtype] - 1)
    for i in (0, 1, n // 2, n - 1):
        _, r = ref.split_word(dtype, int(x[i]))
        assert int.from_bytes(plane[i].tobytes(), "little") == r
    assert coded_off <= h["total"]


# ------------------------------------------------------ localized table
def _check_table(count, n_b):
    f, cum = ref.build_table(count, n_b)
    k = int((count > 0).sum())
    assert int(f.sum()) == M                          # a valid ANS table
    assert np.array_equal(f > 0, count > 0)           # every present symbol codable
    assert int(f.max()) <= M
    base = np.where(count > 0, 1 + (count.astype(np.int64) * (M - k)) // max(n_b, 1), 0)
    d = M - int(base.sum())
    assert 0 <= d < k
    order = np.argsort(count)
    for a, b in zip(order[:-1], order[1:]):           # monotone in the count
        if count[b] > count[a]:
            assert f[b] >= f[a]
    assert np.array_equal(cum, np.concatenate([[0], np.cumsum(f)[:-1]]))
    return f


def test_table_exhaustive_small():
    syms = [0, 1, 7, 128, 255]
    for k in range(1, 5):
        for chosen in itertools.combinations(syms, k):
            for counts in itertools.product(range(1, 10), repeat=k):
                if sum(counts) > 12:
                    continue
                c = np.zeros(256, np.uint32)
                c[list(chosen)] = counts
                _check_table(c, int(c.sum()))


def test_table_random_wide():
    rng = np.random.default_rng(3)
    for _ in range(300):
        k = int(rng.integers(1, 257))
        c = np.zeros(256, np.uint32)
        idx = rng.choice(256, k, replace=False)
        c[idx] = rng.geometric(rng.uniform(0.001, 0.9), k)
        _check_table(c, int(c.sum()))


def test_table_single_symbol():
    c = np.zeros(256, np.uint32)
    c[131] = 32768
    f, cum = ref.build_table(c, 32768)
    assert f[131] == M and f.sum() == M


# ---------------------------------------------------------------- rANS
def _table_for(sym):
    c = np.bincount(sym, minlength=256).astype(np.uint32)
    return ref.build_table(c, len(sym))


def test_rans_bruteforce_three_symbols():
    """Every sequence over a 3-symbol alphabet up to length 7 round-trips
    and the decoder ends in the initial state (checked inside decode)."""
    alphabet = [3, 100, 250]
    for n in range(1, 8):
        for seq in itertools.product(alphabet, repeat=n):
            sym = np.array(seq, np.uint8)
            f, cum = _table_for(sym)
            st, words = ref.rans_encode(sym, f, cum)
            out = ref.rans_decode(st, words, f, cum, n)
            assert out is not None and np.array_equal(out[0], sym)
            assert out[1] == len(words)


def _information(sym, f):
    return float(np.sum(np.log2(M / f[sym].astype(np.float64))))


def test_rans_size_against_information_content():
    """ANS is an entropy coder: the coded bits (16 W plus the bits held in
    the final states above L) follow the information content Q of the
    block under its own table.  With states kept at >= 16 f before coding,
    each symbol costs log2(M/f) + [log2(15/16), log2(17/16)) bits and each
    16-bit renormalisation loses less than log2(17/16) bits."""
    rng = np.random.default_rng(7)
    lo_s, hi_s = math.log2(15 / 16), math.log2(17 / 16)
    for trial in range(60):
        n = int(rng.integers(1, 40000))
        kind = trial % 4
        if kind == 0:
            sym = rng.integers(0, 256, n).astype(np.uint8)
        elif kind == 1:
            sym = (120 + rng.geometric(0.5, n)).clip(0, 255).astype(np.uint8)
        elif kind == 2:
            sym = rng.choice([5, 6], n, p=[0.999, 0.001]).astype(np.uint8)
        else:
            sym = np.clip(rng.normal(120, 3, n), 0, 255).astype(np.uint8)
        f, cum = _table_for(sym)
        st, words = ref.rans_encode(sym, f, cum)
        nw = len(words)
        coded = 16 * nw + float(np.sum(np.log2(st.astype(np.float64) / L_STATE)))
        Q = _information(sym, f)
        assert Q + n * lo_s - 1e-6 <= coded <= Q + n * hi_s + nw * hi_s + 1e-6
        # Gibbs: the table can only cost bits relative to the empirical entropy
        p = np.bincount(sym, minlength=256) / n
        H = -float(np.sum(p[p > 0] * np.log2(p[p > 0])))
        assert n * H <= Q + 1e-6
        # every present symbol gets f >= c (M - k) / n_b, so the table costs
        # at most log2(M / (M - k)) bits per symbol above the entropy
        k = int((p > 0).sum())
        assert Q <= n * H + n * math.log2(M / (M - k)) + 1e-6
        if n > 5000 and kind != 0:
            assert coded <= 1.005 * Q + 64 * 16
        out = ref.rans_decode(st, words, f, cum, n)
        assert out is not None and np.array_equal(out[0], sym)


def test_rans_rejects_tampering():
    rng = np.random.default_rng(9)
    sym = np.clip(rng.normal(120, 2, 5000), 0, 255).astype(np.uint8)
    f, cum = _table_for(sym)
    st, words = ref.rans_encode(sym, f, cum)
    bad = st.copy()
    bad[5] ^= 1 << 3
    res = ref.rans_decode(bad, words, f, cum, len(sym))
    assert res is None or not np.array_equal(res[0], sym)
    assert ref.rans_decode(st, words[:-1], f, cum, len(sym)) is None


# --------------------------------------------------------- closed forms
def test_single_symbol_block_closed_form():
    """k = 1: the table is f = M, coding is the identity on the states, no
    words: section = 64 states (all L) + bitmap + one f = 290 -> 304 bytes."""
    x = np.full(32768, 0x3F80, np.uint16)      # bf16 1.0 everywhere
    sec, stored = ref.block_section(x, "bf16", 65536, 0)
    assert not stored and len(sec) == 304
    states = np.frombuffer(sec[:256].tobytes(), np.uint32)
    assert np.all(states == L_STATE)
    assert np.frombuffer(sec[288:290].tobytes(), np.uint16)[0] == M
    assert np.all(sec[290:] == 0)


def test_largest_block_closed_forms():
    """A 4 MiB block holds 2^21 16-bit symbols, the most of any block.  One
    symbol throughout: f = M, no words, a 304-byte section.  With one
    outlier the counts are 2^21 - 1 and 1: f = 1 + floor((2^21 - 1)(M - 2)
    / 2^21) = 2046 and 1 + floor((M - 2) / 2^21) = 1, and the remainder 1
    goes to the most frequent symbol: (2047, 1) -- c (M - k) at its
    largest, just under 2^32."""
    n = 1 << 21
    x = np.full(n, 0x3F80, np.uint16)          # bf16 1.0: symbol (exponent) 127
    sec, stored = ref.block_section(x, "bf16", 1 << 22, 0)
    assert not stored and len(sec) == 304
    assert np.all(np.frombuffer(sec[:256].tobytes(), np.uint32) == L_STATE)
    assert np.frombuffer(sec[288:290].tobytes(), np.uint16)[0] == M
    x[12345] = 0x4000                          # bf16 2.0: symbol 128
    sec, stored = ref.block_section(x, "bf16", 1 << 22, 0)
    assert not stored
    present = np.unpackbits(sec[256:288], bitorder="little")
    assert list(np.flatnonzero(present)) == [127, 128]
    assert list(np.frombuffer(sec[288:292].tobytes(), np.uint16)) == [2047, 1]
    s = ref.compress(x, "bf16", 1 << 22)
    assert np.array_equal(ref.decompress(s, "bf16", n), x)


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
def test_stored_coded_boundary_closed_form(dtype):
    """One symbol, no words: the coded section would be 288 + 2 = 290 bytes,
    so a block of 290 elements is STORED (290 symbol bytes are not more)
    and one of 291 is CODED (pad16(290) = 304 bytes) -- the strict
    inequality of the STORED rule, at its edge."""
    one = {"bf16": 0x3F80, "fp16": 0x3C00, "fp32": 0x3F800000}[dtype]
    for n, stored, sec_len in ((290, True, 304), (291, False, 304), (289, True, 304), (300, False, 304)):
        x = np.full(n, one, np.uint32 if dtype == "fp32" else np.uint16)
        s = ref.compress(x, dtype, 65536)
        h = header(s)
        d = struct.unpack_from("<I", s.tobytes(), 32)[0]
        assert bool(d >> 31) == stored, (dtype, n)
        assert 16 * (d & 0x7FFFFFFF) == sec_len
        assert h["total"] == s.size
        raw_off = 32 + pad16(4)
        coded_off = raw_off + pad16((EB[dtype] - 1) * n)
        assert s.size == coded_off + sec_len
        if not stored:
            states = np.frombuffer(s[coded_off:coded_off + 256].tobytes(), np.uint32)
            assert np.all(states == L_STATE)
        assert np.array_equal(ref.decompress(s, dtype, n), x)


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
def test_uniform_random_words_all_stored(dtype):
    """Uniformly random words carry 8 bits per symbol plus the table, so
    every block is STORED and the size has a closed form."""
    n = 150_001
    x = W.random_bits(n, 8 * EB[dtype], seed=21)
    bb = 65536
    s = ref.compress(x, dtype, bb)
    be = bb // EB[dtype]
    nb = -(-n // be)
    expect = 32 + pad16(4 * nb) + pad16((EB[dtype] - 1) * n) + sum(
        pad16(min(be, n - b * be)) for b in range(nb))
    assert len(s) == expect == ref.max_compressed_size(dtype, n, bb)
    dirs = np.frombuffer(s[32:32 + 4 * nb].tobytes(), np.uint32)
    assert np.all(dirs >> 31 == 1)


def test_empty_tensor_stream():
    s = ref.compress(np.zeros(0, np.uint16), "bf16", 65536)
    assert len(s) == 32
    h = header(s)
    assert h["nb"] == 0 and h["n"] == 0 and h["total"] == 32
    assert ref.decompress(s, "bf16", 0).size == 0


def test_tiny_blocks_are_stored():
    x = W.normal_bf16(200, seed=4)
    s = ref.compress(x, "bf16", 4096)
    assert np.frombuffer(s[32:36].tobytes(), np.uint32)[0] >> 31 == 1
    assert np.array_equal(ref.decompress(s, "bf16", 200), x)


# ------------------------------------------------------ paper's ratio
def test_ratio_bf16_uniform_matches_paper():
    """Section 5.2.1 reports a compression ratio of about 0.64 for bf16
    tensors drawn from U[-1, 1].  Their exponent law P(126 - m) = 2^-(m+1)
    has 2 bits of entropy, so the ratio sits just above (8 + 2) / 16."""
    n = 1 << 21
    x = W.uniform_bf16(n, seed=11)
    s = ref.compress(x, "bf16", 65536)
    ratio = len(s) / (2 * n)
    sym = (x >> 7) & 0xFF
    p = np.bincount(sym, minlength=256) / n
    H = -float(np.sum(p[p > 0] * np.log2(p[p > 0])))
    assert (8 + H) / 16 <= ratio <= (8 + H) / 16 + 0.01
    assert abs(ratio - 0.64) <= 0.02


def test_ratio_bounded_by_exponent_entropy():
    for x, dtype, bb in [(W.normal_bf16(1 << 20, seed=2), "bf16", 65536),
                         (W.grad_fp32(1 << 19, seed=3), "fp32", 262144),
                         (W.grad_fp16(1 << 19, seed=3), "fp16", 262144),
                         (W.normal_bf16(5 << 20, seed=4), "bf16", 1 << 22),
                         (W.grad_fp32((1 << 20) + 4321, seed=5), "fp32", 1 << 20)]:
        e = EB[dtype]
        n = x.size
        be = bb // e
        s = ref.compress(x, dtype, bb)
        bits = 8 * e
        sym = (((x.astype(np.uint64) << 1) | (x.astype(np.uint64) >> (bits - 1))) >> (bits - 8)) & 0xFF
        Hsum = 0.0
        for b in range(0, n, be):
            blk = sym[b:b + be]
            p = np.bincount(blk, minlength=256) / blk.size
            Hsum += -blk.size * float(np.sum(p[p > 0] * np.log2(p[p > 0])))
        lower = ((e - 1) * 8 * n + Hsum) / 8
        assert lower <= len(s) <= lower * 1.01 + 1024 * (n // be + 1)


# ----------------------------------------------- FP8 pairs (section 4.1)
def _fp8_value_table(fmt):
    """Float value of every FP8 byte, decoded by torch (independent of the
    oracle's bit handling)."""
    b = torch.arange(256, dtype=torch.uint8)
    t = {"e4m3fn": torch.float8_e4m3fn, "e5m2": torch.float8_e5m2}[fmt]
    return b.view(t).to(torch.float64).numpy()


@pytest.mark.parametrize("fmt", ["e4m3fn", "e5m2"])
def test_fp8_pair_symbol_is_the_joint_exponent(fmt):
    """Every 16-bit unit of two FP8 values: the symbol's nibbles locate the
    two values' binades (the exponent fields of section 4.1; for e5m2 the
    exponent without its lowest bit, i.e. a pair of binades), the raw byte
    keeps the signs, and the split is a bijection."""
    vals = _fp8_value_table(fmt)
    bias, pair = (7, 1) if fmt == "e4m3fn" else (15, 2)   # e5m2: a nibble spans two binades
    seen = set()
    for w in range(1 << 16):
        s, r = ref.split_word(fmt, w)
        assert 0 <= s < 256 and 0 <= r < 256
        seen.add((s, r))
        assert ref.merge_word(fmt, s, r) == w
        for k in range(2):
            v = vals[(w >> (8 * k)) & 0xFF]
            nib, rnib = (s >> (4 * k)) & 15, (r >> (4 * k)) & 15
            if np.isnan(v) or np.isinf(v):
                continue
            assert (rnib >> 3) == (1 if math.copysign(1.0, v) < 0 else 0), (w, k)
            a = abs(v)
            if a == 0:
                assert nib == 0
                continue
            lo = 2.0 ** (pair * nib - bias) if nib > 0 else 0.0
            hi = 2.0 ** (pair * nib + pair - bias)
            # nibble 0 holds the subnormals (and for e5m2 also the first normal binade)
            assert lo <= a < hi, (fmt, w, k, v, nib)
    assert len(seen) == 1 << 16


@pytest.mark.parametrize("fmt", ["e4m3fn", "e5m2"])
def test_fp8_ratio_bounded_by_pair_exponent_entropy(fmt):
    """FP8 N(0,1) pairs: half the bytes stay raw; the coded part is the
    symbols' empirical entropy per block plus the bounded rANS overhead."""
    x = W.normal_fp8_pairs(1 << 19, fmt, seed=21)
    n, bb = x.size, 65536
    be = bb // 2
    s = ref.compress(x, fmt, bb)
    sym = np.array([ref.split_word(fmt, int(w))[0] for w in x[:1 << 16]])
    sym = np.concatenate([sym, ((x[1 << 16:] >> 3) & 15) | (((x[1 << 16:] >> 11) & 15) << 4)])
    Hsum = 0.0
    for b in range(0, n, be):
        blk = sym[b:b + be]
        p = np.bincount(blk, minlength=256) / blk.size
        Hsum += -blk.size * float(np.sum(p[p > 0] * np.log2(p[p > 0])))
    lower = (8 * n + Hsum) / 8
    assert lower <= len(s) <= lower * 1.01 + 1024 * (n // be + 1)
    assert np.array_equal(ref.decompress(s, fmt, n), x)


@pytest.mark.parametrize("fmt", ["e4m3fn", "e5m2"])
def test_fp8_specials_and_random_bits_roundtrip(fmt):
    rng = np.random.default_rng(5)
    x = W.normal_fp8_pairs(70_001, fmt, seed=9)
    specials = np.array([0x0000, 0x8080, 0x7F7F, 0xFFFF, 0x7E00, 0x007C, 0xFC7B, 0x0101], np.uint16)
    pos = rng.integers(0, x.size, x.size // 10)
    x[pos] = rng.choice(specials, pos.size)
    r = W.random_bits(9000, 16, seed=3)
    for arr in (x, r):
        for bb in (4096, 65536):
            st = ref.compress(arr, fmt, bb)
            assert np.array_equal(ref.decompress(st, fmt, arr.size), arr)


# ------------------------------------------------------- losslessness
def _special_words(dtype, n, seed):
    rng = np.random.default_rng(seed)
    bits = 8 * EB[dtype]
    if dtype == "bf16":
        specials = [0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC0, 0x7F81, 0xFFFF, 0x0001, 0x807F, 0x3F80]
    elif dtype == "fp16":
        specials = [0x0000, 0x8000, 0x7C00, 0xFC00, 0x7E00, 0x7C01, 0xFFFF, 0x0001, 0x83FF, 0x3C00]
    elif dtype in ("e4m3fn", "e5m2"):
        specials = [0x0000, 0x8080, 0x7F7F, 0xFFFF, 0x7E00, 0x007C, 0xFC7B, 0x0101, 0x3838, 0x3C3C]
    else:
        specials = [0, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 0x7F800001, 0xFFFFFFFF, 1,
                    0x807FFFFF, 0x3F800000]
    if dtype in ("e4m3fn", "e5m2"):
        x = W.normal_fp8_pairs(n, dtype, seed=seed)
    else:
        x = W.normal_bf16(n, seed=seed) if dtype == "bf16" else (
            W.grad_fp16(n, seed=seed) if dtype == "fp16" else W.grad_fp32(n, seed=seed))
    pos = rng.integers(0, n, n // 10)
    x[pos] = rng.choice(specials, pos.size)
    noise = rng.integers(0, n, n // 50)
    x[noise] = rng.integers(0, 1 << bits, noise.size, dtype=np.uint64).astype(x.dtype)
    return x


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
@pytest.mark.parametrize("n", [1, 511, 512, 513, 4097, 70_001])
def test_roundtrip_lossless(dtype, n):
    x = _special_words(dtype, n, seed=n)
    for bb in (4096, 65536):
        s = ref.compress(x, dtype, bb)
        y = ref.decompress(s, dtype, n)
        assert y is not None and np.array_equal(x, y)


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32", "e4m3fn"])
def test_roundtrip_lossless_large_blocks(dtype):
    """1 MiB and 4 MiB blocks with a partial last block."""
    n = (1 << 21) + 3 * (1 << 18) + 777
    x = _special_words(dtype, n, seed=5)
    for bb in (1 << 20, 1 << 22):
        s = ref.compress(x, dtype, bb)
        assert len(s) <= ref.max_compressed_size(dtype, n, bb)
        y = ref.decompress(s, dtype, n)
        assert y is not None and np.array_equal(x, y)


def test_corrupt_headers_detected():
    x = W.normal_bf16(50_000, seed=8)
    s = ref.compress(x, "bf16", 4096)
    assert ref.decompress(s, "bf16", 50_000) is not None
    for off in (0, 4, 5, 6, 7, 8, 12, 16, 24):
        bad = s.copy()
        bad[off] ^= 0x5A
        assert ref.decompress(bad, "bf16", 50_000) is None
    assert ref.decompress(s[:-16], "bf16", 50_000) is None
    assert ref.decompress(s, "fp16", 50_000) is None
    assert ref.decompress(s, "bf16", 50_001) is None


def test_corrupt_payload_never_crashes():
    rng = np.random.default_rng(4)
    x = W.normal_bf16(40_000, seed=9)
    s = ref.compress(x, "bf16", 4096)
    detected = 0
    for _ in range(200):
        bad = s.copy()
        pos = int(rng.integers(32, len(s)))
        bad[pos] ^= 1 << int(rng.integers(0, 8))
        y = ref.decompress(bad, "bf16", 40_000)
        detected += y is None or not np.array_equal(x, y)
    assert detected > 150


# ----------------------------------------------------- fused reduce
def _f32(dtype, bits):
    if dtype == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32)
    if dtype == "fp16":
        return bits.view(np.float16).astype(np.float32)
    return bits.view(np.float32)


def _round(dtype, acc):
    """numpy/torch rounding of float32 to the storage type, NaN canonical."""
    nan = np.isnan(acc)
    if dtype == "bf16":
        out = torch.from_numpy(acc.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        out = out.copy()
        out[nan] = 0x7FC0
    elif dtype == "fp16":
        out = acc.astype(np.float16).view(np.uint16).copy()
        out[nan] = 0x7E00
    else:
        out = acc.view(np.uint32).copy()
        out[nan] = 0x7FC00000
    return out


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
def test_reduce_matches_numpy_sequential_sum(dtype):
    n = 30_017
    xs = [_special_words(dtype, n, seed=100 + i) for i in range(5)]
    local = _special_words(dtype, n, seed=99)
    streams = [ref.compress(x, dtype, 4096) for x in xs]
    out, y = ref.reduce(streams, dtype, n, 4096, local=local)
    with np.errstate(all="ignore"):
        acc = _f32(dtype, xs[0]).copy()
        for x in xs[1:]:
            acc = (acc + _f32(dtype, x)).astype(np.float32)
        acc = (acc + _f32(dtype, local)).astype(np.float32)
    assert np.array_equal(y, _round(dtype, acc))
    assert np.array_equal(out, ref.compress(y, dtype, 4096))


def test_reduce_single_input_is_identity():
    x = W.normal_bf16(100_000, seed=12)
    s = ref.compress(x, "bf16", 65536)
    out, y = ref.reduce([s], "bf16", x.size, 65536)
    assert np.array_equal(y, x) and np.array_equal(out, s)


def test_reduce_eight_copies_scales_exponents():
    """8 copies of x sum to 8x exactly (no rounding for values with 8
    significant bits); the raw plane is unchanged, every exponent symbol
    moves up by 3, so the coded words and states are the same."""
    rng = np.random.default_rng(13)
    v = rng.normal(0, 1, 70_000).astype(np.float32)
    x = W.to_bf16_bits(v)
    s = ref.compress(x, "bf16", 65536)
    out, y = ref.reduce([s] * 8, "bf16", x.size, 65536)
    assert np.array_equal(_f32("bf16", y), 8 * _f32("bf16", x))
    h = header(s)
    raw_off = 32 + pad16(4 * h["nb"])
    coded = raw_off + pad16(x.size)
    assert np.array_equal(out[raw_off:coded], s[raw_off:coded])
    for b in range(h["nb"]):
        a_sec, _ = ref.block_section(x, "bf16", 65536, b)
        b_sec, _ = ref.block_section(y, "bf16", 65536, b)
        assert len(a_sec) == len(b_sec)
        assert np.array_equal(a_sec[:256], b_sec[:256])          # states
        assert np.array_equal(a_sec[288:], b_sec[288:])          # f[] and words
        bits_a = np.unpackbits(a_sec[256:288], bitorder="little")
        bits_b = np.unpackbits(b_sec[256:288], bitorder="little")
        assert np.array_equal(np.roll(bits_a, 3), bits_b)


def test_reduce_x_plus_minus_x_is_positive_zero():
    x = W.normal_bf16(20_000, seed=14)
    s1 = ref.compress(x, "bf16", 4096)
    s2 = ref.compress(x ^ np.uint16(0x8000), "bf16", 4096)
    _, y = ref.reduce([s1, s2], "bf16", x.size, 4096)
    assert np.all(y == 0)


def test_scalar_conversions_against_numpy_and_torch():
    all16 = np.arange(1 << 16, dtype=np.uint32)
    want = all16.astype(np.uint16).view(np.float16).astype(np.float32)
    for h in range(0, 1 << 16, 7):
        got = ref.half_to_float(h)
        w = want[h]
        assert (np.isnan(got) and np.isnan(w)) or np.float32(got).view(np.uint32) == w.view(np.uint32)
    rng = np.random.default_rng(1)
    vals = np.concatenate([
        rng.integers(0, 1 << 32, 20000, dtype=np.uint64).astype(np.uint32).view(np.float32),
        (rng.normal(0, 1e-5, 5000)).astype(np.float32),
        np.array([65504, 65519.996, 65520, 65536, 6.1035156e-05, 5.9604645e-08, 2.9802322e-08,
                  2.9802326e-08, 1.0 + 2 ** -11, 1.0 + 3 * 2 ** -11], np.float32)])
    h_np = vals.astype(np.float16).view(np.uint16)
    b_t = torch.from_numpy(vals.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    for i, v in enumerate(vals):
        if np.isnan(v):
            assert ref.float_to_half(float(v)) == 0x7E00
            assert ref.float_to_bf16(float(v)) == 0x7FC0
            continue
        assert ref.float_to_half(float(v)) == h_np[i], (v, hex(h_np[i]))
        assert ref.float_to_bf16(float(v)) == b_t[i], v


# ------------------------------------ second CPU reading (micro-model)
def test_c_oracle_matches_python_model():
    rng = np.random.default_rng(17)
    for trial in range(30):
        dtype = ["bf16", "fp16", "fp32", "e4m3fn", "e5m2"][trial % 5]
        n = int(rng.integers(0, 9000))
        if trial % 4 == 0:
            x = W.random_bits(n, 8 * EB[dtype], seed=trial)
        else:
            x = _special_words(dtype, max(n, 1), seed=trial)[:n]
        a = ref.compress(x, dtype, 4096).tobytes()
        b = model.compress([int(v) for v in x], dtype, 4096)
        assert a == b, (trial, n, dtype)
        assert model.decompress(b, dtype, n) == [int(v) for v in x]
    # one 1 MiB block and part of a second: the model's arithmetic at a
    # block size past the register path's
    x = W.grad_fp32((1 << 18) + 777, seed=8)
    assert ref.compress(x, "fp32", 1 << 20).tobytes() == model.compress([int(v) for v in x], "fp32", 1 << 20)


# ------------------------------------------------------ golden fixtures
def test_golden_streams_stable():
    """Fixtures written by tests/golden/make_golden.py from the oracle."""
    import hashlib
    import json
    import os
    here = os.path.join(os.path.dirname(__file__), "golden")
    meta = json.load(open(os.path.join(here, "streams.json")))
    gens = {"normal_bf16_5000_b4096": lambda: W.normal_bf16(5000, seed=7),
            "grad_fp32_3000_b4096": lambda: W.grad_fp32(3000, seed=7),
            "grad_fp16_6000_b4096": lambda: W.grad_fp16(6000, seed=7),
            "normal_e4m3fn_6000_b4096": lambda: W.normal_fp8_pairs(6000, "e4m3fn", seed=7),
            "normal_e5m2_6000_b4096": lambda: W.normal_fp8_pairs(6000, "e5m2", seed=7),
            "normal_bf16_5000_b4096_sampled": lambda: W.normal_bf16(5000, seed=7)}
    assert set(meta) == set(gens)
    for name, m in meta.items():
        x = gens[name]()
        assert hashlib.sha256(x.tobytes()).hexdigest() == m["input_sha256"]
        hexs = "".join(open(os.path.join(here, name + ".hex")).read().split())
        stored = np.frombuffer(bytes.fromhex(hexs), np.uint8)
        assert stored.size == m["stream_bytes"]
        mode = m.get("table_mode", "per_block")
        assert np.array_equal(ref.compress_table(x, m["dtype"], m["block_bytes"], mode), stored)
        assert np.array_equal(ref.decompress_table(stored, m["dtype"], m["n"]), x)
