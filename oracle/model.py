"""Pure-Python micro-model of the codec, for tiny inputs only.

TEST INFRASTRUCTURE ONLY.  A second, independently written CPU reading of
the same stream format as ``uzip_ref.c`` (Python integers, lists and
``struct``), used to cross-check the C oracle byte for byte on small random
streams.  It pins the C code against slips in writing the reading down; it
does not pin the reading against the paper (the pins in the test suite do
that).

Method steps, as in the paper: the exponent/sign+fraction split of section
2.1.2 (Step 1), a localized table per block (section 3.3.1), per-block ANS
(Step 2), concatenation into one stream (Step 3), metadata of section 4.1.
"""
from __future__ import annotations

import struct

M = 1 << 11
L = 1 << 15
LANES, PER_LANE = 64, 8
ROUND = LANES * PER_LANE
EB = {"bf16": 2, "fp16": 2, "fp32": 4, "e4m3fn": 2, "e5m2": 2}
CODE = {"bf16": 0, "fp16": 1, "fp32": 2, "e4m3fn": 3, "e5m2": 4}
# FP8 value fields (sign, exponent bits, fraction bits)
FP8_FIELDS = {"e4m3fn": (4, 3), "e5m2": (5, 2)}


def fp8_pair_planes(dtype: str, w: int) -> tuple[int, int]:
    """Section 4.1: two FP8 values in one 16-bit unit, their exponent fields
    taken together as the 8-bit symbol.  Written from the value fields: for
    e4m3fn the symbol is the two exponents; for e5m2 the two exponents'
    top four bits, the lowest exponent bit going with sign and fraction."""
    ebits, mbits = FP8_FIELDS[dtype]
    sym = raw = 0
    for k in range(2):
        v = (w >> (8 * k)) & 0xFF
        sign, exp, frac = v >> 7, (v >> mbits) & ((1 << ebits) - 1), v & ((1 << mbits) - 1)
        keep = ebits - 4  # exponent bits that do not fit the symbol nibble
        sym |= (exp >> keep) << (4 * k)
        raw |= ((sign << 3) | ((exp & ((1 << keep) - 1)) << mbits) | frac) << (4 * k)
    return sym, raw


def fp8_pair_value(dtype: str, sym: int, raw: int) -> int:
    ebits, mbits = FP8_FIELDS[dtype]
    keep = ebits - 4
    w = 0
    for k in range(2):
        s4, r4 = (sym >> (4 * k)) & 15, (raw >> (4 * k)) & 15
        exp = (s4 << keep) | ((r4 >> mbits) & ((1 << keep) - 1))
        v = ((r4 >> 3) << 7) | (exp << mbits) | (r4 & ((1 << mbits) - 1))
        w |= v << (8 * k)
    return w


def to_planes(dtype: str, w: int) -> tuple[int, int]:
    if dtype in FP8_FIELDS:
        return fp8_pair_planes(dtype, w)
    bits = 8 * EB[dtype]
    full = (1 << bits) - 1
    r = ((w << 1) & full) | (w >> (bits - 1))
    return r >> (bits - 8), r & ((1 << (bits - 8)) - 1)


def from_planes(dtype: str, sym: int, raw: int) -> int:
    if dtype in FP8_FIELDS:
        return fp8_pair_value(dtype, sym, raw)
    bits = 8 * EB[dtype]
    full = (1 << bits) - 1
    r = (sym << (bits - 8)) | raw
    return (r >> 1) | ((r & 1) << (bits - 1)) & full


def table(symbols: list[int]) -> list[int]:
    n = len(symbols)
    c = [0] * 256
    for s in symbols:
        c[s] += 1
    present = [s for s in range(256) if c[s]]
    k = len(present)
    f = [0] * 256
    for s in present:
        f[s] = 1 + (c[s] * (M - k)) // n
    top = max(range(256), key=lambda s: (c[s], -s))
    f[top] += M - sum(f)
    return f


def cumulative(f: list[int]) -> list[int]:
    out, run = [], 0
    for v in f:
        out.append(run)
        run += v
    return out


def order(n: int):
    """(round, sub-step, lane, index) in decode order."""
    for r in range((n + ROUND - 1) // ROUND):
        for t in range(PER_LANE):
            for j in range(LANES):
                i = r * ROUND + j * PER_LANE + t
                if i < n:
                    yield r, t, j, i


def encode(symbols: list[int], f: list[int]):
    cum = cumulative(f)
    n = len(symbols)
    x = [L] * LANES
    steps = {}
    for r, t, j, i in reversed(list(order(n))):
        s = symbols[i]
        out = steps.setdefault((r, t), [])
        if x[j] >= f[s] << 20:
            out.append((j, x[j] & 0xFFFF))
            x[j] >>= 16
        q, rem = divmod(x[j], f[s])
        x[j] = q * M + rem + cum[s]
    words = []
    for key in sorted(steps):
        words.extend(w for _, w in sorted(steps[key]))
    return x, words


def decode(states: list[int], words: list[int], f: list[int], n: int):
    cum = cumulative(f)
    owner = []
    for s in range(256):
        owner.extend([s] * f[s])
    x = list(states)
    pos = 0
    out = [0] * n
    for _, _, j, i in order(n):
        slot = x[j] % M
        s = owner[slot]
        x[j] = f[s] * (x[j] // M) + slot - cum[s]
        if x[j] < L:
            x[j] = (x[j] << 16) | words[pos]
            pos += 1
        out[i] = s
    assert all(v == L for v in x)
    return out


def pad16(v: int) -> int:
    return -(-v // 16) * 16


def section(symbols: list[int]) -> tuple[bytes, bool]:
    n = len(symbols)
    f = table(symbols)
    states, words = encode(symbols, f)
    present = [s for s in range(256) if f[s]]
    if 288 + 2 * len(present) + 2 * len(words) < n:
        bitmap = bytearray(32)
        for s in present:
            bitmap[s // 8] |= 1 << (s % 8)
        body = (struct.pack("<64I", *states) + bytes(bitmap)
                + struct.pack(f"<{len(present)}H", *[f[s] for s in present])
                + struct.pack(f"<{len(words)}H", *words))
        return body + bytes(pad16(len(body)) - len(body)), False
    body = bytes(symbols)
    return body + bytes(pad16(n) - n), True


def compress(words_in: list[int], dtype: str, block_bytes: int) -> bytes:
    e = EB[dtype]
    n = len(words_in)
    be = block_bytes // e
    nb = -(-n // be)
    planes = [to_planes(dtype, w) for w in words_in]
    raw = b"".join(r.to_bytes(e - 1, "little") for _, r in planes)
    sections, directory, end = [], [], 0
    for b in range(nb):
        sec, stored = section([s for s, _ in planes[b * be:(b + 1) * be]])
        sections.append(sec)
        end += len(sec)
        directory.append((0x80000000 if stored else 0) | (end // 16))
    dir_bytes = struct.pack(f"<{nb}I", *directory)
    body = (dir_bytes + bytes(pad16(len(dir_bytes)) - len(dir_bytes))
            + raw + bytes(pad16(len(raw)) - len(raw)) + b"".join(sections))
    header = struct.pack("<IBBBBIIQQ", 0x31505A55, 1, CODE[dtype], 11, 0, be, nb, n, 32 + len(body))
    return header + body


def decompress(stream: bytes, dtype: str, n: int) -> list[int]:
    e = EB[dtype]
    magic, ver, code, pb, flg, be, nb, n2, total = struct.unpack_from("<IBBBBIIQQ", stream, 0)
    assert (magic, ver, code, pb, flg, n2) == (0x31505A55, 1, CODE[dtype], 11, 0, n)
    raw_off = 32 + pad16(4 * nb)
    coded = raw_off + pad16((e - 1) * n)
    out, start = [], 0
    for b in range(nb):
        d = struct.unpack_from("<I", stream, 32 + 4 * b)[0]
        end = 16 * (d & 0x7FFFFFFF)
        sec = stream[coded + start:coded + end]
        nbk = min(be, n - b * be)
        if d >> 31:
            syms = list(sec[:nbk])
        else:
            states = list(struct.unpack_from("<64I", sec, 0))
            present = [s for s in range(256) if sec[256 + s // 8] >> (s % 8) & 1]
            fv = struct.unpack_from(f"<{len(present)}H", sec, 288)
            f = [0] * 256
            for s, v in zip(present, fv):
                f[s] = v
            wstart = 288 + 2 * len(present)
            words = list(struct.unpack_from(f"<{(len(sec) - wstart) // 2}H", sec, wstart))
            syms = decode(states, words, f, nbk)
        for q, s in enumerate(syms):
            i = b * be + q
            raw = int.from_bytes(stream[raw_off + (e - 1) * i: raw_off + (e - 1) * (i + 1)], "little")
            out.append(from_planes(dtype, s, raw))
        start = end
    assert coded + start == total
    return out


# --------------------------------------------------------------------------
# Stream-wide tables (section 3.3.1's table from a sample of the range,
# section 3.4's table sent once and reused): one table codes every block.
# Mode 1 keeps it in the stream after the directory, mode 2 leaves it to
# the caller.  Every symbol keeps a nonzero frequency, so symbols that the
# sample (the first 256 KiB) missed can still be coded.
# --------------------------------------------------------------------------
SAMPLE_BYTES = 256 * 1024


def table_all(sample: list[int]) -> list[int]:
    n = len(sample)
    if n == 0:
        return [M // 256] * 256
    c = [sample.count(s) for s in range(256)]
    f = [1 + (c[s] * (M - 256)) // n for s in range(256)]
    top = max(range(256), key=lambda s: (c[s], -s))
    f[top] += M - sum(f)
    return f


def shared_section(symbols: list[int], f: list[int]) -> tuple[bytes, bool]:
    n = len(symbols)
    states, words = encode(symbols, f)
    if 256 + 2 * len(words) < n:
        body = struct.pack("<64I", *states) + struct.pack(f"<{len(words)}H", *words)
        return body + bytes(pad16(len(body)) - len(body)), False
    return bytes(symbols) + bytes(pad16(n) - n), True


def compress_shared(words_in: list[int], dtype: str, block_bytes: int, mode: int, ext=None) -> bytes:
    e = EB[dtype]
    n = len(words_in)
    be = block_bytes // e
    nb = -(-n // be)
    planes = [to_planes(dtype, w) for w in words_in]
    f = table_all([s for s, _ in planes[:SAMPLE_BYTES // e]]) if mode == 1 else list(ext)
    secs = [shared_section([s for s, _ in planes[b * be:(b + 1) * be]], f) for b in range(nb)]
    ends, end = [], 0
    for sec, stored in secs:
        end += len(sec)
        ends.append((0x80000000 if stored else 0) | (end // 16))
    dir_bytes = struct.pack(f"<{nb}I", *ends)
    table_bytes = struct.pack("<256H", *f) if (mode == 1 and nb) else b""
    raw = b"".join(r.to_bytes(e - 1, "little") for _, r in planes)
    body = (dir_bytes + bytes(pad16(len(dir_bytes)) - len(dir_bytes)) + table_bytes
            + raw + bytes(pad16(len(raw)) - len(raw)) + b"".join(sec for sec, _ in secs))
    return struct.pack("<IBBBBIIQQ", 0x31505A55, 1, CODE[dtype], 11, mode, be, nb, n, 32 + len(body)) + body


def decompress_shared(stream: bytes, dtype: str, n: int, ext=None) -> list[int]:
    e = EB[dtype]
    magic, ver, code, pb, mode, be, nb, n2, total = struct.unpack_from("<IBBBBIIQQ", stream, 0)
    assert (magic, ver, code, pb, n2) == (0x31505A55, 1, CODE[dtype], 11, n) and mode in (1, 2)
    tab_off = 32 + pad16(4 * nb)
    if mode == 1:
        f = list(struct.unpack_from("<256H", stream, tab_off)) if nb else [M // 256] * 256
        raw_off = tab_off + (512 if nb else 0)
    else:
        f, raw_off = list(ext), tab_off
    assert min(f) >= 1 and sum(f) == M
    coded = raw_off + pad16((e - 1) * n)
    out, start = [], 0
    for b in range(nb):
        d = struct.unpack_from("<I", stream, 32 + 4 * b)[0]
        end = 16 * (d & 0x7FFFFFFF)
        sec = stream[coded + start:coded + end]
        nbk = min(be, n - b * be)
        if d >> 31:
            syms = list(sec[:nbk])
        else:
            states = list(struct.unpack_from("<64I", sec, 0))
            words = list(struct.unpack_from(f"<{(len(sec) - 256) // 2}H", sec, 256))
            syms = decode(states, words, f, nbk)
        for q, s in enumerate(syms):
            i = b * be + q
            raw = int.from_bytes(stream[raw_off + (e - 1) * i: raw_off + (e - 1) * (i + 1)], "little")
            out.append(from_planes(dtype, s, raw))
        start = end
    assert coded + start == total
    return out
