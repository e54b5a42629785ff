"""Seeded synthetic inputs shaped like the paper's workloads.

The paper measures on tensors that are not available here (GLM4-9B
gradients, activations and weights, Table 1; RL weight updates and vLLM
KV-cache transfers, section 5.3).  These generators stand in for them with
the shapes and value distributions of those workloads.  They hold none of
the codec's arithmetic: they only draw numbers and convert them to the
storage type with library conversions, and both the GPU path and the CPU
oracle consume what they return.

Every generator is a pure function of (seed, sizes).  Large tensors are
drawn in pieces of ``PIECE`` elements; piece p draws from
``SeedSequence(seed, spawn_key=(p,))`` so that any prefix of a buffer is
the same whatever its total length, and pieces can be drawn in parallel.

Results are numpy arrays of bit patterns: ``uint16`` for bf16 and fp16,
``uint32`` for fp32.

Workloads (sizes are those the benchmark and the full-size tests use):

  normal_bf16      4 MiB bf16, N(0, 0.02) (a single activation/weight tensor)
  weight_sync      1 GiB bf16 buffer laid out like a 0.5B-parameter
                   transformer (RL weight synchronisation)
  grad_fp32        fp32 gradient: Laplace(0, 1e-4), 1% of entries x100;
                   grad_fp16 is the same values rounded to fp16
  kv_cache         [layers, K/V, tokens, kv_heads, head_dim] bf16 with
                   log-normal per-channel scales and 4 outlier channels/head
  reduce_slices    n_in bf16 shares [tokens, hidden] with per-token scales
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

PIECE = 1 << 22
_THREADS = min(16, os.cpu_count() or 1)


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=tuple(key))))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (round to nearest even), via torch."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def to_fp16_bits(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def _pieces(n: int, fn, out: np.ndarray) -> np.ndarray:
    """Fill out[0:n] piece by piece; fn(p, lo, hi) returns out[lo:hi]."""
    count = (n + PIECE - 1) // PIECE

    def work(p: int) -> None:
        lo = p * PIECE
        hi = min(n, lo + PIECE)
        out[lo:hi] = fn(p, lo, hi)

    if count <= 1:
        for p in range(count):
            work(p)
    else:
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(work, range(count)))
    return out


# --------------------------------------------------------------------------
# normal_bf16: one bf16 tensor with N(0, sigma) values
# --------------------------------------------------------------------------
def normal_bf16(n: int = 2_097_152, sigma: float = 0.02, seed: int = 1) -> np.ndarray:
    def fn(p, lo, hi):
        z = _rng(seed, p).standard_normal(hi - lo, dtype=np.float32)
        return to_bf16_bits(z * np.float32(sigma))
    return _pieces(n, fn, np.empty(n, np.uint16))


def uniform_bf16(n: int, lo: float = -1.0, hi: float = 1.0, seed: int = 11) -> np.ndarray:
    """bf16 U[lo, hi]: the paper's synthetic P2P tensors (section 5.2.1)."""
    def fn(p, a, b):
        u = _rng(seed, p).random(b - a, dtype=np.float32)
        return to_bf16_bits(np.float32(lo) + u * np.float32(hi - lo))
    return _pieces(n, fn, np.empty(n, np.uint16))


FP8_TORCH = {"e4m3fn": torch.float8_e4m3fn, "e5m2": torch.float8_e5m2}


def normal_fp8_pairs(n_pairs: int, fmt: str = "e4m3fn", sigma: float = 1.0, seed: int = 13) -> np.ndarray:
    """FP8 values N(0, sigma^2), converted by torch (round to nearest even,
    saturating), as 16-bit pairs (value 2i in the low byte): the element the
    codec takes for FP8 (section 4.1)."""
    def fn(p, lo, hi):
        z = _rng(seed, p).standard_normal(2 * (hi - lo), dtype=np.float32) * np.float32(sigma)
        b = torch.from_numpy(z).to(FP8_TORCH[fmt]).view(torch.uint8).numpy()
        return b.view(np.uint16)
    return _pieces(n_pairs, fn, np.empty(n_pairs, np.uint16))


def random_bits(n: int, bits: int, seed: int = 12) -> np.ndarray:
    dt = np.uint16 if bits == 16 else np.uint32

    def fn(p, lo, hi):
        return _rng(seed, p).integers(0, 1 << bits, hi - lo, dtype=np.uint64).astype(dt)
    return _pieces(n, fn, np.empty(n, dt))


# IEEE layouts (exponent bits, fraction bits) of the types whose exponent
# field is exactly 8 bits wide
_EXP8 = {"bf16": (16, 7), "fp32": (32, 23)}


def exponent_multiset(counts: dict, dtype: str = "bf16", seed: int = 21) -> np.ndarray:
    """Values whose biased exponent fields form the given multiset
    ({exponent: count}), with uniformly random signs and fractions, in a
    seeded random order.  bf16 or fp32 bit patterns."""
    bits, fbits = _EXP8[dtype]
    dt = np.uint16 if bits == 16 else np.uint32
    rng = _rng(seed, 0)
    exps = np.concatenate([np.full(c, e, np.uint64) for e, c in sorted(counts.items())])
    rng.shuffle(exps)
    n = exps.size
    sign = rng.integers(0, 2, n, dtype=np.uint64)
    frac = rng.integers(0, 1 << fbits, n, dtype=np.uint64)
    return ((sign << (bits - 1)) | (exps << fbits) | frac).astype(dt)


# --------------------------------------------------------------------------
# weight_sync: 1 GiB bf16 buffer shaped like a 0.5B-parameter transformer
# --------------------------------------------------------------------------
WEIGHT_SYNC_ELEMS = 1 << 29
HIDDEN, FFN, VOCAB, LAYERS = 896, 4864, 151936, 24


def weight_sync_layout(total: int = WEIGHT_SYNC_ELEMS):
    """[(name, start, length, mean, std)] in buffer order.

    Embedding [151936 x 896] N(0, 1); 24 layers of q, o [896 x 896],
    gate, up [896 x 4864], down [4864 x 896] N(0, 0.02) and two norm
    vectors [896] N(1, 0.05); the rest of the 1 GiB buffer N(0, 0.02)
    (standing in for the omitted k/v projections and other tensors)."""
    segs = []
    pos = 0

    def add(name, length, mean, std):
        nonlocal pos
        segs.append((name, pos, length, mean, std))
        pos += length

    add("embed", VOCAB * HIDDEN, 0.0, 1.0)
    for layer in range(LAYERS):
        add(f"l{layer}.q", HIDDEN * HIDDEN, 0.0, 0.02)
        add(f"l{layer}.o", HIDDEN * HIDDEN, 0.0, 0.02)
        add(f"l{layer}.gate", HIDDEN * FFN, 0.0, 0.02)
        add(f"l{layer}.up", HIDDEN * FFN, 0.0, 0.02)
        add(f"l{layer}.down", FFN * HIDDEN, 0.0, 0.02)
        add(f"l{layer}.input_norm", HIDDEN, 1.0, 0.05)
        add(f"l{layer}.post_norm", HIDDEN, 1.0, 0.05)
    assert pos <= total
    add("rest", total - pos, 0.0, 0.02)
    return segs


def weight_sync(n: int = WEIGHT_SYNC_ELEMS, seed: int = 2) -> np.ndarray:
    """The first n elements of the weight-sync buffer."""
    segs = weight_sync_layout()
    starts = np.array([s[1] for s in segs], np.int64)
    means = np.array([s[3] for s in segs], np.float32)
    stds = np.array([s[4] for s in segs], np.float32)

    def fn(p, lo, hi):
        z = _rng(seed, p).standard_normal(hi - lo, dtype=np.float32)
        idx = np.searchsorted(starts, np.arange(lo, hi, dtype=np.int64), side="right") - 1
        return to_bf16_bits(means[idx] + stds[idx] * z)
    return _pieces(n, fn, np.empty(n, np.uint16))


# --------------------------------------------------------------------------
# grad_fp32 / grad_fp16: gradient-like values
# --------------------------------------------------------------------------
def grad_fp32(n: int = 1 << 28, seed: int = 3) -> np.ndarray:
    """Laplace(0, 1e-4); each entry independently scaled x100 with
    probability 0.01 (outliers at random positions)."""
    def fn(p, lo, hi):
        g = _rng(seed, p)
        x = g.laplace(0.0, 1e-4, hi - lo)
        x[g.random(hi - lo) < 0.01] *= 100.0
        return x.astype(np.float32).view(np.uint32)
    return _pieces(n, fn, np.empty(n, np.uint32))


def grad_fp16(n: int = 1 << 28, seed: int = 3) -> np.ndarray:
    """The same values as grad_fp32, rounded to fp16 (many fp16 subnormals)."""
    def fn(p, lo, hi):
        g = _rng(seed, p)
        x = g.laplace(0.0, 1e-4, hi - lo)
        x[g.random(hi - lo) < 0.01] *= 100.0
        return to_fp16_bits(x.astype(np.float32))
    return _pieces(n, fn, np.empty(n, np.uint16))


# --------------------------------------------------------------------------
# kv_cache: [layers, 2, tokens, kv_heads, head_dim] bf16
# --------------------------------------------------------------------------
def kv_cache(layers: int = 32, tokens: int = 16384, kv_heads: int = 8, head_dim: int = 128,
             seed: int = 4) -> np.ndarray:
    """Per (layer, K/V, head, channel) scale ~ LogNormal(0, 0.5); in each
    head 4 channels (chosen without replacement) are outliers at 20x scale;
    values = scale * N(0, 1).  One (layer, K/V) slab per seed child."""
    slab = tokens * kv_heads * head_dim
    out = np.empty(layers * 2 * slab, np.uint16)

    def work(s: int) -> None:
        g = _rng(seed, s)
        sigma = g.lognormal(0.0, 0.5, (kv_heads, head_dim)).astype(np.float32)
        for h in range(kv_heads):
            sigma[h, g.choice(head_dim, 4, replace=False)] *= 20.0
        z = g.standard_normal((tokens, kv_heads, head_dim), dtype=np.float32)
        out[s * slab:(s + 1) * slab] = to_bf16_bits((z * sigma[None]).ravel())

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, range(layers * 2)))
    return out


# --------------------------------------------------------------------------
# reduce_slices: one rank's share of an 8-way all-reduce
# --------------------------------------------------------------------------
def reduce_slices(n_in: int = 8, tokens: int = 1024, hidden: int = 8192, seed: int = 5):
    """n_in bf16 shares [tokens, hidden] of an activation tensor: per-token
    scale s_t ~ U(0.5, 2) drawn once, share r = s_t * N(0, 1)."""
    scale = _rng(seed, 0).uniform(0.5, 2.0, tokens).astype(np.float32)
    outs = [np.empty(tokens * hidden, np.uint16) for _ in range(n_in)]

    def work(r: int) -> None:
        z = _rng(seed, r + 1).standard_normal((tokens, hidden), dtype=np.float32)
        outs[r][:] = to_bf16_bits((z * scale[:, None]).ravel())

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, range(n_in)))
    return outs


# --------------------------------------------------------------------------
# the five measured configurations
# --------------------------------------------------------------------------
CONFIGS = {
    "normal_bf16_4MiB": dict(dtype="bf16", block_bytes=65536, n=2_097_152),
    "weight_sync_bf16_1GiB": dict(dtype="bf16", block_bytes=65536, chunk_bytes=4 << 20,
                                  n=WEIGHT_SYNC_ELEMS),
    "grad_fp32_1GiB": dict(dtype="fp32", block_bytes=262144, n=1 << 28),
    "grad_fp16_512MiB": dict(dtype="fp16", block_bytes=262144, n=1 << 28),
    "kv_cache_bf16_2GiB": dict(dtype="bf16", block_bytes=65536, chunk_bytes=1 << 20, n=1 << 30),
    "reduce_8x_bf16_16MiB": dict(dtype="bf16", block_bytes=65536, n=1 << 23, n_in=8),
}


def generate(name: str):
    if name == "normal_bf16_4MiB":
        return normal_bf16()
    if name == "weight_sync_bf16_1GiB":
        return weight_sync()
    if name == "grad_fp32_1GiB":
        return grad_fp32()
    if name == "grad_fp16_512MiB":
        return grad_fp16()
    if name == "kv_cache_bf16_2GiB":
        return kv_cache()
    if name == "reduce_8x_bf16_16MiB":
        return reduce_slices()
    raise KeyError(name)
