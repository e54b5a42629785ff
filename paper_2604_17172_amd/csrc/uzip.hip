// uzip.hip -- gfx950 kernels and C ABI of the block-wise lossless float codec.
//
// Method (arXiv 2604.17172): section 2.1.2 (split, per-block ANS, one
// contiguous stream), section 3.3.1 (localized per-block tables, all steps
// fused in one launch, no third coalescing pass), section 3.2.3 (split-send:
// the raw plane is published before coding ends), section 3.4 (fused
// decompress -> reduce -> recompress), section 4.1 (metadata with dtype and
// sizes).  Stream layout: include/uzip.h.
//
// Kernel design (one wave64 per codec block, as the paper runs one warp per
// compression block):
//   encode_kernel   pass 1 streams the block once (16-byte loads), writes
//                   the raw plane to its final place and builds the block
//                   histogram in LDS sub-histograms; the table is built with
//                   wave reductions and scans; pass 2 runs the 64 interleaved
//                   rANS states backwards over the block, compacting the
//                   emitted 16-bit words with ballot/mbcnt into an LDS
//                   staging area; the block's output offset comes from a
//                   single-pass scan with decoupled look-back over blocks
//                   taken in ticket order; the section is then stored with
//                   16-byte writes straight into the final stream.
//   decode_kernel   grid-stride over blocks; each block's offset is read
//                   from the directory, its decode table (2048 x u32) is
//                   built in LDS and the 64 states decode forwards.
//   encode_kernel<REDUCE>  pass 1 decodes block b of every input in lock
//                   step round by round and adds in binary32 in input order.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "../../include/uzip.h"
#include "uzip_device.h"

using namespace uzip;

namespace {

constexpr int kMaxInputs = 16;
constexpr uint32_t kMinBlockBytes = 4096, kMaxBlockBytes = 262144;

struct EncodeArgs {
  const uint8_t *in;        // elements to compress (compress modes)
  uint64_t n;               // total elements
  uint64_t chunk_elems;     // elements per stream (one stream: >= n)
  uint32_t block_elems;
  uint32_t blocks_per_chunk;
  uint32_t n_blocks;        // over all chunks
  uint32_t wcap;            // word capacity of the LDS staging area
  uint32_t pass2_off;       // LDS byte offset of the staging area
  uint32_t epoch;
  uint8_t *out;
  uint64_t slot_bytes;      // distance between chunk streams
  uint64_t *sizes;          // per-stream total bytes (may be null)
  uint32_t *flags;          // split-send flags (may be null)
  uint32_t *ticket;         // workspace: block ticket counter
  uint64_t *status;         // workspace: look-back status per block
  uint32_t *chunk_cnt;      // workspace: [2 * chunks] completion counters
  // fused reduce only
  int n_in;
  const uint8_t *ins[kMaxInputs];
  uint64_t in_bytes[kMaxInputs];
  const uint8_t *local_raw;
  uint8_t *ybuf;            // reduced tensor, re-read by pass 2
  uint32_t *dstatus;
};

struct DecodeArgs {
  const uint8_t *in;
  uint64_t in_bytes;
  uint64_t n;
  uint32_t dtype;
  uint8_t *out;
  uint32_t *dstatus;
};

// first error wins
__device__ inline void report(uint32_t *dstatus, int code) {
  if (dstatus != nullptr) {
    uint32_t expected = 0;
    __hip_atomic_compare_exchange_strong(dstatus, &expected, (uint32_t)code, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ inline uint32_t ld32(const uint8_t *p) { return *(const uint32_t *)p; }
__device__ inline uint64_t ld64(const uint8_t *p) {
  return (uint64_t)ld32(p) | ((uint64_t)ld32(p + 4) << 32);
}

// ---------------------------------------------------------------------------
// Element groups: lane j of round r owns elements 512 r + 8 j .. +7 of a block
// ---------------------------------------------------------------------------
template <int E>
__device__ inline void load_words(const uint8_t *base, uint64_t first, uint32_t valid, uint32_t w[4 * (E / 2)]) {
  // first: element index of the group; valid: how many of its 8 elements exist
  if (valid >= 8) {
    const uint4 *p = (const uint4 *)(base + first * E);
    uint4 a = p[0];
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    if (E == 4) {
      uint4 b = p[1];
      w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4 * (E / 2); ++q) w[q] = 0;
#pragma unroll
    for (uint32_t q = 0; q < 8; ++q) {
      if (q < valid) {
        if (E == 2) {
          uint32_t v = ((const uint16_t *)base)[first + q];
          w[q >> 1] |= v << (16 * (q & 1));
        } else {
          w[q] = ((const uint32_t *)base)[first + q];
        }
      }
    }
  }
}

template <int E>
__device__ inline void split_group(const uint32_t w[4 * (E / 2)], Group &g) {
  if (E == 2)
    split16(w, g);
  else
    split32(w, g);
}

// raw plane bytes of a group: 8 (E = 2) or 24 (E = 4) bytes at plane + (E-1) first
template <int E>
__device__ inline void store_raw(uint8_t *plane, uint64_t first, uint32_t valid, const Group &g) {
  uint8_t *p = plane + (uint64_t)(E - 1) * first;
  if (valid >= 8) {
    uint2 *q = (uint2 *)p;
    q[0] = make_uint2(g.raw[0], g.raw[1]);
    if (E == 4) {
      q[1] = make_uint2(g.raw[2], g.raw[3]);
      q[2] = make_uint2(g.raw[4], g.raw[5]);
    }
  } else {
#pragma unroll
    for (uint32_t b = 0; b < 8 * (E - 1); ++b)
      if (b < (E - 1) * valid) p[b] = (uint8_t)(g.raw[b >> 2] >> (8 * (b & 3)));
  }
}

template <int E>
__device__ inline void load_raw(const uint8_t *plane, uint64_t first, uint32_t valid, uint32_t raw[6]) {
  const uint8_t *p = plane + (uint64_t)(E - 1) * first;
  if (valid >= 8) {
    const uint2 *q = (const uint2 *)p;
    uint2 a = q[0];
    raw[0] = a.x; raw[1] = a.y;
    if (E == 4) {
      uint2 b = q[1], c = q[2];
      raw[2] = b.x; raw[3] = b.y; raw[4] = c.x; raw[5] = c.y;
    }
  } else {
#pragma unroll
    for (int q = 0; q < 6; ++q) raw[q] = 0;
#pragma unroll
    for (uint32_t b = 0; b < 8 * (E - 1); ++b)
      if (b < (E - 1) * valid) raw[b >> 2] |= (uint32_t)p[b] << (8 * (b & 3));
  }
}

template <int E>
__device__ inline void merge_group(const uint32_t sym[2], const uint32_t raw[6], uint32_t w[4 * (E / 2)]) {
  if (E == 2)
    merge16(sym, raw, w);
  else
    merge32(sym, raw, w);
}

template <int E>
__device__ inline void store_words(uint8_t *base, uint64_t first, uint32_t valid, const uint32_t w[4 * (E / 2)]) {
  if (valid >= 8) {
    uint4 *p = (uint4 *)(base + first * E);
    p[0] = make_uint4(w[0], w[1], w[2], w[3]);
    if (E == 4) p[1] = make_uint4(w[4], w[5], w[6], w[7]);
  } else {
#pragma unroll
    for (uint32_t q = 0; q < 8; ++q) {
      if (q < valid) {
        if (E == 2)
          ((uint16_t *)base)[first + q] = (uint16_t)(w[q >> 1] >> (16 * (q & 1)));
        else
          ((uint32_t *)base)[first + q] = w[q];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Decode side: table of one coded block -> 2048-entry lookup table in LDS.
// Entry for slot: f | (slot - cum) << 12 | sym << 24.
// Returns false (uniformly) if the stored table is not a valid ANS table.
// ---------------------------------------------------------------------------
__device__ bool build_lut(const uint8_t *sec, uint64_t sec_len, uint32_t *lut, uint16_t *cum_s,
                          uint16_t *f_s, uint32_t &k_out) {
  const uint32_t lane = lane_id();
  if (sec_len < kSectionFixed) return false;
  // presence bits of symbols 4 lane .. 4 lane + 3
  uint32_t byte = sec[256 + (lane >> 1)];
  uint32_t nib = (byte >> (4 * (lane & 1))) & 0xFu;
  uint32_t pres = __popc(nib);
  uint32_t k = wave_sum(pres);
  uint32_t rank0 = wave_excl_scan(pres);
  bool ok = k >= 1 && (uint64_t)kSectionFixed + 2ull * k <= sec_len;
  uint32_t f[4] = {0, 0, 0, 0};
  uint32_t r = rank0, total = 0;
  if (ok) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (nib & (1u << q)) {
        const uint8_t *p = sec + kSectionFixed + 2 * r;
        f[q] = (uint32_t)p[0] | ((uint32_t)p[1] << 8);
        ++r;
      }
      total += f[q];
    }
  }
  uint32_t bad = (nib & 1 && f[0] == 0) | (nib & 2 && f[1] == 0) | (nib & 4 && f[2] == 0) |
                 (nib & 8 && f[3] == 0);
  ok = ok && !__any(bad) && wave_sum(total) == kM;
  if (!ok) return false;
  uint32_t c = wave_excl_scan(total);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    cum_s[4 * lane + q] = (uint16_t)c;
    f_s[4 * lane + q] = (uint16_t)f[q];
    c += f[q];
  }
  __syncthreads();
  // lane fills slots 32 lane .. 32 lane + 31: find the owner of the first one
  uint32_t slot = 32 * lane;
  uint32_t lo = 0, hi = 255;  // largest s with cum[s] <= slot
  while (lo < hi) {
    uint32_t mid = (lo + hi + 1) >> 1;
    if (cum_s[mid] <= slot)
      lo = mid;
    else
      hi = mid - 1;
  }
  uint32_t s = lo;
  for (uint32_t q = 0; q < 32; ++q, ++slot) {
    while (slot >= (uint32_t)cum_s[s] + f_s[s]) ++s;
    uint32_t fs = f_s[s];
    lut[slot] = fs | ((slot - cum_s[s]) << 12) | (s << 24);
  }
  __syncthreads();
  k_out = k;
  return true;
}

// One decode sub-step of one lane; returns the symbol.
__device__ inline uint32_t decode_step(uint32_t &x, bool valid, const uint32_t *lut, const uint16_t *words,
                                       uint32_t &p, uint32_t w_avail, bool &bad) {
  uint32_t s = 0;
  if (valid) {
    uint32_t e = lut[x & (kM - 1)];
    uint32_t f = e & 0xFFFu;
    uint32_t bias = (e >> 12) & 0x7FFu;
    s = e >> 24;
    x = __umul24(f, x >> kProbBits) + bias;
  }
  bool need = valid && x < kStateLo;
  uint64_t m = __ballot(need);
  if (need) {
    uint32_t idx = p + mbcnt(m);
    uint32_t w = 0;
    if (idx < w_avail)
      w = words[idx];
    else
      bad = true;
    x = (x << 16) | w;
  }
  p += (uint32_t)__popcll(m);
  return s;
}

// ---------------------------------------------------------------------------
// Encode side
// ---------------------------------------------------------------------------
struct Table {
  uint32_t k;          // present symbols
  uint32_t f[4];       // frequencies of symbols 4 lane .. +3
  uint32_t rank0;      // rank of this lane's first present symbol
  uint64_t present[4]; // ballots: bit j of present[q] = symbol 4 j + q present
};

// Localized table of one block (section 3.3.1): f[s] = 1 + floor(c(M-k)/n_b)
// for present symbols, the remainder to the most frequent symbol (ties to
// the smallest), cum in ascending symbol order.  Writes the encoder table
// {reciprocal, f << 20, (M - f) | shift << 24, cum (+2047 if f == 1)}.
__device__ void build_enc_table(const uint32_t *hist, uint32_t n_b, uint4 *enc, Table &t) {
  const uint32_t lane = lane_id();
  uint32_t c[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t s = 4 * lane + q, acc = 0;
#pragma unroll
    for (uint32_t rep = 0; rep < kHistReplicas; ++rep) acc += hist[rep * kHistStride + s];
    c[q] = acc;
  }
  uint32_t pres = (c[0] > 0) + (c[1] > 0) + (c[2] > 0) + (c[3] > 0);
  uint32_t k = wave_sum(pres);
  uint32_t lt = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    t.f[q] = c[q] ? 1u + (uint32_t)(((uint64_t)c[q] * (kM - k)) / n_b) : 0u;
    lt += t.f[q];
  }
  uint32_t d = kM - wave_sum(lt);
  uint32_t key = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t kq = (c[q] << 8) | (255u - (4 * lane + q));
    key = kq > key ? kq : key;
  }
  key = wave_max(key);
  uint32_t best = 255u - (key & 0xFFu);
#pragma unroll
  for (uint32_t q = 0; q < 4; ++q)
    if (best == 4 * lane + q) t.f[q] += d;
  lt = t.f[0] + t.f[1] + t.f[2] + t.f[3];
  uint32_t cum = wave_excl_scan(lt);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t f = t.f[q];
    uint4 e = make_uint4(0, 0, 0, 0);
    if (f > 0) {
      uint32_t l = 32 - __clz(f - 1);  // ceil(log2 f) for f >= 2
      if (f == 1) {
        // floor(x / 1) = x = mulhi(x, 2^32 - 1) + 1 for 1 <= x < 2^32; the
        // missing (M - 1) is folded into the additive term
        e = make_uint4(0xFFFFFFFFu, 1u << 20, (kM - 1) | (0u << 24), cum + (kM - 1));
      } else {
        // floor(x / f) = mulhi(x, m) >> (l - 1), m = ceil(2^(31+l) / f),
        // exact for x < 2^31 (division by invariant integers)
        uint32_t m = (uint32_t)(((1ull << (31 + l)) + f - 1) / f);
        e = make_uint4(m, f << 20, (kM - f) | ((l - 1) << 24), cum);
      }
      enc[4 * lane + q] = e;
    }
    cum += f;
  }
  t.k = k;
  t.rank0 = wave_excl_scan(pres);
#pragma unroll
  for (int q = 0; q < 4; ++q) t.present[q] = __ballot(c[q] > 0);
}

// Decoupled look-back over the blocks of one stream: returns the exclusive
// prefix (16-byte units) of block b, whose stream's first block is `first`.
// Every block publishes its status, and blocks are taken in ticket order, so
// the wait always ends; the spin is bounded anyway, and a wait that runs out
// raises the workspace error word instead of hanging.
constexpr uint32_t kSpinLimit = 1u << 22;
__device__ uint64_t lookback(uint64_t *status, uint32_t b, uint32_t first, uint64_t len16, uint32_t *err) {
  const uint32_t lane = lane_id();
  if (b == first) {
    if (lane == 0) __hip_atomic_store(&status[b], kFlagInclusive | len16, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return 0;
  }
  if (lane == 0) __hip_atomic_store(&status[b], kFlagAggregate | len16, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  uint64_t excl = 0;
  int64_t look = (int64_t)b - 1;
  uint32_t spins = 0;
  while (true) {
    int64_t idx = look - (int64_t)lane;
    uint64_t st = kFlagInclusive;  // before the stream's first block: inclusive 0
    if (idx >= (int64_t)first) st = __hip_atomic_load(&status[idx], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint32_t flag = (uint32_t)(st >> 62);
    uint64_t inc = __ballot(flag == 2);
    uint64_t upto = inc ? ((inc & (~inc + 1)) << 1) - 1 : ~0ull;  // lanes up to the first inclusive
    uint64_t notready = __ballot(flag == 0) & upto;
    if (notready) {
      if (++spins < kSpinLimit) {
        __builtin_amdgcn_s_sleep(2);
        continue;
      }
      if (lane == 0) __hip_atomic_store(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    uint64_t v = ((upto >> lane) & 1) ? (st & kValueMask) : 0;
    excl += wave_sum64(v);
    if (inc) break;
    look -= 64;
  }
  if (lane == 0)
    __hip_atomic_store(&status[b], kFlagInclusive | (excl + len16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return excl;
}

// Counter of finished blocks of a chunk; the last one publishes the flag.
__device__ void publish_chunk(uint32_t *cnt, uint32_t need, uint32_t *flag, uint32_t epoch) {
  if (lane_id() == 0) {
    uint32_t old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_SYSTEM);
    if (old + 1 == need) __hip_atomic_store(flag, epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// Fused reduce, pass 1 helpers: per-input state of the block being reduced.
struct InBlock {
  const uint8_t *sec;
  const uint16_t *words;
  const uint8_t *raw_plane;
  uint32_t w_avail;
  uint32_t stored;
};

template <int DT>
__device__ inline float to_f32(uint32_t w) {
  if (DT == 0) return bf16_to_f32(w);
  if (DT == 1) return fp16_to_f32(w);
  return __uint_as_float(w);
}

template <int DT>
__device__ inline uint32_t from_f32(float f) {
  if (DT == 0) return f32_to_bf16(f);
  if (DT == 1) return f32_to_fp16(f);
  return (f != f) ? 0x7FC00000u : __float_as_uint(f);
}

// ---------------------------------------------------------------------------
// encode_kernel: compress / split-send producer / fused reduce
// ---------------------------------------------------------------------------
template <int DT, bool REDUCE>
__global__ void __launch_bounds__(64) encode_kernel(EncodeArgs a) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  extern __shared__ __align__(16) uint8_t smem[];
  uint4 *enc = (uint4 *)smem;
  uint32_t *hist = (uint32_t *)(smem + kEncTableBytes);
  uint8_t *stage = smem + a.pass2_off;
  uint16_t *stage16 = (uint16_t *)(stage + kStageHead);
  const uint32_t lane = lane_id();

  uint32_t b = 0;
  if (lane == 0) b = __hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  b = uniform(b);
  if (b >= a.n_blocks) return;

  const uint32_t chunk = b / a.blocks_per_chunk;
  const uint32_t lb = b - chunk * a.blocks_per_chunk;
  const uint32_t first_block = b - lb;
  const uint64_t chunk_first = (uint64_t)chunk * a.chunk_elems;
  const uint64_t chunk_n = (a.n - chunk_first) < a.chunk_elems ? (a.n - chunk_first) : a.chunk_elems;
  const Geom g = make_geom(chunk_n, a.block_elems, E);
  uint8_t *sout = a.out + (uint64_t)chunk * a.slot_bytes;
  const uint64_t blk0 = (uint64_t)lb * a.block_elems;  // chunk-relative
  const uint32_t n_b = (uint32_t)((chunk_n - blk0) < a.block_elems ? (chunk_n - blk0) : a.block_elems);
  const uint32_t rounds = (n_b + kRound - 1) / kRound;
  const bool last_in_chunk = (lb + 1 == g.n_blocks);
  const uint8_t *src = REDUCE ? a.ybuf : a.in + chunk_first * E;  // pass 2 source

  // ---- pass 1: split, raw plane, histogram ----
  for (uint32_t i = lane; i < kHistReplicas * kHistStride; i += 64) hist[i] = 0;
  __syncthreads();

  if constexpr (!REDUCE) {
    for (uint32_t r = 0; r < rounds; ++r) {
      uint32_t i0 = r * kRound + kPerLane * lane;
      uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
      if (valid == 0) continue;
      uint32_t w[NW];
      load_words<E>(src, blk0 + i0, valid, w);
      Group gr;
      split_group<E>(w, gr);
      store_raw<E>(sout + g.raw_off, blk0 + i0, valid, gr);
      uint32_t *h = hist + (lane & (kHistReplicas - 1)) * kHistStride;
#pragma unroll
      for (uint32_t q = 0; q < 8; ++q)
        if (q < valid) atomicAdd(&h[sym_at(gr.sym, q)], 1u);
    }
  } else {
    // fused reduce: decode block b of every input, add in order, round
    uint32_t *luts = (uint32_t *)(smem + kEncTableBytes + kHistBytes);
    uint16_t *cum_s = (uint16_t *)(smem + kEncTableBytes + kHistBytes + a.n_in * kLutBytes);
    uint16_t *f_s = cum_s + 256;
    InBlock ib[kMaxInputs];
    uint32_t x[kMaxInputs], p[kMaxInputs];
    bool bad = false;
#pragma unroll
    for (int i = 0; i < kMaxInputs; ++i) {
      x[i] = kStateLo;
      p[i] = 0;
      ib[i].sec = nullptr;
      ib[i].words = nullptr;
      ib[i].raw_plane = nullptr;
      ib[i].w_avail = 0;
      ib[i].stored = 1;
      if (i < a.n_in) {
        const uint8_t *s = a.ins[i];
        const uint64_t total = ld64(s + 24);
        const uint32_t be = ld32(s + 8), nb = ld32(s + 12);
        bool ok = a.in_bytes[i] >= kHeaderBytes && ld32(s) == kMagic && s[4] == kVersion && s[5] == DT &&
                  s[6] == kProbBits && s[7] == 0 && be == a.block_elems && nb == g.n_blocks &&
                  ld64(s + 16) == chunk_n && total <= a.in_bytes[i] && total >= g.coded_off;
        uint64_t start = 0, end = 0;
        uint32_t d = 0;
        if (ok) {
          d = ld32(s + kHeaderBytes + 4 * lb);
          start = lb ? 16ull * (ld32(s + kHeaderBytes + 4 * (lb - 1)) & ~kStoredBit) : 0;
          end = 16ull * (d & ~kStoredBit);
          ok = end >= start && g.coded_off + end <= total;
        }
        if (ok) {
          ib[i].sec = s + g.coded_off + start;
          ib[i].raw_plane = s + g.raw_off;
          ib[i].stored = d >> 31;
          if (ib[i].stored) {
            ok = end - start >= n_b;
          } else {
            uint32_t k = 0;
            ok = build_lut(ib[i].sec, end - start, luts + i * kM, cum_s, f_s, k);
            if (ok) {
              x[i] = ((const uint32_t *)ib[i].sec)[lane];
              ok = !__any(x[i] < kStateLo || x[i] >= 0x80000000u);
              ib[i].words = (const uint16_t *)(ib[i].sec + kSectionFixed + 2 * k);
              ib[i].w_avail = (uint32_t)((end - start - kSectionFixed - 2 * k) / 2);
            }
          }
        }
        if (!ok) {
          bad = true;
          ib[i].stored = 1;
          ib[i].sec = nullptr;
        }
      }
    }
    __syncthreads();
    for (uint32_t r = 0; r < rounds; ++r) {
      uint32_t i0 = r * kRound + kPerLane * lane;
      uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
      float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < kMaxInputs; ++i) {
        if (i < a.n_in) {
          uint32_t sym[2] = {0, 0};
          if (ib[i].stored) {
            if (ib[i].sec != nullptr && valid > 0)
#pragma unroll
              for (uint32_t q = 0; q < 8; ++q)
                if (q < valid) sym[q >> 2] |= (uint32_t)ib[i].sec[i0 + q] << (8 * (q & 3));
          } else {
#pragma unroll
            for (uint32_t t = 0; t < kPerLane; ++t) {
              uint32_t s = decode_step(x[i], t < valid, luts + i * kM, ib[i].words, p[i], ib[i].w_avail, bad);
              sym[t >> 2] |= s << (8 * (t & 3));
            }
          }
          uint32_t raw[6] = {0, 0, 0, 0, 0, 0};
          if (valid > 0 && ib[i].raw_plane != nullptr) load_raw<E>(ib[i].raw_plane, blk0 + i0, valid, raw);
          uint32_t w[NW];
          merge_group<E>(sym, raw, w);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            uint32_t wq = (E == 2) ? ((w[q >> 1] >> (16 * (q & 1))) & 0xFFFFu) : w[q];
            float v = to_f32<DT>(wq);
            acc[q] = (i == 0) ? v : acc[q] + v;
          }
        }
      }
      if (valid == 0) continue;
      if (a.local_raw != nullptr) {
        uint32_t w[NW];
        load_words<E>(a.local_raw, blk0 + i0, valid, w);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          uint32_t wq = (E == 2) ? ((w[q >> 1] >> (16 * (q & 1))) & 0xFFFFu) : w[q];
          acc[q] = acc[q] + to_f32<DT>(wq);
        }
      }
      uint32_t w[NW];
#pragma unroll
      for (int q = 0; q < NW; ++q) w[q] = 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        uint32_t y = from_f32<DT>(acc[q]);
        if (E == 2)
          w[q >> 1] |= y << (16 * (q & 1));
        else
          w[q] = y;
      }
      store_words<E>(a.ybuf, blk0 + i0, valid, w);
      Group gr;
      split_group<E>(w, gr);
      store_raw<E>(sout + g.raw_off, blk0 + i0, valid, gr);
      uint32_t *h = hist + (lane & (kHistReplicas - 1)) * kHistStride;
#pragma unroll
      for (uint32_t q = 0; q < 8; ++q)
        if (q < valid) atomicAdd(&h[sym_at(gr.sym, q)], 1u);
    }
#pragma unroll
    for (int i = 0; i < kMaxInputs; ++i)
      if (i < a.n_in && !ib[i].stored && x[i] != kStateLo) bad = true;
    if (__any(bad) && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
  }

  if (last_in_chunk && lane < 16) {
    // zero padding after the raw plane (pad16 of (E-1) n bytes)
    uint64_t rb = g.raw_off + (uint64_t)(E - 1) * chunk_n + lane;
    if (rb < g.coded_off) sout[rb] = 0;
  }
  __syncthreads();
  if (a.flags != nullptr) {
    __threadfence_system();
    publish_chunk(&a.chunk_cnt[2 * chunk], g.n_blocks, &a.flags[2 * chunk], a.epoch);
  }

  // ---- table ----
  Table t;
  build_enc_table(hist, n_b, enc, t);
  __syncthreads();

  // ---- pass 2: rANS over the block, backwards; words staged in LDS ----
  for (uint32_t i = lane; i < kStageTail / 4; i += 64)
    ((uint32_t *)(stage + kStageHead + 2 * a.wcap))[i] = 0;
  const uint32_t limit_words = (n_b > kSectionFixed + 2 * t.k) ? (n_b - kSectionFixed - 2 * t.k + 1) / 2 : 0;
  uint32_t pos = a.wcap;  // stage16[pos .. wcap) hold the words written so far
  uint32_t x = kStateLo;
  bool stored = (limit_words == 0);
  for (int r = (int)rounds - 1; r >= 0 && !stored; --r) {
    uint32_t i0 = (uint32_t)r * kRound + kPerLane * lane;
    uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
    uint32_t w[NW];
    Group gr;
    gr.sym[0] = gr.sym[1] = 0;
    if (valid > 0) {
      load_words<E>(src, blk0 + i0, valid, w);
      split_group<E>(w, gr);
    }
#pragma unroll
    for (int tt = kPerLane - 1; tt >= 0; --tt) {
      const bool v = (uint32_t)tt < valid;
      uint4 e = enc[sym_at(gr.sym, tt)];
      const bool emit = v && x >= e.y;
      const uint64_t m = __ballot(emit);
      const uint32_t cnt = (uint32_t)__popcll(m);
      if (emit) {
        stage16[pos - cnt + mbcnt(m)] = (uint16_t)x;
        x >>= 16;
      }
      pos -= cnt;
      if (v) {
        uint32_t q = __umulhi(x, e.x) >> (e.z >> 24);
        x = x + __umul24(q, e.z & 0xFFFFu) + e.w;
      }
    }
    if (a.wcap - pos >= limit_words) stored = true;  // coded section no smaller than n_b
  }
  const uint32_t n_words = a.wcap - pos;
  const uint64_t img = kSectionFixed + 2ull * t.k + 2ull * n_words;
  const uint64_t sec_len = stored ? pad16(n_b) : pad16(img);

  // ---- output offset: single-pass scan over the stream's blocks ----
  const uint64_t excl = lookback(a.status, b, first_block, sec_len / 16, a.ticket + 1);
  uint8_t *sec = sout + g.coded_off + 16 * excl;
  if (lane == 0)
    *(uint32_t *)(sout + kHeaderBytes + 4 * lb) = (stored ? kStoredBit : 0u) | (uint32_t)(excl + sec_len / 16);

  if (!stored) {
    // assemble states | bitmap | f[k] in front of the words, then copy out
    const uint32_t A = kStageHead + 2 * pos - (kSectionFixed + 2 * t.k);
    uint16_t *h16 = (uint16_t *)(stage + A);
    h16[2 * lane] = (uint16_t)x;
    h16[2 * lane + 1] = (uint16_t)(x >> 16);
    if (lane < 16) {
      uint32_t word = 0;
      for (uint32_t bit = 0; bit < 16; ++bit) {
        uint32_t s = 16 * lane + bit;
        word |= (uint32_t)((t.present[s & 3] >> (s >> 2)) & 1u) << bit;
      }
      h16[128 + lane] = (uint16_t)word;
    }
    uint32_t rk = t.rank0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (t.f[q]) h16[144 + rk++] = (uint16_t)t.f[q];
    __syncthreads();
    const uint32_t *s32 = (const uint32_t *)(stage + (A & ~3u));
    const uint32_t sh = A & 3u;
    for (uint32_t u = lane; u < sec_len / 16; u += 64) {
      const uint32_t *q = s32 + 4 * u;
      uint4 o;
      o.x = __builtin_amdgcn_alignbyte(q[1], q[0], sh);
      o.y = __builtin_amdgcn_alignbyte(q[2], q[1], sh);
      o.z = __builtin_amdgcn_alignbyte(q[3], q[2], sh);
      o.w = __builtin_amdgcn_alignbyte(q[4], q[3], sh);
      ((uint4 *)sec)[u] = o;
    }
  } else {
    // STORED: the block's symbol bytes, zero-padded to 16
    const uint32_t padded = (uint32_t)pad16(n_b);
    for (uint32_t r = 0; r < rounds; ++r) {
      uint32_t i0 = r * kRound + kPerLane * lane;
      if (i0 >= padded) continue;
      uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
      Group gr;
      gr.sym[0] = gr.sym[1] = 0;
      if (valid > 0) {
        uint32_t w[NW];
        load_words<E>(src, blk0 + i0, valid, w);
        split_group<E>(w, gr);
        if (valid < 8) {
          uint64_t keep = (1ull << (8 * valid)) - 1;
          uint64_t v = ((uint64_t)gr.sym[1] << 32 | gr.sym[0]) & keep;
          gr.sym[0] = (uint32_t)v;
          gr.sym[1] = (uint32_t)(v >> 32);
        }
      }
      *(uint2 *)(sec + i0) = make_uint2(gr.sym[0], gr.sym[1]);
    }
  }

  if (last_in_chunk) {
    const uint64_t total = g.coded_off + 16 * (excl + sec_len / 16);
    if (lane == 0) {
      uint32_t h[8];
      h[0] = kMagic;
      h[1] = kVersion | ((uint32_t)DT << 8) | (kProbBits << 16);
      h[2] = a.block_elems;
      h[3] = g.n_blocks;
      h[4] = (uint32_t)chunk_n;
      h[5] = (uint32_t)(chunk_n >> 32);
      h[6] = (uint32_t)total;
      h[7] = (uint32_t)(total >> 32);
      uint4 *hp = (uint4 *)sout;
      hp[0] = make_uint4(h[0], h[1], h[2], h[3]);
      hp[1] = make_uint4(h[4], h[5], h[6], h[7]);
      if (a.sizes != nullptr) a.sizes[chunk] = total;
    }
    // zero padding after the directory
    uint64_t db = kHeaderBytes + 4ull * g.n_blocks + lane;
    if (lane < 16 && db < g.raw_off) sout[db] = 0;
  }
  if (a.flags != nullptr) {
    __threadfence_system();
    publish_chunk(&a.chunk_cnt[2 * chunk + 1], g.n_blocks, &a.flags[2 * chunk + 1], a.epoch);
  }
}

// ---------------------------------------------------------------------------
// decode_kernel
// ---------------------------------------------------------------------------
template <int DT>
__global__ void __launch_bounds__(64) decode_kernel(DecodeArgs a) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  __shared__ uint32_t lut[kM];
  __shared__ uint16_t cum_s[256], f_s[256];
  const uint32_t lane = lane_id();
  const uint8_t *s = a.in;
  if (a.in_bytes < kHeaderBytes) {
    if (blockIdx.x == 0 && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
    return;
  }
  const uint32_t be = ld32(s + 8);
  const uint32_t nb = ld32(s + 12);
  const uint64_t total = ld64(s + 24);
  bool ok = ld32(s) == kMagic && s[4] == kVersion && s[5] == DT && s[6] == kProbBits && s[7] == 0 &&
            ld64(s + 16) == a.n && be > 0 && (be & (be - 1)) == 0 && (uint64_t)be * E >= kMinBlockBytes &&
            (uint64_t)be * E <= kMaxBlockBytes && (uint64_t)nb == (a.n + be - 1) / be && total <= a.in_bytes;
  Geom g = make_geom(a.n, ok ? be : 1, E);
  ok = ok && total >= g.coded_off;
  if (!ok) {
    if (blockIdx.x == 0 && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
    return;
  }
  if (blockIdx.x == 0 && lane == 0 && nb > 0) {
    uint64_t endall = 16ull * (ld32(s + kHeaderBytes + 4 * (nb - 1)) & ~kStoredBit);
    if (g.coded_off + endall != total) report(a.dstatus, UZIP_ECORRUPT);
  }
  if (blockIdx.x == 0 && lane == 0 && nb == 0 && total != g.coded_off) report(a.dstatus, UZIP_ECORRUPT);

  for (uint32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const uint32_t d = ld32(s + kHeaderBytes + 4 * b);
    const uint64_t start = b ? 16ull * (ld32(s + kHeaderBytes + 4 * (b - 1)) & ~kStoredBit) : 0;
    const uint64_t end = 16ull * (d & ~kStoredBit);
    const uint64_t blk0 = (uint64_t)b * be;
    const uint32_t n_b = (uint32_t)((a.n - blk0) < be ? (a.n - blk0) : be);
    const uint32_t rounds = (n_b + kRound - 1) / kRound;
    bool bad = !(end >= start && g.coded_off + end <= total);
    const uint8_t *sec = s + g.coded_off + start;
    const uint64_t len = bad ? 0 : end - start;
    const bool stored = d >> 31;
    if (!bad && stored && len < n_b) bad = true;
    uint32_t k = 0, x = kStateLo, p = 0, w_avail = 0;
    const uint16_t *words = nullptr;
    if (!bad && !stored) {
      if (len < kSectionFixed || !build_lut(sec, len, lut, cum_s, f_s, k)) {
        bad = true;
      } else {
        x = ((const uint32_t *)sec)[lane];
        if (__any(x < kStateLo || x >= 0x80000000u)) bad = true;
        words = (const uint16_t *)(sec + kSectionFixed + 2 * k);
        w_avail = (uint32_t)((len - kSectionFixed - 2 * k) / 2);
      }
    }
    if (bad) {
      if (lane == 0) report(a.dstatus, UZIP_ECORRUPT);
      continue;
    }
    for (uint32_t r = 0; r < rounds; ++r) {
      uint32_t i0 = r * kRound + kPerLane * lane;
      uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
      uint32_t sym[2] = {0, 0};
      if (stored) {
        if (valid >= 8) {
          uint2 v = *(const uint2 *)(sec + i0);
          sym[0] = v.x;
          sym[1] = v.y;
        } else {
#pragma unroll
          for (uint32_t q = 0; q < 8; ++q)
            if (q < valid) sym[q >> 2] |= (uint32_t)sec[i0 + q] << (8 * (q & 3));
        }
      } else {
#pragma unroll
        for (uint32_t t = 0; t < kPerLane; ++t) {
          uint32_t sy = decode_step(x, t < valid, lut, words, p, w_avail, bad);
          sym[t >> 2] |= sy << (8 * (t & 3));
        }
      }
      if (valid == 0) continue;
      uint32_t raw[6];
      load_raw<E>(s + g.raw_off, blk0 + i0, valid, raw);
      uint32_t w[NW];
      merge_group<E>(sym, raw, w);
      store_words<E>(a.out, blk0 + i0, valid, w);
    }
    if (!stored && x != kStateLo) bad = true;
    if (__any(bad) && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
    __syncthreads();
  }
}

// zero the ticket, the look-back status words and the chunk counters
__global__ void clear_kernel(uint32_t *p, uint64_t words) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// n == 0: the stream is the 32-byte header alone
__global__ void empty_stream_kernel(uint8_t *out, uint32_t dt, uint32_t block_elems, uint64_t *size_out) {
  if (threadIdx.x == 0) {
    uint4 *hp = (uint4 *)out;
    hp[0] = make_uint4(kMagic, kVersion | (dt << 8) | (kProbBits << 16), block_elems, 0);
    hp[1] = make_uint4(0, 0, kHeaderBytes, 0);
    if (size_out != nullptr) *size_out = kHeaderBytes;
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct DeviceInfo {
  int cus = 0;
  bool gfx950 = false;
};

constexpr int kMaxDevices = 64;
DeviceInfo g_info[kMaxDevices];
std::once_flag g_once[kMaxDevices];

uzip_status device_info(DeviceInfo &out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return UZIP_EHIP;
  hipError_t err = hipSuccess;
  std::call_once(g_once[dev], [&]() {
    hipDeviceProp_t prop;
    err = hipGetDeviceProperties(&prop, dev);
    if (err != hipSuccess) return;
    g_info[dev].cus = prop.multiProcessorCount;
    g_info[dev].gfx950 = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    const int lds_max = 160 * 1024;
    (void)hipFuncSetAttribute((const void *)encode_kernel<0, false>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)encode_kernel<1, false>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)encode_kernel<2, false>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)encode_kernel<0, true>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)encode_kernel<1, true>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)encode_kernel<2, true>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
  });
  if (err != hipSuccess) return UZIP_EHIP;
  out = g_info[dev];
  if (!out.gfx950) return UZIP_EUNSUPPORTED;
  return UZIP_OK;
}

uint32_t elem_bytes(uzip_dtype dt) { return dt == UZIP_FP32 ? 4u : 2u; }
bool valid_dtype(uzip_dtype dt) { return dt == UZIP_BF16 || dt == UZIP_FP16 || dt == UZIP_FP32; }
bool valid_block(uint32_t bb) { return bb >= kMinBlockBytes && bb <= kMaxBlockBytes && (bb & (bb - 1)) == 0; }
bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
uint64_t pad256(uint64_t x) { return (x + 255u) & ~uint64_t(255); }

uint64_t max_size(uint32_t E, uint64_t n, uint32_t block_elems) {
  Geom g = make_geom(n, block_elems, E);
  uint64_t full = n / block_elems, tail = n - full * block_elems;
  return g.coded_off + full * pad16(block_elems) + (tail ? pad16(tail) : 0);
}

// LDS bytes of encode_kernel
uint32_t encode_lds(uint32_t block_elems, uint32_t wcap, int n_in, uint32_t &pass2_off) {
  uint32_t pass1 = kHistBytes + (n_in > 0 ? n_in * kLutBytes + 1024 : 0);
  uint32_t pass2 = kStageHead + 2 * wcap + kStageTail;
  pass2_off = kEncTableBytes;
  uint32_t region = pass1 > pass2 ? pass1 : pass2;
  (void)block_elems;
  return kEncTableBytes + region;
}

uint32_t word_cap(uint32_t block_elems) { return block_elems / 2 + kRound + 8; }

struct EncodeWs {
  uint64_t status_off, cnt_off, y_off, total;
};

EncodeWs encode_ws(uint64_t n_blocks, uint64_t n_chunks, uint64_t ybytes) {
  EncodeWs w;
  w.status_off = 256;
  w.cnt_off = pad256(w.status_off + 8 * n_blocks);
  w.y_off = pad256(w.cnt_off + 8 * n_chunks);
  w.total = pad256(w.y_off + ybytes);
  return w;
}

uzip_status launch_encode(EncodeArgs &a, uzip_dtype dt, bool reduce, uint8_t *ws, const EncodeWs &w,
                          hipStream_t stream) {
  a.ticket = (uint32_t *)ws;
  a.status = (uint64_t *)(ws + w.status_off);
  a.chunk_cnt = (uint32_t *)(ws + w.cnt_off);
  a.wcap = word_cap(a.block_elems);
  uint32_t lds = encode_lds(a.block_elems, a.wcap, reduce ? a.n_in : 0, a.pass2_off);
  if (lds > 160 * 1024) return UZIP_EINVAL;
  uint64_t clear_words = w.y_off / 4;
  hipLaunchKernelGGL(clear_kernel, dim3((unsigned)((clear_words + 255) / 256 < 4096 ? (clear_words + 255) / 256 : 4096)),
                     dim3(256), 0, stream, (uint32_t *)ws, clear_words);
  if (hipGetLastError() != hipSuccess) return UZIP_EHIP;
  dim3 grid(a.n_blocks), block(64);
  if (!reduce) {
    if (dt == UZIP_BF16) hipLaunchKernelGGL((encode_kernel<0, false>), grid, block, lds, stream, a);
    if (dt == UZIP_FP16) hipLaunchKernelGGL((encode_kernel<1, false>), grid, block, lds, stream, a);
    if (dt == UZIP_FP32) hipLaunchKernelGGL((encode_kernel<2, false>), grid, block, lds, stream, a);
  } else {
    if (dt == UZIP_BF16) hipLaunchKernelGGL((encode_kernel<0, true>), grid, block, lds, stream, a);
    if (dt == UZIP_FP16) hipLaunchKernelGGL((encode_kernel<1, true>), grid, block, lds, stream, a);
    if (dt == UZIP_FP32) hipLaunchKernelGGL((encode_kernel<2, true>), grid, block, lds, stream, a);
  }
  return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
}

}  // namespace

extern "C" {

size_t uzip_max_compressed_size(uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes)) return 0;
  return (size_t)max_size(elem_bytes(dtype), n_elems, block_bytes / elem_bytes(dtype));
}

size_t uzip_workspace_size(int op, uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, uint64_t aux) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes)) return 0;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t nb = (n_elems + be - 1) / be;
  switch (op) {
    case UZIP_OP_COMPRESS:
      return (size_t)encode_ws(nb, 1, 0).total;
    case UZIP_OP_DECOMPRESS:
      return 0;
    case UZIP_OP_CHUNKED: {
      if (aux == 0 || aux % block_bytes) return 0;
      const uint64_t ce = aux / E;
      const uint64_t chunks = (n_elems + ce - 1) / ce;
      return (size_t)encode_ws(chunks * (ce / be), chunks, 0).total;
    }
    case UZIP_OP_REDUCE: {
      const uint64_t n_in = aux & 0xFFFFu;
      if (n_in < 1 || n_in > kMaxInputs) return 0;
      const uint64_t y = (aux & UZIP_WS_NO_OUT_RAW) ? n_elems * E : 0;
      return (size_t)encode_ws(nb, 1, y).total;
    }
    default:
      return 0;
  }
}

uzip_status uzip_compress(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                          void *d_out, size_t out_cap, uint64_t *d_out_size, void *d_ws, size_t ws_bytes,
                          hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes)) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out) || (n_elems > 0 && (d_in == nullptr || !aligned16(d_in))))
    return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t nb = (n_elems + be - 1) / be;
  if (nb >= 0x7FFFFFFFull) return UZIP_EINVAL;
  if (out_cap < max_size(E, n_elems, be)) return UZIP_ENOSPC;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  if (n_elems == 0) {
    hipLaunchKernelGGL(empty_stream_kernel, dim3(1), dim3(64), 0, stream, (uint8_t *)d_out, (uint32_t)dtype, be,
                       d_out_size);
    return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
  }
  EncodeWs w = encode_ws(nb, 1, 0);
  if (d_ws == nullptr || !aligned16(d_ws) || ws_bytes < w.total) return UZIP_ENOSPC;
  EncodeArgs a;
  memset(&a, 0, sizeof(a));
  a.in = (const uint8_t *)d_in;
  a.n = n_elems;
  a.chunk_elems = (nb * be);
  a.block_elems = be;
  a.blocks_per_chunk = (uint32_t)nb;
  a.n_blocks = (uint32_t)nb;
  a.out = (uint8_t *)d_out;
  a.slot_bytes = 0;
  a.sizes = d_out_size;
  return launch_encode(a, dtype, false, (uint8_t *)d_ws, w, stream);
}

uzip_status uzip_compress_chunked(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                  uint64_t chunk_bytes, void *d_out, size_t slot_bytes, uint64_t *chunk_sizes,
                                  uint32_t *flags, uint32_t epoch, void *d_ws, size_t ws_bytes,
                                  hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes)) return UZIP_EINVAL;
  if (chunk_bytes == 0 || chunk_bytes % block_bytes) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out) || (slot_bytes & 15u) || (n_elems > 0 && (d_in == nullptr || !aligned16(d_in))))
    return UZIP_EINVAL;
  if (chunk_sizes == nullptr || flags == nullptr) return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t ce = chunk_bytes / E;
  if (ce / be >= 0x7FFFFFFFull) return UZIP_EINVAL;
  const uint64_t chunks = (n_elems + ce - 1) / ce;
  if (n_elems == 0) return UZIP_OK;
  if (slot_bytes < max_size(E, n_elems < ce ? n_elems : ce, be)) return UZIP_ENOSPC;
  const uint64_t nb = (chunks - 1) * (ce / be) + ((n_elems - (chunks - 1) * ce) + be - 1) / be;
  if (nb >= 0x7FFFFFFFull) return UZIP_EINVAL;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  EncodeWs w = encode_ws(chunks * (ce / be), chunks, 0);
  if (d_ws == nullptr || !aligned16(d_ws) || ws_bytes < w.total) return UZIP_ENOSPC;
  EncodeArgs a;
  memset(&a, 0, sizeof(a));
  a.in = (const uint8_t *)d_in;
  a.n = n_elems;
  a.chunk_elems = ce;
  a.block_elems = be;
  a.blocks_per_chunk = (uint32_t)(ce / be);
  a.n_blocks = (uint32_t)nb;
  a.out = (uint8_t *)d_out;
  a.slot_bytes = slot_bytes;
  a.sizes = chunk_sizes;
  a.flags = flags;
  a.epoch = epoch;
  return launch_encode(a, dtype, false, (uint8_t *)d_ws, w, stream);
}

uzip_status uzip_decompress(const void *d_in, size_t in_bytes, uzip_dtype dtype, uint64_t n_elems, void *d_out,
                            size_t out_cap, uint32_t *d_status, void *d_ws, size_t ws_bytes, hipStream_t stream) {
  (void)d_ws;
  (void)ws_bytes;
  if (!valid_dtype(dtype) || d_in == nullptr || !aligned16(d_in)) return UZIP_EINVAL;
  if (n_elems > 0 && (d_out == nullptr || !aligned16(d_out))) return UZIP_EINVAL;
  if (out_cap < n_elems * elem_bytes(dtype)) return UZIP_ENOSPC;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  DecodeArgs a;
  a.in = (const uint8_t *)d_in;
  a.in_bytes = in_bytes;
  a.n = n_elems;
  a.dtype = (uint32_t)dtype;
  a.out = (uint8_t *)d_out;
  a.dstatus = d_status;
  // grid-stride: enough waves to fill the device, never more than the smallest block size allows
  const uint64_t most = (n_elems + (kMinBlockBytes / elem_bytes(dtype)) - 1) / (kMinBlockBytes / elem_bytes(dtype));
  uint64_t grid = (uint64_t)info.cus * 16;
  if (grid > most) grid = most;
  if (grid == 0) grid = 1;
  if (dtype == UZIP_BF16) hipLaunchKernelGGL(decode_kernel<0>, dim3((unsigned)grid), dim3(64), 0, stream, a);
  if (dtype == UZIP_FP16) hipLaunchKernelGGL(decode_kernel<1>, dim3((unsigned)grid), dim3(64), 0, stream, a);
  if (dtype == UZIP_FP32) hipLaunchKernelGGL(decode_kernel<2>, dim3((unsigned)grid), dim3(64), 0, stream, a);
  return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
}

uzip_status uzip_reduce_fused(const void *const *d_in, const size_t *in_bytes, int n_in, const void *d_local_raw,
                              uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, void *d_out, size_t out_cap,
                              uint64_t *d_out_size, void *d_out_raw, uint32_t *d_status, void *d_ws,
                              size_t ws_bytes, hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes)) return UZIP_EINVAL;
  if (n_in < 1 || n_in > kMaxInputs || d_in == nullptr || in_bytes == nullptr) return UZIP_EINVAL;
  for (int i = 0; i < n_in; ++i)
    if (d_in[i] == nullptr || !aligned16(d_in[i]) || in_bytes[i] < kHeaderBytes) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out)) return UZIP_EINVAL;
  if ((d_local_raw && !aligned16(d_local_raw)) || (d_out_raw && !aligned16(d_out_raw))) return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t nb = (n_elems + be - 1) / be;
  if (nb >= 0x7FFFFFFFull) return UZIP_EINVAL;
  if (out_cap < max_size(E, n_elems, be)) return UZIP_ENOSPC;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  if (n_elems == 0) {
    hipLaunchKernelGGL(empty_stream_kernel, dim3(1), dim3(64), 0, stream, (uint8_t *)d_out, (uint32_t)dtype, be,
                       d_out_size);
    return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
  }
  EncodeWs w = encode_ws(nb, 1, d_out_raw ? 0 : n_elems * E);
  if (d_ws == nullptr || !aligned16(d_ws) || ws_bytes < w.total) return UZIP_ENOSPC;
  EncodeArgs a;
  memset(&a, 0, sizeof(a));
  a.n = n_elems;
  a.chunk_elems = nb * be;
  a.block_elems = be;
  a.blocks_per_chunk = (uint32_t)nb;
  a.n_blocks = (uint32_t)nb;
  a.out = (uint8_t *)d_out;
  a.sizes = d_out_size;
  a.n_in = n_in;
  for (int i = 0; i < n_in; ++i) {
    a.ins[i] = (const uint8_t *)d_in[i];
    a.in_bytes[i] = in_bytes[i];
  }
  a.local_raw = (const uint8_t *)d_local_raw;
  a.ybuf = d_out_raw ? (uint8_t *)d_out_raw : (uint8_t *)d_ws + w.y_off;
  a.dstatus = d_status;
  return launch_encode(a, dtype, true, (uint8_t *)d_ws, w, stream);
}

const char *uzip_status_str(uzip_status status) {
  switch (status) {
    case UZIP_OK: return "ok";
    case UZIP_EINVAL: return "invalid argument";
    case UZIP_ENOSPC: return "output or workspace too small";
    case UZIP_ECORRUPT: return "corrupt or mismatched stream";
    case UZIP_EHIP: return "HIP runtime error";
    case UZIP_EUNSUPPORTED: return "device is not gfx950";
    default: return "unknown status";
  }
}

}  // extern "C"
