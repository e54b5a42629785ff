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
//                   16-byte writes straight into the final stream.  Blocks
//                   of up to 32768 elements resolve their offset and write
//                   their section only after the wave's next block has
//                   streamed through pass 1.
//   decode_kernel   resident waves walk the blocks grid-stride; each block's
//                   offset is read from the directory, its decode table
//                   (2048 x u32) is built in LDS, its words are staged
//                   through an LDS ring and the 64 states decode forwards.
//                   For the receiver of the split-send producer the walk
//                   covers the blocks of a range of chunk streams at once,
//                   opening each chunk's header when it reaches that chunk.
//   reduce_fused_kernel (fused reduce)  one workgroup per output block
//                   decodes block b of up to eight inputs in parallel waves,
//                   round by round; a further wave adds them in binary32 in
//                   input order, splits the rounded result (raw plane,
//                   histogram, symbols kept in LDS) and then codes the block
//                   and places its section itself.  When the output blocks
//                   outnumber the compute units (or a block's symbols do not
//                   fit in LDS), reduce_decode_kernel does the decoding and
//                   summing and reduce_kernel, the encoder's coding half,
//                   runs over the reduced tensor.
//   split-send producer  encode_kernel with write-through stores and
//                   per-chunk completion counters.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>

#include "../../include/uzip.h"
#include "uzip_device.h"

using namespace uzip;

namespace {

constexpr int kMaxInputs = 16;
constexpr uint32_t kTrashBytes = 256;  // encoder: slots for non-emitted words (2 bytes per lane), free outside coding
constexpr uint32_t kMinBlockBytes = 4096, kMaxBlockBytes = 4194304;

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
  const uint8_t *ybuf;      // the reduced tensor: source of both passes
  const uint32_t *hist_in;  // [n_blocks][256] symbol histograms of the reduced tensor
  // per-workgroup overflow slots for the staged words past the LDS window
  uint16_t *slots;
  uint32_t slot_words;
  uint32_t lds_words;       // staging words held in LDS
  // stream-wide table (table modes 1, 2): frequencies f[256], the mode
  // written to the header's flags byte, and the table bytes in the stream
  const uint16_t *table;
  uint32_t table_stride;  // u16 entries between the tables of consecutive streams (0: one table for all)
  uint32_t table_mode;
  uint32_t table_bytes;
  // split-send producer, XCD-local (n_xcd > 0): chunk c is coded only by
  // waves of XCD c mod n_xcd, which take its blocks from their XCD's own
  // ticket counter; the stream bytes then go out with ordinary stores and
  // the block that completes a chunk's count writes the XCD's L2 back
  // before raising the flag
  uint32_t n_xcd;
};

// The first workspace words of an encoder launch (u32 index), written by the
// clear kernel: the ticket counter, the error word and the count of
// workgroups that have finished; then, in a cache line of their own (the
// ticket's takes an atomic from every wave per block), the single-pass
// scan's bounded wait (polls), a block that never publishes its length
// (fault injection; ~0u: none) and the caller's device status (fused
// reduce; may be null).  Read from memory where used, they take no
// registers in the encoder's loop.
enum : uint32_t { kWsTicket = 0, kWsError = 1, kWsExit = 2, kWsSpin = 32, kWsHold = 33, kWsStatusPtr = 34 };
// the XCD-local producer's ticket counters, one 64-byte line per XCD
constexpr uint32_t kWsXcd = 64, kWsXcdStride = 16, kMaxXcd = 8;
constexpr uint64_t kWsHeaderBytes = 4 * (kWsXcd + kWsXcdStride * kMaxXcd);

constexpr size_t kDecodeWsBytes = 256;   // reserved: the decoder keeps no state there

struct DecodeArgs {
  const uint8_t *in;
  uint64_t in_bytes;
  uint64_t n;
  uint32_t dtype;
  uint8_t *out;
  uint32_t *dstatus;
  const uint16_t *table;  // the caller's table (streams of table mode 2)
  // chunk streams of the split-send producer (bpc > 0): chunk c's stream in
  // the slot at in + c slot_bytes, its elements at out + c chunk_elems E;
  // the launch decodes chunks [first_chunk, first_chunk + n_chunks), bpc
  // blocks of block_elems each (the tensor's last chunk: fewer).  bpc == 0:
  // one stream of n elements at in, its block count from its header.
  uint64_t slot_bytes;
  uint64_t chunk_elems;
  uint64_t first_chunk;
  uint64_t n_chunks;
  uint32_t bpc;
  uint32_t block_elems;
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

// element width of a dtype code: fp32 4 bytes, the rest (bf16, fp16, FP8
// pairs) 2
template <int DT>
constexpr int dt_bytes() { return DT == 2 ? 4 : 2; }

template <int DT>
__device__ inline void split_group(const uint32_t w[4 * (dt_bytes<DT>() / 2)], Group &g) {
  if constexpr (DT >= 3)
    split8x2(w, g);
  else if constexpr (DT == 2)
    split32(w, g);
  else
    split16(w, g);
}

// raw plane bytes of a group: 8 (E = 2) or 24 (E = 4) bytes at plane + (E-1) first
// Stores of stream bytes.  SYS (split-send producer): system-coherent
// stores, written through to memory, so that a block only has to wait for
// its own stores before it counts itself done, instead of writing back the
// whole L2 (a consumer outside this GPU reads the chunk once its flag is set).
// Otherwise the raw plane and the sections go out with non-temporal stores:
// nothing on this GPU reads them back soon, and a stream that does not fill
// the Infinity Cache with dirty lines leaves the next kernel less to drain
// (the decompress that follows a compress ran 2.7% faster, the compress
// itself within 1%; interleaved A/B on the 1 GiB buffer).
template <bool SYS>
__device__ __forceinline__ void out8(uint8_t *p, uint8_t v) {
  if (SYS) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  else *p = v;
}
template <bool SYS>
__device__ __forceinline__ void out32(uint32_t *p, uint32_t v) {
  if (SYS) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  else *p = v;
}
template <bool SYS>
__device__ __forceinline__ void out64(uint8_t *p, uint32_t lo, uint32_t hi) {
  typedef uint32_t v2u __attribute__((ext_vector_type(2)));
  if (SYS) __hip_atomic_store((uint64_t *)p, (uint64_t)hi << 32 | lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  else __builtin_nontemporal_store((v2u){lo, hi}, (v2u *)p);
}
// Header and size words: atomic stores written through the L2 at agent
// scope (system scope for the split-send producer), so that a later store of
// finish_launch to the same words, from any XCD, is the one that stays.
template <bool SYS>
__device__ __forceinline__ void coh64(uint64_t *p, uint64_t v) {
  if (SYS) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  else __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 16 bytes in one store; the split-send producer's is written through to
// memory (sc0 sc1, as its system-scope stores are) in one 16-byte access
// rather than two 8-byte halves.  The memory counter completes in issue
// order, so waits the compiler places for its own accesses stay correct.
template <bool SYS>
__device__ __forceinline__ void out128(uint8_t *p, uint4 v) {
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  const v4u w = {v.x, v.y, v.z, v.w};
  if (SYS) {
    asm volatile("global_store_dwordx4 %0, %1, off sc0 sc1" ::"v"(p), "v"(w) : "memory");
  } else {
    __builtin_nontemporal_store(w, (v4u *)p);
  }
}

template <int E, bool SYS = false>
__device__ inline void store_raw(uint8_t *plane, uint64_t first, uint32_t valid, const Group &g) {
  uint8_t *p = plane + (uint64_t)(E - 1) * first;
  if (valid >= 8) {
    out64<SYS>(p, g.raw[0], g.raw[1]);
    if (E == 4) {
      out64<SYS>(p + 8, g.raw[2], g.raw[3]);
      out64<SYS>(p + 16, g.raw[4], g.raw[5]);
    }
  } else {
#pragma unroll
    for (uint32_t b = 0; b < 8 * (E - 1); ++b)
      if (b < (E - 1) * valid) out8<SYS>(p + b, (uint8_t)(g.raw[b >> 2] >> (8 * (b & 3))));
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

template <int DT>
__device__ inline void merge_group(const uint32_t sym[2], const uint32_t raw[6],
                                   uint32_t w[4 * (dt_bytes<DT>() / 2)]) {
  if constexpr (DT >= 3)
    merge8x2(sym, raw, w);
  else if constexpr (DT == 2)
    merge32(sym, raw, w);
  else
    merge16(sym, raw, w);
}

// Eight elements of one lane out to a tensor.  NT: full groups with
// streaming (non-temporal) stores, for output nothing here reads back.
template <int E, bool NT = false>
__device__ inline void store_words(uint8_t *base, uint64_t first, uint32_t valid, const uint32_t w[4 * (E / 2)]) {
  if (valid >= 8) {
    typedef uint32_t v4u __attribute__((ext_vector_type(4)));
    v4u *p = (v4u *)(base + first * E);
    if (NT) {
      __builtin_nontemporal_store((v4u){w[0], w[1], w[2], w[3]}, p);
      if (E == 4) __builtin_nontemporal_store((v4u){w[4], w[5], w[6], w[7]}, p + 1);
    } else {
      p[0] = (v4u){w[0], w[1], w[2], w[3]};
      if (E == 4) p[1] = (v4u){w[4], w[5], w[6], w[7]};
    }
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

// LDS traffic of one wave is processed in order: between its own stores and
// loads only the compiler has to be kept from reordering (no workgroup
// barrier, so the table build also runs in one wave of a larger group).
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------------------
// Decode side: table of one coded block -> 2048-entry lookup table in LDS.
// Entry for slot: f | (slot - cum) << 12 | sym << 24.
// Returns false (uniformly) if the stored table is not a valid ANS table.
// ---------------------------------------------------------------------------
__device__ void fill_lut(const uint32_t f[4], uint32_t *lut, uint16_t *cum_s, uint16_t *f_s);
// The caller loaded the section's start: `byte` is byte 256 + lane / 2 of
// the section (the presence bits), `fa` its bytes 288 + 8 lane .. + 7 (the
// u16 frequencies of ranks 4 lane .. 4 lane + 3; zero past the section's
// end).
__device__ bool build_lut_pre(uint32_t byte, uint2 fa, uint64_t sec_len, uint32_t *lut, uint16_t *cum_s,
                              uint16_t *f_s, uint32_t &k_out) {
  const uint32_t lane = lane_id();
  if (sec_len < kSectionFixed) return false;
  const uint32_t nib = (byte >> (4 * (lane & 1))) & 0xFu;
  const uint32_t pres = __popc(nib);
  const uint32_t k = wave_sum(pres);
  const uint32_t rank0 = wave_excl_scan(pres);
  const bool ok0 = k >= 1 && (uint64_t)kSectionFixed + 2ull * k <= sec_len;
  // the frequencies of ranks 0 .. 255, staged where the table will go
  ((uint2 *)lut)[lane] = fa;
  wave_lds_fence();
  const uint16_t *fr = (const uint16_t *)lut;
  uint32_t f[4] = {0, 0, 0, 0};
  uint32_t r = rank0, total = 0;
  if (ok0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (nib & (1u << q)) f[q] = fr[r++];
      total += f[q];
    }
  }
  wave_lds_fence();  // read before the table overwrites them
  const uint32_t bad = (nib & 1 && f[0] == 0) | (nib & 2 && f[1] == 0) | (nib & 4 && f[2] == 0) |
                       (nib & 8 && f[3] == 0);
  if (!(ok0 && !__any(bad) && wave_sum(total) == kM)) return false;
  fill_lut(f, lut, cum_s, f_s);
  k_out = k;
  return true;
}

// The lookup table from this lane's frequencies f[4] of symbols 4 lane ..
// 4 lane + 3 (summing to M over the wave).
__device__ void fill_lut(const uint32_t f[4], uint32_t *lut, uint16_t *cum_s, uint16_t *f_s) {
  const uint32_t lane = lane_id();
  uint32_t c = wave_excl_scan(f[0] + f[1] + f[2] + f[3]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    cum_s[4 * lane + q] = (uint16_t)c;
    f_s[4 * lane + q] = (uint16_t)f[q];
    c += f[q];
  }
  wave_lds_fence();
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
  uint32_t c0 = cum_s[s], fs = f_s[s];
  for (uint32_t q = 0; q < 32; ++q, ++slot) {
    while (slot >= c0 + fs) {
      ++s;
      c0 = cum_s[s];
      fs = f_s[s];
    }
    lut[slot] = fs | ((slot - c0) << 12) | (s << 24);
  }
  wave_lds_fence();
}

// Lookup table of a stream-wide table (u16 f[256] in memory): every symbol
// has f >= 1 and the sum is M, else false (uniformly).
__device__ bool build_lut_shared(const uint16_t *table, uint32_t *lut, uint16_t *cum_s, uint16_t *f_s) {
  const uint32_t lane = lane_id();
  const uint2 v = *(const uint2 *)(table + 4 * lane);
  const uint32_t f[4] = {v.x & 0xFFFFu, v.x >> 16, v.y & 0xFFFFu, v.y >> 16};
  const bool bad = f[0] == 0 || f[1] == 0 || f[2] == 0 || f[3] == 0;
  if (__any(bad) || wave_sum(f[0] + f[1] + f[2] + f[3]) != kM) return false;
  fill_lut(f, lut, cum_s, f_s);
  return true;
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
__device__ void enc_entries(const Table &t, uint4 *enc);
template <bool PACKED = false>
__device__ void build_enc_table(const uint32_t *hist, uint32_t n_b, uint4 *enc, Table &t) {
  const uint32_t lane = lane_id();
  uint32_t c[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t s = 4 * lane + q, acc = 0;
#pragma unroll
    for (uint32_t rep = 0; rep < kHistReplicas; ++rep) {
      if constexpr (PACKED)
        acc += (hist[rep * kPackedHistStride + (s & 127u)] >> (16 * (s >> 7))) & 0xFFFFu;
      else
        acc += hist[rep * kHistStride + s];
    }
    c[q] = acc;
  }
  // the counts are read: a packed histogram may share its LDS with `enc`
  uint32_t pres = (c[0] > 0) + (c[1] > 0) + (c[2] > 0) + (c[3] > 0);
  uint32_t k = wave_sum(pres);
  uint32_t lt = 0;
  // c (M - k) <= 2^21 (2^11 - 1) < 2^32 (a block holds at most 2^21
  // symbols): exact in 32 bits; every block but a stream's last has a
  // power-of-two size, a shift
  const bool pow2 = (n_b & (n_b - 1)) == 0;
  const uint32_t lg = 31 - __clz(n_b);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t num = c[q] * (kM - k);
    t.f[q] = c[q] ? 1u + (pow2 ? num >> lg : num / n_b) : 0u;
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
  t.k = k;
  t.rank0 = wave_excl_scan(pres);
#pragma unroll
  for (int q = 0; q < 4; ++q) t.present[q] = __ballot(c[q] > 0);
  enc_entries(t, enc);
}

// Encoder table entries of this lane's frequencies t.f[4].
__device__ void enc_entries(const Table &t, uint4 *enc) {
  const uint32_t lane = lane_id();
  uint32_t cum = wave_excl_scan(t.f[0] + t.f[1] + t.f[2] + t.f[3]);
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
        // 2^(31+l) / f in binary64 is correctly rounded and a non-integer
        // quotient is at least 1/f from the next integer, far more than half
        // an ulp (< 2^-20), so the ceiling of the rounded quotient is exact
        uint32_t m = (uint32_t)ceil((double)(1ull << (31 + l)) / (double)f);
        e = make_uint4(m, f << 20, (kM - f) | ((l - 1) << 24), cum);
      }
      enc[4 * lane + q] = e;
    }
    cum += f;
  }
}

// Decoupled look-back over the blocks of one stream, in two steps: a block
// publishes its section length (its aggregate; for the stream's first block
// already its inclusive prefix), and later resolves its exclusive prefix
// (16-byte units) from its predecessors' states.  Between the two a wave may
// do other work: a wait is only ever for an aggregate, which every taken
// block publishes without waiting, and blocks are taken in ticket order, so
// the wait always ends.  The spin is bounded anyway (a wave of an earlier
// block may be descheduled for long on a shared GPU): a wait that runs out
// returns `failed`, and the launch then marks the stream invalid instead of
// hanging (finish_launch).
constexpr uint32_t kSpinLimit = 1u << 22;
__device__ __forceinline__ void publish_aggregate(uint64_t *status, uint32_t b, uint32_t first, uint64_t len16,
                                                  uint32_t hold) {
  if (lane_id() == 0 && b != hold)
    __hip_atomic_store(&status[b], (b == first ? kFlagInclusive : kFlagAggregate) | len16, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline uint64_t wave_excl_scan64(uint64_t v) {
  const uint32_t lane = lane_id();
  uint64_t inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t w = __shfl_up(inc, o);
    if (lane >= (uint32_t)o) inc += w;
  }
  return inc - v;
}

// Resolves block b's exclusive prefix and publishes its inclusive one.  The
// nearest predecessors (up to 64) that had only published their length get
// their inclusive prefix too, the same value their own look-back publishes:
// later blocks then find an inclusive prefix close by.  A wait that runs out
// after spin_limit polls sets `failed` (uniform) and the error word and
// publishes nothing; the held block (fault injection) publishes nothing.
__device__ uint64_t resolve_prefix(uint64_t *status, uint32_t b, uint32_t first, uint64_t len16,
                                   uint32_t spin_limit, uint32_t hold, uint32_t *err, bool &failed) {
  const uint32_t lane = lane_id();
  failed = false;
  if (b == first) return 0;
  uint64_t excl = 0, near_v = 0;
  bool near_agg = false, near = true;
  int64_t look = (int64_t)b - 1;
  uint32_t spins = 0;
  while (true) {
    const int64_t idx = look - (int64_t)lane;
    uint64_t st = kFlagInclusive;  // before the stream's first block: inclusive 0
    if (idx >= (int64_t)first) st = __hip_atomic_load(&status[idx], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t flag = (uint32_t)(st >> 62);
    const uint64_t inc = __ballot(flag == 2);
    const uint64_t upto = inc ? ((inc & (~inc + 1)) << 1) - 1 : ~0ull;  // lanes up to the first inclusive
    const uint64_t notready = __ballot(flag == 0) & upto;
    if (notready) {
      if (++spins < spin_limit) {
        __builtin_amdgcn_s_sleep(2);
        continue;
      }
      if (lane == 0) __hip_atomic_store(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      failed = true;
      return excl;
    }
    const bool mine = (upto >> lane) & 1;
    const uint64_t v = mine ? (st & kValueMask) : 0;
    if (near) {
      near_v = v;
      near_agg = mine && flag == 1;
      near = false;
    }
    excl += wave_sum64(v);
    if (inc) break;
    look -= 64;
  }
  if (b == hold) return excl;
  if (lane == 0)
    __hip_atomic_store(&status[b], kFlagInclusive | (excl + len16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // lane l of the nearest window is block b-1-l: its inclusive prefix is
  // excl less the lengths of blocks b-l .. b-1
  const uint64_t later = wave_excl_scan64(near_v);
  if (near_agg)
    __hip_atomic_store(&status[b - 1 - lane], kFlagInclusive | (excl - later), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  return excl;
}

// Counter of finished blocks of a chunk; the last one publishes the flag.
// The block's stream bytes were written with system-coherent stores
// (write-through), so waiting for them to complete is what orders them
// before the count; the count is a system-scope atomic at the memory, so the
// block that completes it stores the flag after every block's bytes are in
// memory.
// A block whose look-back failed first sets the counter's top bit (block
// counts stay below 2^31), so no later count can equal `need` and the flag
// is left to finish_launch, which raises it over a zero size.
// A system-scope release: this XCD's L2 written back to memory, then a wait
// for the write-back.  The wait is explicit because the compiler leaves out
// its own after the write-back when an explicit wait precedes the fence.
__device__ __forceinline__ void writeback_l2() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
  __builtin_amdgcn_s_waitcnt(0);
}

// XCD-local producer (wb): the bytes went out with ordinary stores into the
// L2 of the XCD that codes the whole chunk, so the block that completes the
// count first writes that L2 back and then stores the flag.
constexpr uint32_t kChunkFailed = 0x80000000u;
__device__ void publish_chunk(uint32_t *cnt, uint32_t need, uint32_t *flag, uint32_t epoch, bool failed = false,
                              bool wb = false) {
  if (failed && lane_id() == 0) __hip_atomic_fetch_or(cnt, kChunkFailed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __builtin_amdgcn_s_waitcnt(0);
  if (lane_id() == 0 && __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) + 1 == need) {
    if (wb) writeback_l2();
    __hip_atomic_store(flag, epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// The next block of a persistent encoder wave (lane 0 only).  Tickets are
// block indices in order, or, for the XCD-local producer, indices into the
// blocks of this XCD's chunks (c = xcd, xcd + n_xcd, ...) in order; past the
// last block: n_blocks.
__device__ uint32_t take_block(const EncodeArgs &a) {
  if (a.n_xcd == 0) return __hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // HW_REG_XCC_ID (hardware register 20), bits 3..0: the XCD this wave runs on
  const uint32_t xcd = (__builtin_amdgcn_s_getreg(20u | (0u << 6) | ((4u - 1u) << 11)) & 15u) % a.n_xcd;
  uint32_t *ctr = a.ticket + kWsXcd + kWsXcdStride * xcd;
  const uint64_t chunks = ((uint64_t)a.n_blocks + a.blocks_per_chunk - 1) / a.blocks_per_chunk;
  while (true) {
    const uint32_t t = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t q = t / a.blocks_per_chunk;
    const uint64_t c = xcd + (uint64_t)a.n_xcd * q;
    if (c >= chunks) return a.n_blocks;
    const uint64_t b = c * a.blocks_per_chunk + (t - q * a.blocks_per_chunk);
    if (b < a.n_blocks) return (uint32_t)b;
    // past the end of the tensor's last, shorter chunk: take another ticket
  }
}

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
// Symbols of a whole block (up to 64 rounds, block_elems <= 32768) stay in
// registers between the histogram pass and the coding pass, with static
// register indices only: a pass walks the block in 4 groups of 16 rounds
// with the 16 rounds unrolled, always touching vector v3 (pass 1) or v3
// (pass 2), and the four vectors rotate cyclically between groups.
// ---------------------------------------------------------------------------
typedef uint32_t v32u __attribute__((ext_vector_type(32)));
struct SymRegs {
  v32u v0, v1, v2, v3;
};
constexpr uint32_t kRegRounds = 64;

// pass 1: group g was just written to v3; move it down (v0 ends up with group 0)
__device__ __forceinline__ void shift_down(SymRegs &S) {
  S.v0 = S.v1;
  S.v1 = S.v2;
  S.v2 = S.v3;
}
// pass 2: group g in v3 has been coded; bring group g-1 up
__device__ __forceinline__ void shift_up(SymRegs &S) {
  S.v3 = S.v2;
  S.v2 = S.v1;
  S.v1 = S.v0;
}

// Byte K of w shifted left by SH: one SDWA shift (the compiler would emit an
// extract and a shift).
template <int K, int SH>
__device__ __forceinline__ uint32_t byte_shl(uint32_t w) {
  static_assert(K >= 0 && K < 4, "byte index");
  uint32_t r;
  if constexpr (K == 0)
    asm("v_lshlrev_b32_sdwa %0, %2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
        : "=v"(r) : "v"(w), "i"(SH));
  else if constexpr (K == 1)
    asm("v_lshlrev_b32_sdwa %0, %2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
        : "=v"(r) : "v"(w), "i"(SH));
  else if constexpr (K == 2)
    asm("v_lshlrev_b32_sdwa %0, %2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
        : "=v"(r) : "v"(w), "i"(SH));
  else
    asm("v_lshlrev_b32_sdwa %0, %2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
        : "=v"(r) : "v"(w), "i"(SH));
  return r;
}

// The encoder table entries of a lane's 8 symbols (s0: symbols 0-3, s1: 4-7)
__device__ __forceinline__ void enc_lookup8(const uint4 *enc, uint32_t s0, uint32_t s1, uint4 (&e)[8]) {
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) e[tt] = enc[(s0 >> (8 * tt)) & 0xFFu];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) e[4 + tt] = enc[(s1 >> (8 * tt)) & 0xFFu];
}

// 16 bytes at LDS byte address p
__device__ __forceinline__ uint4 lds_load16(uint32_t p) {
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  const v4u v = *(const __attribute__((address_space(3))) v4u *)(uintptr_t)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// The same for a table at the fixed LDS byte address TB: the shifted symbol
// is the address, TB goes into the instruction's offset field (the pointer
// form adds the LDS base in one more instruction).  Read in the order the
// backwards coding round uses them.
template <uint32_t TB>
__device__ __forceinline__ void enc_lookup8_at(uint32_t s0, uint32_t s1, uint4 (&e)[8]) {
  e[7] = lds_load16(TB + byte_shl<3, 4>(s1));
  e[6] = lds_load16(TB + byte_shl<2, 4>(s1));
  e[5] = lds_load16(TB + byte_shl<1, 4>(s1));
  e[4] = lds_load16(TB + byte_shl<0, 4>(s1));
  e[3] = lds_load16(TB + byte_shl<3, 4>(s0));
  e[2] = lds_load16(TB + byte_shl<2, 4>(s0));
  e[1] = lds_load16(TB + byte_shl<1, 4>(s0));
  e[0] = lds_load16(TB + byte_shl<0, 4>(s0));
}

// One encoder sub-step of every lane (rANS coding function with 16-bit
// renormalisation).  Emitted words go to virtual staging index
// pos - cnt + rank, compacted across the wave with ballot + mbcnt.
//
// enc_step_lds: the whole step lands in the LDS staging area (index v lives
// at lds[v - lo]); branch-free: every lane stores, lanes that emit nothing
// store into their own trash slot.
template <bool FULL, bool RANK0>
__device__ __forceinline__ void enc_step_lds(uint32_t &x, const uint4 e, bool valid, uint32_t &pos,
                                             __attribute__((address_space(3))) uint16_t *lds_rel,
                                             __attribute__((address_space(3))) uint16_t *trash) {
  const bool emit = (FULL || valid) && x >= e.y;
  const uint64_t m = __ballot(emit);
  const uint32_t base = pos - (uint32_t)__popcll(m);
  __attribute__((address_space(3))) uint16_t *dst;
  if constexpr (RANK0) {
    // the lane's rank among the emitting lanes, and the wave-uniform row
    // address formed on the scalar unit (one vector move fewer; the large
    // blocks' coding loops spill more with it)
    const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    __attribute__((address_space(3))) uint16_t *row = lds_rel + base;
    dst = emit ? row + rank : trash;
  } else {
    const uint32_t v = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, base));
    dst = emit ? lds_rel + v : trash;
  }
  *dst = (uint16_t)x;
  x = emit ? x >> 16 : x;
  pos = base;
  if (FULL || valid) {
    const uint32_t q = __umulhi(x, e.x) >> (e.z >> 24);
    x = x + __umul24(q, e.z) + e.w;
  }
}

// One round of 8 sub-steps, backwards.
template <bool FULL, bool RANK0 = false>
__device__ __forceinline__ void enc_round(uint32_t &x, const uint4 (&e)[8], uint32_t valid, uint32_t &pos,
                                          __attribute__((address_space(3))) uint16_t *lds_rel,
                                          __attribute__((address_space(3))) uint16_t *trash) {
#pragma unroll
  for (int tt = kPerLane - 1; tt >= 0; --tt)
    enc_step_lds<FULL, RANK0>(x, e[tt], (uint32_t)tt < valid, pos, lds_rel, trash);
}

// The LDS staging window holds virtual indices [lo, lo + cap) at win[v - lo]
// (lo, cap and the slide x are multiples of 8 words, win and the overflow
// slot are 16-byte aligned).  Before a round that could write below it, the
// window's x oldest words (the highest indices) go to the same indices of
// the workgroup's overflow slot and the rest, from the 16-byte unit holding
// pos up, moves up by x: the window then covers [lo - x, lo - x + cap).
constexpr uint32_t kSlideWords = 2048;
// A window slide moves indices of at least lo + cap - x >= cap (x <= lo)
// out, so a slot holds [lds_words, wcap).  The copy-out reads the 16-byte
// units around the LDS/slot seam and one unit past the last word: a slot
// has kSlotLead words before the first index and kSlotTail after the last.
constexpr uint32_t kSlotLead = 8, kSlotTail = 16;
__device__ __forceinline__ void slide_window(__attribute__((address_space(3))) uint16_t *win, uint16_t *ovf_lo,
                                             uint32_t cap, uint32_t x, uint32_t pos_rel) {
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4u lds_u4;
  const uint32_t lane = lane_id();
  for (uint32_t i = 8 * lane; i < x; i += 8 * kLanes)
    *(v4u *)(ovf_lo + cap - x + i) = *(const lds_u4 *)(win + cap - x + i);
  // top chunk first: every word is read before its old place is written
  const int32_t start = (int32_t)(pos_rel & ~7u);
  for (int32_t c = (int32_t)(cap - x) - (int32_t)(8 * kLanes); c + (int32_t)(8 * kLanes) > start;
       c -= (int32_t)(8 * kLanes)) {
    const int32_t i = c + 8 * (int32_t)lane;
    if (i >= start) *(lds_u4 *)(win + i + x) = *(const lds_u4 *)(win + i);
  }
}

// 16 bytes starting `sh` bytes into p0 (sh even, < 16), continuing into p1
__device__ __forceinline__ uint4 funnel16(const uint4 p0, const uint4 p1, uint32_t sh) {
  uint32_t q0, q1, q2, q3, q4;
  switch (sh >> 2) {
    case 0: q0 = p0.x; q1 = p0.y; q2 = p0.z; q3 = p0.w; q4 = p1.x; break;
    case 1: q0 = p0.y; q1 = p0.z; q2 = p0.w; q3 = p1.x; q4 = p1.y; break;
    case 2: q0 = p0.z; q1 = p0.w; q2 = p1.x; q3 = p1.y; q4 = p1.z; break;
    default: q0 = p0.w; q1 = p1.x; q2 = p1.y; q3 = p1.z; q4 = p1.w; break;
  }
  const uint32_t b = sh & 3u;
  return make_uint4(__builtin_amdgcn_alignbyte(q1, q0, b), __builtin_amdgcn_alignbyte(q2, q1, b),
                    __builtin_amdgcn_alignbyte(q3, q2, b), __builtin_amdgcn_alignbyte(q4, q3, b));
}

// zero the bytes of a 16-byte unit at or past byte `keep` (even, < 16)
__device__ __forceinline__ uint4 keep_bytes(uint4 o, uint32_t keep) {
  uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
  for (uint32_t j = 0; j < 4; ++j) {
    if (4 * j >= keep)
      w[j] = 0;
    else if (4 * j + 2 == keep)
      w[j] &= 0xFFFFu;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Full groups addressed as a wave-uniform round base (kept in scalar
// registers) plus a 32-bit lane offset: round r of a block starts at
// elements blk0 + 512 r; lane j owns 16 (E = 2) or 32 (E = 4) bytes of it.
template <int E, bool NT = false>
__device__ __forceinline__ void load_round(const uint8_t *round_base, uint32_t w[4 * (E / 2)]) {
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  const v4u *p = (const v4u *)round_base + (E / 2) * lane_id();
  // NT for a last read: a block whose symbols stay in registers is read
  // once, so its lines need not stay in the caches (compress alone 0.586 ->
  // 0.548 ms, interleaved A/B on the 1 GiB buffer); a block re-read in the
  // coding pass keeps ordinary loads in pass 1 and takes NT ones there
  const v4u a = NT ? __builtin_nontemporal_load(p) : p[0];
  w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
  if (E == 4) {
    const v4u b = NT ? __builtin_nontemporal_load(p + 1) : p[1];
    w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
  }
}

template <int E, bool SYS>
__device__ __forceinline__ void store_raw_round(uint8_t *raw_round_base, const Group &g) {
  uint8_t *q = raw_round_base + 8 * (E - 1) * lane_id();
  out64<SYS>(q, g.raw[0], g.raw[1]);
  if (E == 4) {
    out64<SYS>(q + 8, g.raw[2], g.raw[3]);
    out64<SYS>(q + 16, g.raw[4], g.raw[5]);
  }
}

__device__ __forceinline__ void hist_add8(uint32_t *h, const Group &g, uint32_t valid) {
#pragma unroll
  for (uint32_t q = 0; q < 8; ++q)
    if (q < valid) atomicAdd(&h[sym_at(g.sym, q)], 1u);
}

// Packed 16-bit counts (a block holds at most 32768 symbols): symbols s and
// s + 128 share word s & 127, low and high half.  The bit-field extract is
// written out: the compiler turns it into a shift-and-mask pair.  hs holds,
// per symbol byte, 16 if the symbol's top bit is set and 0 otherwise: the
// increment 1 << that is one SDWA shift of a register holding 1.
template <int O>
__device__ __forceinline__ void hist_add_packed(uint32_t *h, uint32_t w, uint32_t hs, uint32_t one, bool on) {
  uint32_t word, inc;
  asm("v_bfe_u32 %0, %1, %2, 7" : "=v"(word) : "v"(w), "i"(O));  // symbol & 127
  if constexpr (O == 0)
    asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 src1_sel:DWORD"
        : "=v"(inc) : "v"(hs), "v"(one));
  else if constexpr (O == 8)
    asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD"
        : "=v"(inc) : "v"(hs), "v"(one));
  else if constexpr (O == 16)
    asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:DWORD"
        : "=v"(inc) : "v"(hs), "v"(one));
  else
    asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 src1_sel:DWORD"
        : "=v"(inc) : "v"(hs), "v"(one));
  if (on) atomicAdd(&h[word], inc);  // 1 or 1 << 16
}
__device__ __forceinline__ void hist_add8_packed(uint32_t *h, const Group &g, uint32_t valid) {
  const uint32_t hs0 = (g.sym[0] >> 3) & 0x10101010u, hs1 = (g.sym[1] >> 3) & 0x10101010u;
  uint32_t one = 1;
  asm volatile("" : "+v"(one));
  hist_add_packed<0>(h, g.sym[0], hs0, one, 0 < valid);
  hist_add_packed<8>(h, g.sym[0], hs0, one, 1 < valid);
  hist_add_packed<16>(h, g.sym[0], hs0, one, 2 < valid);
  hist_add_packed<24>(h, g.sym[0], hs0, one, 3 < valid);
  hist_add_packed<0>(h, g.sym[1], hs1, one, 4 < valid);
  hist_add_packed<8>(h, g.sym[1], hs1, one, 5 < valid);
  hist_add_packed<16>(h, g.sym[1], hs1, one, 6 < valid);
  hist_add_packed<24>(h, g.sym[1], hs1, one, 7 < valid);
}

// 16 image bytes from LDS: unit u of the image at byte offset sh of s32
__device__ __forceinline__ uint4 lds_unit(const uint32_t *s32, uint32_t u, uint32_t sh) {
  const uint32_t *q = s32 + 4 * u;
  uint4 o;
  o.x = __builtin_amdgcn_alignbyte(q[1], q[0], sh);
  o.y = __builtin_amdgcn_alignbyte(q[2], q[1], sh);
  o.z = __builtin_amdgcn_alignbyte(q[3], q[2], sh);
  o.w = __builtin_amdgcn_alignbyte(q[4], q[3], sh);
  return o;
}

// bytes [0, keep) of o, the rest zero (any keep < 16)
__device__ __forceinline__ uint4 mask_bytes(uint4 o, uint32_t keep) {
  uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int nb = (int)keep - 4 * j;
    w[j] = nb >= 4 ? w[j] : nb <= 0 ? 0u : w[j] & ((1u << (8 * nb)) - 1u);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// bytes [0, m) of a and [m, 16) of b (m even, 0 < m < 16)
__device__ __forceinline__ uint4 splice_bytes(uint4 a, uint4 b, uint32_t m) {
  const uint32_t x[4] = {a.x, a.y, a.z, a.w}, y[4] = {b.x, b.y, b.z, b.w};
  uint32_t w[4];
#pragma unroll
  for (uint32_t j = 0; j < 4; ++j)
    w[j] = (4 * j + 4 <= m) ? x[j] : (4 * j >= m) ? y[j] : ((x[j] & 0xFFFFu) | (y[j] & 0xFFFF0000u));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// What the copy-out of a coded block needs once its offset is known, all
// wave-uniform.  Small blocks keep it across the next block's first pass:
// the offset is resolved only then, when the predecessors have long
// published their lengths.
struct Fin {
  uint8_t *sout;       // the block's stream
  const uint8_t *src;  // the stream's input (a STORED block re-reads its symbols)
  uint64_t coded_off;  // stream offset of the coded sections
  uint64_t dir_end;    // end of the directory (a stored table follows)
  uint64_t chunk_n;    // elements of the stream
  uint64_t blk0;       // first element of the block, stream-relative
  uint64_t sec_len;    // section bytes, a multiple of 16
  uint32_t img;        // section image bytes (header + words) of a coded block
  uint32_t b, chunk, lb, first_block, n_blocks, n_b, rounds;
  uint32_t A;          // staging-area byte offset of the image
  uint32_t lds_bytes;  // image bytes in LDS; the rest is in the overflow slot
  uint32_t slot_delta; // slot byte = image byte + slot_delta (mod 2^32)
  const uint8_t *sym_lds;  // fused reduce: the block's symbols in LDS (a STORED block copies them)
  bool stored, spilled, last;
};

// The section head right before a coded block's words in the staging area
// (image byte offset A): the 64 states, and for a table of its own the
// presence bitmap and the frequencies.
template <bool SHARED>
__device__ __forceinline__ void write_section_head(uint8_t *stage, uint32_t A, uint32_t x, const Table &t) {
  const uint32_t lane = lane_id();
  uint16_t *h16 = (uint16_t *)(stage + A);
  h16[2 * lane] = (uint16_t)x;
  h16[2 * lane + 1] = (uint16_t)(x >> 16);
  if constexpr (!SHARED) {
    if (lane < 16) {
      uint32_t word = 0;
      for (uint32_t bit = 0; bit < 16; ++bit) {
        uint32_t sy = 16 * lane + bit;
        word |= (uint32_t)((t.present[sy & 3] >> (sy >> 2)) & 1u) << bit;
      }
      h16[128 + lane] = (uint16_t)word;
    }
    uint32_t rk = t.rank0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (t.f[q]) h16[144 + rk++] = (uint16_t)t.f[q];
  }
}

// Resolve the block's offset, write its directory entry and section, and for
// a stream's last block the stream header.
template <int DT, bool SYS>
__device__ __forceinline__ void finish_block(const EncodeArgs &a, const Fin &f, const uint8_t *stage,
                                             const uint16_t *ovf) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  const uint32_t lane = lane_id();
  bool failed;
  const uint64_t excl = resolve_prefix(a.status, f.b, f.first_block, f.sec_len / 16, a.ticket[kWsSpin],
                                       a.ticket[kWsHold], a.ticket + kWsError, failed);
  uint8_t *sec = f.sout + f.coded_off + 16 * excl;
  if (lane == 0)
    out32<SYS>((uint32_t *)(f.sout + kHeaderBytes + 4 * f.lb),
               (f.stored ? kStoredBit : 0u) | (uint32_t)(excl + f.sec_len / 16));

  if (!f.stored) {
    const uint32_t *s32 = (const uint32_t *)(stage + (f.A & ~3u));
    const uint32_t sh = f.A & 3u;
    if (!f.spilled) {
      // the whole image is contiguous in LDS
      for (uint32_t u = lane; u < f.sec_len / 16; u += 64) out128<SYS>(sec + 16 * u, lds_unit(s32, u, sh));
    } else {
      // image bytes [0, lds_bytes) are in LDS, bytes [lds_bytes, img) in
      // the workgroup's overflow slot
      const uint32_t lb = f.lds_bytes, imgb = f.img, d = f.slot_delta;
      const uint8_t *ovb = (const uint8_t *)ovf;
      for (uint32_t u = lane; u < f.sec_len / 16; u += 64) {
        uint4 o;
        if (16 * u + 16 <= lb) {
          o = lds_unit(s32, u, sh);
        } else {
          const uint32_t off = 16 * u + d;
          const uint4 *p = (const uint4 *)(ovb + (off & ~15u));
          o = funnel16(p[0], p[1], off & 15u);
          // the unit where LDS and slot bytes meet (lb is even; the LDS
          // reads stay within the staging area's zeroed tail)
          if (16 * u < lb) o = splice_bytes(lds_unit(s32, u, sh), o, lb - 16 * u);
          if (16 * u + 16 > imgb) o = keep_bytes(o, imgb - 16 * u);
        }
        out128<SYS>(sec + 16 * u, o);
      }
    }
  } else if (f.sym_lds != nullptr) {
    // STORED, fused reduce: the block's symbol bytes from LDS, zero-padded
    for (uint32_t u = lane; u < f.sec_len / 16; u += 64) {
      uint4 o = *(const uint4 *)(f.sym_lds + 16 * u);
      if (16 * u + 16 > f.n_b) o = mask_bytes(o, f.n_b - 16 * u);
      out128<SYS>(sec + 16 * u, o);
    }
  } else {
    // STORED: the block's symbol bytes, zero-padded to 16, re-read from the
    // input (the coding pass consumed the register copy)
    const uint32_t padded = (uint32_t)pad16(f.n_b);
    for (uint32_t r = 0; r < f.rounds; ++r) {
      const uint32_t i0 = r * kRound + kPerLane * lane;
      const uint32_t valid = i0 < f.n_b ? (f.n_b - i0 < 8 ? f.n_b - i0 : 8) : 0;
      uint32_t s0 = 0, s1 = 0;
      if (valid > 0) {
        uint32_t w[NW];
        Group gr;
        load_words<E>(f.src, f.blk0 + i0, valid, w);
        split_group<DT>(w, gr);
        s0 = gr.sym[0];
        s1 = gr.sym[1];
      }
      if (i0 >= padded) continue;
      if (valid < 8) {
        const uint64_t keep = valid ? (~0ull >> (64 - 8 * valid)) : 0ull;
        const uint64_t v = ((uint64_t)s1 << 32 | s0) & keep;
        s0 = (uint32_t)v;
        s1 = (uint32_t)(v >> 32);
      }
      out64<SYS>(sec + i0, s0, s1);
    }
  }

  if (f.last) {
    const uint64_t total = f.coded_off + 16 * (excl + f.sec_len / 16);
    if (lane == 0) {
      uint32_t hh[8];
      hh[0] = kMagic;
      hh[1] = kVersion | ((uint32_t)DT << 8) | (kProbBits << 16) | (a.table_mode << 24);
      hh[2] = a.block_elems;
      hh[3] = f.n_blocks;
      hh[4] = (uint32_t)f.chunk_n;
      hh[5] = (uint32_t)(f.chunk_n >> 32);
      hh[6] = (uint32_t)total;
      hh[7] = (uint32_t)(total >> 32);
      uint64_t *hp = (uint64_t *)f.sout;
#pragma unroll
      for (int q = 0; q < 4; ++q) coh64<SYS>(hp + q, (uint64_t)hh[2 * q + 1] << 32 | hh[2 * q]);
      if (a.sizes != nullptr) coh64<SYS>(&a.sizes[f.chunk], total);
    }
    // zero padding after the directory
    const uint64_t db = kHeaderBytes + 4ull * f.n_blocks + lane;
    if (lane < 16 && db < f.dir_end) out8<SYS>(f.sout + db, 0);
  }
  if (a.flags != nullptr)
    publish_chunk(&a.chunk_cnt[2 * f.chunk + 1], f.n_blocks, &a.flags[2 * f.chunk + 1], a.epoch, failed, !SYS);
}

// End of a persistent encoder workgroup.  The last one out (its stores and
// every other workgroup's complete: each waits for its own before counting
// itself) marks every stream that had a failed look-back invalid: magic and
// size 0 -- a stream is never shorter than its 32-byte header, so a zero
// size is the error -- the split-send producer's DONE flag raised over it,
// and the fused reduce's status set.  The split-send producer also marks a
// chunk that no wave finished so (under the XCD-local producer, an XCD that
// received no workgroup; a stream-wide table found invalid), rather than
// leave its flags down.
template <bool SYS, bool REDUCE>
__device__ void finish_launch(const EncodeArgs &a) {
  const uint32_t lane = lane_id();
  __builtin_amdgcn_s_waitcnt(0);
  uint32_t last = 0;
  if (lane == 0)
    last = __hip_atomic_fetch_add(a.ticket + kWsExit, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1 == gridDim.x;
  if (!uniform(last)) return;
  const bool err = __hip_atomic_load(a.ticket + kWsError, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
  if (!err && a.flags == nullptr) return;
  const uint32_t streams = (a.n_blocks + a.blocks_per_chunk - 1) / a.blocks_per_chunk;
  for (uint32_t c = lane; c < streams; c += 64) {
    bool bad = a.flags == nullptr, raw_short = false;
    if (!bad) {
      const uint32_t left = a.n_blocks - c * a.blocks_per_chunk;
      const uint32_t need = left < a.blocks_per_chunk ? left : a.blocks_per_chunk;
      const uint32_t cnt = __hip_atomic_load(&a.chunk_cnt[2 * c + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      raw_short = __hip_atomic_load(&a.chunk_cnt[2 * c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != need;
      bad = (cnt & kChunkFailed) || (cnt & ~kChunkFailed) != need;
    }
    if (!bad) continue;
    coh64<SYS>((uint64_t *)(a.out + (uint64_t)c * a.slot_bytes), 0);
    if (a.sizes != nullptr) coh64<SYS>(&a.sizes[c], 0);
    if (a.flags != nullptr) {
      __builtin_amdgcn_s_waitcnt(0);
      if (!SYS) writeback_l2();
      // a chunk that no wave coded has not raised RAW_READY either
      if (raw_short) __hip_atomic_store(&a.flags[2 * c], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(&a.flags[2 * c + 1], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
  if (REDUCE && lane == 0) report(*(uint32_t *const *)(a.ticket + kWsStatusPtr), UZIP_ETIMEOUT);
}

// ---------------------------------------------------------------------------
// encode_kernel: compress / split-send producer / fused reduce.
// Persistent workgroups of one wave take blocks in ticket order.
// SMALL: block_elems <= 32768, the block's symbols stay in registers and the
//   LDS staging area holds a.lds_words words, the rest spills to the
//   workgroup's overflow slot.  Otherwise the coding pass re-reads the block
//   and LDS holds the whole staging area.
// ---------------------------------------------------------------------------
template <int DT, bool REDUCE, bool SMALL, bool SYS, bool SHARED = false>
__device__ __forceinline__ void encode_body(const EncodeArgs &a) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  // pass-1 load pipeline depth (rounds; it must divide 16): 16 KiB in flight
  // per wave for 16-bit elements (8 KiB where the stream-wide table's
  // variants would spill), 8 KiB for fp32
  constexpr int D = (E == 2) ? (SHARED ? 8 : 16) : 4;
  extern __shared__ __align__(16) uint8_t smem_base[];
  uint8_t *smem = smem_base + kTrashBytes;  // [trash | encoder table | histogram / staging]
  uint4 *enc = (uint4 *)smem;  // at LDS byte kTrashBytes: the kernel has no static LDS (the host checks)
  uint32_t *hist = (uint32_t *)(smem + kEncTableBytes);
  uint8_t *stage = smem + a.pass2_off;
  uint16_t *stage16 = (uint16_t *)(stage + kStageHead);
  const uint32_t lane = lane_id();
  // the workgroup's overflow slot holds the staging indices that can leave
  // the LDS window, [lds_words, wcap), after kSlotLead words of margin:
  // ovf[v] is index v
  uint16_t *ovf = a.slots + (uint64_t)blockIdx.x * a.slot_words + kSlotLead - a.lds_words;
  typedef __attribute__((address_space(3))) uint16_t lds16_t;
  // one private 2-byte slot per lane for words that are not emitted (64
  // slots in 32 consecutive words: every bank once)
  lds16_t *trash = (lds16_t *)smem_base + lane;
  // small blocks: a block's offset is resolved and its section written
  // after the next block's first pass, so the wait for slower predecessors
  // overlaps streaming.  The staging area then still holds the pending
  // block's image during the first pass: the histogram takes packed 16-bit
  // counts in the trash slots and encoder table instead, which are free
  // until the coding pass (the table is built from the counts in place).
  constexpr bool DEFER = SMALL && !REDUCE;
  // larger blocks keep their last 64 rounds' symbols in registers, so the
  // coding pass reads the rest of the block again instead of all of it
  // (interleaved A/B, 256 KiB blocks: 1 GiB fp32 gradient 0.748 -> 0.680 ms,
  // 1 GiB bf16 buffer 0.816 -> 0.775 ms, 512 MiB fp16 gradient 0.484 ->
  // 0.480 ms)
  constexpr bool KEEP = !SMALL && !REDUCE;
  static_assert(kHistReplicas * kPackedHistStride * 4 <= kTrashBytes + kEncTableBytes, "packed histogram");
  uint32_t *phist = (uint32_t *)smem_base;
  Fin pend;
  bool have_pend = false;
  // a stream-wide table codes every block of its stream: the wave derives
  // its encoder entries when it moves to a block of another stream
  uint32_t table_chunk = ~0u;
  // deferred copy-out: the next block's ticket is taken before the table and
  // the coding pass, which hide the atomic's latency (lane 0 holds it)
  uint32_t next_ticket = 0;
  if constexpr (DEFER) {
    if (lane == 0) next_ticket = take_block(a);
  }

  while (true) {
    uint32_t b = 0;
    if constexpr (DEFER) b = next_ticket;
    else if (lane == 0) b = take_block(a);
    b = uniform(b);
    if (b >= a.n_blocks) break;

    const uint32_t chunk = b / a.blocks_per_chunk;
    const uint32_t lb = b - chunk * a.blocks_per_chunk;
    const uint32_t first_block = b - lb;
    if constexpr (SHARED) {
      if (chunk != table_chunk && (a.table_stride != 0 || table_chunk == ~0u)) {
        Table ts;
        const uint2 v = *(const uint2 *)(a.table + (uint64_t)chunk * a.table_stride + 4 * lane);
        ts.f[0] = v.x & 0xFFFFu;
        ts.f[1] = v.x >> 16;
        ts.f[2] = v.y & 0xFFFFu;
        ts.f[3] = v.y >> 16;
        // a table that is not an all-symbol table (some f = 0, or a sum
        // other than M) codes nothing: the block is skipped (every block of
        // the stream is, the table being the stream's) and the stream size
        // reads 0; the wave goes on with its next ticket, so that every
        // stream of the call has its size set
        const bool bad = ts.f[0] == 0 || ts.f[1] == 0 || ts.f[2] == 0 || ts.f[3] == 0;
        if (__any(bad) || wave_sum(ts.f[0] + ts.f[1] + ts.f[2] + ts.f[3]) != kM) {
          if (lane == 0 && a.sizes != nullptr) a.sizes[chunk] = 0;
          if constexpr (DEFER) {
            // a pending block belongs to an earlier stream with a valid table
            if (have_pend) finish_block<DT, SYS>(a, pend, stage, ovf);
            have_pend = false;
            if (lane == 0) next_ticket = take_block(a);
          }
          __syncthreads();
          continue;
        }
        __syncthreads();  // the previous block's coding pass is done with the entries
        enc_entries(ts, enc);
        __syncthreads();
      }
      table_chunk = chunk;
    }
    const uint64_t chunk_first = (uint64_t)chunk * a.chunk_elems;
    const uint64_t chunk_n = (a.n - chunk_first) < a.chunk_elems ? (a.n - chunk_first) : a.chunk_elems;
    Geom g = make_geom(chunk_n, a.block_elems, E);
    const uint64_t dir_end = g.raw_off;  // a stored stream-wide table sits between the directory and the raw plane
    g.raw_off += a.table_bytes;
    g.coded_off += a.table_bytes;
    uint8_t *sout = a.out + (uint64_t)chunk * a.slot_bytes;
    const uint64_t blk0 = (uint64_t)lb * a.block_elems;  // chunk-relative
    const uint32_t n_b = (uint32_t)((chunk_n - blk0) < a.block_elems ? (chunk_n - blk0) : a.block_elems);
    const uint32_t rounds = (n_b + kRound - 1) / kRound;
    uint32_t full = n_b / kRound;
    // small blocks: an opaque scalar, or the compiler folds the prefetch
    // clamps (r + D < full) back into 64-bit vector compares on n (the
    // large blocks' loops come out slower with it)
    if constexpr (SMALL) asm volatile("" : "+s"(full));
    const bool last_in_chunk = (lb + 1 == g.n_blocks);
    const uint8_t *src = REDUCE ? a.ybuf : a.in + chunk_first * E;  // pass-2 source (large blocks)
    uint8_t *raw_plane = sout + g.raw_off;
    const uint8_t *src_blk = src + blk0 * E;           // wave-uniform
    uint8_t *raw_blk = raw_plane + blk0 * (E - 1);      // wave-uniform
    uint32_t *h = hist + (lane & (kHistReplicas - 1)) * kHistStride;
    SymRegs S;

    // The first pass (memory-bound) runs at raised wave priority, the rest
    // at normal: a SIMD's two waves then overlap streaming with coding
    // instead of the older wave winning both.
    __builtin_amdgcn_s_setprio(1);
    // ---- pass 1: split, raw plane to its final place, histogram ----
    if constexpr (!DEFER) {
      for (uint32_t i = lane; i < kHistReplicas * kHistStride; i += 64) hist[i] = 0;
      __syncthreads();
    } else if constexpr (!SHARED) {
      for (uint32_t i = lane; i < kHistReplicas * kPackedHistStride; i += 64) phist[i] = 0;
      __syncthreads();
      h = phist + (lane & (kHistReplicas - 1)) * kPackedHistStride;
    }
    // one histogram update of `valid` symbols
    auto hist_upd = [&](const Group &gr, uint32_t valid) {
      if constexpr (DEFER) hist_add8_packed(h, gr, valid);
      else hist_add8(h, gr, valid);
    };

    uint32_t psym0 = 0, psym1 = 0;  // symbols of a partial last round
    if constexpr (!REDUCE) {
      auto partial_round = [&]() {
        const uint32_t i0 = full * kRound + kPerLane * lane;
        const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
        Group gr;
        gr.sym[0] = gr.sym[1] = 0;
        if (valid > 0) {
          uint32_t w[NW];
          load_words<E>(src, blk0 + i0, valid, w);
          split_group<DT>(w, gr);
          store_raw<E, SYS>(raw_plane, blk0 + i0, valid, gr);
          if constexpr (!SHARED) hist_upd(gr, valid);
        }
        psym0 = gr.sym[0];
        psym1 = gr.sym[1];
      };
      uint32_t buf[D][NW];
      if (full > 0) {
#pragma unroll
        for (int u = 0; u < D; ++u)
          load_round<E, SMALL>(src_blk + (uint64_t)(u < (int)full ? u : full - 1) * kRound * E, buf[u]);
      }
      if constexpr (SMALL) {
        // Fully unrolled and free of value-carrying branches: loads, the
        // split and the register writes run for all 64 rounds (addresses
        // clamped to a real round), only the side effects are guarded.  A
        // prefetch buffer that crossed a branch join would be copied right
        // after its load, and the copy would wait for the load.
        if (full > 0) {
#pragma unroll
          for (uint32_t gi = 0; gi < 4; ++gi) {
#pragma unroll
            for (int rr = 0; rr < 16; ++rr) {
              const uint32_t r = 16 * gi + rr;
              uint32_t w[NW];
#pragma unroll
              for (int q = 0; q < NW; ++q) w[q] = buf[rr % D][q];
              const uint32_t rn = (r + D < full) ? r + D : full - 1;
              // the round's address as a scalar base plus the lane's offset
              // (scalar-base loads and stores; the compiler would otherwise
              // keep a per-lane 64-bit pointer and add each round's offset
              // to it with vector adds)
              const __attribute__((address_space(1))) uint8_t *rsrc =
                  (const __attribute__((address_space(1))) uint8_t *)(src_blk + (uint64_t)rn * kRound * E);
              asm("" : "+s"(rsrc));
              load_round<E, SMALL>((const uint8_t *)rsrc, buf[rr % D]);
              Group gr;
              split_group<DT>(w, gr);
              // the compiler would otherwise carry the split words (four;
              // eight for fp32) to the coding pass instead of the two symbol
              // words and spill, when no histogram update takes the symbols
              // here or fp32's wider words crowd the registers: make the
              // symbols now
              if constexpr (SHARED || DT == 2) asm volatile("" : "+v"(gr.sym[0]), "+v"(gr.sym[1]));
              S.v3[2 * rr] = gr.sym[0];
              S.v3[2 * rr + 1] = gr.sym[1];
              if (r < full) {
                __attribute__((address_space(1))) uint8_t *rdst =
                    (__attribute__((address_space(1))) uint8_t *)(raw_blk + (uint64_t)r * kRound * (E - 1));
                asm("" : "+s"(rdst));
                store_raw_round<E, SYS>((uint8_t *)rdst, gr);
                if constexpr (!SHARED) hist_upd(gr, 8);
              }
            }
            if (gi < 3) shift_down(S);
          }
        }
        if (full < rounds) partial_round();  // its symbols stay in psym0/psym1
      } else {
        // rounds below kb stream through (the coding pass reads them
        // again); the last 64 then keep their symbols in registers as a
        // small block's do, and the coding pass starts with them
        const uint32_t kb = KEEP ? (full > kRegRounds ? full - kRegRounds : 0) : full;
        if (kb > 0) {
          uint32_t r = 0;
          for (; r + D <= kb; r += D) {
#pragma unroll
            for (int u = 0; u < D; ++u) {
              uint32_t w[NW];
#pragma unroll
              for (int q = 0; q < NW; ++q) w[q] = buf[u][q];
              const uint32_t rn = (r + u + D < kb) ? r + u + D : kb - 1;
              load_round<E>(src_blk + (uint64_t)rn * kRound * E, buf[u]);
              Group gr;
              split_group<DT>(w, gr);
              store_raw_round<E, SYS>(raw_blk + (uint64_t)(r + u) * kRound * (E - 1), gr);
              if constexpr (!SHARED) hist_add8(h, gr, 8);
            }
          }
#pragma unroll
          for (int u = 0; u < D - 1; ++u) {
            if (r + u < kb) {
              Group gr;
              split_group<DT>(buf[u], gr);
              store_raw_round<E, SYS>(raw_blk + (uint64_t)(r + u) * kRound * (E - 1), gr);
              if constexpr (!SHARED) hist_add8(h, gr, 8);
            }
          }
        }
        if constexpr (KEEP) {
          if (full > 0) {
            // the small-block loop above, from round kb (the block is not
            // read again after these rounds: non-temporal loads)
#pragma unroll
            for (int u = 0; u < D; ++u)
              load_round<E, true>(src_blk + (uint64_t)(kb + u < full ? kb + u : full - 1) * kRound * E, buf[u]);
#pragma unroll
            for (uint32_t gi = 0; gi < 4; ++gi) {
#pragma unroll
              for (int rr = 0; rr < 16; ++rr) {
                const uint32_t r = kb + 16 * gi + rr;
                uint32_t w[NW];
#pragma unroll
                for (int q = 0; q < NW; ++q) w[q] = buf[rr % D][q];
                const uint32_t rn = (r + D < full) ? r + D : full - 1;
                load_round<E, true>(src_blk + (uint64_t)rn * kRound * E, buf[rr % D]);
                Group gr;
                split_group<DT>(w, gr);
                asm volatile("" : "+v"(gr.sym[0]), "+v"(gr.sym[1]));
                S.v3[2 * rr] = gr.sym[0];
                S.v3[2 * rr + 1] = gr.sym[1];
                if (r < full) {
                  store_raw_round<E, SYS>(raw_blk + (uint64_t)r * kRound * (E - 1), gr);
                  if constexpr (!SHARED) hist_add8(h, gr, 8);
                }
              }
              if (gi < 3) shift_down(S);
            }
          }
        }
        if (full < rounds) partial_round();
      }
    } else {
      // fused reduce: the decode-reduce kernel left the reduced tensor (the
      // source of the coding pass), the raw plane and this block's histogram
      for (uint32_t sy = lane; sy < 256; sy += 64) hist[sy] = a.hist_in[(uint64_t)b * 256 + sy];
    }

    if (last_in_chunk && lane < 16) {
      // zero padding after the raw plane (pad16 of (E-1) n bytes)
      uint64_t rb = g.raw_off + (uint64_t)(E - 1) * chunk_n + lane;
      if (rb < g.coded_off) out8<SYS>(sout + rb, 0);
    }
    __syncthreads();
    if (a.flags != nullptr) {
      publish_chunk(&a.chunk_cnt[2 * chunk], g.n_blocks, &a.flags[2 * chunk], a.epoch, false, !SYS);
    }

    __builtin_amdgcn_s_setprio(0);
    if constexpr (DEFER) {
      // the previous block's section leaves the staging area
      if (have_pend) finish_block<DT, SYS>(a, pend, stage, ovf);
      have_pend = false;
      if (lane == 0) next_ticket = take_block(a);
      __syncthreads();
    }
    // ---- table ----
    Table t;
    if constexpr (SHARED) {
      t.k = 256;  // only the section head differs: no bitmap, no frequencies
    } else {
      if constexpr (DEFER) build_enc_table<true>(phist, n_b, enc, t);
      else build_enc_table(hist, n_b, enc, t);
      t.k = uniform(t.k);
      __syncthreads();
    }
    // section bytes before the words: states, and for a table of its own
    // the presence bitmap and the frequencies
    const uint32_t hdr = SHARED ? kSharedSectionFixed : kSectionFixed + 2 * t.k;

    // ---- pass 2: rANS over the block, backwards; words staged ----
    for (uint32_t i = lane; i < kStageTail / 4; i += 64)
      ((uint32_t *)(stage + kStageHead + 2 * a.lds_words))[i] = 0;
    const uint32_t limit_words = (n_b > hdr) ? (n_b - hdr + 1) / 2 : 0;
    uint32_t pos = a.wcap;  // virtual staging indices [pos, wcap) hold the words written so far
    // LDS window over virtual indices [lo, lo + lds_words); lds_rel[v] is index v
    uint32_t lo = a.wcap - a.lds_words;
    lds16_t *lds_rel = (lds16_t *)stage16 - lo;
    uint32_t spilled = a.wcap;  // indices [spilled, wcap) live in the overflow slot
    uint32_t x = kStateLo;
    bool stored = (limit_words == 0);
    if (full < rounds && !stored) {  // the partial last round comes first
      const uint32_t i0 = full * kRound + kPerLane * lane;
      const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
      uint32_t s0 = psym0, s1 = psym1;
      if (REDUCE && valid > 0) {
        uint32_t w[NW];
        Group gr;
        load_words<E>(src, blk0 + i0, valid, w);
        split_group<DT>(w, gr);
        s0 = gr.sym[0];
        s1 = gr.sym[1];
      }
      const uint32_t sy[2] = {s0, s1};
      uint4 e[8];
      if constexpr (SMALL) {  // (the large blocks' loops spill more with the fixed-address form)
        enc_lookup8_at<kTrashBytes>(sy[0], sy[1], e);
      } else {
#pragma unroll
        for (int tt = 0; tt < 8; ++tt) e[tt] = enc[sym_at(sy, tt)];
      }
      enc_round<false, SMALL>(x, e, valid, pos, lds_rel, trash);
      if (a.wcap - pos >= limit_words) stored = true;
    }
    if constexpr (SMALL) {
      for (int gi = 3; gi >= 0; --gi) {
#pragma unroll
        for (int rr = 15; rr >= 0; --rr) {
          const int r = 16 * gi + rr;
          if (r < (int)full && !stored) {
            if (pos < lo + kRound && lo > 0) {  // the LDS window is full: slide it down
              const uint32_t x = lo < kSlideWords ? lo : kSlideWords;
              slide_window((lds16_t *)stage16, ovf + lo, a.lds_words, x, pos - lo);
              lo -= x;
              spilled = lo + a.lds_words;
              lds_rel = (lds16_t *)stage16 - lo;
            }
            const uint32_t s0 = S.v3[2 * rr], s1 = S.v3[2 * rr + 1];
            uint4 e[8];
            enc_lookup8_at<kTrashBytes>(s0, s1, e);
            enc_round<true, true>(x, e, 8, pos, lds_rel, trash);
            if (a.wcap - pos >= limit_words) stored = true;
          }
        }
        if (gi > 0) shift_up(S);
      }
    } else if constexpr (!REDUCE) {
      // larger blocks: the last 64 rounds from the register store (as for a
      // small block, from round kb), then the rest of the block
      // re-read backwards, four rounds ahead (its last read: non-temporal;
      // fp16 in 256 KiB blocks 0.503 -> 0.457 ms, fp32 0.749 -> 0.733 ms,
      // interleaved A/B), and the LDS window sliding into the workgroup's
      // slot as for small ones
      const uint32_t kb = KEEP ? (full > kRegRounds ? full - kRegRounds : 0) : full;
      if constexpr (KEEP) {
        for (int gi = 3; gi >= 0; --gi) {
#pragma unroll
          for (int rr = 15; rr >= 0; --rr) {
            const int r = (int)kb + 16 * gi + rr;
            if (r < (int)full && !stored) {
              if (pos < lo + kRound && lo > 0) {  // the LDS window is full: slide it down
                const uint32_t x = lo < kSlideWords ? lo : kSlideWords;
                slide_window((lds16_t *)stage16, ovf + lo, a.lds_words, x, pos - lo);
                lo -= x;
                spilled = lo + a.lds_words;
                lds_rel = (lds16_t *)stage16 - lo;
              }
              const uint32_t s0 = S.v3[2 * rr], s1 = S.v3[2 * rr + 1];
              uint4 e[8];
              enc_lookup8(enc, s0, s1, e);
              enc_round<true>(x, e, 8, pos, lds_rel, trash);
              if (a.wcap - pos >= limit_words) stored = true;
            }
          }
          if (gi > 0) shift_up(S);
        }
      }
      constexpr int P = 4;
      uint32_t pb[P][NW];
      if (kb > 0) {
#pragma unroll
        for (int u = 0; u < P; ++u)
          load_round<E, true>(src_blk + (uint64_t)((int)kb - 1 - u >= 0 ? (int)kb - 1 - u : 0) * kRound * E, pb[u]);
      }
      for (int r0 = (int)kb - 1; r0 >= 0 && !stored; r0 -= P) {
#pragma unroll
        for (int u = 0; u < P; ++u) {
          const int r = r0 - u;
          if (r >= 0 && !stored) {
            if (pos < lo + kRound && lo > 0) {  // the LDS window is full: slide it down
              const uint32_t x = lo < kSlideWords ? lo : kSlideWords;
              slide_window((lds16_t *)stage16, ovf + lo, a.lds_words, x, pos - lo);
              lo -= x;
              spilled = lo + a.lds_words;
              lds_rel = (lds16_t *)stage16 - lo;
            }
            Group gr;
            split_group<DT>(pb[u], gr);
            // round r - P into the buffer just used (round 0 again once below it)
            const int rn = r - P;
            load_round<E, true>(src_blk + (uint64_t)(rn >= 0 ? rn : 0) * kRound * E, pb[u]);
            uint4 e[8];
            enc_lookup8(enc, gr.sym[0], gr.sym[1], e);
            enc_round<true>(x, e, 8, pos, lds_rel, trash);
            if (a.wcap - pos >= limit_words) stored = true;
          }
        }
      }
    } else {
      // the fused reduce's coding pass: the reduced block re-read backwards,
      // one round ahead, and the LDS window sliding into the workgroup's
      // slot as for compress
      uint32_t wa[NW], wbuf[NW];
      if (full > 0) load_round<E>(src_blk + (uint64_t)(full - 1) * kRound * E, wa);
      int r = (int)full - 1;
      for (; r >= 1 && !stored; r -= 2) {
        if (pos < lo + kRound && lo > 0) {  // the LDS window is full: slide it down
          const uint32_t x = lo < kSlideWords ? lo : kSlideWords;
          slide_window((lds16_t *)stage16, ovf + lo, a.lds_words, x, pos - lo);
          lo -= x;
          spilled = lo + a.lds_words;
          lds_rel = (lds16_t *)stage16 - lo;
        }
        load_round<E>(src_blk + (uint64_t)(r - 1) * kRound * E, wbuf);
        Group gr;
        split_group<DT>(wa, gr);
        uint4 e[8];
        enc_lookup8(enc, gr.sym[0], gr.sym[1], e);
        enc_round<true>(x, e, 8, pos, lds_rel, trash);
        if (a.wcap - pos >= limit_words) stored = true;
        if (stored) break;
        if (pos < lo + kRound && lo > 0) {  // the LDS window is full: slide it down
          const uint32_t x = lo < kSlideWords ? lo : kSlideWords;
          slide_window((lds16_t *)stage16, ovf + lo, a.lds_words, x, pos - lo);
          lo -= x;
          spilled = lo + a.lds_words;
          lds_rel = (lds16_t *)stage16 - lo;
        }
        const uint32_t rn = r >= 2 ? (uint32_t)(r - 2) : 0u;
        load_round<E>(src_blk + (uint64_t)rn * kRound * E, wa);
        split_group<DT>(wbuf, gr);
        enc_lookup8(enc, gr.sym[0], gr.sym[1], e);
        enc_round<true>(x, e, 8, pos, lds_rel, trash);
        if (a.wcap - pos >= limit_words) stored = true;
      }
      if (r == 0 && !stored) {  // wa holds round 0
        if (pos < lo + kRound && lo > 0) {  // the LDS window is full: slide it down
          const uint32_t x = lo < kSlideWords ? lo : kSlideWords;
          slide_window((lds16_t *)stage16, ovf + lo, a.lds_words, x, pos - lo);
          lo -= x;
          spilled = lo + a.lds_words;
          lds_rel = (lds16_t *)stage16 - lo;
        }
        Group gr;
        split_group<DT>(wa, gr);
        uint4 e[8];
        enc_lookup8(enc, gr.sym[0], gr.sym[1], e);
        enc_round<true>(x, e, 8, pos, lds_rel, trash);
        if (a.wcap - pos >= limit_words) stored = true;
      }
    }
    pos = uniform(pos);
    const uint32_t n_words = a.wcap - pos;
    const uint64_t img = hdr + 2ull * n_words;
    const uint64_t sec_len = stored ? pad16(n_b) : pad16(img);

    // ---- the section image goes to LDS, the length is published ----
    Fin f;
    f.sout = sout;
    f.src = src;
    f.coded_off = g.coded_off;
    f.dir_end = dir_end;
    f.chunk_n = chunk_n;
    f.blk0 = blk0;
    f.sec_len = sec_len;
    f.img = (uint32_t)img;
    f.b = b;
    f.chunk = chunk;
    f.lb = lb;
    f.first_block = first_block;
    f.n_blocks = g.n_blocks;
    f.n_b = n_b;
    f.rounds = rounds;
    f.A = kStageHead + 2 * (pos - lo) - hdr;
    f.lds_bytes = hdr + 2 * (spilled - pos);
    f.slot_delta = 2 * spilled - f.lds_bytes;
    f.stored = stored;
    f.spilled = spilled != a.wcap;
    f.last = last_in_chunk;
    f.sym_lds = nullptr;
    if (!stored) {
      // header bytes right before the words: states | bitmap | f[k] (states
      // only with a stream-wide table)
      write_section_head<SHARED>(stage, f.A, x, t);
      // the overflow slot was written by this wave: order its stores before
      // the copy-out's reads (one wave per workgroup, one CU: no cache in between)
      if (f.spilled) __threadfence_block();
    }
    __syncthreads();
    publish_aggregate(a.status, b, first_block, sec_len / 16, a.ticket[kWsHold]);
    if constexpr (DEFER) {
      pend = f;
      have_pend = true;
    } else {
      finish_block<DT, SYS>(a, f, stage, ovf);
    }
    __syncthreads();
  }
  if constexpr (DEFER) {
    if (have_pend) finish_block<DT, SYS>(a, pend, stage, ovf);
  }
}

// Compress kernels keep two waves per SIMD (the LDS budget allows eight
// workgroups per CU); the fused reduce holds many more per-input states.
template <int DT, bool SMALL, bool SYS, bool SHARED = false>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) encode_kernel(EncodeArgs a) {
  encode_body<DT, false, SMALL, SYS, SHARED>(a);
  finish_launch<SYS, false>(a);
}
template <int DT>
__global__ void __launch_bounds__(64) reduce_kernel(EncodeArgs a) {
  encode_body<DT, true, false, false>(a);
  finish_launch<false, true>(a);
}

// ---------------------------------------------------------------------------
// Table decoding: the decode sub-step shared by decode_kernel and the fused
// reduce's decoding waves, and the fused reduce's word ring.
//
// In the fused reduce the words of a coded block are staged through a 4 KB
// LDS ring in 1 KB chunks read with one 16-byte load per lane: a chunk is
// loaded as soon as the ring has room and written to LDS only when the
// decoder is about to need it, so the serial decode chain only ever waits on
// LDS.  The raw plane of the next round is loaded one round ahead.
// decode_kernel's own ring (2 KB, more waves per CU) is described with it.
// ---------------------------------------------------------------------------
constexpr uint32_t kRingBytes = 4096;
constexpr uint32_t kRingMirror = 128;  // ring[0, 128) repeated past the end: one step's reads never wrap
constexpr uint32_t kChunkBytes = 1024;

// One decode sub-step of every lane (inverse of the coding function, then
// 16-bit renormalisation).  Returns the lane's table entry (its symbol in the
// top byte; 0 for a lane without an element).  Branch-free: every lane reads
// the ring at its would-be word position rb + 2 * rank (rb: ring offset of
// the next unread word, uniform); lanes that need no word keep their state.
// Positions past the section's words stay inside the ring and are caught
// once per block by p <= w_avail.
template <bool FULL, uint32_t RB = kRingBytes, bool MIRROR = true>
__device__ __forceinline__ uint32_t decode_step_ring(uint32_t &x, bool valid, const uint32_t *lut,
                                                     const uint8_t *ring, uint32_t &rb, uint32_t &p) {
  uint32_t e = 0;
  if (FULL || valid) {
    e = lut[x & (kM - 1)];
    x = __umul24(e & 0xFFFu, x >> kProbBits) + ((e >> 12) & 0x7FFu);
  }
  const bool need = (FULL || valid) && x < kStateLo;
  const uint64_t m = __ballot(need);
  const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
  uint32_t w = *(const uint16_t *)(ring + (MIRROR ? rb + 2 * rank : (rb + 2 * rank) & (RB - 1)));
  asm volatile("" : "+v"(w));  // keep the read unconditional: no exec-mask branch around it
  x = need ? ((x << 16) | w) : x;
  const uint32_t c = (uint32_t)__popcll(m);
  p += c;
  rb = (rb + 2 * c) & (RB - 1);
  // the ring offset stays a scalar of its own: the compiler would rebuild it
  // from p with one more vector add per sub-step
  rb = __builtin_amdgcn_readfirstlane(rb);
  return e;
}

// 16 bytes of section words into the ring at pos and, for the first 128
// bytes, into the mirror (the other lanes store to pos twice: no branch)
__device__ __forceinline__ void ring_put(uint8_t *ring, uint32_t pos, uint4 v) {
  *(uint4 *)(ring + pos) = v;
  *(uint4 *)(ring + (pos < kRingMirror ? kRingBytes + pos : pos)) = v;
}

// Eight decoded elements of one lane from their table entries (symbols in
// the top bytes) and raw bytes: the inverse of the byte-plane split.
template <int DT>
__device__ inline void merge_entries(const uint32_t e[8], const uint32_t raw[6],
                                     uint32_t w[4 * (dt_bytes<DT>() / 2)]) {
  if constexpr (DT <= 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // [raw, sym, raw, sym] of elements 2j, 2j + 1, then rotate each half back
      const uint32_t t = __builtin_amdgcn_perm(e[2 * j], raw[j >> 1], (j & 1) ? 0x07030702u : 0x07010700u);
      w[j] = rotr16x2(__builtin_amdgcn_perm(e[2 * j + 1], t, 0x07020100u));
    }
  } else {
    uint32_t sym[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t lo = __builtin_amdgcn_perm(e[4 * h + 1], e[4 * h], 0x07070703u);
      const uint32_t hi = __builtin_amdgcn_perm(e[4 * h + 3], e[4 * h + 2], 0x07030303u);
      sym[h] = __builtin_amdgcn_perm(hi, lo, 0x07060100u);
    }
    merge_group<DT>(sym, raw, w);
  }
}


// Ring bookkeeping of one coded block (all members wave-uniform).
struct Ring {
  uint32_t written;  // section bytes [written - 4096, written) are in the ring
  uint32_t len;      // section length (a multiple of 16)
  uint4 pv;          // this lane's 16 bytes of the chunk at `written`, loaded a round ahead
};

// 16 bytes of this lane's part of the chunk at section offset o (clamped to
// the section: a chunk past the end is never decoded from)
__device__ __forceinline__ uint4 ring_fetch(const uint8_t *sec, uint32_t o, uint32_t len) {
  return *(const uint4 *)(sec + (o + 16 <= len ? o : len - 16));
}

// A stream header's eight words (loaded by the caller, ahead of their use).
struct Hdr {
  uint4 lo, hi;
};
__device__ inline Hdr load_hdr(const uint8_t *s) { return Hdr{((const uint4 *)s)[0], ((const uint4 *)s)[1]}; }

// Modes of a decoding wave's input block in the fused reduce.
enum : uint32_t { kBad = 0, kStored = 1, kCoded = 2 };

// Opens block b of one input stream s (in_bytes long) of the fused reduce:
// checks the header against the call (n elements, blocks of be) and the
// block's directory entries, and for a coded block builds the lookup table
// and fills the ring.  The loads come in two rounds: the header with the
// directory entries, then the start of the section -- states, presence
// bits, frequencies and the 4096 bytes from the end of the fixed part,
// which hold the first two ring chunks and the first pending one (the
// words begin at most 512 bytes in) -- instead of five dependent ones.
// Returns kBad, kStored or kCoded; sets sec, raw_plane, the states x, the
// word start wb, the words available and the ring.
template <int DT>
__device__ uint32_t open_input_block(const uint8_t *s, uint64_t in_bytes, uint64_t n, uint32_t be, uint32_t b,
                                     uint32_t n_b, uint32_t *lut, uint8_t *ring, const uint8_t *&sec,
                                     const uint8_t *&raw_plane, uint32_t &x, uint32_t &wb, uint32_t &w_avail,
                                     Ring &rg) {
  constexpr int E = (DT == 2) ? 4 : 2;
  const uint32_t lane = lane_id();
  const Geom g = make_geom(n, be, E);
  if (in_bytes < kHeaderBytes) return kBad;
  // round 1: header and directory entries (inside the stream's bytes)
  const Hdr h = load_hdr(s);
  const uint64_t de = kHeaderBytes + 4ull * (b + 1);
  const uint32_t d = de <= in_bytes ? ld32(s + de - 4) : 0u;
  const uint32_t dp = (b > 0 && de <= in_bytes) ? ld32(s + de - 8) : 0u;
  const uint64_t start = b ? 16ull * (dp & ~kStoredBit) : 0;
  const uint64_t end = 16ull * (d & ~kStoredBit);
  const bool stored = d >> 31;
  const uint32_t len = end >= start ? (uint32_t)(end - start) : 0u;
  // round 2: the section's start, read inside the stream's bytes (16-byte
  // loads of a section of 16-byte units are whole inside it or skipped)
  uint32_t pbyte = 0;
  uint2 pfa = make_uint2(0u, 0u);
  uint4 pre[4] = {make_uint4(0u, 0u, 0u, 0u), make_uint4(0u, 0u, 0u, 0u), make_uint4(0u, 0u, 0u, 0u),
                  make_uint4(0u, 0u, 0u, 0u)};
  const uint8_t *sc = s + g.coded_off + start;
  uint32_t xs = kStateLo;
  x = kStateLo;
  if (end >= start && g.coded_off + end <= in_bytes && !stored && len >= kSectionFixed) {
    xs = ((const uint32_t *)sc)[lane];
    pbyte = sc[256 + (lane >> 1)];
    if (kSectionFixed + 8 * lane + 8 <= len) pfa = *(const uint2 *)(sc + kSectionFixed + 8 * lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t o = kSectionFixed + 1024 * j + 16 * lane;
      if (o + 16 <= len) pre[j] = *(const uint4 *)(sc + o);
    }
  }
  const uint64_t total = (uint64_t)h.hi.z | (uint64_t)h.hi.w << 32;
  const bool ok = h.lo.x == kMagic && h.lo.y == (kVersion | ((uint32_t)DT << 8) | (kProbBits << 16)) &&
                  h.lo.z == be && h.lo.w == g.n_blocks && ((uint64_t)h.hi.x | (uint64_t)h.hi.y << 32) == n &&
                  total <= in_bytes && total >= g.coded_off && de <= in_bytes && end >= start &&
                  g.coded_off + end <= total;
  if (!ok) return kBad;
  sec = sc;
  raw_plane = s + g.raw_off;
  if (stored) return len >= n_b ? kStored : kBad;
  uint32_t k = 0;
  if (!build_lut_pre(pbyte, pfa, len, lut, (uint16_t *)ring, (uint16_t *)ring + 256, k)) return kBad;
  k = uniform(k);
  x = xs;
  wb = kSectionFixed + 2 * k;
  w_avail = (len - wb) / 2;
  rg.len = len;
  // section bytes [288, 288 + 4096) fill the ring (the table build's
  // scratch until now): it then holds the two chunks from the word start's
  // 16-byte unit on, and the third is the first pending one
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t o = kSectionFixed + 1024 * j + 16 * lane;
    ring_put(ring, o & (kRingBytes - 1), pre[j]);
  }
  wave_lds_fence();
  rg.written = (wb & ~15u) + 2 * kChunkBytes;
  rg.pv = *(const uint4 *)(ring + ((rg.written + 16 * lane) & (kRingBytes - 1)));
  return kCoded;
}

// Before a round: make sure the next 1 KB of words (from section offset cur)
// is in LDS, then load the following chunk for the next round.  Every round
// stores the loaded chunk at its ring position and loads the chunk at
// `written` again, also when neither has moved (a repeat store of the same
// bytes; a cache hit): every path through a round then issues the same
// memory operations, so no wait for them lands inside the decode chain.
// The store never overwrites unread words: written < cur + 2048 always.
__device__ __forceinline__ void ring_maintain(Ring &rg, uint8_t *ring, const uint8_t *sec, uint32_t cur) {
  const uint32_t lane = lane_id();
  ring_put(ring, (rg.written + 16 * lane) & (kRingBytes - 1), rg.pv);
  asm volatile("" ::: "memory");  // the ring stores stay before the round's ring reads
  rg.written += rg.written < cur + kChunkBytes ? kChunkBytes : 0;
  rg.pv = ring_fetch(sec, rg.written + 16 * lane, rg.len);
}

// decode_kernel's ring: 2 KB without a mirror (8 KB table + 2 KB ring =
// 10 KB of LDS per wave, 16 waves per CU), 512-byte chunks read with one
// 8-byte load per lane.  A half round (4 sub-steps) reads at most 512 bytes;
// each half round stores the chunk its slot fetched a round earlier and
// fetches the next chunk if it will fit when stored (front < cur + 1536),
// else re-fetches the newest chunk.  Two slots alternate by half round.  The
// stored frontier then stays at least 512 bytes ahead of the words a half
// round reads, and a store never overwrites unread words.
constexpr uint32_t kDecRingBytes = 2048;
constexpr uint32_t kDecChunk = 512;

struct RingD {
  uint32_t len;
  uint32_t front;
  uint32_t pos[2];
  uint2 pv[2];
};

template <int X>
__device__ __forceinline__ void ringd_half(RingD &rg, uint8_t *ring, const uint8_t *sec, uint32_t cur) {
  const uint32_t lane = lane_id();
  *(uint2 *)(ring + ((rg.pos[X] + 8 * lane) & (kDecRingBytes - 1))) = rg.pv[X];
  asm volatile("" ::: "memory");  // the ring stores stay before the half round's ring reads
  rg.front += rg.front < cur + 3 * kDecChunk ? kDecChunk : 0;
  rg.pos[X] = rg.front - kDecChunk;
  const uint32_t o = rg.pos[X] + 8 * lane;
  rg.pv[X] = *(const uint2 *)(sec + (o + 8 <= rg.len ? o : rg.len - 8));
}

template <int E>
__device__ inline void load_raw_full(const uint8_t *plane, uint64_t first, uint32_t raw[6]) {
  const uint2 *q = (const uint2 *)(plane + (uint64_t)(E - 1) * first);
  uint2 a = q[0];
  raw[0] = a.x;
  raw[1] = a.y;
  if (E == 4) {
    uint2 b = q[1], c = q[2];
    raw[2] = b.x;
    raw[3] = b.y;
    raw[4] = c.x;
    raw[5] = c.y;
  }
}

// The header of one stream checked (and, for a stream-wide table, its
// lookup table built): its place and geometry.
struct DecStream {
  const uint8_t *s;
  uint8_t *out;
  uint64_t n, total;
  uint32_t be, nb;
  Geom g;
};
// Checks stream c's header h (words: magic | version, dtype, probability
// bits, flags | block elements | blocks | elements (2) | total bytes (2))
// and sets up its geometry; builds the stream-wide lookup table.
template <int DT, bool SHARED>
__device__ bool open_stream(const DecodeArgs &a, uint64_t c, const Hdr &h, DecStream &st, uint32_t *lut,
                            uint16_t *cum_s, uint16_t *f_s) {
  constexpr int E = (DT == 2) ? 4 : 2;
  const bool chunked = a.bpc != 0;
  st.s = a.in + (chunked ? c * a.slot_bytes : 0);
  st.out = a.out + (chunked ? c * a.chunk_elems * E : 0);
  st.n = chunked ? ((a.n - c * a.chunk_elems) < a.chunk_elems ? a.n - c * a.chunk_elems : a.chunk_elems) : a.n;
  const uint64_t cap = chunked ? a.slot_bytes : a.in_bytes;
  const uint8_t *s = st.s;
  if (cap < kHeaderBytes) {
    st.nb = 0;
    return false;
  }
  const uint32_t be = h.lo.z;
  const uint32_t nb = h.lo.w;
  const uint64_t total = (uint64_t)h.hi.z | (uint64_t)h.hi.w << 32;
  // flags byte: the table mode (0: a table per block; 1: a stream-wide
  // table after the directory; 2: the caller's stream-wide table)
  const uint32_t mode = h.lo.y >> 24;
  bool ok = h.lo.x == kMagic && (h.lo.y & 0xFFu) == kVersion && ((h.lo.y >> 8) & 0xFFu) == DT &&
            ((h.lo.y >> 16) & 0xFFu) == kProbBits &&
            (SHARED ? ((mode == 1) || (mode == 2 && a.table != nullptr)) : mode == 0) &&
            ((uint64_t)h.hi.x | (uint64_t)h.hi.y << 32) == st.n && be > 0 && (be & (be - 1)) == 0 &&
            (uint64_t)be * E >= kMinBlockBytes &&
            (uint64_t)be * E <= kMaxBlockBytes && (uint64_t)nb == (st.n + be - 1) / be && total <= cap &&
            (!chunked || be == a.block_elems);
  Geom g = make_geom(st.n, ok ? be : 1, E);
  const uint64_t table_off = g.raw_off;
  if (SHARED && mode == 1 && nb > 0) {
    g.raw_off += kTableBytes;
    g.coded_off += kTableBytes;
  }
  ok = ok && total >= g.coded_off;
  if (SHARED && ok && nb > 0) {
    // one lookup table for every block of the stream
    ok = build_lut_shared(mode == 1 ? (const uint16_t *)(s + table_off) : a.table, lut, cum_s, f_s);
    __syncthreads();
  }
  st.be = be;
  st.nb = ok ? nb : 0;
  st.total = total;
  st.g = g;
  return ok;
}

// the stream's sections end where its header says it ends
__device__ inline bool stream_end_ok(const DecStream &st) {
  const uint64_t endall = st.nb ? 16ull * (ld32(st.s + kHeaderBytes + 4 * (st.nb - 1)) & ~kStoredBit) : 0;
  return st.g.coded_off + endall == st.total;
}

template <int DT, bool SHARED = false>
__global__ void __launch_bounds__(64) decode_kernel(DecodeArgs a) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  __shared__ uint32_t lut[kM];
  __shared__ __align__(16) uint8_t ring[kDecRingBytes];
  // the table-build scratch (cum, f) lives in the ring before the ring fills
  uint16_t *cum_s = (uint16_t *)ring, *f_s = (uint16_t *)ring + 256;
  const uint32_t lane = lane_id();
  DecStream st;
  uint64_t cur = 0, n_work = 0;
  bool ok = true;
  if (a.bpc == 0) {
    // one stream
    Hdr h = {};
    if (a.in_bytes >= kHeaderBytes) h = load_hdr(a.in);
    ok = open_stream<DT, SHARED>(a, 0, h, st, lut, cum_s, f_s);
    if (!ok) {
      if (blockIdx.x == 0 && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
      return;
    }
    if (blockIdx.x == 0 && lane == 0 && !stream_end_ok(st)) report(a.dstatus, UZIP_ECORRUPT);
    n_work = st.nb;
  } else {
    // chunk streams: a header is opened when the walk reaches its chunk
    cur = ~0ull;
    n_work = a.n_chunks * a.bpc;
  }

  // The next block's directory entries, and over chunk streams its chunk's
  // header, are loaded a block ahead: a block then starts from its section
  // instead of a chain of dependent loads.  Directory words are only read
  // inside the stream's bytes (a valid header puts the directory there).
  struct Ahead {
    Hdr h;
    uint32_t d, dp;
  };
  auto fetch = [&](uint64_t g2, Ahead &nx) {
    const uint8_t *s2 = a.in;
    uint64_t cap = a.in_bytes;
    uint32_t b2 = (uint32_t)g2;
    if (a.bpc != 0) {
      const uint64_t q = g2 / a.bpc;
      b2 = (uint32_t)(g2 - q * a.bpc);
      s2 = a.in + (a.first_chunk + q) * a.slot_bytes;
      cap = a.slot_bytes;
      nx.h = load_hdr(s2);
    }
    const uint64_t de = kHeaderBytes + 4ull * (b2 + 1);
    nx.d = de <= cap ? ld32(s2 + de - 4) : 0u;
    nx.dp = (b2 > 0 && de <= cap) ? ld32(s2 + de - 8) : 0u;
  };

  // blocks are independent: a grid-stride walk, no ticket (one counter for
  // every wave costs more in queueing than it recovers in balance)
  Ahead nx = {};
  if (blockIdx.x < n_work) fetch(blockIdx.x, nx);
  for (uint64_t gb = blockIdx.x; gb < n_work; gb += gridDim.x) {
    const Ahead here = nx;
    if (gb + gridDim.x < n_work) fetch(gb + gridDim.x, nx);
    uint32_t b = (uint32_t)gb;
    if (a.bpc != 0) {
      const uint64_t q = gb / a.bpc;
      const uint64_t c = a.first_chunk + q;
      b = (uint32_t)(gb - q * a.bpc);
      if (c != cur) {
        cur = c;
        ok = open_stream<DT, SHARED>(a, c, here.h, st, lut, cum_s, f_s);
      }
      if (!ok) {
        if (b == 0 && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
        continue;
      }
      if (b >= st.nb) continue;  // the tensor's last chunk has fewer blocks
      if (b == 0 && lane == 0 && !stream_end_ok(st)) report(a.dstatus, UZIP_ECORRUPT);
    }
    const uint8_t *s = st.s;
    const Geom &g = st.g;
    const uint32_t be = st.be;
    const uint64_t total = st.total;
    const uint8_t *raw_plane = s + g.raw_off;
    const uint32_t d = here.d;
    const uint64_t start = b ? 16ull * (here.dp & ~kStoredBit) : 0;
    const uint64_t end = 16ull * (d & ~kStoredBit);
    const uint64_t blk0 = (uint64_t)b * be;
    const uint32_t n_b = (uint32_t)((st.n - blk0) < be ? (st.n - blk0) : be);
    const uint32_t rounds = (n_b + kRound - 1) / kRound;
    bool bad = !(end >= start && g.coded_off + end <= total);
    const uint8_t *sec = s + g.coded_off + start;
    const uint32_t len = bad ? 0 : (uint32_t)(end - start);
    const bool stored = d >> 31;
    if (!bad && stored && len < n_b) bad = true;
    // The start of a coded section in one round of loads: the states, the
    // presence bits and frequencies, and the 2048 bytes that follow the
    // fixed part (the first three ring chunks start within its first 512:
    // the words begin at most 2 x 256 bytes of frequencies in).  Sections
    // are 16-byte units, so a 16-byte load is either whole inside it or
    // skipped.
    constexpr uint32_t P0 = SHARED ? kSharedSectionFixed : kSectionFixed;
    uint32_t x = 0, pbyte = 0;
    uint2 pfa = make_uint2(0u, 0u);
    uint4 pre0 = make_uint4(0u, 0u, 0u, 0u), pre1 = pre0;
    if (!bad && !stored && len >= P0) {
      x = ((const uint32_t *)sec)[lane];
      if constexpr (!SHARED) {
        pbyte = sec[256 + (lane >> 1)];
        if (kSectionFixed + 8 * lane + 8 <= len) pfa = *(const uint2 *)(sec + kSectionFixed + 8 * lane);
      }
      const uint32_t o0 = P0 + 32 * lane;
      if (o0 + 16 <= len) pre0 = *(const uint4 *)(sec + o0);
      if (o0 + 32 <= len) pre1 = *(const uint4 *)(sec + o0 + 16);
    }
    if (bad) {
      if (lane == 0) report(a.dstatus, UZIP_ECORRUPT);
      continue;
    }
    if (stored) {
      for (uint32_t r = 0; r < rounds; ++r) {
        uint32_t i0 = r * kRound + kPerLane * lane;
        uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
        if (valid == 0) continue;
        uint32_t sym[2] = {0, 0};
        if (valid == 8) {
          uint2 v = *(const uint2 *)(sec + i0);
          sym[0] = v.x;
          sym[1] = v.y;
        } else {
#pragma unroll
          for (uint32_t q = 0; q < 8; ++q)
            if (q < valid) sym[q >> 2] |= (uint32_t)sec[i0 + q] << (8 * (q & 3));
        }
        uint32_t raw[6];
        load_raw<E>(raw_plane, blk0 + i0, valid, raw);
        uint32_t w[NW];
        merge_group<DT>(sym, raw, w);
        store_words<E>(st.out, blk0 + i0, valid, w);
      }
      continue;
    }
    uint32_t k = 0;
    if constexpr (SHARED) {
      if (len < kSharedSectionFixed) {
        if (lane == 0) report(a.dstatus, UZIP_ECORRUPT);
        continue;
      }
    } else {
      if (!build_lut_pre(pbyte, pfa, len, lut, cum_s, f_s, k)) {
        if (lane == 0) report(a.dstatus, UZIP_ECORRUPT);
        continue;
      }
      k = uniform(k);
    }
    const uint32_t x0 = x;  // checked at the end of the block: no wait for it here
    const uint32_t wb = SHARED ? kSharedSectionFixed : kSectionFixed + 2 * k;  // section offset of word 0
    const uint32_t w_avail = (len - wb) / 2;
    RingD rg;
    rg.len = len;
    {
      // section bytes [P0, P0 + 2048) fill the ring (which held the table
      // build's scratch until now), so it holds the three chunks from the
      // word start's 16-byte unit on; the third chunk is also the first
      // pending refill
      const uint32_t base = wb & ~15u;
      const uint32_t o0 = P0 + 32 * lane;
      *(uint4 *)(ring + (o0 & (kDecRingBytes - 1))) = pre0;
      *(uint4 *)(ring + ((o0 + 16) & (kDecRingBytes - 1))) = pre1;
      wave_lds_fence();
      rg.front = base + 3 * kDecChunk;
      rg.pos[0] = rg.pos[1] = base + 2 * kDecChunk;
      rg.pv[0] = rg.pv[1] = *(const uint2 *)(ring + ((base + 2 * kDecChunk + 8 * lane) & (kDecRingBytes - 1)));
    }
    __syncthreads();
    uint32_t p = 0, rb = wb & (kDecRingBytes - 1);
    const uint32_t full = n_b / kRound;
    uint8_t *outp = st.out + blk0 * E;
    const uint8_t *rawp = raw_plane + blk0 * (E - 1);
    uint32_t rawA[6] = {0, 0, 0, 0, 0, 0}, rawB[6] = {0, 0, 0, 0, 0, 0};
    // round 0's raw bytes; with no full round a dummy load of the stream
    // header, so that the loop below is always entered with the same loads
    // in flight and waits only for what it uses
    load_raw_full<E>(full > 0 ? rawp : s, full > 0 ? kPerLane * lane : 0, rawA);
    // round 1's (clamped to a full round) likewise
    load_raw_full<E>(full > 0 ? rawp : s, full > 1 ? (kRound + kPerLane * lane) : (full > 0 ? kPerLane * lane : 0),
                     rawB);
    // one more memory operation in flight, standing in for the store that
    // ends every round, so that both ways into the loops match
    const uint32_t pad_load = *(const uint32_t *)(s + 4 * lane);
    uint32_t r = 0;
    // full rounds, four per iteration with four raw buffers: each round's
    // raw bytes are loaded two rounds before their use
    uint32_t rawC[6] = {0, 0, 0, 0, 0, 0}, rawD[6] = {0, 0, 0, 0, 0, 0};
    auto clampr = [&](uint32_t q) { return q < full ? q : full - 1; };
    for (; r + 4 <= full; r += 4) {
      if ((r & 15u) == 0) {
        // a wave's priority steps down with every 16 rounds of a block it
        // decodes and wraps after four steps: a SIMD issues for its oldest
        // wave first, and with equal shares the waves that arrived last on a
        // SIMD would finish last (the fourth ~10% after the first); a wave
        // that lags gets the issue slots until it has caught up (1 GiB
        // buffer 0.413 -> 0.407 ms, its chunk streams 0.425 -> 0.421 ms,
        // interleaved A/B)
        switch ((r >> 4) & 3u) {
          case 0: __builtin_amdgcn_s_setprio(3); break;
          case 1: __builtin_amdgcn_s_setprio(2); break;
          case 2: __builtin_amdgcn_s_setprio(1); break;
          default: __builtin_amdgcn_s_setprio(0); break;
        }
      }
      uint32_t e[kPerLane], w[NW];
#define UZIP_DEC_ROUND(RAWUSE, RAWLOAD, DR, AHEAD)                                              \
  ringd_half<0>(rg, ring, sec, wb + 2 * p);                                                     \
  load_raw_full<E>(rawp, clampr(r + (AHEAD)) * kRound + kPerLane * lane, RAWLOAD);              \
  _Pragma("unroll") for (uint32_t t = 0; t < kPerLane; ++t) {                                   \
    if (t == kPerLane / 2) ringd_half<1>(rg, ring, sec, wb + 2 * p);                            \
    e[t] = decode_step_ring<true, kDecRingBytes, false>(x, true, lut, ring, rb, p);             \
  }                                                                                             \
  merge_entries<DT>(e, RAWUSE, w);                                                              \
  store_words<E, true>(outp, (r + (DR)) * kRound + kPerLane * lane, 8, w);
      UZIP_DEC_ROUND(rawA, rawC, 0, 2)
      UZIP_DEC_ROUND(rawB, rawD, 1, 3)
      UZIP_DEC_ROUND(rawC, rawA, 2, 4)
      UZIP_DEC_ROUND(rawD, rawB, 3, 5)
#undef UZIP_DEC_ROUND
    }
    // full rounds, two per iteration with ping-pong raw registers: every
    // load is issued a round before its use and no register is copied
    // the rest in twos (rawA, rawB hold rounds r, r + 1 here)
    for (; r + 2 <= full; r += 2) {
      ringd_half<0>(rg, ring, sec, wb + 2 * p);
      load_raw_full<E>(rawp, (r + 1) * kRound + kPerLane * lane, rawB);
      uint32_t e[kPerLane];
#pragma unroll
      for (uint32_t t = 0; t < kPerLane; ++t) {
        if (t == kPerLane / 2) ringd_half<1>(rg, ring, sec, wb + 2 * p);
        e[t] = decode_step_ring<true, kDecRingBytes, false>(x, true, lut, ring, rb, p);
      }
      uint32_t w[NW];
      merge_entries<DT>(e, rawA, w);
      store_words<E, true>(outp, r * kRound + kPerLane * lane, 8, w);

      ringd_half<0>(rg, ring, sec, wb + 2 * p);
      const uint32_t rn = (r + 2 < full) ? r + 2 : r + 1;  // always a full round: no branch around the load
      load_raw_full<E>(rawp, rn * kRound + kPerLane * lane, rawA);
#pragma unroll
      for (uint32_t t = 0; t < kPerLane; ++t) {
        if (t == kPerLane / 2) ringd_half<1>(rg, ring, sec, wb + 2 * p);
        e[t] = decode_step_ring<true, kDecRingBytes, false>(x, true, lut, ring, rb, p);
      }
      merge_entries<DT>(e, rawB, w);
      store_words<E, true>(outp, (r + 1) * kRound + kPerLane * lane, 8, w);
    }
    if (r < full) {  // odd number of full rounds: rawA holds round r
      ringd_half<0>(rg, ring, sec, wb + 2 * p);
      uint32_t e[kPerLane];
#pragma unroll
      for (uint32_t t = 0; t < kPerLane; ++t) {
        if (t == kPerLane / 2) ringd_half<1>(rg, ring, sec, wb + 2 * p);
        e[t] = decode_step_ring<true, kDecRingBytes, false>(x, true, lut, ring, rb, p);
      }
      uint32_t w[NW];
      merge_entries<DT>(e, rawA, w);
      store_words<E, true>(outp, r * kRound + kPerLane * lane, 8, w);
      ++r;
    }
    if (r < rounds) {  // partial last round
      ringd_half<0>(rg, ring, sec, wb + 2 * p);
      const uint32_t i0 = r * kRound + kPerLane * lane;
      const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
      uint32_t e[kPerLane];
#pragma unroll
      for (uint32_t t = 0; t < kPerLane; ++t) {
        if (t == kPerLane / 2) ringd_half<1>(rg, ring, sec, wb + 2 * p);
        e[t] = decode_step_ring<false, kDecRingBytes, false>(x, t < valid, lut, ring, rb, p);
      }
      if (valid > 0) {
        uint32_t raw[6];
        load_raw<E>(raw_plane, blk0 + i0, valid, raw);
        uint32_t w[NW];
        merge_entries<DT>(e, raw, w);
        store_words<E>(st.out, blk0 + i0, valid, w);
      }
    }
    asm volatile("" ::"v"(pad_load));
    if (x != kStateLo || p > w_avail || x0 < kStateLo || x0 >= 0x80000000u) bad = true;
    if (__any(bad) && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// reduce_decode_kernel: the decode and reduce half of the fused reduce
// (section 3.4).  One workgroup per output block, one wave per input of a
// group of up to 8 inputs plus one reducing wave.  Input wave i decodes block
// b of its stream round by round into an LDS slab (its own lookup table and
// word ring, as in decode_kernel); after every round the reducing wave adds
// the slabs in input order in fp32, continuing the partial sums of earlier
// groups.  The group that finishes the sum adds the local contribution,
// rounds to the element type and writes the reduced tensor, the raw plane
// of the output stream and the block's symbol histogram; encode_kernel then
// codes the reduced tensor from there.  Slabs are double-buffered, so one
// barrier per round suffices.
// ---------------------------------------------------------------------------
constexpr int kReduceGroup = 8;
constexpr uint32_t kDecLds = kLutBytes + kRingBytes + kRingMirror;  // per decoding wave

struct ReduceArgs {
  const uint8_t *ins[kReduceGroup];
  uint64_t in_bytes[kReduceGroup];
  int n_in;              // inputs of this group
  int first;             // this group starts the sums
  int last;              // this group ends them
  const float *acc_in;   // partial sums of the groups before (first == 0)
  float *acc_out;        // partial sums for the next group (last == 0)
  const uint8_t *local_raw;
  uint64_t n;
  uint32_t block_elems;
  uint8_t *out_raw_plane;  // raw plane of the output stream
  uint8_t *ybuf;           // reduced tensor, read again by the coding pass
  uint8_t *yout;           // caller's copy of it (may be null or ybuf)
  uint32_t *hist_out;      // [n_blocks][256]
  uint32_t *dstatus;
  // reduce_fused_kernel: byte offsets of its LDS regions (the decoders'
  // tables and rings, later the coding pass's staging area, start at 0)
  uint32_t lds_slabs, lds_hist, lds_syms, lds_enc, lds_trash;
};

uint32_t reduce_lds(int n_in, uint32_t E) { return n_in * (kDecLds + 2 * kRound * E) + kHistBytes; }

template <int DT>
__global__ void __launch_bounds__(64 * (kReduceGroup + 1)) reduce_decode_kernel(ReduceArgs a) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  extern __shared__ __align__(16) uint8_t smem_base[];
  const uint32_t wave = threadIdx.x >> 6;
  const uint32_t lane = lane_id();
  const int n_in = a.n_in;
  const bool decoder = (int)wave < n_in;
  uint8_t *slabs = smem_base + n_in * kDecLds;  // [2][n_in][512 elements]
  constexpr uint32_t kSlab = kRound * E;
  uint32_t *hist = (uint32_t *)(slabs + 2 * n_in * kSlab);
  const uint32_t be = a.block_elems;
  const uint32_t b = blockIdx.x;
  const uint64_t blk0 = (uint64_t)b * be;
  const uint32_t n_b = (uint32_t)((a.n - blk0) < be ? (a.n - blk0) : be);
  const uint32_t rounds = (n_b + kRound - 1) / kRound;
  const uint32_t full = n_b / kRound;

  // ---- decoding waves: block b of input `wave` ----
  uint32_t *lut = (uint32_t *)(smem_base + wave * kDecLds);
  uint8_t *ring = smem_base + wave * kDecLds + kLutBytes;
  uint32_t mode = kBad;
  const uint8_t *sec = nullptr, *raw_plane = nullptr;
  uint32_t x = kStateLo, x0 = kStateLo, p = 0, rb = 0, wb = 0, w_avail = 0;
  Ring rg;
  rg.written = 0;
  rg.len = 16;
  rg.pv = make_uint4(0, 0, 0, 0);
  if (decoder) {
    mode = open_input_block<DT>(a.ins[wave], a.in_bytes[wave], a.n, be, b, n_b, lut, ring, sec, raw_plane, x, wb,
                                w_avail, rg);
    x0 = x;
    rb = wb & (kRingBytes - 1);
    if (mode == kBad && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
  } else {
    for (uint32_t i = lane; i < kHistReplicas * kHistStride; i += 64) hist[i] = 0;
  }
  uint32_t *h = hist + (lane & (kHistReplicas - 1)) * kHistStride;
  __syncthreads();

  for (uint32_t r = 0; r < rounds; ++r) {
    uint8_t *slab = slabs + (r & 1) * n_in * kSlab;
    const uint32_t i0 = r * kRound + kPerLane * lane;
    const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
    if (decoder) {
      uint32_t w[NW];
#pragma unroll
      for (int q = 0; q < NW; ++q) w[q] = 0;
      if (mode == kCoded) {
        ring_maintain(rg, ring, sec, wb + 2 * p);
        uint32_t e[kPerLane];
        if (r < full) {
#pragma unroll
          for (uint32_t t = 0; t < kPerLane; ++t) e[t] = decode_step_ring<true>(x, true, lut, ring, rb, p);
        } else {
#pragma unroll
          for (uint32_t t = 0; t < kPerLane; ++t) e[t] = decode_step_ring<false>(x, t < valid, lut, ring, rb, p);
        }
        uint32_t raw[6] = {0, 0, 0, 0, 0, 0};
        load_raw<E>(raw_plane, blk0 + i0, valid, raw);
        merge_entries<DT>(e, raw, w);
      } else if (mode == kStored && valid > 0) {
        uint32_t sym[2] = {0, 0};
#pragma unroll
        for (uint32_t q = 0; q < 8; ++q)
          if (q < valid) sym[q >> 2] |= (uint32_t)sec[i0 + q] << (8 * (q & 3));
        uint32_t raw[6] = {0, 0, 0, 0, 0, 0};
        load_raw<E>(raw_plane, blk0 + i0, valid, raw);
        merge_group<DT>(sym, raw, w);
      }
      uint4 *dst = (uint4 *)(slab + wave * kSlab + kPerLane * E * lane);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      if (E == 4) dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
    __syncthreads();
    if (!decoder && valid > 0) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (!a.first) {
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] = (uint32_t)q < valid ? a.acc_in[blk0 + i0 + q] : 0.f;
      }
      for (int i = 0; i < n_in; ++i) {
        const uint4 *src = (const uint4 *)(slabs + (r & 1) * n_in * kSlab + i * kSlab + kPerLane * E * lane);
        uint32_t w[NW];
        const uint4 v0 = src[0];
        w[0] = v0.x, w[1] = v0.y, w[2] = v0.z, w[3] = v0.w;
        if (E == 4) {
          const uint4 v1 = src[1];
          w[4] = v1.x, w[5] = v1.y, w[6] = v1.z, w[7] = v1.w;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint32_t wq = (E == 2) ? ((w[q >> 1] >> (16 * (q & 1))) & 0xFFFFu) : w[q];
          const float v = to_f32<DT>(wq);
          acc[q] = (a.first && i == 0) ? v : acc[q] + v;
        }
      }
      if (a.last) {
        if (a.local_raw != nullptr) {
          uint32_t w[NW];
          load_words<E>(a.local_raw, blk0 + i0, valid, w);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const uint32_t wq = (E == 2) ? ((w[q >> 1] >> (16 * (q & 1))) & 0xFFFFu) : w[q];
            acc[q] = acc[q] + to_f32<DT>(wq);
          }
        }
        uint32_t w[NW];
#pragma unroll
        for (int q = 0; q < NW; ++q) w[q] = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint32_t y = from_f32<DT>(acc[q]);
          if (E == 2)
            w[q >> 1] |= y << (16 * (q & 1));
          else
            w[q] = y;
        }
        store_words<E>(a.ybuf, blk0 + i0, valid, w);
        if (a.yout != nullptr && a.yout != a.ybuf) store_words<E>(a.yout, blk0 + i0, valid, w);
        Group gr;
        split_group<DT>(w, gr);
        store_raw<E>(a.out_raw_plane, blk0 + i0, valid, gr);
        hist_add8(h, gr, valid);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if ((uint32_t)q < valid) a.acc_out[blk0 + i0 + q] = acc[q];
      }
    }
  }
  __syncthreads();
  if (decoder && mode == kCoded) {
    const bool bad = x != kStateLo || p > w_avail || x0 < kStateLo || x0 >= 0x80000000u;
    if (__any(bad) && lane == 0) report(a.dstatus, UZIP_ECORRUPT);
  }
  if (!decoder && a.last) {
    for (uint32_t sy = lane; sy < 256; sy += 64) {
      uint32_t c = 0;
#pragma unroll
      for (uint32_t rep = 0; rep < kHistReplicas; ++rep) c += hist[rep * kHistStride + sy];
      a.hist_out[(uint64_t)b * 256 + sy] = c;
    }
  }
}

// ---------------------------------------------------------------------------
// reduce_fused_kernel: the whole fused reduce of one output block per
// workgroup (section 3.4's receive-reduce-send step with the codec fused
// in), for the last (or only) group of up to eight inputs.  Workgroups take
// output blocks by ticket.  Waves 0 .. n_in-1 decode block b of their input
// round by round into double-buffered LDS slabs (lookup table and word ring
// as in reduce_decode_kernel, raw bytes loaded a round ahead); wave n_in adds
// the slabs in input order in binary32 (after the partial sums of earlier
// input groups), adds the local share, rounds to the element type, writes
// the output stream's raw plane (and the caller's copy of the reduced
// tensor), and keeps the block's symbols and histogram in LDS.  After the
// last round the decoding waves end and the reducing wave codes the block
// from LDS -- table, the 64 rANS states backwards, words staged where the
// lookup tables were -- and places its section with the single-pass scan.
// The reduced tensor does not go through HBM.
// ---------------------------------------------------------------------------
template <int DT>
__global__ void __launch_bounds__(64 * (kReduceGroup + 1)) reduce_fused_kernel(ReduceArgs r, EncodeArgs a) {
  constexpr int E = (DT == 2) ? 4 : 2;
  constexpr int NW = 4 * (E / 2);
  constexpr uint32_t kSlab = kRound * E;
  extern __shared__ __align__(16) uint8_t smem_base[];
  __shared__ uint32_t s_block;
  typedef __attribute__((address_space(3))) uint16_t lds16_t;
  const uint32_t wave = threadIdx.x >> 6;
  const uint32_t lane = lane_id();
  const int n_in = r.n_in;
  const bool decoder = (int)wave < n_in;
  uint8_t *slabs = smem_base + r.lds_slabs;  // [2][n_in][512 elements]
  uint32_t *hist = (uint32_t *)(smem_base + r.lds_hist);
  uint8_t *syms = smem_base + r.lds_syms;    // the block's symbols, 512 per round
  const uint32_t be = r.block_elems;

  // the output block: taken in ticket order, so a workgroup only ever waits
  // in the scan for blocks of workgroups that started before it
  if (!decoder) {
    if (lane == 0) s_block = __hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (uint32_t i = lane; i < kHistReplicas * kHistStride; i += 64) hist[i] = 0;
  }
  __syncthreads();
  const uint32_t b = uniform(s_block);
  if (b >= a.n_blocks) return;  // (the grid has exactly one workgroup per block)
  const uint64_t blk0 = (uint64_t)b * be;
  const uint32_t n_b = (uint32_t)((r.n - blk0) < be ? (r.n - blk0) : be);
  const uint32_t rounds = (n_b + kRound - 1) / kRound;
  const uint32_t full = n_b / kRound;
  const Geom g = make_geom(r.n, be, E);

  // ---- decoding waves: block b of input `wave` ----
  uint32_t *lut = (uint32_t *)(smem_base + wave * kDecLds);
  uint8_t *ring = smem_base + wave * kDecLds + kLutBytes;
  uint32_t mode = kBad;
  const uint8_t *sec = nullptr, *raw_plane = nullptr;
  uint32_t x = kStateLo, x0 = kStateLo, p = 0, rb = 0, wb = 0, w_avail = 0;
  Ring rg;
  rg.written = 0;
  rg.len = 16;
  rg.pv = make_uint4(0, 0, 0, 0);
  if (decoder) {
    mode = open_input_block<DT>(r.ins[wave], r.in_bytes[wave], r.n, be, b, n_b, lut, ring, sec, raw_plane, x, wb,
                                w_avail, rg);
    x0 = x;
    rb = wb & (kRingBytes - 1);
    if (mode == kBad && lane == 0) report(r.dstatus, UZIP_ECORRUPT);
  }
  uint32_t *h = hist + (lane & (kHistReplicas - 1)) * kHistStride;
  // raw bytes of this lane's group of round q (the output's for a partial
  // round are masked by `valid`)
  auto load_raw_round = [&](uint32_t q, uint32_t raw[6]) {
    const uint32_t i0 = q * kRound + kPerLane * lane;
    const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
    if (q < full) load_raw_full<E>(raw_plane, blk0 + i0, raw);
    else load_raw<E>(raw_plane, blk0 + i0, valid, raw);
  };
  uint32_t rawA[6] = {0, 0, 0, 0, 0, 0}, rawB[6] = {0, 0, 0, 0, 0, 0};
  if (decoder && mode != kBad && rounds > 0) load_raw_round(0, rawA);
  __syncthreads();

  // one round: decoders fill slab (q & 1) (raw bytes of round q in `cur`,
  // round q + 1's loaded into `nxt`), one barrier, the reducing wave takes
  // the slab while the decoders go on with round q + 1
  auto round_body = [&](uint32_t q, uint32_t cur[6], uint32_t nxt[6]) {
    uint8_t *slab = slabs + (q & 1) * n_in * kSlab;
    const uint32_t i0 = q * kRound + kPerLane * lane;
    const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
    if (decoder) {
      uint32_t w[NW];
#pragma unroll
      for (int t = 0; t < NW; ++t) w[t] = 0;
      if (mode != kBad && q + 1 < rounds) load_raw_round(q + 1, nxt);
      if (mode == kCoded) {
        ring_maintain(rg, ring, sec, wb + 2 * p);
        uint32_t e[kPerLane];
        if (q < full) {
#pragma unroll
          for (uint32_t t = 0; t < kPerLane; ++t) e[t] = decode_step_ring<true>(x, true, lut, ring, rb, p);
        } else {
#pragma unroll
          for (uint32_t t = 0; t < kPerLane; ++t) e[t] = decode_step_ring<false>(x, t < valid, lut, ring, rb, p);
        }
        merge_entries<DT>(e, cur, w);
      } else if (mode == kStored && valid > 0) {
        uint32_t sy[2] = {0, 0};
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t)
          if (t < valid) sy[t >> 2] |= (uint32_t)sec[i0 + t] << (8 * (t & 3));
        merge_group<DT>(sy, cur, w);
      }
      uint4 *dst = (uint4 *)(slab + wave * kSlab + kPerLane * E * lane);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      if (E == 4) dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
    __syncthreads();
    if (!decoder && valid > 0) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (!r.first) {
#pragma unroll
        for (int t = 0; t < 8; ++t) acc[t] = (uint32_t)t < valid ? r.acc_in[blk0 + i0 + t] : 0.f;
      }
      for (int i = 0; i < n_in; ++i) {
        const uint4 *src = (const uint4 *)(slab + i * kSlab + kPerLane * E * lane);
        uint32_t w[NW];
        const uint4 v0 = src[0];
        w[0] = v0.x, w[1] = v0.y, w[2] = v0.z, w[3] = v0.w;
        if (E == 4) {
          const uint4 v1 = src[1];
          w[4] = v1.x, w[5] = v1.y, w[6] = v1.z, w[7] = v1.w;
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const uint32_t wt = (E == 2) ? ((w[t >> 1] >> (16 * (t & 1))) & 0xFFFFu) : w[t];
          const float v = to_f32<DT>(wt);
          acc[t] = (r.first && i == 0) ? v : acc[t] + v;
        }
      }
      if (r.local_raw != nullptr) {
        uint32_t w[NW];
        load_words<E>(r.local_raw, blk0 + i0, valid, w);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const uint32_t wt = (E == 2) ? ((w[t >> 1] >> (16 * (t & 1))) & 0xFFFFu) : w[t];
          acc[t] = acc[t] + to_f32<DT>(wt);
        }
      }
      uint32_t w[NW];
#pragma unroll
      for (int t = 0; t < NW; ++t) w[t] = 0;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t y = (uint32_t)t < valid ? from_f32<DT>(acc[t]) : 0u;
        if (E == 2)
          w[t >> 1] |= y << (16 * (t & 1));
        else
          w[t] = y;
      }
      if (r.yout != nullptr) store_words<E>(r.yout, blk0 + i0, valid, w);
      Group gr;
      split_group<DT>(w, gr);
      store_raw<E>(r.out_raw_plane, blk0 + i0, valid, gr);
      hist_add8(h, gr, valid);
      *(uint2 *)(syms + q * kRound + kPerLane * lane) = make_uint2(gr.sym[0], gr.sym[1]);
    }
  };
  uint32_t q = 0;
  for (; q + 2 <= rounds; q += 2) {
    round_body(q, rawA, rawB);
    round_body(q + 1, rawB, rawA);
  }
  if (q < rounds) round_body(q, rawA, rawB);
  __syncthreads();
  if (decoder) {
    if (mode == kCoded) {
      const bool bad = x != kStateLo || p > w_avail || x0 < kStateLo || x0 >= 0x80000000u;
      if (__any(bad) && lane == 0) report(r.dstatus, UZIP_ECORRUPT);
    }
    return;
  }

  // ---- the reducing wave codes the block (the decoding waves have ended) ----
  uint4 *enc = (uint4 *)(smem_base + r.lds_enc);
  lds16_t *trash = (lds16_t *)(smem_base + r.lds_trash) + lane;
  uint8_t *stage = smem_base;  // where the lookup tables and rings were
  uint16_t *stage16 = (uint16_t *)(stage + kStageHead);
  if (b + 1 == a.n_blocks && lane < 16) {
    // zero padding after the raw plane (pad16 of (E-1) n bytes)
    const uint64_t rbyte = g.raw_off + (uint64_t)(E - 1) * r.n + lane;
    if (rbyte < g.coded_off) a.out[rbyte] = 0;
  }
  wave_lds_fence();
  Table t;
  build_enc_table(hist, n_b, enc, t);
  t.k = uniform(t.k);
  wave_lds_fence();
  const uint32_t hdr = kSectionFixed + 2 * t.k;
  for (uint32_t i = lane; i < kStageTail / 4; i += 64) ((uint32_t *)(stage16 + a.wcap))[i] = 0;
  const uint32_t limit_words = (n_b > hdr) ? (n_b - hdr + 1) / 2 : 0;
  uint32_t pos = a.wcap;  // staging indices [pos, wcap) hold the words so far; the block's words all fit
  lds16_t *lds_rel = (lds16_t *)stage16;
  uint32_t xs = kStateLo;
  bool stored = (limit_words == 0);
  if (full < rounds && !stored) {  // the partial last round comes first
    const uint32_t i0 = full * kRound + kPerLane * lane;
    const uint32_t valid = i0 < n_b ? (n_b - i0 < 8 ? n_b - i0 : 8) : 0;
    const uint2 sv = *(const uint2 *)(syms + full * kRound + kPerLane * lane);
    const uint32_t sy[2] = {sv.x, sv.y};
    uint4 e[8];
    enc_lookup8(enc, sy[0], sy[1], e);
    enc_round<false>(xs, e, valid, pos, lds_rel, trash);
    if (a.wcap - pos >= limit_words) stored = true;
  }
  for (int q2 = (int)full - 1; q2 >= 0 && !stored; --q2) {
    const uint2 sv = *(const uint2 *)(syms + (uint32_t)q2 * kRound + kPerLane * lane);
    uint4 e[8];
    enc_lookup8(enc, sv.x, sv.y, e);
    enc_round<true>(xs, e, 8, pos, lds_rel, trash);
    if (a.wcap - pos >= limit_words) stored = true;
  }
  pos = uniform(pos);
  const uint32_t n_words = a.wcap - pos;
  const uint64_t img = hdr + 2ull * n_words;
  const uint64_t sec_len = stored ? pad16(n_b) : pad16(img);
  Fin f;
  f.sout = a.out;
  f.src = nullptr;
  f.coded_off = g.coded_off;
  f.dir_end = g.raw_off;
  f.chunk_n = r.n;
  f.blk0 = blk0;
  f.sec_len = sec_len;
  f.img = (uint32_t)img;
  f.b = b;
  f.chunk = 0;
  f.lb = b;
  f.first_block = 0;
  f.n_blocks = g.n_blocks;
  f.n_b = n_b;
  f.rounds = rounds;
  f.A = kStageHead + 2 * pos - hdr;
  f.lds_bytes = (uint32_t)img;
  f.slot_delta = 0;
  f.sym_lds = syms;
  f.stored = stored;
  f.spilled = false;
  f.last = b + 1 == a.n_blocks;
  if (!stored) write_section_head<false>(stage, f.A, xs, t);
  wave_lds_fence();
  publish_aggregate(a.status, b, 0, sec_len / 16, a.ticket[kWsHold]);
  finish_block<DT, false>(a, f, stage, nullptr);
  finish_launch<false, true>(a);
}

// zero the ticket, the look-back status words and the chunk counters
__global__ void clear_kernel(uint32_t *p, uint64_t words, uint32_t spin, uint32_t hold, uint64_t status_ptr) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = i == kWsSpin                ? spin
           : i == kWsHold              ? hold
           : i == kWsStatusPtr         ? (uint32_t)status_ptr
           : i == kWsStatusPtr + 1     ? (uint32_t)(status_ptr >> 32)
                                       : 0u;
}

// n == 0: the stream is the 32-byte header alone
__global__ void empty_stream_kernel(uint8_t *out, uint32_t dt, uint32_t block_elems, uint64_t *size_out,
                                    uint32_t mode = 0) {
  if (threadIdx.x == 0) {
    uint4 *hp = (uint4 *)out;
    hp[0] = make_uint4(kMagic, kVersion | (dt << 8) | (kProbBits << 16) | (mode << 24), block_elems, 0);
    hp[1] = make_uint4(0, 0, kHeaderBytes, 0);
    if (size_out != nullptr) *size_out = kHeaderBytes;
  }
}

// The stream-wide table from the counts c[4] of symbols 4 lane .. 4 lane + 3
// of an n_s-element sample (one wave): f[s] = 1 + floor(c[s](M - 256)/n_s),
// the remainder to the most frequent symbol (ties: the smallest); written to
// dst0 and, if given, dst1.
__device__ void write_table(const uint32_t c[4], uint32_t n_s, uint16_t *dst0, uint16_t *dst1) {
  const uint32_t lane = lane_id();
  uint32_t f[4], lt = 0, key = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    // c (M - 256) < 2^17 * 2^11: the quotient is exact in 32 bits
    f[q] = n_s ? 1u + (c[q] * (kM - 256u)) / n_s : kM / 256u;
    lt += f[q];
    const uint32_t kq = (c[q] << 8) | (255u - (4 * lane + q));
    key = kq > key ? kq : key;
  }
  const uint32_t d = kM - wave_sum(lt);
  const uint32_t best = 255u - (wave_max(key) & 0xFFu);
#pragma unroll
  for (uint32_t q = 0; q < 4; ++q)
    if (best == 4 * lane + q) f[q] += d;
  const uint2 v = make_uint2(f[0] | (f[1] << 16), f[2] | (f[3] << 16));
  *(uint2 *)(dst0 + 4 * lane) = v;
  if (dst1 != nullptr) *(uint2 *)(dst1 + 4 * lane) = v;
}

// ---------------------------------------------------------------------------
// table_kernel: the stream-wide table of a tensor (section 3.3.1's table from
// a sample of the range): histogram of the symbols of its first
// min(n, 256 KiB / E) elements, then f[s] = 1 + floor(c[s](M - 256)/n_s) for
// all 256 symbols, the remainder to the most frequent (ties: the smallest).
// One workgroup of 4 waves per stream (workgroup c: the stream of elements
// [c chunk_elems, ...)).  Every thread counts into a histogram of its own
// (16-bit counts packed as in the encoder, a thread sees at most 512
// symbols), so skewed exponents cost no atomic conflicts; the 256 private
// histograms are then summed bin by bin.  The table is written to
// dst0 + 256 c and, if `out` is given, to its place in stream c
// (out + c slot_bytes, after its directory).
// ---------------------------------------------------------------------------
constexpr uint32_t kTableThreads = 256;
constexpr uint32_t kLaneHist = 129;  // 128 packed words + 1: a bin of consecutive threads in distinct banks
constexpr uint32_t kTableLds = kTableThreads * kLaneHist * 4;
template <int DT>
__global__ void __launch_bounds__(kTableThreads) table_kernel(const uint8_t *in_all, uint64_t n_all,
                                                             uint64_t chunk_elems, uint32_t block_elems,
                                                             uint16_t *dst0_all, uint8_t *out, uint64_t slot_bytes) {
  constexpr int E = dt_bytes<DT>();
  constexpr int NW = 4 * (E / 2);
  extern __shared__ __align__(16) uint32_t hl[];  // [thread][kLaneHist]
  const uint64_t first = (uint64_t)blockIdx.x * chunk_elems;
  const uint8_t *in = in_all + first * E;
  const uint64_t n = n_all - first < chunk_elems ? n_all - first : chunk_elems;
  uint16_t *dst0 = dst0_all + 256ull * blockIdx.x;
  uint16_t *dst1 = out == nullptr ? nullptr
                                  : (uint16_t *)(out + blockIdx.x * slot_bytes + kHeaderBytes +
                                                 pad16(4 * ((n + block_elems - 1) / block_elems)));
  for (uint32_t i = threadIdx.x; i < kTableThreads * kLaneHist / 4; i += kTableThreads)
    ((uint4 *)hl)[i] = make_uint4(0, 0, 0, 0);
  __syncthreads();
  const uint64_t n_s = n < kSampleBytes / E ? n : kSampleBytes / E;
  uint32_t *mine = hl + threadIdx.x * kLaneHist;
  // the sample in batches of 16 groups of 8 elements per thread, every
  // load of a batch issued before its first use
  constexpr uint32_t kBatch = 16;
  constexpr uint32_t kBatches = kSampleBytes / E / (kPerLane * kTableThreads * kBatch);
  static_assert(kBatches * kBatch * kPerLane <= 65535, "private 16-bit counts");
  for (uint32_t bt = 0; bt < kBatches; ++bt) {
    uint32_t w[kBatch][NW];
    uint32_t valid[kBatch];
#pragma unroll
    for (uint32_t it = 0; it < kBatch; ++it) {
      const uint64_t i0 = (uint64_t)kPerLane * (threadIdx.x + (bt * kBatch + it) * kTableThreads);
      valid[it] = i0 < n_s ? (uint32_t)(n_s - i0 < kPerLane ? n_s - i0 : kPerLane) : 0u;
      load_words<E>(in, i0, valid[it], w[it]);
    }
#pragma unroll
    for (uint32_t it = 0; it < kBatch; ++it) {
      Group gr;
      split_group<DT>(w[it], gr);
      hist_add8_packed(mine, gr, valid[it]);
    }
  }
  __syncthreads();
  // thread t sums word t & 127 (symbols t & 127 and (t & 127) + 128) over
  // half of the private histograms, the two halves of each word apart
  const uint32_t wd = threadIdx.x & 127u, part = threadIdx.x >> 7;
  uint32_t lo = 0, hi = 0;
  for (uint32_t r = 0; r < kTableThreads / 2; ++r) {
    const uint32_t v = hl[(part * (kTableThreads / 2) + r) * kLaneHist + wd];
    lo += v & 0xFFFFu;
    hi += v >> 16;
  }
  __syncthreads();
  uint32_t *sums = hl;  // [2][256]: per half, the count of every symbol
  sums[256 * part + wd] = lo;
  sums[256 * part + wd + 128] = hi;
  __syncthreads();
  if (threadIdx.x >= 64) return;
  uint32_t c[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) c[q] = sums[4 * threadIdx.x + q] + sums[256 + 4 * threadIdx.x + q];
  write_table(c, (uint32_t)n_s, dst0, dst1);
}

// Each stream's sample split over kTableParts workgroups (one workgroup per
// stream would count a whole sample on one CU): workgroup kTableParts c + p
// counts elements [p S, (p + 1) S) of the sample of stream c (elements
// [c chunk_elems, ...) of the tensor), S = (256 KiB / E) / kTableParts, into
// 8 sub-histograms per wave and writes its 256 counts to
// part_out + 256 (kTableParts c + p); table_merge_kernel sums the parts.
constexpr uint32_t kTableParts = 16;
template <int DT>
__global__ void __launch_bounds__(kTableThreads) table_part_kernel(const uint8_t *in_all, uint64_t n_all,
                                                                  uint64_t chunk_elems, uint32_t *part_out) {
  constexpr int E = dt_bytes<DT>();
  constexpr int NW = 4 * (E / 2);
  constexpr uint32_t kReps = (kTableThreads / 64) * kHistReplicas;
  constexpr uint32_t kSlice = kSampleBytes / E / kTableParts;
  constexpr uint32_t kGroups = kSlice / (kPerLane * kTableThreads);
  static_assert(kGroups * kPerLane * kTableThreads == kSlice, "slice cover");
  __shared__ uint32_t h[kReps * kHistStride];
  for (uint32_t i = threadIdx.x; i < kReps * kHistStride; i += kTableThreads) h[i] = 0;
  __syncthreads();
  const uint32_t chunk = blockIdx.x / kTableParts, part = blockIdx.x % kTableParts;
  const uint64_t first = (uint64_t)chunk * chunk_elems;
  const uint8_t *in = in_all + first * E;
  const uint64_t n = n_all - first < chunk_elems ? n_all - first : chunk_elems;
  const uint64_t n_s = n < kSampleBytes / E ? n : kSampleBytes / E;
  uint32_t *hw = h + ((threadIdx.x / 64) * kHistReplicas + (threadIdx.x & (kHistReplicas - 1))) * kHistStride;
  uint32_t w[kGroups][NW], valid[kGroups];
#pragma unroll
  for (uint32_t it = 0; it < kGroups; ++it) {
    const uint64_t i0 = (uint64_t)part * kSlice + (uint64_t)kPerLane * (threadIdx.x + it * kTableThreads);
    valid[it] = i0 < n_s ? (uint32_t)(n_s - i0 < kPerLane ? n_s - i0 : kPerLane) : 0u;
    load_words<E>(in, i0, valid[it], w[it]);
  }
#pragma unroll
  for (uint32_t it = 0; it < kGroups; ++it) {
    Group gr;
    split_group<DT>(w[it], gr);
    hist_add8(hw, gr, valid[it]);
  }
  __syncthreads();
  for (uint32_t sy = threadIdx.x; sy < 256; sy += kTableThreads) {
    uint32_t acc = 0;
    for (uint32_t rp = 0; rp < kReps; ++rp) acc += h[rp * kHistStride + sy];
    part_out[256ull * blockIdx.x + sy] = acc;
  }
}

// One wave per stream c: its parts' counts summed, then the table, written
// to dst0 + 256 c and, if `out` is given, to its place in stream c (as
// table_kernel).
__global__ void __launch_bounds__(64) table_merge_kernel(const uint32_t *parts_all, uint64_t n_all,
                                                         uint64_t chunk_elems, uint32_t block_elems, uint32_t e_bytes,
                                                         uint16_t *dst0_all, uint8_t *out, uint64_t slot_bytes) {
  const uint64_t first = (uint64_t)blockIdx.x * chunk_elems;
  const uint64_t n = n_all - first < chunk_elems ? n_all - first : chunk_elems;
  const uint64_t cap = kSampleBytes / e_bytes;
  const uint32_t n_s = (uint32_t)(n < cap ? n : cap);
  uint16_t *dst0 = dst0_all + 256ull * blockIdx.x;
  uint16_t *dst1 = out == nullptr ? nullptr
                                  : (uint16_t *)(out + blockIdx.x * slot_bytes + kHeaderBytes +
                                                 pad16(4 * ((n + block_elems - 1) / block_elems)));
  const uint32_t *parts = parts_all + 256ull * kTableParts * blockIdx.x;
  uint32_t c[4] = {0, 0, 0, 0};
  for (uint32_t p = 0; p < kTableParts; ++p) {
    const uint4 v = *(const uint4 *)(parts + 256 * p + 4 * threadIdx.x);
    c[0] += v.x;
    c[1] += v.y;
    c[2] += v.z;
    c[3] += v.w;
  }
  write_table(c, n_s, dst0, dst1);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
// Device scratch of uzip_compress_noalloc, for callers that cannot allocate:
// the encoder's workspace (ticket and counters, look-back status words,
// overflow slots).  Every GPU the library runs on holds its own copy until
// the process ends; host code reaches it only through the address that
// hipGetSymbolAddress returns for the current device.
constexpr uint64_t kScratchBytes = 64ull << 20;
constexpr uint64_t kScratchMaxBlocks = 4194304;  // status words: 32 MiB
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
// encoder kernels: index = dt * 4 + kind, kind 0/1 = compress large/small
// blocks, 2/3 = split-send producer large/small blocks; fused reduce apart
constexpr int kEncodeKernels = 20;
const void *encode_kernel_ptr(int k) {
  static const void *const tab[kEncodeKernels] = {
      (const void *)encode_kernel<0, false, false>, (const void *)encode_kernel<0, true, false>,
      (const void *)encode_kernel<0, false, true>,  (const void *)encode_kernel<0, true, true>,
      (const void *)encode_kernel<1, false, false>, (const void *)encode_kernel<1, true, false>,
      (const void *)encode_kernel<1, false, true>,  (const void *)encode_kernel<1, true, true>,
      (const void *)encode_kernel<2, false, false>, (const void *)encode_kernel<2, true, false>,
      (const void *)encode_kernel<2, false, true>,  (const void *)encode_kernel<2, true, true>,
      (const void *)encode_kernel<3, false, false>, (const void *)encode_kernel<3, true, false>,
      (const void *)encode_kernel<3, false, true>,  (const void *)encode_kernel<3, true, true>,
      (const void *)encode_kernel<4, false, false>, (const void *)encode_kernel<4, true, false>,
      (const void *)encode_kernel<4, false, true>,  (const void *)encode_kernel<4, true, true>};
  return tab[k];
}
// encoders with stream-wide tables: index = dt * 4 + kind (as above)
constexpr int kSharedKernels = 20;
const void *shared_kernel_ptr(int k) {
  static const void *const tab[kSharedKernels] = {
      (const void *)encode_kernel<0, false, false, true>, (const void *)encode_kernel<0, true, false, true>,
      (const void *)encode_kernel<0, false, true, true>,  (const void *)encode_kernel<0, true, true, true>,
      (const void *)encode_kernel<1, false, false, true>, (const void *)encode_kernel<1, true, false, true>,
      (const void *)encode_kernel<1, false, true, true>,  (const void *)encode_kernel<1, true, true, true>,
      (const void *)encode_kernel<2, false, false, true>, (const void *)encode_kernel<2, true, false, true>,
      (const void *)encode_kernel<2, false, true, true>,  (const void *)encode_kernel<2, true, true, true>,
      (const void *)encode_kernel<3, false, false, true>, (const void *)encode_kernel<3, true, false, true>,
      (const void *)encode_kernel<3, false, true, true>,  (const void *)encode_kernel<3, true, true, true>,
      (const void *)encode_kernel<4, false, false, true>, (const void *)encode_kernel<4, true, false, true>,
      (const void *)encode_kernel<4, false, true, true>,  (const void *)encode_kernel<4, true, true, true>};
  return tab[k];
}
const void *reduce_kernel_ptr(int dt) {
  static const void *const tab[3] = {(const void *)reduce_kernel<0>, (const void *)reduce_kernel<1>,
                                     (const void *)reduce_kernel<2>};
  return tab[dt];
}

struct DeviceInfo {
  int cus = 0;
  bool gfx950 = false;
  uint8_t *scratch = nullptr;  // this device's copy of `scratch` (uzip_compress_noalloc)
  // the encoder kernels have no static LDS, so their dynamic LDS (and the
  // encoder table they read at a fixed LDS address) starts at address 0
  bool enc_lds_at0 = false;
};

// fault injection (uzip_inject_scan_stall)
std::atomic<uint32_t> g_spin_limit{kSpinLimit};
std::atomic<uint32_t> g_hold_block{~0u};

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
    // the device address of this device's copy of the static scratch (in
    // host code the array's name is only a stand-in); null on failure, and
    // uzip_compress_noalloc then reports UZIP_EHIP
    void *sp = nullptr;
    if (hipGetSymbolAddress(&sp, HIP_SYMBOL(scratch)) == hipSuccess) g_info[dev].scratch = (uint8_t *)sp;
    const int lds_max = 160 * 1024;
    for (int k = 0; k < kEncodeKernels; ++k)
      (void)hipFuncSetAttribute(encode_kernel_ptr(k), hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    for (int k = 0; k < kSharedKernels; ++k)
      (void)hipFuncSetAttribute(shared_kernel_ptr(k), hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    for (int k = 0; k < 3; ++k)
      (void)hipFuncSetAttribute(reduce_kernel_ptr(k), hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    bool at0 = true;
    auto no_static_lds = [](const void *f) {
      hipFuncAttributes fa;
      return hipFuncGetAttributes(&fa, f) == hipSuccess && fa.sharedSizeBytes == 0;
    };
    for (int k = 0; k < kEncodeKernels; ++k) at0 = at0 && no_static_lds(encode_kernel_ptr(k));
    for (int k = 0; k < kSharedKernels; ++k) at0 = at0 && no_static_lds(shared_kernel_ptr(k));
    for (int k = 0; k < 3; ++k) at0 = at0 && no_static_lds(reduce_kernel_ptr(k));
    g_info[dev].enc_lds_at0 = at0;
    (void)hipFuncSetAttribute((const void *)reduce_decode_kernel<0>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)reduce_decode_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    (void)hipFuncSetAttribute((const void *)reduce_decode_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    // (reduce_fused_kernel has a few bytes of static LDS besides)
    (void)hipFuncSetAttribute((const void *)reduce_fused_kernel<0>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max - 1024);
    (void)hipFuncSetAttribute((const void *)reduce_fused_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max - 1024);
    (void)hipFuncSetAttribute((const void *)reduce_fused_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max - 1024);
    (void)hipFuncSetAttribute((const void *)table_kernel<0>, hipFuncAttributeMaxDynamicSharedMemorySize, kTableLds);
    (void)hipFuncSetAttribute((const void *)table_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize, kTableLds);
    (void)hipFuncSetAttribute((const void *)table_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize, kTableLds);
    (void)hipFuncSetAttribute((const void *)table_kernel<3>, hipFuncAttributeMaxDynamicSharedMemorySize, kTableLds);
    (void)hipFuncSetAttribute((const void *)table_kernel<4>, hipFuncAttributeMaxDynamicSharedMemorySize, kTableLds);
    // an attribute the runtime refused must not surface as the error of a
    // later launch
    (void)hipGetLastError();
  });
  if (err != hipSuccess) return UZIP_EHIP;
  out = g_info[dev];
  if (!out.gfx950) return UZIP_EUNSUPPORTED;
  return UZIP_OK;
}

uint32_t elem_bytes(uzip_dtype dt) { return dt == UZIP_FP32 ? 4u : 2u; }
bool valid_dtype(uzip_dtype dt) { return dt >= UZIP_BF16 && dt <= UZIP_E5M2; }
// the fused reduction adds values, which FP8 pairs are not given for
bool valid_reduce_dtype(uzip_dtype dt) { return dt >= UZIP_BF16 && dt <= UZIP_FP32; }
bool valid_block(uint32_t bb) { return bb >= kMinBlockBytes && bb <= kMaxBlockBytes && (bb & (bb - 1)) == 0; }
// element counts up to 2^48: every size computed from one stays far from
// 64-bit overflow
constexpr uint64_t kMaxElems = 1ull << 48;
bool valid_n(uint64_t n) { return n <= kMaxElems; }
bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
uint64_t pad256(uint64_t x) { return (x + 255u) & ~uint64_t(255); }

uint64_t max_size(uint32_t E, uint64_t n, uint32_t block_elems) {
  Geom g = make_geom(n, block_elems, E);
  uint64_t full = n / block_elems, tail = n - full * block_elems;
  return g.coded_off + full * pad16(block_elems) + (tail ? pad16(tail) : 0);
}

constexpr uint32_t kSmallMaxElems = kRegRounds * kRound;  // symbols fit the register store
constexpr uint32_t kSmallStageWords = 7424;                // LDS staging window (words), compress
constexpr uint32_t kMaxSlots = 2048;                        // persistent workgroups, compress

bool small_path(uint32_t block_elems) { return block_elems <= kSmallMaxElems; }
uint32_t word_cap(uint32_t block_elems) { return block_elems / 2 + kRound + 8; }
uint32_t stage_words(uint32_t block_elems) {
  const uint32_t w = word_cap(block_elems);
  return w > kSmallStageWords ? kSmallStageWords : w;
}
// words of one overflow slot: the staging indices that can leave the LDS
// window (none when the window holds a whole block's words)
uint32_t slot_words(uint32_t block_elems) {
  const uint32_t w = word_cap(block_elems), l = stage_words(block_elems);
  return w > l ? (kSlotLead + (w - l) + kSlotTail + 127u) & ~127u : 0u;
}
// overflow slots of a coding pass (compress, the split-send producer, the
// fused reduce's separate coding pass): one per persistent workgroup
uint64_t n_slots(uint64_t n_blocks, uint32_t block_elems) {
  (void)block_elems;
  return n_blocks < kMaxSlots ? n_blocks : kMaxSlots;
}

// LDS bytes of encode_kernel and reduce_kernel: the pass-1 histogram or the
// coding pass's staging window
uint32_t encode_lds(uint32_t block_elems) {
  const uint32_t pass1 = kHistBytes;
  const uint32_t pass2 = kStageHead + 2 * stage_words(block_elems) + kStageTail;
  return kTrashBytes + kEncTableBytes + (pass1 > pass2 ? pass1 : pass2);
}

struct EncodeWs {
  uint64_t status_off, cnt_off, slot_off, y_off, total;
  uint64_t slots;  // overflow slots: the persistent grid's upper bound
};

// workspace: ticket, error word, exit counter | look-back status per block |
// chunk counters | overflow slots (blocks whose words can exceed the LDS
// window) | reduced tensor (fused reduce without a caller buffer).
// [0, slot_off) is cleared per call.
// `slots`: how many overflow slots to lay out (0: n_slots of the call)
EncodeWs encode_ws(uint64_t n_blocks, uint64_t n_chunks, uint32_t block_elems, uint64_t ybytes, uint64_t slots = 0) {
  EncodeWs w;
  w.status_off = kWsHeaderBytes;
  w.cnt_off = pad256(w.status_off + 8 * n_blocks);
  w.slot_off = pad256(w.cnt_off + 8 * n_chunks);
  w.slots = slots ? slots : n_slots(n_blocks, block_elems);
  w.y_off = pad256(w.slot_off + 2ull * w.slots * slot_words(block_elems));
  w.total = pad256(w.y_off + ybytes);
  return w;
}

// Fused reduce workspace: the coding pass's (status words, the reduced
// tensor if the caller keeps no copy), the per-block histograms, and fp32
// partial sums when the inputs come in more than one group.
struct ReduceWs {
  EncodeWs enc;
  uint64_t hist_off, acc_off, total;
};
ReduceWs reduce_ws(uint64_t n_blocks, uint32_t block_elems, uint64_t n, uint32_t E, int n_in, bool need_y) {
  ReduceWs w;
  w.enc = encode_ws(n_blocks, 1, block_elems, need_y ? n * E : 0);
  w.hist_off = w.enc.total;
  w.acc_off = pad256(w.hist_off + 1024 * n_blocks);
  w.total = pad256(w.acc_off + (n_in > kReduceGroup ? 4 * n : 0));
  return w;
}

// LDS of reduce_fused_kernel for n_in decoding waves: the decoders' tables
// and rings (or, once they are done, the staging area of a whole block's
// words), the slabs, the histogram, the block's symbols, the encoder table
// and the trash slots; 0 if the block does not fit (larger blocks take the
// decode-reduce kernel and the encoder's coding pass instead).
constexpr uint32_t kLdsMax = 160 * 1024;
uint32_t fused_layout(int n_in, uint32_t E, uint32_t block_elems, ReduceArgs *r) {
  const uint32_t stage = kStageHead + 2 * word_cap(block_elems) + kStageTail;
  const uint32_t dec = (uint32_t)n_in * kDecLds;
  uint32_t o = (dec > stage ? dec : stage);
  o = (o + 15u) & ~15u;
  const uint32_t slabs = o;
  o += 2u * (uint32_t)n_in * kRound * E;
  const uint32_t hist = o;
  o += kHistBytes;
  const uint32_t syms = o;
  o += (block_elems + 15u) & ~15u;
  const uint32_t enc = o;
  o += kEncTableBytes;
  const uint32_t trash = o;
  o += kTrashBytes;
  if (o + 1024 > kLdsMax) return 0;  // (the kernel's own static bytes besides)
  if (r != nullptr) {
    r->lds_slabs = slabs;
    r->lds_hist = hist;
    r->lds_syms = syms;
    r->lds_enc = enc;
    r->lds_trash = trash;
  }
  return o;
}

uzip_status launch_table(const void *d_in, uint64_t n, uzip_dtype dt, uint64_t chunk_elems, uint32_t block_elems,
                         uint64_t chunks, uint16_t *dst0, uint8_t *out, uint64_t slot_bytes, hipStream_t stream) {
  static const void *const tab[5] = {(const void *)table_kernel<0>, (const void *)table_kernel<1>,
                                     (const void *)table_kernel<2>, (const void *)table_kernel<3>,
                                     (const void *)table_kernel<4>};
  const uint8_t *in = (const uint8_t *)d_in;
  void *args[] = {&in, &n, &chunk_elems, &block_elems, &dst0, &out, &slot_bytes};
  if (hipLaunchKernel(tab[(int)dt], dim3((unsigned)chunks), dim3(kTableThreads), args, kTableLds, stream) != hipSuccess)
    return UZIP_EHIP;
  return UZIP_OK;
}

// The tables of `chunks` streams (as launch_table) with each sample split
// over kTableParts workgroups; `parts`: chunks * kTableParts * 256 u32 of
// workspace.
uzip_status launch_table_split(const void *d_in, uint64_t n, uzip_dtype dt, uint64_t chunk_elems,
                               uint32_t block_elems, uint64_t chunks, uint16_t *dst0, uint8_t *out,
                               uint64_t slot_bytes, uint32_t *parts, hipStream_t stream) {
  static const void *const tab[5] = {(const void *)table_part_kernel<0>, (const void *)table_part_kernel<1>,
                                     (const void *)table_part_kernel<2>, (const void *)table_part_kernel<3>,
                                     (const void *)table_part_kernel<4>};
  const uint8_t *in = (const uint8_t *)d_in;
  void *args[] = {&in, &n, &chunk_elems, &parts};
  if (hipLaunchKernel(tab[(int)dt], dim3((unsigned)(chunks * kTableParts)), dim3(kTableThreads), args, 0, stream) !=
      hipSuccess)
    return UZIP_EHIP;
  hipLaunchKernelGGL(table_merge_kernel, dim3((unsigned)chunks), dim3(64), 0, stream, (const uint32_t *)parts, n,
                     chunk_elems, block_elems, elem_bytes(dt), dst0, out, slot_bytes);
  return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
}

uzip_status launch_encode(EncodeArgs &a, uzip_dtype dt, bool reduce, uint8_t *ws, const EncodeWs &w,
                          const DeviceInfo &info, hipStream_t stream, bool shared = false,
                          uint32_t *dstatus = nullptr) {
  if (!info.enc_lds_at0) return UZIP_EHIP;
  const bool small = !reduce && small_path(a.block_elems);
  a.ticket = (uint32_t *)ws;  // the kWs* words, then the look-back status
  a.status = (uint64_t *)(ws + w.status_off);
  a.chunk_cnt = (uint32_t *)(ws + w.cnt_off);
  a.slots = (uint16_t *)(ws + w.slot_off);
  a.slot_words = slot_words(a.block_elems);
  a.wcap = word_cap(a.block_elems);
  a.lds_words = stage_words(a.block_elems);
  a.pass2_off = kEncTableBytes;
  const uint32_t lds = encode_lds(a.block_elems);
  if (lds > 160 * 1024) return UZIP_EINVAL;
  // The split-send producer keeps each chunk on one XCD when the chip runs
  // as one device of 8 XCDs and the grid gives every XCD 32 workgroups
  // (workgroups go to the XCDs in turn): its stream bytes then need no
  // write-through stores, one write-back of the XCD's L2 per chunk does.
  // The XCDs get equal numbers of chunks, or numbers at most 1/8 apart.
  const uint64_t chunks = ((uint64_t)a.n_blocks + a.blocks_per_chunk - 1) / a.blocks_per_chunk;
  const uint64_t most = a.n_blocks < w.slots ? a.n_blocks : w.slots;
  const bool even = chunks >= 8 * kMaxXcd || (chunks >= kMaxXcd && chunks % kMaxXcd == 0);
  a.n_xcd = (!reduce && a.flags != nullptr && info.cus == 32 * (int)kMaxXcd && even && most >= (uint64_t)info.cus)
                ? kMaxXcd
                : 0;
  const int kind = (a.flags != nullptr && a.n_xcd == 0 ? 2 : 0) + (small ? 1 : 0);
  const void *fn = reduce   ? reduce_kernel_ptr((int)dt)
                   : shared ? shared_kernel_ptr((int)dt * 4 + kind)
                            : encode_kernel_ptr((int)dt * 4 + kind);
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, 64, lds) != hipSuccess || occ < 1) occ = 1;
  uint64_t grid = (uint64_t)info.cus * (uint64_t)occ;
  if (grid > a.n_blocks) grid = a.n_blocks;
  if (grid > w.slots) grid = w.slots;
  if (grid == 0) grid = 1;
  const uint64_t clear_words = w.slot_off / 4;
  const uint64_t cgrid = (clear_words + 255) / 256 < 4096 ? (clear_words + 255) / 256 : 4096;
  hipLaunchKernelGGL(clear_kernel, dim3((unsigned)cgrid), dim3(256), 0, stream, (uint32_t *)ws, clear_words,
                     g_spin_limit.load(std::memory_order_relaxed), g_hold_block.load(std::memory_order_relaxed),
                     (uint64_t)(uintptr_t)dstatus);
  if (hipGetLastError() != hipSuccess) return UZIP_EHIP;
  void *args[] = {&a};
  if (hipLaunchKernel(fn, dim3((unsigned)grid), dim3(64), args, lds, stream) != hipSuccess) return UZIP_EHIP;
  return UZIP_OK;
}

}  // namespace

extern "C" {

size_t uzip_max_compressed_size(uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return 0;
  return (size_t)max_size(elem_bytes(dtype), n_elems, block_bytes / elem_bytes(dtype));
}

size_t uzip_workspace_size(int op, uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, uint64_t aux) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return 0;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t nb = (n_elems + be - 1) / be;
  switch (op) {
    case UZIP_OP_COMPRESS:
      return (size_t)encode_ws(nb, 1, be, 0).total;
    case UZIP_OP_DECOMPRESS:
      return kDecodeWsBytes;
    case UZIP_OP_COMPRESS_TABLE:
      return (size_t)encode_ws(nb, 1, be, 0).total + kTableBytes + kTableParts * 256 * 4;
    case UZIP_OP_CHUNKED_TABLE: {
      if (aux == 0 || aux % block_bytes) return 0;
      const uint64_t ce = aux / E;
      const uint64_t chunks = (n_elems + ce - 1) / ce;
      return (size_t)(encode_ws(chunks * (ce / be), chunks, be, 0).total + chunks * (kTableBytes + kTableParts * 256 * 4));
    }
    case UZIP_OP_CHUNKED: {
      if (aux == 0 || aux % block_bytes) return 0;
      const uint64_t ce = aux / E;
      const uint64_t chunks = (n_elems + ce - 1) / ce;
      return (size_t)encode_ws(chunks * (ce / be), chunks, be, 0).total;
    }
    case UZIP_OP_REDUCE: {
      if (!valid_reduce_dtype(dtype)) return 0;
      const uint64_t n_in = aux & 0xFFFFu;
      if (n_in < 1 || n_in > kMaxInputs) return 0;
      return (size_t)reduce_ws(nb, be, n_elems, E, (int)n_in, (aux & UZIP_WS_NO_OUT_RAW) != 0).total;
    }
    default:
      return 0;
  }
}

uzip_status uzip_compress(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                          void *d_out, size_t out_cap, uint64_t *d_out_size, void *d_ws, size_t ws_bytes,
                          hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return UZIP_EINVAL;
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
  EncodeWs w = encode_ws(nb, 1, be, 0);
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
  return launch_encode(a, dtype, false, (uint8_t *)d_ws, w, info, stream);
}

uzip_status uzip_compress_noalloc(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                  void *d_out, size_t out_cap, uint64_t *d_out_size, hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out) || (n_elems > 0 && (d_in == nullptr || !aligned16(d_in))))
    return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t nb = (n_elems + be - 1) / be;
  if (nb > kScratchMaxBlocks) return UZIP_ENOSPC;  // beyond the scratch's status words
  if (out_cap < max_size(E, n_elems, be)) return UZIP_ENOSPC;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  if (info.scratch == nullptr) return UZIP_EHIP;
  if (n_elems == 0) {
    hipLaunchKernelGGL(empty_stream_kernel, dim3(1), dim3(64), 0, stream, (uint8_t *)d_out, (uint32_t)dtype, be,
                       d_out_size);
    return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
  }
  // as many overflow slots as the scratch holds after the status words, up
  // to the usual one per persistent workgroup (fewer only shrink the grid)
  const EncodeWs full = encode_ws(nb, 1, be, 0);
  uint64_t slots = full.slots;
  const uint64_t sw = 2ull * slot_words(be);
  if (sw > 0 && full.slot_off + slots * sw > kScratchBytes) slots = (kScratchBytes - full.slot_off) / sw;
  if (slots == 0) return UZIP_ENOSPC;
  const EncodeWs w = encode_ws(nb, 1, be, 0, slots);
  if (w.total > kScratchBytes) return UZIP_ENOSPC;
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
  return launch_encode(a, dtype, false, info.scratch, w, info, stream);
}

uzip_status uzip_compress_chunked(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                  uint64_t chunk_bytes, void *d_out, size_t slot_bytes, uint64_t *chunk_sizes,
                                  uint32_t *flags, uint32_t epoch, void *d_ws, size_t ws_bytes,
                                  hipStream_t stream) {
  return uzip_compress_chunked_table(d_in, n_elems, dtype, block_bytes, chunk_bytes, UZIP_TABLE_PER_BLOCK, nullptr,
                                     d_out, slot_bytes, chunk_sizes, flags, epoch, d_ws, ws_bytes, stream);
}

uzip_status uzip_compress_chunked_table(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                        uint64_t chunk_bytes, uzip_table_mode mode, const uint16_t *d_table,
                                        void *d_out, size_t slot_bytes, uint64_t *chunk_sizes, uint32_t *flags,
                                        uint32_t epoch, void *d_ws, size_t ws_bytes, hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return UZIP_EINVAL;
  if (mode != UZIP_TABLE_PER_BLOCK && mode != UZIP_TABLE_SAMPLED && mode != UZIP_TABLE_EXTERNAL) return UZIP_EINVAL;
  if (mode == UZIP_TABLE_EXTERNAL && (d_table == nullptr || !aligned16(d_table))) return UZIP_EINVAL;
  if (chunk_bytes == 0 || chunk_bytes % block_bytes) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out) || (slot_bytes & 15u) || (n_elems > 0 && (d_in == nullptr || !aligned16(d_in))))
    return UZIP_EINVAL;
  if (chunk_sizes == nullptr || flags == nullptr) return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t ce = chunk_bytes / E;
  if (ce / be >= 0x7FFFFFFFull) return UZIP_EINVAL;
  const uint64_t chunks = (n_elems + ce - 1) / ce;
  if (n_elems == 0) return UZIP_OK;
  const uint32_t tb = mode == UZIP_TABLE_SAMPLED ? kTableBytes : 0;  // every chunk has a block
  if (slot_bytes < max_size(E, n_elems < ce ? n_elems : ce, be) + tb) return UZIP_ENOSPC;
  const uint64_t nb = (chunks - 1) * (ce / be) + ((n_elems - (chunks - 1) * ce) + be - 1) / be;
  if (nb >= 0x7FFFFFFFull) return UZIP_EINVAL;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  EncodeWs w = encode_ws(chunks * (ce / be), chunks, be, 0);
  const uint64_t ws_need = w.total + (mode == UZIP_TABLE_SAMPLED ? chunks * (kTableBytes + kTableParts * 256 * 4) : 0);
  if (d_ws == nullptr || !aligned16(d_ws) || ws_bytes < ws_need) return UZIP_ENOSPC;
  const uint16_t *table = d_table;
  if (mode == UZIP_TABLE_SAMPLED) {
    // each chunk's table from its own first 256 KiB, into the workspace
    // and its place in the chunk's stream
    uint16_t *t = (uint16_t *)((uint8_t *)d_ws + w.total);
    st = launch_table_split(d_in, n_elems, dtype, ce, be, chunks, t, (uint8_t *)d_out, slot_bytes,
                            (uint32_t *)((uint8_t *)d_ws + w.total + chunks * kTableBytes), stream);
    if (st != UZIP_OK) return st;
    table = t;
  }
  EncodeArgs a;
  memset(&a, 0, sizeof(a));
  a.table = table;
  a.table_stride = mode == UZIP_TABLE_SAMPLED ? 256 : 0;
  a.table_mode = (uint32_t)mode;
  a.table_bytes = tb;
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
  return launch_encode(a, dtype, false, (uint8_t *)d_ws, w, info, stream, mode != UZIP_TABLE_PER_BLOCK);
}

}  // extern "C"

namespace {
uzip_status launch_decode_args(DecodeArgs &a, uzip_dtype dtype, uint64_t most, const DeviceInfo &info,
                               hipStream_t stream, bool shared);

uzip_status launch_decode(const void *d_in, size_t in_bytes, uzip_dtype dtype, uint64_t n_elems, void *d_out,
                          size_t out_cap, uint32_t *d_status, void *d_ws, size_t ws_bytes, hipStream_t stream,
                          bool shared, const uint16_t *d_table) {
  if (!valid_dtype(dtype) || !valid_n(n_elems) || d_in == nullptr || !aligned16(d_in)) return UZIP_EINVAL;
  if (d_table != nullptr && !aligned16(d_table)) return UZIP_EINVAL;
  if (n_elems > 0 && (d_out == nullptr || !aligned16(d_out))) return UZIP_EINVAL;
  if (out_cap < n_elems * elem_bytes(dtype)) return UZIP_ENOSPC;
  (void)d_ws;  // the decoder keeps no state in a workspace
  (void)ws_bytes;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  a.in = (const uint8_t *)d_in;
  a.in_bytes = in_bytes;
  a.n = n_elems;
  a.dtype = (uint32_t)dtype;
  a.out = (uint8_t *)d_out;
  a.dstatus = d_status;
  a.table = d_table;
  // at most one wave per block of the smallest size
  const uint64_t most = (n_elems + (kMinBlockBytes / elem_bytes(dtype)) - 1) / (kMinBlockBytes / elem_bytes(dtype));
  return launch_decode_args(a, dtype, most, info, stream, shared);
}

uzip_status launch_decode_args(DecodeArgs &a, uzip_dtype dtype, uint64_t most, const DeviceInfo &info,
                               hipStream_t stream, bool shared) {
  // an occupancy-sized grid; its waves walk the blocks grid-stride
  static const void *const dec_tab[10] = {
      (const void *)decode_kernel<0>,       (const void *)decode_kernel<1>,       (const void *)decode_kernel<2>,
      (const void *)decode_kernel<3>,       (const void *)decode_kernel<4>,       (const void *)decode_kernel<0, true>,
      (const void *)decode_kernel<1, true>, (const void *)decode_kernel<2, true>, (const void *)decode_kernel<3, true>,
      (const void *)decode_kernel<4, true>};
  const void *fn = dec_tab[(int)dtype + (shared ? 5 : 0)];
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, 64, 0) != hipSuccess || occ < 1) occ = 1;
  uint64_t grid = (uint64_t)info.cus * (uint64_t)occ;
  if (grid > most) grid = most;
  if (grid == 0) grid = 1;
  void *args[] = {&a};
  if (hipLaunchKernel(fn, dim3((unsigned)grid), dim3(64), args, 0, stream) != hipSuccess) return UZIP_EHIP;
  return UZIP_OK;
}

uzip_status launch_decode_chunked(const void *d_in, size_t slot_bytes, uint64_t first_chunk, uint64_t n_chunks,
                                  uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, uint64_t chunk_bytes,
                                  void *d_out, size_t out_cap, uint32_t *d_status, hipStream_t stream, bool shared,
                                  const uint16_t *d_table) {
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return UZIP_EINVAL;
  if (chunk_bytes == 0 || chunk_bytes % block_bytes) return UZIP_EINVAL;
  if (d_table != nullptr && !aligned16(d_table)) return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t ce = chunk_bytes / E;
  if (ce / be >= 0x7FFFFFFFull) return UZIP_EINVAL;
  const uint64_t chunks = (n_elems + ce - 1) / ce;
  if (first_chunk > chunks || n_chunks > chunks - first_chunk) return UZIP_EINVAL;
  if (n_chunks == 0) return UZIP_OK;
  if (d_in == nullptr || !aligned16(d_in) || (slot_bytes & 15u) || slot_bytes < kHeaderBytes) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out)) return UZIP_EINVAL;
  // the output covers the tensor up to the end of the last chunk decoded
  const uint64_t end = (first_chunk + n_chunks) * ce < n_elems ? (first_chunk + n_chunks) * ce : n_elems;
  if (out_cap < end * E) return UZIP_ENOSPC;
  if (n_chunks * (ce / be) >= 0x7FFFFFFFull) return UZIP_EINVAL;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  a.in = (const uint8_t *)d_in;
  a.n = n_elems;
  a.dtype = (uint32_t)dtype;
  a.out = (uint8_t *)d_out;
  a.dstatus = d_status;
  a.table = d_table;
  a.slot_bytes = slot_bytes;
  a.chunk_elems = ce;
  a.first_chunk = first_chunk;
  a.n_chunks = n_chunks;
  a.bpc = (uint32_t)(ce / be);
  a.block_elems = be;
  return launch_decode_args(a, dtype, n_chunks * a.bpc, info, stream, shared);
}
}  // namespace

extern "C" {

uzip_status uzip_decompress(const void *d_in, size_t in_bytes, uzip_dtype dtype, uint64_t n_elems, void *d_out,
                            size_t out_cap, uint32_t *d_status, void *d_ws, size_t ws_bytes, hipStream_t stream) {
  return launch_decode(d_in, in_bytes, dtype, n_elems, d_out, out_cap, d_status, d_ws, ws_bytes, stream, false,
                       nullptr);
}

uzip_status uzip_decompress_table(const void *d_in, size_t in_bytes, uzip_dtype dtype, uint64_t n_elems,
                                  const uint16_t *d_table, void *d_out, size_t out_cap, uint32_t *d_status,
                                  void *d_ws, size_t ws_bytes, hipStream_t stream) {
  return launch_decode(d_in, in_bytes, dtype, n_elems, d_out, out_cap, d_status, d_ws, ws_bytes, stream, true,
                       d_table);
}

uzip_status uzip_decompress_chunked(const void *d_in, size_t slot_bytes, uint64_t first_chunk, uint64_t n_chunks,
                                    uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, uint64_t chunk_bytes,
                                    void *d_out, size_t out_cap, uint32_t *d_status, hipStream_t stream) {
  return launch_decode_chunked(d_in, slot_bytes, first_chunk, n_chunks, dtype, n_elems, block_bytes, chunk_bytes,
                               d_out, out_cap, d_status, stream, false, nullptr);
}

uzip_status uzip_decompress_chunked_table(const void *d_in, size_t slot_bytes, uint64_t first_chunk,
                                          uint64_t n_chunks, uzip_dtype dtype, uint64_t n_elems,
                                          uint32_t block_bytes, uint64_t chunk_bytes, const uint16_t *d_table,
                                          void *d_out, size_t out_cap, uint32_t *d_status, hipStream_t stream) {
  return launch_decode_chunked(d_in, slot_bytes, first_chunk, n_chunks, dtype, n_elems, block_bytes, chunk_bytes,
                               d_out, out_cap, d_status, stream, true, d_table);
}

uzip_status uzip_build_table(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint16_t *d_table,
                             hipStream_t stream) {
  if (!valid_dtype(dtype) || !valid_n(n_elems) || d_table == nullptr || !aligned16(d_table)) return UZIP_EINVAL;
  if (n_elems > 0 && (d_in == nullptr || !aligned16(d_in))) return UZIP_EINVAL;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  const uint32_t be = kMinBlockBytes / elem_bytes(dtype);  // no stream: only the sample matters
  return launch_table(d_in, n_elems, dtype, n_elems ? n_elems : 1, be, 1, d_table, nullptr, 0, stream);
}

uzip_status uzip_compress_table(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                uzip_table_mode mode, const uint16_t *d_table, void *d_out, size_t out_cap,
                                uint64_t *d_out_size, void *d_ws, size_t ws_bytes, hipStream_t stream) {
  if (mode == UZIP_TABLE_PER_BLOCK)
    return uzip_compress(d_in, n_elems, dtype, block_bytes, d_out, out_cap, d_out_size, d_ws, ws_bytes, stream);
  if (mode != UZIP_TABLE_SAMPLED && mode != UZIP_TABLE_EXTERNAL) return UZIP_EINVAL;
  if (!valid_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return UZIP_EINVAL;
  if (d_out == nullptr || !aligned16(d_out) || (n_elems > 0 && (d_in == nullptr || !aligned16(d_in))))
    return UZIP_EINVAL;
  if (mode == UZIP_TABLE_EXTERNAL && (d_table == nullptr || !aligned16(d_table))) return UZIP_EINVAL;
  const uint32_t E = elem_bytes(dtype), be = block_bytes / E;
  const uint64_t nb = (n_elems + be - 1) / be;
  if (nb >= 0x7FFFFFFFull) return UZIP_EINVAL;
  const uint32_t tb = (mode == UZIP_TABLE_SAMPLED && nb > 0) ? kTableBytes : 0;
  if (out_cap < max_size(E, n_elems, be) + tb) return UZIP_ENOSPC;
  DeviceInfo info;
  uzip_status st = device_info(info);
  if (st != UZIP_OK) return st;
  if (n_elems == 0) {
    hipLaunchKernelGGL(empty_stream_kernel, dim3(1), dim3(64), 0, stream, (uint8_t *)d_out, (uint32_t)dtype, be,
                       d_out_size, (uint32_t)mode);
    return hipGetLastError() == hipSuccess ? UZIP_OK : UZIP_EHIP;
  }
  EncodeWs w = encode_ws(nb, 1, be, 0);
  if (d_ws == nullptr || !aligned16(d_ws) || ws_bytes < w.total + kTableBytes + kTableParts * 256 * 4)
    return UZIP_ENOSPC;
  uint8_t *ws = (uint8_t *)d_ws;
  const uint16_t *table = d_table;
  if (mode == UZIP_TABLE_SAMPLED) {
    // the table, into the workspace and its place in the stream (after the
    // directory)
    uint16_t *t = (uint16_t *)(ws + w.total);
    st = launch_table_split(d_in, n_elems, dtype, n_elems, be, 1, t, (uint8_t *)d_out, 0,
                            (uint32_t *)(ws + w.total + kTableBytes), stream);
    if (st != UZIP_OK) return st;
    table = t;
  }
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
  a.table = table;
  a.table_mode = (uint32_t)mode;
  a.table_bytes = tb;
  return launch_encode(a, dtype, false, ws, w, info, stream, true);
}

uzip_status uzip_reduce_fused(const void *const *d_in, const size_t *in_bytes, int n_in, const void *d_local_raw,
                              uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, void *d_out, size_t out_cap,
                              uint64_t *d_out_size, void *d_out_raw, uint32_t *d_status, void *d_ws,
                              size_t ws_bytes, hipStream_t stream) {
  if (!valid_reduce_dtype(dtype) || !valid_block(block_bytes) || !valid_n(n_elems)) return UZIP_EINVAL;
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
  const bool need_y = d_out_raw == nullptr;
  const ReduceWs w = reduce_ws(nb, be, n_elems, E, n_in, need_y);
  if (d_ws == nullptr || !aligned16(d_ws) || ws_bytes < w.total) return UZIP_ENOSPC;
  uint8_t *ws = (uint8_t *)d_ws;
  uint8_t *ybuf = d_out_raw ? (uint8_t *)d_out_raw : ws + w.enc.y_off;
  const Geom g = make_geom(n_elems, be, E);
  // decode + reduce, inputs in groups of up to kReduceGroup
  const int groups = (n_in + kReduceGroup - 1) / kReduceGroup;
  const int n_last = n_in - (groups - 1) * kReduceGroup;
  // One kernel for the last group (the whole call for up to eight inputs)
  // when a block's symbols and words fit in LDS and every output block gets
  // a compute unit of its own at once (one workgroup per CU; its coding pass
  // then costs one block's coding).  With more blocks the decode-reduce
  // kernel and a separate coding pass at higher occupancy overlap better.
  const bool fused = fused_layout(n_last, E, be, nullptr) != 0 && nb <= (uint64_t)info.cus;
  const void *dfn = dtype == UZIP_BF16   ? (const void *)reduce_decode_kernel<0>
                    : dtype == UZIP_FP16 ? (const void *)reduce_decode_kernel<1>
                                         : (const void *)reduce_decode_kernel<2>;
  if (fused) {
    // the scan's workspace words (ticket, error word, exit counter, the
    // fault settings, the status pointer, the per-block status) start clear
    const uint64_t clear_words = w.enc.slot_off / 4;
    const uint64_t cgrid = (clear_words + 255) / 256 < 4096 ? (clear_words + 255) / 256 : 4096;
    hipLaunchKernelGGL(clear_kernel, dim3((unsigned)cgrid), dim3(256), 0, stream, (uint32_t *)ws, clear_words,
                       g_spin_limit.load(std::memory_order_relaxed), g_hold_block.load(std::memory_order_relaxed),
                       (uint64_t)(uintptr_t)d_status);
    if (hipGetLastError() != hipSuccess) return UZIP_EHIP;
  }
  for (int gi = 0; gi < groups; ++gi) {
    ReduceArgs r;
    memset(&r, 0, sizeof(r));
    const int i0 = gi * kReduceGroup;
    r.n_in = n_in - i0 < kReduceGroup ? n_in - i0 : kReduceGroup;
    for (int i = 0; i < r.n_in; ++i) {
      r.ins[i] = (const uint8_t *)d_in[i0 + i];
      r.in_bytes[i] = in_bytes[i0 + i];
    }
    r.first = gi == 0;
    r.last = gi == groups - 1;
    r.acc_in = (const float *)(ws + w.acc_off);
    r.acc_out = (float *)(ws + w.acc_off);
    r.local_raw = (const uint8_t *)d_local_raw;
    r.n = n_elems;
    r.block_elems = be;
    r.out_raw_plane = (uint8_t *)d_out + g.raw_off;
    r.ybuf = ybuf;
    r.yout = (uint8_t *)d_out_raw;
    r.hist_out = (uint32_t *)(ws + w.hist_off);
    r.dstatus = d_status;
    if (fused && r.last) {
      EncodeArgs a;
      memset(&a, 0, sizeof(a));
      a.n = n_elems;
      a.chunk_elems = nb * be;
      a.block_elems = be;
      a.blocks_per_chunk = (uint32_t)nb;
      a.n_blocks = (uint32_t)nb;
      a.out = (uint8_t *)d_out;
      a.sizes = d_out_size;
      a.ticket = (uint32_t *)ws;
      a.status = (uint64_t *)(ws + w.enc.status_off);
      a.chunk_cnt = (uint32_t *)(ws + w.enc.cnt_off);
      a.wcap = word_cap(be);
      a.lds_words = a.wcap;
      const uint32_t lds = fused_layout(r.n_in, E, be, &r);
      static const void *const ftab[3] = {(const void *)reduce_fused_kernel<0>, (const void *)reduce_fused_kernel<1>,
                                          (const void *)reduce_fused_kernel<2>};
      void *args[] = {&r, &a};
      if (hipLaunchKernel(ftab[(int)dtype], dim3((unsigned)nb), dim3(64 * (r.n_in + 1)), args, lds, stream) !=
          hipSuccess)
        return UZIP_EHIP;
      return UZIP_OK;
    }
    const uint32_t lds = reduce_lds(r.n_in, E);
    void *args[] = {&r};
    if (hipLaunchKernel(dfn, dim3((unsigned)nb), dim3(64 * (r.n_in + 1)), args, lds, stream) != hipSuccess)
      return UZIP_EHIP;
  }
  // coding pass over the reduced tensor
  EncodeArgs a;
  memset(&a, 0, sizeof(a));
  a.n = n_elems;
  a.chunk_elems = nb * be;
  a.block_elems = be;
  a.blocks_per_chunk = (uint32_t)nb;
  a.n_blocks = (uint32_t)nb;
  a.out = (uint8_t *)d_out;
  a.sizes = d_out_size;
  a.ybuf = ybuf;
  a.hist_in = (const uint32_t *)(ws + w.hist_off);
  return launch_encode(a, dtype, true, ws, w.enc, info, stream, false, d_status);
}

uzip_status uzip_inject_scan_stall(uint32_t spin_limit, uint32_t held_block) {
  g_spin_limit.store(spin_limit ? spin_limit : kSpinLimit, std::memory_order_relaxed);
  g_hold_block.store(held_block, std::memory_order_relaxed);
  return UZIP_OK;
}

const char *uzip_status_str(uzip_status status) {
  switch (status) {
    case UZIP_OK: return "ok";
    case UZIP_EINVAL: return "invalid argument";
    case UZIP_ENOSPC: return "output or workspace too small";
    case UZIP_ECORRUPT: return "corrupt or mismatched stream";
    case UZIP_EHIP: return "HIP runtime error";
    case UZIP_EUNSUPPORTED: return "device is not gfx950";
    case UZIP_ETIMEOUT: return "encoder wait for an earlier block ran out; stream invalid";
    default: return "unknown status";
  }
}

}  // extern "C"
