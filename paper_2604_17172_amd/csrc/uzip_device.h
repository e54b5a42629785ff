// uzip_device.h -- device building blocks of the gfx950 codec kernels.
//
// Wave64 primitives, the element transform of the split step (section
// 2.1.2, Step 1), stream geometry and the per-block table helpers shared by
// the compress, decompress and fused-reduce kernels.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uzip {

// ---- format constants (stream version 1) ----
constexpr uint32_t kProbBits = 11;          // table resolution: frequencies sum to 2^11
constexpr uint32_t kM = 1u << kProbBits;
constexpr uint32_t kStateLo = 1u << 15;     // coder state interval [2^15, 2^31)
constexpr uint32_t kLanes = 64;             // interleaved states per block (one wave64)
constexpr uint32_t kPerLane = 8;            // consecutive elements per lane and round
constexpr uint32_t kRound = kLanes * kPerLane;
constexpr uint32_t kHeaderBytes = 32;
constexpr uint32_t kSectionFixed = 288;     // 64 states + 32-byte presence bitmap
constexpr uint32_t kSharedSectionFixed = 256;  // 64 states (stream-wide table)
constexpr uint32_t kTableBytes = 512;          // a stream-wide table: u16 f[256]
constexpr uint32_t kSampleBytes = 262144;      // the sample a stream-wide table is built from
constexpr uint32_t kMagic = 0x31505A55u;
constexpr uint32_t kVersion = 1;
constexpr uint32_t kStoredBit = 0x80000000u;

// status words of the single-pass scan over block sizes (decoupled look-back)
constexpr uint64_t kFlagAggregate = 1ull << 62;
constexpr uint64_t kFlagInclusive = 2ull << 62;
constexpr uint64_t kValueMask = (1ull << 62) - 1;

// LDS layout constants
constexpr uint32_t kHistReplicas = 8;       // sub-histograms, lane & 7
// Replica strides of the LDS sub-histograms.  LDS serves 32 banks; a block's
// exponents crowd a narrow band of adjacent symbols, so with an odd stride
// (replica r's bin s in bank r + s) the hot bins of neighbouring replicas
// pile up on the same banks.  A stride of 4 mod 32 shifts each replica's
// band by four banks and the eight replicas go once round the banks
// (measured on weight-buffer exponents: 10.2 -> 4.4 conflict cycles per
// wave-wide atomic).
constexpr uint32_t kHistStride = 260;       // 256 bins, 4 mod 32
constexpr uint32_t kPackedHistStride = 132; // packed 16-bit counts, two bins per word, 4 mod 32
constexpr uint32_t kHistBytes = kHistReplicas * kHistStride * 4;
constexpr uint32_t kEncTableBytes = 256 * 16;
constexpr uint32_t kLutBytes = kM * 4;
constexpr uint32_t kStageHead = 800;        // room for state/bitmap/f[256] before the words
constexpr uint32_t kStageTail = 32;         // zero bytes after the words

__host__ __device__ constexpr uint64_t pad16(uint64_t x) { return (x + 15u) & ~uint64_t(15); }

// Geometry of one stream (a whole tensor or one chunk of it).
struct Geom {
  uint64_t n;          // elements in the stream
  uint32_t n_blocks;
  uint64_t raw_off;    // byte offset of the raw plane
  uint64_t coded_off;  // byte offset of the coded plane
};

__host__ __device__ inline Geom make_geom(uint64_t n, uint32_t block_elems, uint32_t E) {
  Geom g;
  g.n = n;
  g.n_blocks = (uint32_t)((n + block_elems - 1) / block_elems);
  g.raw_off = kHeaderBytes + pad16(4ull * g.n_blocks);
  g.coded_off = g.raw_off + pad16((uint64_t)(E - 1) * n);
  return g;
}

// ---- wave64 primitives ----
__device__ inline uint32_t lane_id() { return __lane_id(); }

__device__ inline uint32_t mbcnt(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Wave-wide scans and reductions with DPP lane moves (VALU operands, a few
// cycles each) rather than LDS-routed lane shuffles: row shifts by 1, 2, 4
// and 8 scan each row of 16 lanes, then row broadcasts of lanes 15 and 31
// carry the row totals into the later rows.  Lanes without a source read 0.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, true);
}
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;

// inclusive prefix sum over lanes
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += dpp_mov<kRowShr1>(v);
  v += dpp_mov<kRowShr2>(v);
  v += dpp_mov<kRowShr4>(v);
  v += dpp_mov<kRowShr8>(v);
  v += dpp_mov<kRowBcast15, 0xA>(v);
  v += dpp_mov<kRowBcast31, 0xC>(v);
  return v;
}

// sum over the wave, the same in every lane
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(v), 63);
}

__device__ inline uint64_t wave_sum64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// maximum over the wave, the same in every lane (a running maximum along
// the same row shifts and broadcasts; a missing source reads 0, the least
// unsigned value)
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  v = max(v, dpp_mov<kRowShr1>(v));
  v = max(v, dpp_mov<kRowShr2>(v));
  v = max(v, dpp_mov<kRowShr4>(v));
  v = max(v, dpp_mov<kRowShr8>(v));
  v = max(v, dpp_mov<kRowBcast15, 0xA>(v));
  v = max(v, dpp_mov<kRowBcast31, 0xC>(v));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// exclusive prefix sum over lanes
__device__ __forceinline__ uint32_t wave_excl_scan(uint32_t v) { return wave_incl_scan(v) - v; }

__device__ inline uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// ---- element transform (section 2.1.2, Step 1) ----
// A value is rotated left by one bit so that the sign lands in bit 0; the
// top byte is then the coded symbol (the exponent byte) and the remaining
// low bytes are the raw sign+fraction part.
__device__ inline uint32_t rotl16x2(uint32_t v) {
  return ((v << 1) & 0xFFFEFFFEu) | ((v >> 15) & 0x00010001u);
}
__device__ inline uint32_t rotr16x2(uint32_t v) {
  return ((v >> 1) & 0x7FFF7FFFu) | ((v << 15) & 0x80008000u);
}
__device__ inline uint32_t rotl32(uint32_t v) { return (v << 1) | (v >> 31); }
__device__ inline uint32_t rotr32(uint32_t v) { return (v >> 1) | (v << 31); }

// Eight consecutive elements of one lane, split into symbols and raw bytes.
// sym: 8 bytes; raw: 8 bytes (16-bit types) or 24 bytes (fp32).
struct Group {
  uint32_t sym[2];
  uint32_t raw[6];
};

// 16-bit elements packed two per word (element 2q in the low half).
__device__ inline void split16(const uint32_t w[4], Group &g) {
  uint32_t r0 = rotl16x2(w[0]), r1 = rotl16x2(w[1]), r2 = rotl16x2(w[2]), r3 = rotl16x2(w[3]);
  g.sym[0] = __builtin_amdgcn_perm(r1, r0, 0x07050301u);
  g.sym[1] = __builtin_amdgcn_perm(r3, r2, 0x07050301u);
  g.raw[0] = __builtin_amdgcn_perm(r1, r0, 0x06040200u);
  g.raw[1] = __builtin_amdgcn_perm(r3, r2, 0x06040200u);
}

__device__ inline void merge16(const uint32_t sym[2], const uint32_t raw[2], uint32_t w[4]) {
  w[0] = rotr16x2(__builtin_amdgcn_perm(sym[0], raw[0], 0x05010400u));
  w[1] = rotr16x2(__builtin_amdgcn_perm(sym[0], raw[0], 0x07030602u));
  w[2] = rotr16x2(__builtin_amdgcn_perm(sym[1], raw[1], 0x05010400u));
  w[3] = rotr16x2(__builtin_amdgcn_perm(sym[1], raw[1], 0x07030602u));
}

// FP8 pairs (section 4.1): element = 16-bit unit of two FP8 values, the
// first in the low byte.  Per value byte, bits 6..3 form its symbol nibble
// and bit 7 with bits 2..0 its raw nibble; a unit's symbol (raw byte) is
// the first value's nibble | the second's << 4.
__device__ inline void split8x2(const uint32_t w[4], Group &g) {
  uint32_t s[4], r[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t t = (w[q] >> 3) & 0x0F0F0F0Fu;                            // symbol nibble per byte
    s[q] = t | (t >> 4);                                                      // units' symbols: bytes 0, 2
    const uint32_t u = ((w[q] >> 4) & 0x08080808u) | (w[q] & 0x07070707u);  // raw nibble per byte
    r[q] = u | (u >> 4);
  }
  g.sym[0] = __builtin_amdgcn_perm(s[1], s[0], 0x06040200u);
  g.sym[1] = __builtin_amdgcn_perm(s[3], s[2], 0x06040200u);
  g.raw[0] = __builtin_amdgcn_perm(r[1], r[0], 0x06040200u);
  g.raw[1] = __builtin_amdgcn_perm(r[3], r[2], 0x06040200u);
}

__device__ inline void merge8x2(const uint32_t sym[2], const uint32_t raw[2], uint32_t w[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    // units 2q, 2q + 1: each unit byte twice, then one nibble per value byte
    const uint32_t sel = (q & 1) ? 0x03030202u : 0x01010000u;
    const uint32_t sp = __builtin_amdgcn_perm(0u, sym[q >> 1], sel);
    const uint32_t rp = __builtin_amdgcn_perm(0u, raw[q >> 1], sel);
    const uint32_t sn = (sp & 0x000F000Fu) | ((sp >> 4) & 0x0F000F00u);
    const uint32_t rn = (rp & 0x000F000Fu) | ((rp >> 4) & 0x0F000F00u);
    w[q] = ((rn << 4) & 0x80808080u) | (sn << 3) | (rn & 0x07070707u);
  }
}

__device__ inline void split32(const uint32_t w[8], Group &g) {
  uint32_t r[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) r[q] = rotl32(w[q]);
  g.sym[0] = (r[0] >> 24) | ((r[1] >> 24) << 8) | ((r[2] >> 24) << 16) | (r[3] & 0xFF000000u);
  g.sym[1] = (r[4] >> 24) | ((r[5] >> 24) << 8) | ((r[6] >> 24) << 16) | (r[7] & 0xFF000000u);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t a = r[4 * h] & 0xFFFFFFu, b = r[4 * h + 1] & 0xFFFFFFu;
    uint32_t c = r[4 * h + 2] & 0xFFFFFFu, d = r[4 * h + 3] & 0xFFFFFFu;
    g.raw[3 * h + 0] = a | (b << 24);
    g.raw[3 * h + 1] = (b >> 8) | (c << 16);
    g.raw[3 * h + 2] = (c >> 16) | (d << 8);
  }
}

__device__ inline void merge32(const uint32_t sym[2], const uint32_t raw[6], uint32_t w[8]) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t r0 = raw[3 * h], r1 = raw[3 * h + 1], r2 = raw[3 * h + 2];
    uint32_t a = r0 & 0xFFFFFFu;
    uint32_t b = (r0 >> 24) | ((r1 & 0xFFFFu) << 8);
    uint32_t c = (r1 >> 16) | ((r2 & 0xFFu) << 16);
    uint32_t d = r2 >> 8;
    uint32_t s = sym[h];
    w[4 * h + 0] = rotr32(a | (s << 24));
    w[4 * h + 1] = rotr32(b | ((s >> 8) << 24));
    w[4 * h + 2] = rotr32(c | ((s >> 16) << 24));
    w[4 * h + 3] = rotr32(d | ((s >> 24) << 24));
  }
}

__device__ inline uint32_t sym_at(const uint32_t sym[2], uint32_t t) {
  return (sym[t >> 2] >> (8 * (t & 3))) & 0xFFu;
}

// ---- scalar conversions for the fused reduce ----
__device__ inline float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }
__device__ inline uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if (f != f) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ inline float fp16_to_f32(uint32_t h) {
  return __half2float(__ushort_as_half((unsigned short)h));
}
__device__ inline uint32_t f32_to_fp16(float f) {
  if (f != f) return 0x7E00u;
  return (uint32_t)__half_as_ushort(__float2half_rn(f));
}

}  // namespace uzip
