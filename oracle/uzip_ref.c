/*
 * uzip_ref.c -- CPU oracle for the block-wise lossless float codec.
 *
 * TEST INFRASTRUCTURE ONLY (see uzip_ref.h).  Plain scalar C, no intrinsics,
 * no blocking, no fusion: every step below is written in the order the
 * method takes it, so that it can be read against the paper.
 *
 * The stream format (our reading where the paper is silent):
 *
 *   Element transform (section 2.1.2, Step 1).  A value of B = 8E bits is
 *   rotated left by one bit, which moves the sign to bit 0.  The top byte of
 *   the rotated word is the symbol (for bf16 and fp32 exactly the 8-bit
 *   exponent field; for fp16 the 5-bit exponent and the top 3 fraction
 *   bits); the low E-1 bytes are the raw sign+fraction part, stored as-is.
 *
 *   FP8 pairs (section 4.1: two FP8 values packed in a 16-bit unit, their
 *   exponent fields extracted jointly into one 8-bit symbol).  Element = the
 *   16-bit unit v0 | v1 << 8 of two consecutive values.  From each value
 *   byte, bits 6..3 go to the symbol and bit 7 (sign) with bits 2..0 to the
 *   raw byte: symbol = n(v0) | n(v1) << 4 with n(v) = (v >> 3) & 15, raw =
 *   r(v0) | r(v1) << 4 with r(v) = (v >> 7) << 3 | (v & 7).  For e4m3fn the
 *   symbol nibbles are the two 4-bit exponent fields; for e5m2 (5-bit
 *   exponent, 2-bit fraction) they are the top four exponent bits of each
 *   value, and the lowest exponent bit travels in the raw byte with the
 *   sign and fraction (our reading: 2 x 5 exponent bits do not fit a byte).
 *
 *   Localized table (section 3.3.1).  Each block of n_b symbols gets its own
 *   table from its own histogram c[256]: with k present symbols and
 *   M = 2^11, f[s] = 1 + floor(c[s](M-k)/n_b) for present s (0 otherwise);
 *   the remainder M - sum(f) goes to the most frequent symbol (ties: the
 *   smallest symbol); cum[s] is the exclusive prefix sum of f in ascending
 *   symbol order.
 *
 *   ANS coding (section 2.1.2, Step 2; one wavefront per block as in the
 *   warp-level execution of section 3.4).  rANS in the sense of Duda
 *   (arXiv:1311.2540) with 64 interleaved 32-bit states (Giesen,
 *   arXiv:1402.3392).  States live in [L, 2^31) with L = 2^15; a state is
 *   renormalised by writing out its low 16 bits.  Symbol i of a block
 *   belongs to round r = i / 512, lane j = (i % 512) / 8, sub-step
 *   t = i % 8.  The encoder walks rounds and sub-steps backwards; the words
 *   one sub-step writes, in ascending lane order, go in front of all words
 *   written before, so that the decoder reads them front to back.
 *
 *   Stream (Step 3, plus the metadata of section 4.1).  32-byte header,
 *   a u32 directory entry per block, the raw plane of all elements, then
 *   the block sections back to back (all little-endian, 16-byte padding
 *   filled with zeros):
 *     0  u32 magic 0x31505A55        4  u8 version (1)   5 u8 dtype
 *     6  u8 prob_bits (11)           7  u8 flags (0)
 *     8  u32 block_elems            12  u32 n_blocks
 *    16  u64 n_elems                24  u64 total_bytes
 *    32  u32 dir[n_blocks]: bit 31 = STORED, bits 30..0 = end offset of the
 *        block's section from the start of the coded plane, in 16-byte units
 *    raw_off   = 32 + pad16(4 n_blocks):  element i's raw bytes at
 *                raw_off + (E-1) i
 *    coded_off = raw_off + pad16((E-1) n): sections of blocks 0..n_blocks-1
 *   A CODED section is u32 state[64] | u8 present[32] (bit s%8 of byte s/8)
 *   | u16 f[k] (present symbols, ascending) | u16 word[W] (decode order) |
 *   zero pad to 16.  A block is CODED iff 288 + 2k + 2W < n_b; otherwise it
 *   is STORED: its n_b symbol bytes, zero-padded to 16.
 *
 *   Stream-wide tables (the sampled localized table of section 3.3.1 and
 *   the table sent once per collective of section 3.4; our reading).  The
 *   header's flags byte names the table mode: 0 = a table per block (as
 *   above), 1 = SAMPLED, 2 = EXTERNAL.  SAMPLED: one table for the whole
 *   stream from the histogram c[256] of its first n_s = min(n, 262144 / E)
 *   elements (the first 256 KiB); every symbol is covered, f[s] = 1 +
 *   floor(c[s](M-256)/n_s) for all 256 symbols, the remainder to the most
 *   frequent (ties: smallest), so a symbol the sample missed stays codable;
 *   the table (u16 f[256], 512 bytes) follows the directory (when there is
 *   at least one block) and the raw plane moves behind it.  EXTERNAL: the
 *   caller's table (any f[256] >= 1 summing to M, e.g. a SAMPLED table of
 *   an earlier call) codes every block and is not in the stream.  With a
 *   stream-wide table a CODED section is u32 state[64] | u16 word[W] | zero
 *   pad to 16, and a block is CODED iff 256 + 2W < n_b.
 *
 *   Fused reduce (section 3.4: decompress, reduce, recompress).  Element by
 *   element, acc = x_0, then acc = acc + x_i for i = 1.. in input order in
 *   IEEE binary32 (round to nearest even, subnormals kept), the optional raw
 *   local addend last; acc is rounded to nearest even into the storage type
 *   (NaN becomes the canonical quiet NaN of that type) and the result is
 *   compressed with the same block size.
 */
#include "uzip_ref.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define M_TOTAL 2048u      /* table total M = 2^11 */
#define PROB_BITS 11u
#define STATE_LO 32768u    /* L = 2^15: lower end of the state interval */
#define LANES 64u
#define PER_LANE 8u
#define ROUND (LANES * PER_LANE)
#define HEADER_BYTES 32u
#define SECTION_FIXED 288u /* 64 states + 32-byte presence bitmap */
#define MAGIC 0x31505A55u

static uint32_t elem_bytes(int dtype) { return dtype == REF_FP32 ? 4u : 2u; }
static uint64_t pad16(uint64_t x) { return (x + 15u) & ~(uint64_t)15u; }

static void put16(uint8_t *p, uint32_t v) {
  p[0] = (uint8_t)v;
  p[1] = (uint8_t)(v >> 8);
}
static void put32(uint8_t *p, uint32_t v) {
  for (int i = 0; i < 4; ++i) p[i] = (uint8_t)(v >> (8 * i));
}
static void put64(uint8_t *p, uint64_t v) {
  for (int i = 0; i < 8; ++i) p[i] = (uint8_t)(v >> (8 * i));
}
static uint32_t get16(const uint8_t *p) { return (uint32_t)p[0] | ((uint32_t)p[1] << 8); }
static uint32_t get32(const uint8_t *p) {
  uint32_t v = 0;
  for (int i = 0; i < 4; ++i) v |= (uint32_t)p[i] << (8 * i);
  return v;
}
static uint64_t get64(const uint8_t *p) {
  uint64_t v = 0;
  for (int i = 0; i < 8; ++i) v |= (uint64_t)p[i] << (8 * i);
  return v;
}

static uint32_t load_elem(const void *in, int dtype, uint64_t i) {
  if (dtype == REF_FP32) return ((const uint32_t *)in)[i];
  return ((const uint16_t *)in)[i];
}
static void store_elem(void *out, int dtype, uint64_t i, uint32_t w) {
  if (dtype == REF_FP32)
    ((uint32_t *)out)[i] = w;
  else
    ((uint16_t *)out)[i] = (uint16_t)w;
}

/* ------------------------------------------------------------------ */
/* Step 1: split a value into symbol (exponent byte) and raw part.      */
/* ------------------------------------------------------------------ */
static int is_fp8(int dtype) { return dtype == REF_E4M3FN || dtype == REF_E5M2; }

/* one FP8 value byte: symbol nibble (bits 6..3), raw nibble (bit 7, bits 2..0) */
static uint32_t fp8_sym_nibble(uint32_t v) { return (v >> 3) & 15u; }
static uint32_t fp8_raw_nibble(uint32_t v) { return ((v >> 7) << 3) | (v & 7u); }
static uint32_t fp8_value(uint32_t sym_nibble, uint32_t raw_nibble) {
  return ((raw_nibble >> 3) << 7) | (sym_nibble << 3) | (raw_nibble & 7u);
}

void ref_split_word(int dtype, uint32_t w, uint32_t *sym, uint32_t *raw) {
  if (is_fp8(dtype)) {
    uint32_t v0 = w & 0xFFu, v1 = (w >> 8) & 0xFFu;
    *sym = fp8_sym_nibble(v0) | (fp8_sym_nibble(v1) << 4);
    *raw = fp8_raw_nibble(v0) | (fp8_raw_nibble(v1) << 4);
    return;
  }
  uint32_t bits = 8u * elem_bytes(dtype);
  uint64_t mask = (bits == 32u) ? 0xFFFFFFFFull : ((1ull << bits) - 1ull);
  uint64_t v = (uint64_t)w & mask;
  uint64_t rot = ((v << 1) | (v >> (bits - 1u))) & mask; /* rotate left 1 */
  *sym = (uint32_t)(rot >> (bits - 8u));
  *raw = (uint32_t)(rot & ((1ull << (bits - 8u)) - 1ull));
}

uint32_t ref_merge_word(int dtype, uint32_t sym, uint32_t raw) {
  if (is_fp8(dtype)) {
    uint32_t v0 = fp8_value(sym & 15u, raw & 15u);
    uint32_t v1 = fp8_value((sym >> 4) & 15u, (raw >> 4) & 15u);
    return v0 | (v1 << 8);
  }
  uint32_t bits = 8u * elem_bytes(dtype);
  uint64_t mask = (bits == 32u) ? 0xFFFFFFFFull : ((1ull << bits) - 1ull);
  uint64_t rot = ((uint64_t)sym << (bits - 8u)) | (uint64_t)raw;
  uint64_t v = ((rot >> 1) | (rot << (bits - 1u))) & mask; /* rotate right 1 */
  return (uint32_t)v;
}

/* ------------------------------------------------------------------ */
/* Localized frequency table of one block (section 3.3.1).             */
/* ------------------------------------------------------------------ */
void ref_build_table(const uint32_t *count, uint32_t n_b, uint32_t *freq,
                     uint32_t *cum) {
  uint32_t k = 0;
  for (int s = 0; s < 256; ++s)
    if (count[s] > 0) ++k;
  uint32_t total = 0;
  for (int s = 0; s < 256; ++s) {
    if (count[s] > 0)
      freq[s] = 1u + (uint32_t)(((uint64_t)count[s] * (M_TOTAL - k)) / n_b);
    else
      freq[s] = 0;
    total += freq[s];
  }
  int best = 0;
  for (int s = 1; s < 256; ++s)
    if (count[s] > count[best]) best = s;
  freq[best] += M_TOTAL - total;
  uint32_t run = 0;
  for (int s = 0; s < 256; ++s) {
    cum[s] = run;
    run += freq[s];
  }
}

/* ------------------------------------------------------------------ */
/* Step 2: interleaved rANS over one block.                            */
/* ------------------------------------------------------------------ */
int64_t ref_rans_encode(const uint8_t *sym, uint32_t n_b, const uint32_t *freq,
                        const uint32_t *cum, uint32_t *state, uint16_t *words,
                        uint64_t max_words) {
  uint64_t rounds = ((uint64_t)n_b + ROUND - 1) / ROUND;
  for (uint32_t j = 0; j < LANES; ++j) state[j] = STATE_LO;
  uint64_t front = max_words; /* words[front..max_words) are written */
  for (int64_t r = (int64_t)rounds - 1; r >= 0; --r) {
    for (int t = (int)PER_LANE - 1; t >= 0; --t) {
      uint16_t step_words[LANES];
      uint32_t g = 0;
      for (uint32_t j = 0; j < LANES; ++j) {
        uint64_t i = (uint64_t)r * ROUND + (uint64_t)j * PER_LANE + (uint64_t)t;
        if (i >= n_b) continue;
        uint32_t s = sym[i];
        uint32_t f = freq[s];
        uint32_t x = state[j];
        /* renormalise: keep x below f * 2^20 so the coded state stays < 2^31 */
        if ((uint64_t)x >= ((uint64_t)f << 20)) {
          step_words[g++] = (uint16_t)(x & 0xFFFFu);
          x >>= 16;
        }
        /* rANS coding function C(s, x) = floor(x / f) M + (x mod f) + cum */
        x = (x / f) * M_TOTAL + (x % f) + cum[s];
        state[j] = x;
      }
      if (g > front) return -1;
      front -= g;
      for (uint32_t q = 0; q < g; ++q) words[front + q] = step_words[q];
    }
  }
  uint64_t w = max_words - front;
  memmove(words, words + front, (size_t)w * sizeof(uint16_t));
  return (int64_t)w;
}

int64_t ref_rans_decode(const uint32_t *state_in, const uint16_t *words,
                        uint64_t n_words, const uint32_t *freq,
                        const uint32_t *cum, uint32_t n_b, uint8_t *sym_out) {
  uint32_t x[LANES];
  for (uint32_t j = 0; j < LANES; ++j) {
    x[j] = state_in[j];
    if (x[j] < STATE_LO || x[j] >= 0x80000000u) return REF_ECORRUPT;
  }
  uint64_t p = 0;
  uint64_t rounds = ((uint64_t)n_b + ROUND - 1) / ROUND;
  for (uint64_t r = 0; r < rounds; ++r) {
    for (uint32_t t = 0; t < PER_LANE; ++t) {
      for (uint32_t j = 0; j < LANES; ++j) {
        uint64_t i = r * ROUND + (uint64_t)j * PER_LANE + t;
        if (i >= n_b) continue;
        uint32_t slot = x[j] & (M_TOTAL - 1u);
        int s = -1;
        for (int c = 0; c < 256; ++c) {
          if (freq[c] > 0 && cum[c] <= slot && slot < cum[c] + freq[c]) {
            s = c;
            break;
          }
        }
        if (s < 0) return REF_ECORRUPT;
        /* decoding function D(x): inverse of C */
        x[j] = freq[s] * (x[j] >> PROB_BITS) + slot - cum[s];
        if (x[j] < STATE_LO) {
          if (p >= n_words) return REF_ECORRUPT;
          x[j] = (x[j] << 16) | words[p++];
        }
        sym_out[i] = (uint8_t)s;
      }
    }
  }
  for (uint32_t j = 0; j < LANES; ++j)
    if (x[j] != STATE_LO) return REF_ECORRUPT;
  return (int64_t)p;
}

/* ------------------------------------------------------------------ */
/* Stream layout helpers                                               */
/* ------------------------------------------------------------------ */
static int valid_block_bytes(uint32_t block_bytes) {
  if (block_bytes < 4096u || block_bytes > 4194304u) return 0;
  return (block_bytes & (block_bytes - 1u)) == 0;
}

static uint64_t raw_offset(uint64_t n_blocks) { return HEADER_BYTES + pad16(4u * n_blocks); }

static uint64_t coded_offset(int dtype, uint64_t n, uint64_t n_blocks) {
  return raw_offset(n_blocks) + pad16((uint64_t)(elem_bytes(dtype) - 1u) * n);
}

uint64_t ref_max_compressed_size(int dtype, uint64_t n, uint32_t block_bytes) {
  uint64_t be = block_bytes / elem_bytes(dtype);
  uint64_t nb = (n + be - 1) / be;
  uint64_t total = coded_offset(dtype, n, nb);
  for (uint64_t b = 0; b < nb; ++b) {
    uint64_t lo = b * be, hi = lo + be < n ? lo + be : n;
    total += pad16(hi - lo);
  }
  return total;
}

int64_t ref_block_section(const void *in, uint64_t n, int dtype,
                          uint32_t block_bytes, uint64_t b, uint8_t *sec,
                          uint64_t sec_cap, int *stored) {
  uint64_t be = block_bytes / elem_bytes(dtype);
  uint64_t lo = b * be;
  if (lo >= n) return REF_EINVAL;
  uint32_t n_b = (uint32_t)((lo + be < n ? lo + be : n) - lo);
  if (sec_cap < pad16(n_b)) return REF_ENOSPC;

  uint8_t *sym = (uint8_t *)malloc(n_b);
  uint16_t *words = (uint16_t *)malloc((size_t)n_b * sizeof(uint16_t) + 16);
  uint32_t count[256] = {0}, freq[256], cum[256], state[LANES];
  for (uint32_t i = 0; i < n_b; ++i) {
    uint32_t s, raw;
    ref_split_word(dtype, load_elem(in, dtype, lo + i), &s, &raw);
    sym[i] = (uint8_t)s;
    count[s] += 1;
  }
  ref_build_table(count, n_b, freq, cum);
  uint32_t k = 0;
  for (int s = 0; s < 256; ++s)
    if (freq[s] > 0) ++k;
  int64_t w = ref_rans_encode(sym, n_b, freq, cum, state, words, n_b);
  uint64_t coded_len = SECTION_FIXED + 2u * k + (w < 0 ? 2u * (uint64_t)n_b : 2u * (uint64_t)w);
  int64_t len;
  if (w >= 0 && coded_len < n_b) {
    len = (int64_t)pad16(coded_len);
    memset(sec, 0, (size_t)len);
    for (uint32_t j = 0; j < LANES; ++j) put32(sec + 4 * j, state[j]);
    for (int s = 0; s < 256; ++s)
      if (freq[s] > 0) sec[256 + s / 8] |= (uint8_t)(1u << (s % 8));
    uint64_t o = SECTION_FIXED;
    for (int s = 0; s < 256; ++s)
      if (freq[s] > 0) {
        put16(sec + o, freq[s]);
        o += 2;
      }
    for (int64_t q = 0; q < w; ++q) put16(sec + o + 2 * q, words[q]);
    *stored = 0;
  } else {
    len = (int64_t)pad16(n_b);
    memset(sec, 0, (size_t)len);
    memcpy(sec, sym, n_b);
    *stored = 1;
  }
  free(sym);
  free(words);
  return len;
}

int64_t ref_compress(const void *in, uint64_t n, int dtype,
                     uint32_t block_bytes, uint8_t *out, uint64_t out_cap) {
  if (dtype < 0 || dtype > 4 || !valid_block_bytes(block_bytes)) return REF_EINVAL;
  uint32_t E = elem_bytes(dtype);
  uint64_t be = block_bytes / E;
  uint64_t nb = (n + be - 1) / be;
  if (nb >= 0x80000000ull) return REF_EINVAL;
  if (out_cap < ref_max_compressed_size(dtype, n, block_bytes)) return REF_ENOSPC;
  uint64_t raw_off = raw_offset(nb), coded_off = coded_offset(dtype, n, nb);
  memset(out, 0, (size_t)coded_off);

  /* raw (uncompressed) plane */
  for (uint64_t i = 0; i < n; ++i) {
    uint32_t s, raw;
    ref_split_word(dtype, load_elem(in, dtype, i), &s, &raw);
    for (uint32_t q = 0; q + 1 < E; ++q)
      out[raw_off + (uint64_t)(E - 1) * i + q] = (uint8_t)(raw >> (8 * q));
  }
  /* block sections, concatenated (Step 3) */
  uint64_t off = 0;
  for (uint64_t b = 0; b < nb; ++b) {
    int stored = 0;
    int64_t len = ref_block_section(in, n, dtype, block_bytes, b, out + coded_off + off,
                                    out_cap - coded_off - off, &stored);
    if (len < 0) return len;
    off += (uint64_t)len;
    put32(out + HEADER_BYTES + 4 * b, (stored ? 0x80000000u : 0u) | (uint32_t)(off / 16));
  }
  uint64_t total = coded_off + off;
  put32(out + 0, MAGIC);
  out[4] = 1;
  out[5] = (uint8_t)dtype;
  out[6] = (uint8_t)PROB_BITS;
  out[7] = 0;
  put32(out + 8, (uint32_t)be);
  put32(out + 12, (uint32_t)nb);
  put64(out + 16, n);
  put64(out + 24, total);
  return (int64_t)total;
}

int ref_decompress(const uint8_t *in, uint64_t in_bytes, int dtype, uint64_t n,
                   void *out) {
  if (in_bytes < HEADER_BYTES) return REF_ECORRUPT;
  if (get32(in) != MAGIC || in[4] != 1 || in[5] != dtype || in[6] != PROB_BITS || in[7] != 0)
    return REF_ECORRUPT;
  uint32_t E = elem_bytes(dtype);
  uint64_t be = get32(in + 8), nb = get32(in + 12);
  if (get64(in + 16) != n || be == 0 || !valid_block_bytes((uint32_t)(be * E)))
    return REF_ECORRUPT;
  if (nb != (n + be - 1) / be) return REF_ECORRUPT;
  uint64_t total = get64(in + 24);
  uint64_t raw_off = raw_offset(nb), coded_off = coded_offset(dtype, n, nb);
  if (total > in_bytes || total < coded_off) return REF_ECORRUPT;

  uint8_t *sym = (uint8_t *)malloc(be ? be : 1);
  uint64_t start = 0;
  int rc = 0;
  for (uint64_t b = 0; b < nb && rc == 0; ++b) {
    uint32_t d = get32(in + HEADER_BYTES + 4 * b);
    uint64_t end = 16ull * (d & 0x7FFFFFFFu);
    if (end < start || coded_off + end > total) {
      rc = REF_ECORRUPT;
      break;
    }
    const uint8_t *sec = in + coded_off + start;
    uint64_t len = end - start;
    uint64_t lo = b * be;
    uint32_t n_b = (uint32_t)((lo + be < n ? lo + be : n) - lo);
    if (d & 0x80000000u) {
      if (len < n_b) {
        rc = REF_ECORRUPT;
        break;
      }
      memcpy(sym, sec, n_b);
    } else {
      if (len < SECTION_FIXED) {
        rc = REF_ECORRUPT;
        break;
      }
      uint32_t state[LANES], freq[256], cum[256];
      for (uint32_t j = 0; j < LANES; ++j) state[j] = get32(sec + 4 * j);
      uint32_t k = 0;
      for (int s = 0; s < 256; ++s)
        if (sec[256 + s / 8] & (1u << (s % 8))) ++k;
      if (k == 0 || len < SECTION_FIXED + 2ull * k) {
        rc = REF_ECORRUPT;
        break;
      }
      uint64_t o = SECTION_FIXED, sum = 0;
      for (int s = 0; s < 256; ++s) {
        if (sec[256 + s / 8] & (1u << (s % 8))) {
          freq[s] = get16(sec + o);
          o += 2;
          if (freq[s] == 0) rc = REF_ECORRUPT;
        } else {
          freq[s] = 0;
        }
        sum += freq[s];
      }
      if (rc != 0 || sum != M_TOTAL) {
        rc = REF_ECORRUPT;
        break;
      }
      uint32_t run = 0;
      for (int s = 0; s < 256; ++s) {
        cum[s] = run;
        run += freq[s];
      }
      uint64_t n_words = (len - o) / 2;
      uint16_t *words = (uint16_t *)malloc((size_t)(n_words + 1) * sizeof(uint16_t));
      for (uint64_t q = 0; q < n_words; ++q) words[q] = (uint16_t)get16(sec + o + 2 * q);
      int64_t used = ref_rans_decode(state, words, n_words, freq, cum, n_b, sym);
      free(words);
      if (used < 0) {
        rc = REF_ECORRUPT;
        break;
      }
    }
    for (uint32_t i = 0; i < n_b; ++i) {
      uint32_t raw = 0;
      for (uint32_t q = 0; q + 1 < E; ++q)
        raw |= (uint32_t)in[raw_off + (uint64_t)(E - 1) * (lo + i) + q] << (8 * q);
      store_elem(out, dtype, lo + i, ref_merge_word(dtype, sym[i], raw));
    }
    start = end;
  }
  if (rc == 0 && coded_off + start != total) rc = REF_ECORRUPT;
  free(sym);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Stream-wide tables (sections 3.3.1 and 3.4)                         */
/* ------------------------------------------------------------------ */
#define SAMPLE_BYTES 262144u
#define SHARED_SECTION_FIXED 256u /* 64 states */

void ref_build_table_all(const uint32_t *count, uint64_t n_s, uint32_t *freq) {
  if (n_s == 0) {
    for (int s = 0; s < 256; ++s) freq[s] = M_TOTAL / 256u;
    return;
  }
  uint32_t total = 0;
  for (int s = 0; s < 256; ++s) {
    freq[s] = 1u + (uint32_t)(((uint64_t)count[s] * (M_TOTAL - 256u)) / n_s);
    total += freq[s];
  }
  int best = 0;
  for (int s = 1; s < 256; ++s)
    if (count[s] > count[best]) best = s;
  freq[best] += M_TOTAL - total;
}

void ref_sampled_table(const void *in, uint64_t n, int dtype, uint32_t *freq) {
  uint64_t n_s = SAMPLE_BYTES / elem_bytes(dtype);
  if (n_s > n) n_s = n;
  uint32_t count[256] = {0};
  for (uint64_t i = 0; i < n_s; ++i) {
    uint32_t s, raw;
    ref_split_word(dtype, load_elem(in, dtype, i), &s, &raw);
    count[s] += 1;
  }
  ref_build_table_all(count, n_s, freq);
}

static int table_ok(const uint32_t *freq) {
  uint32_t sum = 0;
  for (int s = 0; s < 256; ++s) {
    if (freq[s] == 0 || freq[s] > M_TOTAL) return 0;
    sum += freq[s];
  }
  return sum == M_TOTAL;
}

static uint64_t table_bytes(int mode, uint64_t nb) {
  return (mode == REF_TABLE_SAMPLED && nb > 0) ? REF_TABLE_BYTES : 0;
}

uint64_t ref_max_compressed_size_mode(int dtype, uint64_t n, uint32_t block_bytes, int mode) {
  uint64_t be = block_bytes / elem_bytes(dtype);
  return ref_max_compressed_size(dtype, n, block_bytes) + table_bytes(mode, (n + be - 1) / be);
}

/* one block's section under a stream-wide table */
static int64_t shared_block_section(const void *in, uint64_t n, int dtype, uint64_t be, uint64_t b,
                                    const uint32_t *freq, const uint32_t *cum, uint8_t *sec,
                                    int *stored) {
  uint64_t lo = b * be;
  uint32_t n_b = (uint32_t)((lo + be < n ? lo + be : n) - lo);
  uint8_t *sym = (uint8_t *)malloc(n_b);
  uint16_t *words = (uint16_t *)malloc((size_t)n_b * sizeof(uint16_t) + 16);
  uint32_t state[LANES];
  for (uint32_t i = 0; i < n_b; ++i) {
    uint32_t s, raw;
    ref_split_word(dtype, load_elem(in, dtype, lo + i), &s, &raw);
    sym[i] = (uint8_t)s;
  }
  int64_t w = ref_rans_encode(sym, n_b, freq, cum, state, words, n_b);
  uint64_t coded_len = SHARED_SECTION_FIXED + (w < 0 ? 2u * (uint64_t)n_b : 2u * (uint64_t)w);
  int64_t len;
  if (w >= 0 && coded_len < n_b) {
    len = (int64_t)pad16(coded_len);
    memset(sec, 0, (size_t)len);
    for (uint32_t j = 0; j < LANES; ++j) put32(sec + 4 * j, state[j]);
    for (int64_t q = 0; q < w; ++q) put16(sec + SHARED_SECTION_FIXED + 2 * q, words[q]);
    *stored = 0;
  } else {
    len = (int64_t)pad16(n_b);
    memset(sec, 0, (size_t)len);
    memcpy(sec, sym, n_b);
    *stored = 1;
  }
  free(sym);
  free(words);
  return len;
}

int64_t ref_compress_table(const void *in, uint64_t n, int dtype, uint32_t block_bytes,
                           int mode, const uint16_t *table, uint8_t *out, uint64_t out_cap) {
  if (mode == REF_TABLE_PER_BLOCK) return ref_compress(in, n, dtype, block_bytes, out, out_cap);
  if (dtype < 0 || dtype > 4 || !valid_block_bytes(block_bytes)) return REF_EINVAL;
  if (mode != REF_TABLE_SAMPLED && mode != REF_TABLE_EXTERNAL) return REF_EINVAL;
  uint32_t E = elem_bytes(dtype);
  uint64_t be = block_bytes / E;
  uint64_t nb = (n + be - 1) / be;
  if (nb >= 0x80000000ull) return REF_EINVAL;
  if (out_cap < ref_max_compressed_size_mode(dtype, n, block_bytes, mode)) return REF_ENOSPC;
  uint32_t freq[256], cum[256];
  if (mode == REF_TABLE_SAMPLED) {
    ref_sampled_table(in, n, dtype, freq);
  } else {
    if (table == NULL) return REF_EINVAL;
    for (int s = 0; s < 256; ++s) freq[s] = table[s];
    if (!table_ok(freq)) return REF_EINVAL;
  }
  uint32_t run = 0;
  for (int s = 0; s < 256; ++s) {
    cum[s] = run;
    run += freq[s];
  }
  uint64_t table_off = raw_offset(nb);
  uint64_t raw_off = table_off + table_bytes(mode, nb);
  uint64_t coded_off = raw_off + pad16((uint64_t)(E - 1) * n);
  memset(out, 0, (size_t)coded_off);
  if (table_bytes(mode, nb))
    for (int s = 0; s < 256; ++s) put16(out + table_off + 2 * s, freq[s]);
  for (uint64_t i = 0; i < n; ++i) {
    uint32_t s, raw;
    ref_split_word(dtype, load_elem(in, dtype, i), &s, &raw);
    for (uint32_t q = 0; q + 1 < E; ++q)
      out[raw_off + (uint64_t)(E - 1) * i + q] = (uint8_t)(raw >> (8 * q));
  }
  uint64_t off = 0;
  for (uint64_t b = 0; b < nb; ++b) {
    int stored = 0;
    int64_t len = shared_block_section(in, n, dtype, be, b, freq, cum, out + coded_off + off, &stored);
    off += (uint64_t)len;
    put32(out + HEADER_BYTES + 4 * b, (stored ? 0x80000000u : 0u) | (uint32_t)(off / 16));
  }
  uint64_t total = coded_off + off;
  put32(out + 0, MAGIC);
  out[4] = 1;
  out[5] = (uint8_t)dtype;
  out[6] = (uint8_t)PROB_BITS;
  out[7] = (uint8_t)mode;
  put32(out + 8, (uint32_t)be);
  put32(out + 12, (uint32_t)nb);
  put64(out + 16, n);
  put64(out + 24, total);
  return (int64_t)total;
}

int ref_decompress_table(const uint8_t *in, uint64_t in_bytes, int dtype, uint64_t n,
                         const uint16_t *table, void *out) {
  if (in_bytes < HEADER_BYTES) return REF_ECORRUPT;
  int mode = in[7];
  if (mode == REF_TABLE_PER_BLOCK) return ref_decompress(in, in_bytes, dtype, n, out);
  if (mode != REF_TABLE_SAMPLED && mode != REF_TABLE_EXTERNAL) return REF_ECORRUPT;
  if (mode == REF_TABLE_EXTERNAL && table == NULL) return REF_EINVAL;
  if (get32(in) != MAGIC || in[4] != 1 || in[5] != dtype || in[6] != PROB_BITS) return REF_ECORRUPT;
  uint32_t E = elem_bytes(dtype);
  uint64_t be = get32(in + 8), nb = get32(in + 12);
  if (get64(in + 16) != n || be == 0 || !valid_block_bytes((uint32_t)(be * E))) return REF_ECORRUPT;
  if (nb != (n + be - 1) / be) return REF_ECORRUPT;
  uint64_t total = get64(in + 24);
  uint64_t table_off = raw_offset(nb);
  uint64_t raw_off = table_off + table_bytes(mode, nb);
  uint64_t coded_off = raw_off + pad16((uint64_t)(E - 1) * n);
  if (total > in_bytes || total < coded_off) return REF_ECORRUPT;
  uint32_t freq[256], cum[256];
  for (int s = 0; s < 256; ++s)
    freq[s] = mode == REF_TABLE_SAMPLED ? (nb > 0 ? get16(in + table_off + 2 * s) : M_TOTAL / 256u)
                                        : table[s];
  if (!table_ok(freq)) return mode == REF_TABLE_SAMPLED ? REF_ECORRUPT : REF_EINVAL;
  uint32_t run = 0;
  for (int s = 0; s < 256; ++s) {
    cum[s] = run;
    run += freq[s];
  }
  uint8_t *sym = (uint8_t *)malloc(be ? be : 1);
  uint64_t start = 0;
  int rc = 0;
  for (uint64_t b = 0; b < nb && rc == 0; ++b) {
    uint32_t d = get32(in + HEADER_BYTES + 4 * b);
    uint64_t end = 16ull * (d & 0x7FFFFFFFu);
    if (end < start || coded_off + end > total) {
      rc = REF_ECORRUPT;
      break;
    }
    const uint8_t *sec = in + coded_off + start;
    uint64_t len = end - start;
    uint64_t lo = b * be;
    uint32_t n_b = (uint32_t)((lo + be < n ? lo + be : n) - lo);
    if (d & 0x80000000u) {
      if (len < n_b) {
        rc = REF_ECORRUPT;
        break;
      }
      memcpy(sym, sec, n_b);
    } else {
      if (len < SHARED_SECTION_FIXED) {
        rc = REF_ECORRUPT;
        break;
      }
      uint32_t state[LANES];
      for (uint32_t j = 0; j < LANES; ++j) state[j] = get32(sec + 4 * j);
      uint64_t n_words = (len - SHARED_SECTION_FIXED) / 2;
      uint16_t *words = (uint16_t *)malloc((size_t)(n_words + 1) * sizeof(uint16_t));
      for (uint64_t q = 0; q < n_words; ++q) words[q] = (uint16_t)get16(sec + SHARED_SECTION_FIXED + 2 * q);
      int64_t used = ref_rans_decode(state, words, n_words, freq, cum, n_b, sym);
      free(words);
      if (used < 0) {
        rc = REF_ECORRUPT;
        break;
      }
    }
    for (uint32_t i = 0; i < n_b; ++i) {
      uint32_t raw = 0;
      for (uint32_t q = 0; q + 1 < E; ++q)
        raw |= (uint32_t)in[raw_off + (uint64_t)(E - 1) * (lo + i) + q] << (8 * q);
      store_elem(out, dtype, lo + i, ref_merge_word(dtype, sym[i], raw));
    }
    start = end;
  }
  if (rc == 0 && coded_off + start != total) rc = REF_ECORRUPT;
  free(sym);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Scalar conversions (IEEE binary16 / bfloat16 <-> binary32)          */
/* ------------------------------------------------------------------ */
float ref_half_to_float(uint32_t h) {
  uint32_t sign = (h >> 15) & 1u, e = (h >> 10) & 31u, m = h & 1023u;
  float v;
  if (e == 0)
    v = ldexpf((float)m, -24); /* zero or subnormal: m * 2^-24 */
  else if (e == 31)
    v = (m == 0) ? INFINITY : NAN;
  else
    v = ldexpf((float)(1024u + m), (int)e - 25); /* (1 + m/1024) 2^(e-15) */
  return sign ? -v : v;
}

/* round a non-negative double that holds an exact value to the nearest
 * integer, ties to even */
static double round_half_even(double v) {
  double fl = floor(v);
  double diff = v - fl;
  if (diff > 0.5) return fl + 1.0;
  if (diff < 0.5) return fl;
  return (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
}

uint32_t ref_float_to_half(float f) {
  if (isnan(f)) return 0x7E00u;
  uint32_t sign = signbit(f) ? 0x8000u : 0u;
  double a = fabs((double)f);
  if (a >= 65520.0) return sign | 0x7C00u; /* rounds past the largest finite half */
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: multiple of 2^-24 (1024 * 2^-24 becomes the smallest normal) */
    uint32_t m = (uint32_t)round_half_even(a * ldexp(1.0, 24));
    return sign | m;
  }
  int e2;
  (void)frexp(a, &e2); /* a = m * 2^e2, m in [0.5, 1): exponent of a is e2 - 1 */
  int e = e2 - 1;
  uint32_t mant = (uint32_t)round_half_even(ldexp(a, 10 - e)); /* in [1024, 2048] */
  if (mant == 2048u) {
    mant = 1024u;
    e += 1;
  }
  if (e + 15 >= 31) return sign | 0x7C00u;
  return sign | ((uint32_t)(e + 15) << 10) | (mant - 1024u);
}

float ref_bf16_to_float(uint32_t b) {
  uint32_t u = (b & 0xFFFFu) << 16; /* bfloat16 is the upper half of binary32 */
  float f;
  memcpy(&f, &u, 4);
  return f;
}

uint32_t ref_float_to_bf16(float f) {
  if (isnan(f)) return 0x7FC0u;
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t upper = u >> 16, lower = u & 0xFFFFu;
  if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;
  return upper;
}

static float elem_to_float(int dtype, uint32_t w) {
  if (dtype == REF_BF16) return ref_bf16_to_float(w);
  if (dtype == REF_FP16) return ref_half_to_float(w);
  float f;
  memcpy(&f, &w, 4);
  return f;
}

static uint32_t float_to_elem(int dtype, float f) {
  if (dtype == REF_BF16) return ref_float_to_bf16(f);
  if (dtype == REF_FP16) return ref_float_to_half(f);
  if (isnan(f)) return 0x7FC00000u;
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

/* ------------------------------------------------------------------ */
/* Fused reduce: decompress -> fixed-order binary32 sum -> recompress  */
/* ------------------------------------------------------------------ */
int64_t ref_reduce(const uint8_t *const *ins, const uint64_t *in_bytes,
                   int n_in, const void *local_raw, int dtype, uint64_t n,
                   uint32_t block_bytes, void *y, uint8_t *out,
                   uint64_t out_cap) {
  if (n_in < 1 || n_in > 16 || dtype < 0 || dtype > 2) return REF_EINVAL;
  uint32_t E = elem_bytes(dtype);
  void *x = malloc((size_t)(n ? n : 1) * E);
  float *acc = (float *)malloc((size_t)(n ? n : 1) * sizeof(float));
  for (int i = 0; i < n_in; ++i) {
    int rc = ref_decompress(ins[i], in_bytes[i], dtype, n, x);
    if (rc != 0) {
      free(x);
      free(acc);
      return rc;
    }
    for (uint64_t e = 0; e < n; ++e) {
      float v = elem_to_float(dtype, load_elem(x, dtype, e));
      acc[e] = (i == 0) ? v : acc[e] + v;
    }
  }
  if (local_raw != NULL)
    for (uint64_t e = 0; e < n; ++e) acc[e] = acc[e] + elem_to_float(dtype, load_elem(local_raw, dtype, e));
  for (uint64_t e = 0; e < n; ++e) store_elem(y, dtype, e, float_to_elem(dtype, acc[e]));
  free(x);
  free(acc);
  return ref_compress(y, n, dtype, block_bytes, out, out_cap);
}
