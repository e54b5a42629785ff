/*
 * uzip_ref.h -- CPU oracle for the block-wise lossless float codec.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, scalar C reading of the
 * codec that exists to check the GPU library byte for byte.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it.
 * It shares no code, header, table or constant with the GPU library.
 *
 * What it computes (the paper's method, section 2.1.2 "GPU compression
 * algorithm for floating-point tensors" and section 3.3.1 "Localized
 * frequency tables"):
 *   - Step 1: split every value into its exponent byte (the "compressed
 *     part", one 8-bit symbol per value) and its sign+fraction bits (the
 *     "uncompressed part"), written to two separate planes.
 *   - a frequency table per block, built from that block's own symbols and
 *     used for both directions (localized tables instead of one global one);
 *   - Step 2: ANS coding of each block's symbols, independently per block;
 *   - Step 3: the variable-length block outputs concatenated into one
 *     contiguous stream;
 *   - metadata carrying dtype and sizes (section 4.1, P2P implementation);
 *   - the fused reduce of section 3.4: decompress each input, add in a fixed
 *     order in binary32, round to the storage type, compress again.
 * Where the paper leaves the bit-level encoding open, the reading written
 * out in uzip_ref.c is used (rotate-by-one byte planes, rANS with 64
 * interleaved states, an 11-bit table, a 32-byte header, per-block STORED
 * fallback).
 */
#ifndef UZIP_REF_H
#define UZIP_REF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* dtype codes used by the stream header.  The two FP8 formats (section
 * 4.1) are coded as pairs: one codec element is a 16-bit unit holding two
 * consecutive FP8 values (the first in the low byte), and element counts
 * of FP8 streams count pairs. */
#define REF_BF16 0
#define REF_FP16 1
#define REF_FP32 2
#define REF_E4M3FN 3
#define REF_E5M2 4

/* error codes (negative returns) */
#define REF_EINVAL (-1)
#define REF_ENOSPC (-2)
#define REF_ECORRUPT (-3)

/* ---- single-element transform (Step 1 split) ---- */
void ref_split_word(int dtype, uint32_t w, uint32_t *sym, uint32_t *raw);
uint32_t ref_merge_word(int dtype, uint32_t sym, uint32_t raw);

/* ---- per-block frequency table ---- */
/* count[256] -> freq[256] (sums to 2048) and cum[256]; n_b = sum(count) */
void ref_build_table(const uint32_t *count, uint32_t n_b, uint32_t *freq,
                     uint32_t *cum);

/* ---- rANS coding of one block of symbols ----
 * Encode: returns the number of 16-bit words W written to words[0..W) in
 * decode order, or -1 if more than max_words would be needed.  state[64]
 * receives the final encoder states. */
int64_t ref_rans_encode(const uint8_t *sym, uint32_t n_b, const uint32_t *freq,
                        const uint32_t *cum, uint32_t *state, uint16_t *words,
                        uint64_t max_words);
/* Decode: returns the number of words consumed, or REF_ECORRUPT. */
int64_t ref_rans_decode(const uint32_t *state_in, const uint16_t *words,
                        uint64_t n_words, const uint32_t *freq,
                        const uint32_t *cum, uint32_t n_b, uint8_t *sym_out);

/* ---- whole streams ---- */
uint64_t ref_max_compressed_size(int dtype, uint64_t n, uint32_t block_bytes);
/* One block's section: writes it to sec (capacity sec_cap, at least
 * pad16(n_b) bytes), returns its length and sets *stored. */
int64_t ref_block_section(const void *in, uint64_t n, int dtype,
                          uint32_t block_bytes, uint64_t b, uint8_t *sec,
                          uint64_t sec_cap, int *stored);
/* Returns total stream bytes or a negative error. */
int64_t ref_compress(const void *in, uint64_t n, int dtype,
                     uint32_t block_bytes, uint8_t *out, uint64_t out_cap);
/* Returns 0 or a negative error. */
int ref_decompress(const uint8_t *in, uint64_t in_bytes, int dtype, uint64_t n,
                   void *out);

/* ---- stream-wide tables (sections 3.3.1 and 3.4) ----
 * Table modes: REF_TABLE_PER_BLOCK is the stream above.  REF_TABLE_SAMPLED
 * builds one table for the whole stream from its first
 * min(n, 262144 / E) elements (the first 256 KiB) and stores it once, after
 * the directory.  REF_TABLE_EXTERNAL codes with a table the caller holds
 * (built once, reused across calls) and leaves it out of the stream.
 * A stream-wide table gives every one of the 256 symbols a frequency of
 * at least 1, so symbols outside the sample stay codable. */
#define REF_TABLE_PER_BLOCK 0
#define REF_TABLE_SAMPLED 1
#define REF_TABLE_EXTERNAL 2
#define REF_TABLE_BYTES 512u
/* freq[256] of the sampled table of the first min(n, 262144 / E) elements
 * (sums to 2048, every entry >= 1) */
void ref_sampled_table(const void *in, uint64_t n, int dtype, uint32_t *freq);
/* counts[256] over n_s symbols -> all-symbol table freq[256] */
void ref_build_table_all(const uint32_t *count, uint64_t n_s, uint32_t *freq);
/* largest stream of a mode (SAMPLED adds the table) */
uint64_t ref_max_compressed_size_mode(int dtype, uint64_t n, uint32_t block_bytes, int mode);
/* table: freq[256] as u16, required for EXTERNAL (ignored otherwise).
 * Returns total stream bytes or a negative error. */
int64_t ref_compress_table(const void *in, uint64_t n, int dtype, uint32_t block_bytes,
                           int mode, const uint16_t *table, uint8_t *out, uint64_t out_cap);
/* Decodes any mode; table is required for EXTERNAL streams. */
int ref_decompress_table(const uint8_t *in, uint64_t in_bytes, int dtype, uint64_t n,
                         const uint16_t *table, void *out);

/* ---- fused reduce (section 3.4) ----
 * ins[i] are n_in streams of the same dtype, n and block size.  local_raw
 * (may be NULL) is an uncompressed addend taken last.  y (n elements of
 * dtype) receives the reduced tensor; out receives compress(y).  Returns the
 * output stream size or a negative error. */
int64_t ref_reduce(const uint8_t *const *ins, const uint64_t *in_bytes,
                   int n_in, const void *local_raw, int dtype, uint64_t n,
                   uint32_t block_bytes, void *y, uint8_t *out,
                   uint64_t out_cap);

/* scalar conversions used by the reduce, exposed for their own checks */
float ref_half_to_float(uint32_t h);
uint32_t ref_float_to_half(float f);
float ref_bf16_to_float(uint32_t b);
uint32_t ref_float_to_bf16(float f);

#ifdef __cplusplus
}
#endif
#endif
