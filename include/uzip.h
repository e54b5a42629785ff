/*
 * uzip.h -- C ABI of the MI355X (gfx950) block-wise lossless float codec.
 *
 * The operation is the lossless compression that UCCL-Zip places inside
 * GPU communication (arXiv 2604.17172):
 *   - section 2.1.2: every value is split into its exponent byte (the
 *     "compressed part") and its sign+fraction bits (the "uncompressed
 *     part"); the exponent bytes are ANS-coded block by block and the
 *     variable-length block outputs are concatenated into one stream;
 *   - section 3.3.1: each block codes with its own frequency table built
 *     from its own data (localized tables), in one fused launch with no
 *     third coalescing pass;
 *   - section 3.2.3: split-send -- the uncompressed part is final right
 *     after the split and may be sent before coding finishes;
 *   - section 3.4: the per-hop step of a compressed all-reduce:
 *     decompress, reduce, recompress;
 *   - section 4.1: the metadata carries dtype and the sizes before and
 *     after compression.
 *
 * Stream layout (little-endian; pad16(x) rounds x up to a multiple of 16,
 * padding bytes are zero):
 *     0  u32 magic 0x31505A55   4 u8 version = 1   5 u8 dtype
 *     6  u8 prob_bits = 11      7 u8 flags = the table mode (0 for a table
 *                                 per block; 1, 2: see uzip_table_mode)
 *     8  u32 block_elems       12 u32 n_blocks
 *    16  u64 n_elems           24 u64 total_bytes
 *    32  u32 dir[n_blocks]: bit 31 = STORED, bits 30..0 = end offset of
 *        the block's section within the coded plane, in 16-byte units
 *    raw plane at 32 + pad16(4 n_blocks): (E-1) bytes per element, the low
 *        bytes of the value rotated left by one bit (sign in bit 0)
 *    coded plane at raw_off + pad16((E-1) n): one section per block
 *  A CODED section is u32 state[64] | u8 present[32] | u16 f[k] |
 *  u16 word[W] | pad; the 11-bit table f (sum 2048) comes from the
 *  block's histogram and the words are those of 64 interleaved rANS
 *  states (state interval [2^15, 2^31), 16-bit renormalisation, lane j
 *  codes elements 512 r + 8 j .. +7 of round r).  A block whose coded
 *  section would not be smaller than its n_b symbol bytes is STORED.
 *
 * Conventions for every call:
 *   - All buffers are caller-owned device memory (flags and chunk_sizes may
 *     also be host-mapped memory).  The library never allocates or frees.
 *   - Every call only checks its arguments on the host and enqueues work on
 *     the given stream; it returns before the GPU has run.  Results (and
 *     *d_status) are valid once the stream reaches that point.
 *   - Device pointers must be 16-byte aligned.
 *   - block_bytes is a power of two in [4096, 4194304] (4 KiB to 4 MiB).
 *   - n_elems <= 2^48 (else EINVAL; the size queries return 0).
 *   - Calls that overlap in time need separate workspaces.
 *   - Host-side errors are returned immediately and nothing is enqueued.
 *     Device-side errors (corrupt streams) are written to *d_status (the
 *     first error wins; the caller zeroes it before the call).  No call
 *     writes outside [d_out, d_out + out_cap) or its workspace.
 *   - Encoder failure.  The compressing calls place each block's section
 *     with a single-pass scan in which a block waits, for a bounded number
 *     of polls (2^22, a few seconds), for the sizes of earlier blocks that other
 *     workgroups are coding.  Such a wait always ends when the GPU runs
 *     the call alone; if it runs out (the GPU shared with work that holds
 *     its compute units for longer), the stream is marked invalid: its
 *     magic and its size (*d_out_size, chunk_sizes[c]) read 0 -- a valid
 *     stream is never shorter than its 32-byte header -- the split-send
 *     producer still raises the chunk's DONE flag (and its RAW_READY flag,
 *     had it not risen), and the fused reduce also sets *d_status to
 *     UZIP_ETIMEOUT.  The call may be repeated.
 */
#ifndef UZIP_H
#define UZIP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element types.  The FP8 formats (section 4.1) are coded in pairs: one
 * element is a 16-bit unit holding two FP8 values, the first in the low
 * byte, so for them n_elems counts pairs and an odd count of values is
 * padded by the caller.  Each value gives bits 6..3 (e4m3fn: the exponent;
 * e5m2: its top four exponent bits) to the unit's coded symbol and bit 7
 * with bits 2..0 to its raw byte.  The fused reduction takes bf16, fp16
 * and fp32 only. */
typedef enum {
  UZIP_BF16 = 0,
  UZIP_FP16 = 1,
  UZIP_FP32 = 2,
  UZIP_E4M3FN = 3, /* pairs of float8 e4m3fn */
  UZIP_E5M2 = 4    /* pairs of float8 e5m2 */
} uzip_dtype;

typedef enum {
  UZIP_OK = 0,
  UZIP_EINVAL = -1,      /* bad argument (dtype, sizes, alignment, block size) */
  UZIP_ENOSPC = -2,      /* output capacity or workspace too small */
  UZIP_ECORRUPT = -3,    /* device status: stream corrupt or not matching the call */
  UZIP_EHIP = -4,        /* a HIP runtime call failed */
  UZIP_EUNSUPPORTED = -5, /* the device is not gfx950 */
  UZIP_ETIMEOUT = -6      /* device status: the encoder's bounded wait for an
                             earlier block's size ran out; the stream is invalid */
} uzip_status;

/* operation codes for uzip_workspace_size */
enum {
  UZIP_OP_COMPRESS = 0,
  UZIP_OP_DECOMPRESS = 1, /* also uzip_decompress_table */
  UZIP_OP_REDUCE = 2,
  UZIP_OP_CHUNKED = 3,
  UZIP_OP_COMPRESS_TABLE = 4,
  UZIP_OP_CHUNKED_TABLE = 5 /* aux = chunk_bytes */
};

/* Table modes (sections 3.3.1 and 3.4).  PER_BLOCK: every block carries
 * its own table (the plain stream).  SAMPLED: one table for the whole
 * stream, built from the symbols of its first 256 KiB (min(n, 262144 / E)
 * elements) and stored once after the directory.  EXTERNAL: the caller's
 * table (for example one uzip_build_table made in an earlier call) codes
 * every block and is not stored: section 3.4's table sent once and reused.
 * A stream-wide table is u16 f[256] (UZIP_TABLE_BYTES bytes) with every
 * f >= 1 and sum 2048: f[s] = 1 + floor(c[s] * 1792 / n_s) over the
 * sample's symbol counts c, the remainder to the most frequent symbol
 * (ties: the smallest), so a symbol the sample missed stays codable.  Its
 * sections hold the 64 states and the words only. */
typedef enum { UZIP_TABLE_PER_BLOCK = 0, UZIP_TABLE_SAMPLED = 1, UZIP_TABLE_EXTERNAL = 2 } uzip_table_mode;
#define UZIP_TABLE_BYTES 512

/* Largest possible stream for n_elems values (every block STORED), in
 * bytes.  Section 4.1's "size after compression" never exceeds it.
 * Returns 0 for invalid arguments. */
size_t uzip_max_compressed_size(uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes);

/* Device workspace bytes that `op` needs (section 4.1 bounds the
 * compressor's footprint; this is ours).  For UZIP_OP_CHUNKED pass the
 * chunk size in `aux`; for UZIP_OP_REDUCE pass n_in in `aux` and add the
 * flag UZIP_WS_NO_OUT_RAW (1 << 16) when d_out_raw will be NULL.  Returns
 * 0 for invalid arguments (a zero-byte workspace is never valid for
 * COMPRESS, CHUNKED or REDUCE).  Blocks of more than 7424 words' worth of
 * coded output need an overflow slot of about block_bytes / E bytes for each
 * of up to 2048 workgroups (min(blocks, 2048) slots): e.g. 1 GiB of bf16 in
 * 4 MiB blocks, 256 slots of 2 MiB. */
#define UZIP_WS_NO_OUT_RAW (1u << 16)
size_t uzip_workspace_size(int op, uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes,
                           uint64_t aux);

/* Compress n_elems values at d_in (section 2.1.2 Steps 1-3 with the
 * localized tables of section 3.3.1, fused in one launch).
 *   d_out, out_cap: stream buffer, out_cap >= uzip_max_compressed_size.
 *   d_out_size:     device u64 receiving total_bytes (may be NULL).
 *   d_ws, ws_bytes: workspace of uzip_workspace_size(UZIP_OP_COMPRESS, ...).
 * Errors: EINVAL, ENOSPC, EHIP, EUNSUPPORTED. */
uzip_status uzip_compress(const void *d_in, uint64_t n_elems, uzip_dtype dtype,
                          uint32_t block_bytes, void *d_out, size_t out_cap,
                          uint64_t *d_out_size, void *d_ws, size_t ws_bytes,
                          hipStream_t stream);

/* Decompress a stream (the receiver side of sections 3.2 and 3.4).
 *   d_in, in_bytes: the stream (in_bytes >= its total_bytes).
 *   dtype, n_elems: what the caller expects; the header must agree.
 *   d_out, out_cap: n_elems values, out_cap >= n_elems * element size.
 *   d_status:       device u32, set to UZIP_ECORRUPT if the stream is
 *                   corrupt or does not match (may be NULL).
 *   d_ws, ws_bytes: ignored (the decoder keeps no state in a workspace;
 *                   uzip_workspace_size(UZIP_OP_DECOMPRESS, ...) is 256
 *                   bytes, reserved); may be NULL.
 * Errors: EINVAL, ENOSPC, EHIP, EUNSUPPORTED. */
uzip_status uzip_decompress(const void *d_in, size_t in_bytes, uzip_dtype dtype,
                            uint64_t n_elems, void *d_out, size_t out_cap,
                            uint32_t *d_status, void *d_ws, size_t ws_bytes,
                            hipStream_t stream);

/* The stream-wide table of a tensor (section 3.3.1): from the symbols of
 * its first min(n_elems, 262144 / E) elements, as UZIP_TABLE_SAMPLED builds
 * it.  d_table: UZIP_TABLE_BYTES of device memory, 16-byte aligned.
 * Errors: EINVAL, EHIP, EUNSUPPORTED. */
uzip_status uzip_build_table(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint16_t *d_table,
                             hipStream_t stream);

/* Compress with a table mode (sections 3.3.1 and 3.4).  As uzip_compress,
 * and:
 *   mode:           PER_BLOCK is uzip_compress itself.
 *   d_table:        EXTERNAL only: the table (u16 f[256], 16-byte aligned).
 *                   One that is not an all-symbol table (an f of 0, or a
 *                   sum other than 2048) codes nothing and *d_out_size
 *                   reads 0.
 *   out_cap:        >= uzip_max_compressed_size + UZIP_TABLE_BYTES.
 *   d_ws, ws_bytes: uzip_workspace_size(UZIP_OP_COMPRESS_TABLE, ...).
 * Errors: EINVAL, ENOSPC, EHIP, EUNSUPPORTED. */
uzip_status uzip_compress_table(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                uzip_table_mode mode, const uint16_t *d_table, void *d_out, size_t out_cap,
                                uint64_t *d_out_size, void *d_ws, size_t ws_bytes, hipStream_t stream);

/* The split-send producer (uzip_compress_chunked) with a table mode: with
 * SAMPLED every chunk's stream takes its own table from the chunk's first
 * 256 KiB (the analogue of section 3.3.1's table per CTA range) and stores
 * it; with EXTERNAL every chunk is coded with d_table.  slot_bytes >=
 * uzip_max_compressed_size(one chunk) + UZIP_TABLE_BYTES; workspace:
 * uzip_workspace_size(UZIP_OP_CHUNKED_TABLE, ..., chunk_bytes).  An
 * EXTERNAL table that is not an all-symbol table codes nothing: every
 * chunk is marked invalid as after an encoder failure (magic and size 0,
 * both flags raised).  Otherwise as uzip_compress_chunked
 * (PER_BLOCK is that call).  Each chunk decodes with
 * uzip_decompress_table, or a batch of chunks with
 * uzip_decompress_chunked_table. */
uzip_status uzip_compress_chunked_table(const void *d_in, uint64_t n_elems, uzip_dtype dtype, uint32_t block_bytes,
                                        uint64_t chunk_bytes, uzip_table_mode mode, const uint16_t *d_table,
                                        void *d_out, size_t slot_bytes, uint64_t *chunk_sizes, uint32_t *flags,
                                        uint32_t epoch, void *d_ws, size_t ws_bytes, hipStream_t stream);

/* Decompress a stream of mode SAMPLED or EXTERNAL (a PER_BLOCK stream, or
 * an EXTERNAL one without d_table, sets *d_status to UZIP_ECORRUPT; so
 * does a table that is not an all-symbol table).  d_table: the table the
 * stream was coded with (EXTERNAL; ignored for SAMPLED; may be NULL),
 * 16-byte aligned.  Otherwise as uzip_decompress. */
uzip_status uzip_decompress_table(const void *d_in, size_t in_bytes, uzip_dtype dtype, uint64_t n_elems,
                                  const uint16_t *d_table, void *d_out, size_t out_cap, uint32_t *d_status,
                                  void *d_ws, size_t ws_bytes, hipStream_t stream);

/* Receiver side of the split-send pipeline (section 3.2.3): decompress the
 * chunk streams c = first_chunk .. first_chunk + n_chunks - 1 of a tensor
 * of n_elems values cut into chunks of chunk_bytes, as the producer
 * (uzip_compress_chunked with the same dtype, block_bytes and chunk_bytes)
 * laid them out, in one launch: every block of every chosen chunk is
 * decoded at once, where one uzip_decompress call per chunk runs that
 * chunk's few blocks alone.  A receiver calls it on each batch of chunks
 * whose DONE flags it has seen.
 *   d_in, slot_bytes: chunk c's stream is at d_in + c * slot_bytes and fits
 *                     its slot (slot_bytes a multiple of 16).
 *   d_out, out_cap:   the whole tensor's buffer: chunk c's values go to
 *                     element offset c * chunk_bytes / element size, and
 *                     nothing else is written; out_cap covers the tensor
 *                     up to the end of the last chosen chunk.
 *   d_status:         as for uzip_decompress (one word for all chosen
 *                     chunks; the first error found wins).
 * n_chunks == 0 is a no-op.  Errors: EINVAL (bad sizes, a range past the
 * tensor's chunks), ENOSPC, EHIP, EUNSUPPORTED. */
uzip_status uzip_decompress_chunked(const void *d_in, size_t slot_bytes, uint64_t first_chunk, uint64_t n_chunks,
                                    uzip_dtype dtype, uint64_t n_elems, uint32_t block_bytes, uint64_t chunk_bytes,
                                    void *d_out, size_t out_cap, uint32_t *d_status, hipStream_t stream);

/* uzip_decompress_chunked for chunk streams of uzip_compress_chunked_table
 * (SAMPLED: each chunk's own stored table; EXTERNAL: d_table, the table
 * the chunks were coded with, 16-byte aligned).  d_table is ignored for
 * SAMPLED and may be NULL; a PER_BLOCK chunk stream is reported corrupt. */
uzip_status uzip_decompress_chunked_table(const void *d_in, size_t slot_bytes, uint64_t first_chunk,
                                          uint64_t n_chunks, uzip_dtype dtype, uint64_t n_elems,
                                          uint32_t block_bytes, uint64_t chunk_bytes, const uint16_t *d_table,
                                          void *d_out, size_t out_cap, uint32_t *d_status, hipStream_t stream);

/* Fused decompress -> reduce -> recompress of one rank's share (section
 * 3.4, the CopyReducePacks step with compression fused in).
 *   d_in[i], in_bytes[i] (host arrays of n_in entries, 1 <= n_in <= 16):
 *     streams of the same dtype, n_elems and block size.
 *   d_local_raw: uncompressed local addend, added last (may be NULL; the
 *     selective compression of section 3.4 leaves local data raw).
 *   The sum is taken element by element in IEEE binary32 in input order,
 *   acc = x_0, acc = acc + x_i, rounded to nearest even into dtype (NaN
 *   becomes the canonical quiet NaN), and compressed with block_bytes.
 *   d_out, out_cap, d_out_size: as for uzip_compress.
 *   d_out_raw: receives the reduced tensor (may be NULL).
 *   d_status: as for uzip_decompress.
 * Errors: EINVAL, ENOSPC, EHIP, EUNSUPPORTED. */
uzip_status uzip_reduce_fused(const void *const *d_in, const size_t *in_bytes, int n_in,
                              const void *d_local_raw, uzip_dtype dtype, uint64_t n_elems,
                              uint32_t block_bytes, void *d_out, size_t out_cap,
                              uint64_t *d_out_size, void *d_out_raw, uint32_t *d_status,
                              void *d_ws, size_t ws_bytes, hipStream_t stream);

/* uzip_compress for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the encoder's workspace is the library's own device scratch, a static
 * array of 64 MiB that every GPU the library runs on holds from the
 * library's first call on it until the process ends.  It holds the scan's
 * counters and status words (8 bytes per block) and as many overflow slots
 * as then fit (at most one per persistent workgroup; fewer only shrink the
 * grid).  Each call clears what must start at zero with a kernel of its own
 * (no memset).  Every call on one GPU shares that GPU's scratch: calls that
 * overlap in time on one GPU race, so callers order them (one stream, or
 * events).  The caller still provides d_in, d_out and d_out_size as for
 * uzip_compress, and the stream bytes are the same.  Allocates nothing.
 * Errors: EINVAL; ENOSPC (out_cap too small, or more than 4,194,304 blocks:
 * the scratch's limit); EHIP; EUNSUPPORTED. */
uzip_status uzip_compress_noalloc(const void *d_in, uint64_t n_elems, uzip_dtype dtype,
                                  uint32_t block_bytes, void *d_out, size_t out_cap,
                                  uint64_t *d_out_size, hipStream_t stream);

/* Split-send producer (section 3.2.3): the tensor is cut into chunks of
 * chunk_bytes (a multiple of block_bytes); chunk c is compressed as an
 * independent stream at d_out + c * slot_bytes, byte-identical to
 * uzip_compress of that slice.
 *   slot_bytes >= uzip_max_compressed_size(one full chunk).
 *   flags[2c]   is set to `epoch` once chunk c's raw plane is final
 *               (its offset is computable from dtype and the chunk size),
 *   chunk_sizes[c] receives the chunk's total_bytes, then
 *   flags[2c+1] is set to `epoch` once the whole chunk stream is final.
 *   Both are stored with system-scope release ordering, so host-mapped
 *   flags may be polled by a host thread.  Use a new epoch per call.
 * Errors: EINVAL, ENOSPC, EHIP, EUNSUPPORTED. */
uzip_status uzip_compress_chunked(const void *d_in, uint64_t n_elems, uzip_dtype dtype,
                                  uint32_t block_bytes, uint64_t chunk_bytes, void *d_out,
                                  size_t slot_bytes, uint64_t *chunk_sizes, uint32_t *flags,
                                  uint32_t epoch, void *d_ws, size_t ws_bytes,
                                  hipStream_t stream);

/* Static string naming a status code. */
const char *uzip_status_str(uzip_status status);

/* Fault injection, for tests of the encoder's failure path (see the
 * conventions above): calls enqueued after it bound the single-pass scan's
 * wait at spin_limit polls (0 restores the default, 2^22), and the block
 * with the global index held_block (counted over all chunks of a call;
 * UINT32_MAX: none) never publishes its size, so every later block of its
 * stream waits until its bound runs out and the stream is marked invalid
 * (and so is a stream whose block was taken by a workgroup held up in such
 * a wait, when its own later blocks run out of polls in turn); every kernel
 * still ends normally.  Process-wide; not for production use.
 * Errors: none (returns UZIP_OK). */
uzip_status uzip_inject_scan_stall(uint32_t spin_limit, uint32_t held_block);

#ifdef __cplusplus
}
#endif
#endif
