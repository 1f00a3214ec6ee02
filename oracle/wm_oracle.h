/*
 * wm_oracle.h -- plain CPU oracle for the exact-state mover's data path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link,
 * load or call this code; it exists so that tests, the smoke check and the
 * CPU-baseline leg of the benchmark can compare the HIP library against an
 * independent, slow, obviously-correct implementation.  It shares no source
 * with the HIP library: every constant below is restated here from the
 * written payload-format definition, not taken from the library's headers.
 *
 * Paper passages followed (arXiv 2607.10389):
 *   - Contract: the destination is bit-identical to the source or nothing is
 *     installed (§1 Introduction; §4 "Sufficiency": commit only on a
 *     byte-identical fingerprint).
 *   - Checksum: per-chunk CRC of the flattened state, the CRC being zlib's
 *     (§6.5 verification plane: "CPU-side zlib CRC"; hardware CRC is a fold
 *     "of the same polynomial"), per-chunk CRCs combined into one global CRC
 *     (§6.5; Appendix I "single global CRC").
 *   - Dirty set: chunks rewritten since the last shipped round (§6.2
 *     Exhibit 2 and Appendix H, iterative pre-copy).
 *   - Codec: lossless, bf16 exponent plane carries the redundancy, receipts
 *     bind to the decoded bytes so decode sits inside the verified envelope
 *     (§6.4 codec paragraph).  The paper fixes no codec format; the byte
 *     layout implemented here is this project's payload format v1.
 *   - Shadow slot, verify, then commit or roll back (Table 1, session API).
 *   - Flatten and rehydrate: the mover works on one flat buffer made from the
 *     session's manifest of leaves, flattened before the move and rehydrated
 *     after it (§4 "Sufficiency"; §5 "Implementation": 450 leaves).  The
 *     paper fixes no flat layout; this project's layout places leaf i at the
 *     sum of the earlier leaves' sizes, each rounded up to 16 bytes, with
 *     zero bytes in the gaps.
 *
 * Functions return plain integers; no function allocates memory visible to
 * the caller.  Buffers are host memory owned by the caller.
 */
#ifndef WM_ORACLE_H
#define WM_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* CRC kinds */
#define ORC_CRC32_ZLIB 0 /* reflected 0xEDB88320, init/xorout 0xFFFFFFFF */
#define ORC_CRC32C 1     /* reflected 0x82F63B78, init/xorout 0xFFFFFFFF */

/* verdict bits */
#define ORC_V_HEADER 1u   /* header rejected (nothing else examined) */
#define ORC_V_TABLE 2u    /* table rejected (records not examined) */
#define ORC_V_RECORD 4u   /* a record's structure is invalid */
#define ORC_V_DATA 8u     /* a decoded chunk's CRC differs from its receipt */
#define ORC_V_STAGING 16u /* receiver staging too small for the records */
#define ORC_V_REVERIFY 32u /* re-verifying install: a staged record or the
                              resulting state's global CRC disagrees */

/* CRC by its definition: one bit at a time. */
uint32_t orc_crc_bitwise(int kind, const uint8_t *p, uint64_t n);
/* Same function, one byte at a time through a 256-entry table that is
 * derived from the bitwise step (Sarwate's method). */
uint32_t orc_crc(int kind, const uint8_t *p, uint64_t n);

/* Per-chunk CRCs over chunks of chunk_bytes (last chunk may be short) and
 * the CRC of the whole buffer (global_out may be NULL). */
int orc_checksum_chunks(int kind, const uint8_t *data, uint64_t nbytes,
                        uint32_t chunk_bytes, uint32_t *crc_out,
                        uint32_t *global_out, int threads);

/* Ascending indices of chunks whose bytes differ; returns the count. */
uint32_t orc_diff_dirty(const uint8_t *cur, const uint8_t *prev,
                        uint64_t nbytes, uint32_t chunk_bytes,
                        uint32_t *idx_out, int threads);

/* Upper bound on the payload size when n_ship chunks are shipped (each
 * chunk above 64 KiB as its 64 KiB tiles, one record per tile). */
uint64_t orc_payload_bound(uint64_t nbytes, uint32_t chunk_bytes,
                           uint32_t n_ship);

/* Encode the chunks listed in idx (ascending; idx == NULL means every chunk,
 * which also sets the FULL flag) into payload.  Returns payload bytes, or
 * -1 on invalid arguments, -2 when cap is too small. */
int64_t orc_encode(int kind, const uint8_t *state, uint64_t nbytes,
                   uint32_t chunk_bytes, const uint32_t *idx, uint32_t n_idx,
                   uint8_t *payload, uint64_t cap, int threads);

/* Formats v2 and v3 (codecs 2 and 3, chunks of 64 KiB or more): as
 * orc_encode with records RAW or HUF (a per-chunk canonical Huffman code of
 * one byte plane in 512 streams, the other plane raw): v2 codes the
 * exponents, v3 the high bytes (the bf16 byte-plane split).  orc_encode is
 * orc_encode_codec with codec 1. */
#define ORC_HUF_MAX_LEN 11u
int64_t orc_encode_codec(int kind, int codec, const uint8_t *state,
                         uint64_t nbytes, uint32_t chunk_bytes,
                         const uint32_t *idx, uint32_t n_idx, uint8_t *payload,
                         uint64_t cap, int threads);

/* Huffman code lengths (at most ORC_HUF_MAX_LEN) of 256 symbol counts;
 * returns the longest (0 when at most one symbol occurs). */
uint32_t orc_huffman_lengths(const uint32_t *count, uint8_t *len);

/* Plan of one v2 record: mode (0 RAW, 2 HUF), k (longest code length),
 * base (the only exponent when k = 0), n_sb (stream bytes), size. */
int orc_plan_chunk_v2(const uint8_t *chunk, uint32_t len, uint32_t *mode,
                      uint32_t *k, uint32_t *base, uint32_t *n_sb,
                      uint64_t *size);
/* The same for codec 2 or 3 (base: the only coded-plane symbol). */
int orc_plan_chunk_huf(int codec, const uint8_t *chunk, uint32_t len,
                       uint32_t *mode, uint32_t *k, uint32_t *base,
                       uint32_t *n_sb, uint64_t *size);

/* Plan of one chunk's record (exposed for tests): mode, k, base, n_esc and
 * record size in bytes. */
int orc_plan_chunk(const uint8_t *chunk, uint32_t len, uint32_t *mode,
                   uint32_t *k, uint32_t *base, uint32_t *n_esc,
                   uint64_t *size);

/* Validate and decode a payload into staging (record i at i*unit, the unit
 * being the chunk up to 64 KiB and a 64 KiB tile of a larger chunk).
 * rec_status (may be NULL) receives 0, ORC_V_RECORD or ORC_V_DATA per
 * record when the header and table are valid.  Returns the verdict. */
uint32_t orc_decode_verify(int kind, const uint8_t *payload, uint64_t cap,
                           uint64_t nbytes, uint32_t chunk_bytes,
                           uint8_t *staging, uint64_t staging_cap,
                           uint32_t *rec_status, uint32_t n_status,
                           int threads);

/* orc_decode_verify for either format (codec 1 or 2). */
uint32_t orc_decode_verify_codec(int kind, int codec, const uint8_t *payload,
                                 uint64_t cap, uint64_t nbytes,
                                 uint32_t chunk_bytes, uint8_t *staging,
                                 uint64_t staging_cap, uint32_t *rec_status,
                                 uint32_t n_status, int threads);

/* Install: verdict 0 copies each staged record to its unit of live and
 * returns 0; any other verdict leaves live untouched and returns 1. */
int orc_commit(uint8_t *live, uint64_t nbytes, uint32_t chunk_bytes,
               const uint8_t *staging, const uint8_t *payload,
               uint32_t verdict);

/* Re-verifying install: with verdict 0, re-checks every staged record
 * against its receipt and the CRC of the state the install would produce
 * against the header's global CRC; installs only if both hold.  Returns
 * the given verdict if nonzero, else 0 (installed) or ORC_V_REVERIFY (live
 * untouched). */
uint32_t orc_commit_reverify(int kind, uint8_t *live, uint64_t nbytes,
                             uint32_t chunk_bytes, const uint8_t *staging,
                             const uint8_t *payload, uint32_t verdict);

/* Flat layout of a manifest of n leaves of bytes[i] bytes: writes each
 * leaf's offset into off (n entries) and returns the flat size. */
uint64_t orc_flat_layout(const uint64_t *bytes, uint32_t n, uint64_t *off);

/* Flatten: copy leaf i to flat + off_i and zero the gap bytes after it.
 * flat holds orc_flat_layout()'s size. */
void orc_flatten(const uint8_t *const *leaves, const uint64_t *bytes,
                 uint32_t n, uint8_t *flat);

/* Rehydrate: copy flat + off_i back into leaf i (gap bytes are not read). */
void orc_rehydrate(const uint8_t *flat, uint8_t *const *leaves,
                   const uint64_t *bytes, uint32_t n);

#ifdef __cplusplus
}
#endif
#endif
