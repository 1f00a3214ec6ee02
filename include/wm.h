/*
 * wm.h -- C ABI of libwm, the exact-state mover's device hot path on MI355X.
 *
 * The library implements, for a flat multi-gigabyte bf16 state (an attention
 * KV cache) resident in device memory, the mover's data path from
 * arXiv 2607.10389 ("Stateful Worlds, Stateless Elasticity"):
 *
 *   source side       [wm_flatten] -> wm_checksum_chunks -> wm_diff_dirty
 *                     -> wm_encode (or the single-pass wm_encode_step)
 *   destination side  wm_decode_verify -> wm_commit_or_abort -> [wm_rehydrate]
 *
 * a receive that overlaps the payload's copy into device memory with its
 * decode (wm_receive_verify), and one round of iterative pre-copy built from
 * them (wm_precopy_round).
 *
 * under the paper's contract: the destination is bit-identical to the source
 * or nothing is installed (§1; §4 "Sufficiency": commit only on a
 * byte-identical fingerprint; Table 1: migrate stages into a shadow slot,
 * commit re-verifies then swaps, rollback drops the staged copy).
 *
 * Conventions for every call:
 *   - Buffer pointers are DEVICE pointers owned by the caller, unless a
 *     comment says "host".  The library never allocates, frees or keeps a
 *     pointer after returning.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls only enqueue work on it and return without waiting, except
 *     wm_commit_or_abort and wm_precopy_round, which wait for the stream.
 *   - Argument errors are detected on the host before anything is enqueued;
 *     the call then returns a negative status and writes nothing.
 *   - Problems found on the device (a malformed or corrupted payload) are
 *     never crashes: they become bits of the device verdict word.
 *   - Calls on different streams must use different workspaces; calls that
 *     share a workspace must be ordered (same stream).
 *   - Grids are sized to the CUs the stream may use: its CU mask when it was
 *     made with hipExtStreamCreateWithCUMask, every CU otherwise, so
 *     sessions on disjoint CU slices run side by side.
 *   - All functions are thread-safe.  The first call on a device uploads the
 *     library's constant CRC tables to it (wm_init does this eagerly).
 *   - Chunk sizes: chunk_bytes is a power of two in [4 KiB, 16 MiB]; the
 *     kernels take 64 KiB and above (smaller sizes return
 *     WM_ERR_UNSUPPORTED).  A chunk is the unit of dirtiness and of the
 *     per-chunk CRCs; a chunk above 64 KiB (the paper's pre-copy unit is
 *     4 MB, §6.2 Exhibit 2, App. H) is shipped as its 64 KiB tiles, one
 *     record and one receipt per tile, so "record" below means a 64 KiB
 *     unit: the chunk itself at 64 KiB, else one tile of it.  A table that
 *     ships only part of a chunk is rejected (WM_V_TABLE).
 */
#ifndef WM_H
#define WM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t wm_status;
#define WM_OK 0
#define WM_VERIFY_FAILED 1       /* verdict: nothing was installed */
#define WM_ERR_INVALID_ARG (-1)  /* null/misaligned pointer, bad size/param */
#define WM_ERR_CAPACITY (-2)     /* payload_cap below wm_payload_bound() */
#define WM_ERR_HIP (-3)          /* HIP runtime or launch failure */
#define WM_ERR_WORKSPACE (-4)    /* ws_bytes below wm_workspace_bytes() */
#define WM_ERR_UNSUPPORTED (-5)  /* valid but not implemented (chunk size) */

#define WM_CRC32_ZLIB 0 /* reflected 0xEDB88320, init/xorout 0xFFFFFFFF */
#define WM_CRC32C 1     /* reflected 0x82F63B78, init/xorout 0xFFFFFFFF */
/* Payload formats (codec ids).  EXPFOR, format v1: each chunk's exponents
 * as k-bit offsets from a base with escapes.  EXPHUF, format v2: each
 * chunk's exponents in the chunk's own canonical Huffman code (lengths at
 * most 11) in 512 streams, so that 512 decoders work side by side (§6.4: the
 * redundancy of a bf16 cache sits in its exponent plane, which the paper's
 * codec entropy-codes).  BYTEPLANE, format v3: the paper's bf16 byte-plane
 * split (§6.4 codec paragraph) in format v2's layout, the high byte (sign and
 * the exponent's upper seven bits) Huffman-coded and the low byte (the
 * exponent's lowest bit and the mantissa, close to 8 bits of entropy) raw.
 * All fall back to RAW per chunk.  Every call takes any format, except
 * wm_encode_step_static (format v1 only).  Formats v2 and v3 have no
 * single-pass encoder: their wm_encode_step runs the diff, a checksum of
 * every chunk and the list encoder (same outputs), and their pre-copy rounds
 * checksum every chunk. */
#define WM_CODEC_EXPFOR 1
#define WM_CODEC_EXPHUF 2
#define WM_CODEC_BYTEPLANE 3

/* Bits of the device verdict word written by wm_decode_verify. */
#define WM_V_HEADER 1u  /* header rejected; nothing else examined */
#define WM_V_TABLE 2u   /* record table rejected; records not examined */
#define WM_V_RECORD 4u  /* some record's structure is invalid */
#define WM_V_DATA 8u    /* some decoded chunk's CRC differs from its receipt */
#define WM_V_STAGING 16u /* staging_cap too small for the payload's records */
#define WM_V_REVERIFY 32u /* wm_commit_reverify: a staged record no longer
                             matches its receipt, or the installed state
                             would not have the source's global CRC */

/* wm_commit_or_abort modes */
#define WM_COMMIT_NONE 0    /* only read the verdict (full ship: caller swaps) */
#define WM_COMMIT_SCATTER 1 /* copy each staged record into its chunk of live */

typedef struct wm_params {
  uint32_t chunk_bytes; /* bytes per chunk: a power of two, 64 KiB..16 MiB */
  uint32_t crc_kind;    /* WM_CRC32_ZLIB or WM_CRC32C */
  uint32_t codec;       /* WM_CODEC_EXPFOR, WM_CODEC_EXPHUF or WM_CODEC_BYTEPLANE */
  uint32_t flags;       /* must be 0 */
} wm_params;

/* Human-readable name of a status code (static string; never NULL). */
const char *wm_status_str(wm_status s);

/* Upload the constant tables to `device` (the current HIP device if < 0).
 * Optional: every other call does it on first use. */
wm_status wm_init(int device);

/* Bytes of device workspace needed by wm_diff_dirty, wm_encode,
 * wm_encode_step and wm_decode_verify for a state of nbytes (formats v2 and v3 add
 * 692 bytes per chunk and a few hundred more: the record plans and a dirty
 * list).  0 if p is invalid. */
uint64_t wm_workspace_bytes(uint64_t nbytes, const wm_params *p);

/* Largest payload that shipping n_records chunks of a state of nbytes can
 * produce (header + every record RAW + table; a chunk above 64 KiB counts
 * as its tiles).  0 if p is invalid. */
uint64_t wm_payload_bound(uint64_t nbytes, uint32_t n_records,
                          const wm_params *p);

/* Per-chunk CRC of the flat state (§4 "Sufficiency"; §6.5: zlib's CRC per
 * chunk, chunk CRCs GF(2)-combined into one global CRC).
 *   data       : nbytes of state, 16-byte aligned; any nbytes (last chunk
 *                may be short)
 *   crc_out    : ceil(nbytes / chunk_bytes) u32, CRC of each chunk
 *   global_crc : 1 u32, CRC of the whole state, or NULL
 * No workspace.  Errors: WM_ERR_INVALID_ARG, WM_ERR_UNSUPPORTED, WM_ERR_HIP. */
wm_status wm_checksum_chunks(const void *data, uint64_t nbytes,
                             const wm_params *p, uint32_t *crc_out,
                             uint32_t *global_crc, void *stream);

/* Dirty chunks: those whose bytes differ between cur and prev (the last
 * shipped snapshot; §6.2 Exhibit 2 and App. H, iterative pre-copy).  A chunk
 * rewritten with identical bytes is clean.
 *   cur, prev  : nbytes each, 16-byte aligned
 *   dirty_idx  : ceil(nbytes / chunk_bytes) u32; receives the dirty chunk
 *                indices in ascending order
 *   n_dirty    : 1 u32, the number of dirty chunks
 *   ws         : workspace of ws_bytes >= wm_workspace_bytes() */
wm_status wm_diff_dirty(const void *cur, const void *prev, uint64_t nbytes,
                        const wm_params *p, uint32_t *dirty_idx,
                        uint32_t *n_dirty, void *ws, uint64_t ws_bytes,
                        void *stream);

/* Encode chunks of the state into a payload (format v1: 64-byte header,
 * records from offset 64 in ascending chunk order, then the record table;
 * each record RAW or exponent-window PACK, whichever is smaller; §6.4: a
 * lossless codec whose receipts bind to the decoded bytes).
 *   state      : nbytes (even), 16-byte aligned
 *   idx, n_idx : device list of *n_idx ascending chunk indices to encode, or
 *                both NULL to encode every chunk (sets the FULL flag).  The
 *                list is checked on the device: one that is not strictly
 *                ascending, holds an index >= n_chunks or has more than
 *                n_chunks entries yields an empty payload (*payload_bytes =
 *                0, the 64 header bytes zeroed)
 *   crc        : ceil(nbytes/chunk_bytes) u32 chunk CRCs from
 *                wm_checksum_chunks (used as receipts and for the header's
 *                global CRC), or NULL to compute them within the call: in
 *                the encoding pass when idx is NULL; with a list, every
 *                chunk is checksummed first (the global CRC covers the
 *                whole state, listed or not) and the workspace holds the
 *                CRCs.  Chunks above 64 KiB: the receipts are tile CRCs,
 *                which chunk CRCs cannot give, so they are computed within
 *                the call whether crc is given or not; a given crc then
 *                serves only a list's global CRC
 *   payload    : payload_cap bytes, 16-byte aligned; payload_cap must be at
 *                least wm_payload_bound(nbytes, n_chunks, p)
 *   payload_bytes : 1 u64, the payload size written
 * Errors: WM_ERR_INVALID_ARG, WM_ERR_CAPACITY, WM_ERR_WORKSPACE,
 *         WM_ERR_UNSUPPORTED, WM_ERR_HIP. */
wm_status wm_encode(const void *state, uint64_t nbytes, const wm_params *p,
                    const uint32_t *idx, const uint32_t *n_idx,
                    const uint32_t *crc, void *payload, uint64_t payload_cap,
                    uint64_t *payload_bytes, void *ws, uint64_t ws_bytes,
                    void *stream);

/* Single pass over cur (and prev) with outputs byte-identical to
 * wm_checksum_chunks(cur) + wm_diff_dirty(cur, prev) + wm_encode(cur, dirty
 * list, crc).  prev == NULL ships every chunk (outputs identical to
 * wm_checksum_chunks + wm_encode(cur, NULL, NULL, crc); dirty_idx then lists
 * every chunk).
 *   crc_out    : n_chunks u32, or NULL
 *   global_crc : 1 u32, or NULL
 *   dirty_idx  : n_chunks u32, or NULL;  n_dirty : 1 u32, or NULL
 * Chunks above 64 KiB: a chunk is dirty when any of its tiles differs and
 * then ships whole, so with prev the call runs the diff, a checksum of every
 * tile and the list encoder (same outputs, more reads) instead of one pass.
 * Other arguments as wm_encode. */
wm_status wm_encode_step(const void *cur, const void *prev, uint64_t nbytes,
                         const wm_params *p, uint32_t *crc_out,
                         uint32_t *global_crc, uint32_t *dirty_idx,
                         uint32_t *n_dirty, void *payload, uint64_t payload_cap,
                         uint64_t *payload_bytes, void *ws, uint64_t ws_bytes,
                         void *stream);

/* wm_encode_step for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * outputs, byte for byte, with the workspace taken from a built-in device
 * array instead of the caller.  The call allocates nothing, on the host or
 * on the device.
 *   Limit: states of at most 65,536 chunks (4 GiB in 64 KiB chunks); a larger
 *   state returns WM_ERR_WORKSPACE before anything is enqueued.  Format v1
 *   and 64 KiB chunks only (anything else returns WM_ERR_UNSUPPORTED).
 *   Sharing: each device holds one built-in workspace (2 MiB + 256 B, kept
 *   until the process ends) used by every call of this function on that
 *   device, whatever the stream.  Calls that overlap in time on one device
 *   race on it and give undefined results: order them (one stream, or
 *   events).  A call clears what it needs zeroed itself; the workspace keeps
 *   the last call's contents.
 * Other arguments, outputs and errors as wm_encode_step. */
wm_status wm_encode_step_static(const void *cur, const void *prev,
                                uint64_t nbytes, const wm_params *p,
                                uint32_t *crc_out, uint32_t *global_crc,
                                uint32_t *dirty_idx, uint32_t *n_dirty,
                                void *payload, uint64_t payload_cap,
                                uint64_t *payload_bytes, void *stream);

/* Validate and decode a payload into staging, re-checksumming every decoded
 * chunk against its receipt (§6.4: decode sits inside the verified
 * envelope; Table 1: verify).  Reads never leave [payload, payload +
 * payload_cap).
 *   nbytes     : the receiver's state size (must match the header)
 *   staging    : staging_cap bytes, 16-byte aligned; record i is decoded to
 *                staging + i*65536 (a full ship's staging is therefore the
 *                shadow copy of the state)
 *   verdict    : 1 u32, 0 when every check passed, else WM_V_* bits
 *   rec_status : ceil(nbytes / 65536) u32 (0, WM_V_RECORD or WM_V_DATA per
 *                record when header and table are valid), or NULL
 * After a nonzero verdict the staging contents are unspecified. */
wm_status wm_decode_verify(const void *payload, uint64_t payload_cap,
                           uint64_t nbytes, const wm_params *p, void *staging,
                           uint64_t staging_cap, uint32_t *verdict,
                           uint32_t *rec_status, void *ws, uint64_t ws_bytes,
                           void *stream);

/* Install or abort (Table 1: commit / rollback).  Enqueues, for
 * WM_COMMIT_SCATTER, a copy of each staged record into live that runs only
 * if *verdict == 0 on the device, then waits for the stream and returns
 * WM_OK (installed) or WM_VERIFY_FAILED (live untouched).  WM_COMMIT_NONE
 * copies nothing (a full ship's caller then swaps the staging buffer in).
 *   live     : nbytes, 16-byte aligned (SCATTER only)
 *   staging, payload : as passed to wm_decode_verify (SCATTER only)
 *   verdict  : the device verdict word from wm_decode_verify */
wm_status wm_commit_or_abort(void *live, uint64_t nbytes, const wm_params *p,
                             const void *staging, const void *payload,
                             const uint32_t *verdict, uint32_t mode,
                             void *stream);

/* Install with re-verification (Table 1: commit re-verifies, then swaps;
 * §4 "Sufficiency": commit only on a byte-identical fingerprint).  A scatter
 * install (as WM_COMMIT_SCATTER) that runs only if, besides a zero verdict
 * from wm_decode_verify:
 *   - every staged record still has its receipt's CRC (staging unchanged
 *     since it was verified), and
 *   - the state the install would produce (live's other chunks plus the
 *     staged records) has the header's global CRC, the CRC of the source
 *     state: the destination's base is the source's last shipped snapshot.
 * Without it the guarantee of a dirty ship holds only relative to the base
 * the destination already had.  On failure WM_V_REVERIFY is ORed into
 * *verdict and live is untouched.  Costs a read of live and of the staged
 * records (their CRCs) before the install.  Waits for the stream; returns
 * WM_OK (installed) or WM_VERIFY_FAILED.
 *   live, staging, payload, verdict : as for wm_commit_or_abort (SCATTER)
 *   ws : workspace of ws_bytes >= wm_workspace_bytes() (chunk CRCs)
 * Errors: WM_ERR_INVALID_ARG, WM_ERR_WORKSPACE, WM_ERR_UNSUPPORTED,
 *         WM_ERR_HIP. */
wm_status wm_commit_reverify(void *live, uint64_t nbytes, const wm_params *p,
                             const void *staging, const void *payload,
                             uint32_t *verdict, void *ws, uint64_t ws_bytes,
                             void *stream);

/* ---- manifest: flatten and rehydrate --------------------------------------
 * The mover works on one flat buffer; a session's state is a manifest of
 * separate device tensors (the paper's suspend manifest: 450 leaves, the 420
 * movable tensors plus scalar control flags; §5 "Implementation").  The
 * canonical path flattens the live state, moves and verifies it, and
 * rehydrates it (§4 "Sufficiency").
 *
 * Flat layout: leaf i occupies flat[off_i, off_i + bytes_i) with off_0 = 0
 * and off_{i+1} = off_i + round_up(bytes_i, 16); flatten writes zeros into
 * the gaps, so the flat bytes are a function of the leaves alone. */
typedef struct {
  const void *ptr; /* device address, 16-byte aligned (any value if bytes is 0) */
  uint64_t bytes;  /* data bytes of the leaf */
} wm_leaf;

/* Flat size of a manifest (sum of the leaf sizes rounded up to 16); 0 for a
 * NULL table with n_leaves > 0 or a sum beyond 64 bits.  leaves: host array. */
uint64_t wm_flat_bytes(const wm_leaf *leaves, uint32_t n_leaves);

/* Workspace bytes a flatten or rehydrate of n_leaves leaves needs (the
 * library's device copy of the table: 32 bytes per leaf). */
uint64_t wm_manifest_ws_bytes(uint32_t n_leaves);

/* Gather the leaves into flat (flatten).  Enqueues on stream a copy of the
 * table into ws and one kernel; returns without waiting.
 *   leaves   : host array of n_leaves entries (read before returning)
 *   flat     : flat_cap bytes, 16-byte aligned, flat_cap >= wm_flat_bytes()
 *              (bytes past wm_flat_bytes() are not written)
 *   ws       : ws_bytes >= wm_manifest_ws_bytes(n_leaves), 16-byte aligned;
 *              in use until the kernel has run
 * Leaves and flat must not overlap.  A manifest of 0 flat bytes returns
 * WM_OK without device work.
 * Errors: WM_ERR_INVALID_ARG (NULL or misaligned pointer, sizes summing past
 *         64 bits), WM_ERR_CAPACITY, WM_ERR_WORKSPACE, WM_ERR_HIP. */
wm_status wm_flatten(const wm_leaf *leaves, uint32_t n_leaves, void *flat,
                     uint64_t flat_cap, void *ws, uint64_t ws_bytes,
                     void *stream);

/* Scatter flat back into the leaves (rehydrate): the exact inverse of
 * wm_flatten for the same table (gap bytes of flat are ignored).  Arguments
 * and errors as wm_flatten. */
wm_status wm_rehydrate(const void *flat, uint64_t flat_cap,
                       const wm_leaf *leaves, uint32_t n_leaves, void *ws,
                       uint64_t ws_bytes, void *stream);

/* ---- pipelined receive ----------------------------------------------------
 * Verification hidden behind the transfer (§6.5: the per-chunk CRC
 * overlapped with receive and GF(2)-combined leaves one final chunk's check
 * exposed; §6.4: the exposed tail equals one final-chunk CRC).  The payload
 * arrives in host memory (a network receive buffer, ideally pinned with
 * hipHostMalloc so the copies are DMA transfers); its header and table are
 * copied first, then its records in batches of about batch_bytes, each
 * batch decoded and verified as soon as it lands, so only the last batch's
 * decode follows the last copy.
 *
 * Outputs equal wm_decode_verify's on the same bytes, whatever batch_bytes.
 *   host_payload  : payload_bytes of host memory, read by the copies until
 *                   they have run (the caller keeps it unchanged until then)
 *   payload       : device buffer of payload_cap >= payload_bytes, 16-byte
 *                   aligned, receives the payload; device reads stay in
 *                   [payload, payload + payload_bytes)
 *   batch_bytes   : target record bytes per batch (0: one record per batch;
 *                   raised so that there are at most 4096 batches)
 *   copy_stream   : stream of the copies; stream: stream of the decode,
 *                   which waits for each batch's copies through events.  The
 *                   copies start after the work enqueued on stream before
 *                   the call (which may still read payload).  Use two
 *                   different streams (not the legacy null stream) for
 *                   overlap; the same stream gives the sequential schedule.
 * Other arguments as wm_decode_verify.  Returns after enqueueing.  The host
 * reads the header and table only to schedule the copies; a header or table
 * that does not parse is copied as one batch, and validity is decided on the
 * device exactly as in wm_decode_verify.
 * Errors: WM_ERR_INVALID_ARG, WM_ERR_CAPACITY (payload_bytes > payload_cap),
 *         WM_ERR_WORKSPACE, WM_ERR_UNSUPPORTED, WM_ERR_HIP. */
wm_status wm_receive_verify(const void *host_payload, uint64_t payload_bytes,
                            void *payload, uint64_t payload_cap,
                            uint64_t nbytes, const wm_params *p, void *staging,
                            uint64_t staging_cap, uint32_t *verdict,
                            uint32_t *rec_status, void *ws, uint64_t ws_bytes,
                            uint64_t batch_bytes, void *copy_stream,
                            void *stream);

/* ---- iterative pre-copy ---------------------------------------------------
 * Pre-copy ships a state that keeps changing: each round ships the chunks
 * that differ from what the destination already holds, while the source
 * goes on writing; when a round's dirty set is small enough the source
 * pauses and one last round makes the destination exact (§6.2 Exhibit 2;
 * App. H: the per-round dirty set follows the occupancy law
 * N(1 - e^(-w/(N C))) for w bytes written in C-byte chunks).
 *
 * Device buffers of one move, owned by the caller, with the sizes the
 * individual calls require (n = ceil(nbytes / chunk_bytes)). */
typedef struct {
  uint32_t *crc;            /* n u32: chunk CRCs of the round's cur */
  uint32_t *global_crc;     /* 1 u32 or NULL */
  uint32_t *dirty_idx;      /* n u32 */
  uint32_t *n_dirty;        /* 1 u32 */
  void *payload;            /* payload_cap >= wm_payload_bound(nbytes, n) */
  uint64_t payload_cap;
  uint64_t *payload_bytes;  /* 1 u64 */
  void *staging;            /* staging_cap >= ceil(nbytes / 65536) * 65536 */
  uint64_t staging_cap;
  uint32_t *verdict;        /* 1 u32 */
  uint32_t *rec_status;     /* ceil(nbytes / 65536) u32 or NULL */
  void *ws_src;             /* wm_workspace_bytes() each; two different */
  uint64_t ws_src_bytes;
  void *ws_dst;
  uint64_t ws_dst_bytes;
} wm_move_buffers;

/* One pre-copy round: wm_encode_step(cur, shipped) ships the chunks of cur
 * that differ from shipped, wm_decode_verify checks them, and only if the
 * verdict is 0 each verified record is installed into dest (the
 * destination's state) and into shipped (the source's copy of what the
 * destination holds).  Waits for the stream; *n_dirty_host (host) receives
 * the round's dirty count.  Returns WM_OK, or WM_VERIFY_FAILED with dest and
 * shipped untouched.
 *   cur      : nbytes (even), 16-byte aligned; the caller may keep writing
 *              it on other streams during the round: shipped receives the
 *              bytes that were encoded, so a chunk changed after it was read
 *              differs from shipped and is dirty in the next round
 *   shipped, dest : nbytes each, 16-byte aligned, distinct from cur and
 *              from each other; equal to each other before the first round
 *              (e.g. both zero) and kept equal by every round
 *   crc_valid  : 0: every chunk of cur is checksummed in the encoding pass
 *              (wm_encode_step).  1: b->crc holds the CRCs of shipped's
 *              chunks, as the previous round that returned WM_OK on the same
 *              buffers left them; the round then runs wm_diff_dirty and
 *              checksums and encodes only the dirty chunks (each record's
 *              receipt and bytes from one read), and the header's global CRC
 *              combines kept and new CRCs.  After a round that did not return
 *              WM_OK, pass 0.  Chunks above 64 KiB: ignored (the kept chunk
 *              CRCs cannot give the tile receipts; every tile is checksummed).
 * Errors: those of the four calls it makes (WM_ERR_INVALID_ARG for a
 *         missing buffer, WM_ERR_CAPACITY for a short payload or staging,
 *         WM_ERR_WORKSPACE, WM_ERR_HIP). */
wm_status wm_precopy_round(const void *cur, void *shipped, void *dest,
                           uint64_t nbytes, const wm_params *p,
                           const wm_move_buffers *b, uint32_t crc_valid,
                           uint32_t *n_dirty_host, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* WM_H */
