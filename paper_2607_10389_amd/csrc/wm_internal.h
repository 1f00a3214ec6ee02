// wm_internal.h -- shared constants and launch interfaces of libwm.
//
// CRC arithmetic used throughout.  For a reflected CRC with polynomial P the
// register update after one message bit is Z(c) = (c >> 1) ^ (P & -(c & 1)),
// a linear map over GF(2).  F^m denotes m zero bytes (8m applications of Z).
// Feeding four message bytes d (little-endian word) into register c gives
// F^4(c ^ d).  With R(M) the register after M from a zero register, the
// standard CRC with init = xorout = 0xFFFFFFFF is
//     CRC(M) = R(M) ^ F^|M|(0xFFFFFFFF) ^ 0xFFFFFFFF,
// and CRC(A|B) = F^|B|(CRC(A)) ^ CRC(B) (how chunk CRCs combine, §6.5).
// A linear map is stored either as four byte tables (tab[j][b] = M(b << 8j))
// or as its 32 columns (col[i] = M(1 << i)).
#pragma once
#include <cstdint>

namespace wm {

constexpr uint32_t kChunk = 65536;  // bytes per chunk the kernels process
constexpr int kWaves = 8;           // waves per workgroup
constexpr int kThreads = kWaves * 64;
constexpr uint32_t kRow = 1024;             // bytes per wave row: 64 lanes x 16 B
constexpr uint32_t kSub = kChunk / kWaves;  // bytes of a chunk per wave
constexpr int kRows = kSub / kRow;          // rows per lane

// Constant tables for one CRC kind (built on the host, uploaded once).
struct CrcTables {
  uint32_t row[4][256];          // F^kRow   (column-stream step, hot)
  // f4 .. wave_step are contiguous: they are copied to LDS as one block
  uint32_t f4[4][256];           // F^4      (standard 4-byte step)
  uint32_t f8[4][256];           // F^8
  uint32_t f12[4][256];          // F^12     (lane merge)
  // F^(16 (63 - l) + 4), lane l's shift: columns 4q..4q+3 at lane_mat[q][l]
  // (a 16-byte read of the 64 lanes covers 1 KiB of consecutive banks)
  uint32_t lane_mat[8][64][4];
  uint32_t wave_step[4][256];    // F^kSub: one wave's share of a chunk
  uint32_t byte1[256];           // one-byte step of the table method
  uint32_t pow2[48][32];         // F^(2^i) bytes, columns
  uint32_t k_full;               // F^kChunk(~0) ^ ~0
  uint32_t pad_[3];
};

// Host-side table construction (wm_tables.cpp).
void build_crc_tables(uint32_t poly, CrcTables *t);
// Columns of F^m (m may be negative: the inverse shift).
void shift_matrix(uint32_t poly, int64_t m, uint32_t cols[32]);
// F^m applied to v.
uint32_t shift_apply(uint32_t poly, int64_t m, uint32_t v);
uint32_t poly_of(uint32_t crc_kind);

// Per-call parameters passed by value to every kernel.  The kernels work on
// 64 KiB units: a chunk of at most 64 KiB, or a 64 KiB tile of a larger
// chunk (the payload then holds one record and one receipt per tile, and a
// table ships every tile of each chunk it lists).  n_chunks, tail_len and
// the tail shift describe the units; tile_log2 and hdr_n the caller's
// chunks.
struct ChunkGeom {
  uint64_t nbytes;      // state bytes
  uint32_t n_chunks;    // units: ceil(nbytes / kChunk)
  uint32_t tail_len;    // length of the last unit (kChunk if full)
  uint32_t crc_kind;
  uint32_t codec;       // payload format: 1 (v1) or 2 (v2, Huffman exponents)
  uint32_t k_tail;      // F^tail_len(~0) ^ ~0
  uint32_t tail_mat[32];// F^-(kChunk - tail_len), columns
  uint32_t tile_log2;   // log2(chunk_bytes / kChunk): 0 for 64 KiB chunks
  uint32_t hdr_n;       // chunks: ceil(nbytes / chunk_bytes)
};
// Bytes of the caller's chunk.
inline uint32_t geom_chunk_bytes(const ChunkGeom &g) { return kChunk << g.tile_log2; }

// Workspace layout (bytes from the workspace base).
struct WsLayout {
  uint64_t ctl;        // 256 B of counters and flags
  uint64_t status;     // n_chunks x u64 look-back words
  uint64_t table;      // n_chunks x 16 B staged table entries
  uint64_t entry_crc;  // n_chunks x u32 CRC of each table entry
  uint64_t flags;      // n_chunks x u32 (diff flags / record bits)
  uint64_t total;
};
WsLayout ws_layout(uint32_t n_chunks);

// Control block at the start of the workspace.
struct WsCtl {
  uint32_t ticket;       // dynamic work counter
  uint32_t error;        // encode: 1 = look-back gave up, 2 = bad chunk index
  uint32_t hdr_ok;       // decode: header passed
  uint32_t table_bad;    // decode: a table-local rule failed
  uint32_t rec_bits;     // decode: OR of record status bits
  uint32_t n_rec;        // decode: records in the payload
  uint64_t payload_bytes;// decode: from the header
  uint64_t table_off;    // decode: table start
  uint32_t table_crc;    // decode: expected table CRC
  uint32_t verdict_pre;  // decode: header/staging verdict
  uint32_t pad_[52];
};
static_assert(sizeof(WsCtl) == 256, "control block is 256 bytes");

// Kernel launchers (wm_kernels.hip).  All return a hipError_t as int.
int upload_tables(int device, const CrcTables tabs[2]);
// CRC of each of the caller's chunks (hdr_n of them), or with `units` of
// each 64 KiB unit (n_chunks); the global CRC from them.
int launch_checksum(const void *data, const ChunkGeom &g, uint32_t *crc_out,
                    uint32_t *global_crc, int n_cu, void *stream, bool units = false);
// Dirty chunks (the caller's chunks: one is dirty when any of its tiles is).
int launch_diff(const void *cur, const void *prev, const ChunkGeom &g,
                uint32_t *dirty_idx, uint32_t *n_dirty, void *ws,
                const WsLayout &L, void *stream);
// Chunks above 64 KiB: a device list of the caller's chunks as the list of
// their tiles (an invalid list as an over-long one), and chunk CRCs from
// tile CRCs.
int launch_expand_list(const uint32_t *idx, const uint32_t *n_idx, const ChunkGeom &g,
                       uint32_t *out, uint32_t *n_out, void *stream);
int launch_fold_tiles(const uint32_t *tile_crc, const ChunkGeom &g, uint32_t *out, void *stream);
// mode: 0 = list (idx/n_idx), 1 = all chunks, 2 = step (prev may be NULL);
// the encoder works on units (idx lists units, CRCs are units').  The
// header's global CRC combines the unit CRCs (crc_in, else crc_out), or
// global_from: the caller's chunk CRCs.
int launch_encode(int mode, const void *cur, const void *prev,
                  const ChunkGeom &g, const uint32_t *idx,
                  const uint32_t *n_idx, const uint32_t *crc_in,
                  uint32_t *crc_out, uint32_t *global_crc,
                  uint32_t *dirty_idx, uint32_t *n_dirty, void *payload,
                  uint64_t *payload_bytes, void *ws, const WsLayout &L,
                  int n_cu, void *stream, const uint32_t *global_from = nullptr);
int launch_decode(const void *payload, uint64_t payload_cap,
                  const ChunkGeom &g, void *staging, uint64_t staging_cap,
                  uint32_t *verdict, uint32_t *rec_status, void *ws,
                  const WsLayout &L, int n_cu, void *stream);
// The three parts of launch_decode, for a payload decoded in record batches:
// header and table checks, records [r0, r1), table CRC and verdict.
int launch_decode_begin(const void *payload, uint64_t payload_cap, const ChunkGeom &g,
                        uint64_t staging_cap, void *ws, const WsLayout &L, void *stream);
int launch_decode_records(const void *payload, const ChunkGeom &g, void *staging,
                          uint32_t *rec_status, void *ws, const WsLayout &L, int n_cu,
                          uint32_t r0, uint32_t r1, void *stream);
int launch_decode_end(const ChunkGeom &g, uint32_t *verdict, void *ws, const WsLayout &L,
                      void *stream);
int launch_commit(void *live, const ChunkGeom &g, const void *staging,
                  const void *payload, const uint32_t *verdict, int n_cu,
                  void *stream);
// idx[i] = i for i < n (idx may be NULL) and *n_out = n (n_out may be NULL).
int launch_fill_all(uint32_t *idx, uint32_t *n_out, uint32_t n, void *stream);
// Re-verification before an install: CRCs of live's chunks (geometry g) and
// of the staged records (gs: the staged bytes as one state), receipts in
// place of the chunks the install overwrites, their combined global CRC
// against the header's; a failure ORs 32 into the verdict.  Uses the
// workspace's control block, entry CRC and flag arrays.
int launch_reverify(const void *live, const ChunkGeom &g, const void *staging,
                    const ChunkGeom &gs, const void *payload, uint32_t *verdict, void *ws,
                    const WsLayout &L, int n_cu, void *stream);
// One leaf of a manifest as the device sees it (the library's copy of the
// caller's table, with offsets): 32 bytes.
struct ManifestLeaf {
  uint64_t ptr;    // device address, 16-byte aligned
  uint64_t off;    // flat offset, multiple of 16, ascending
  uint64_t bytes;  // data bytes
  uint64_t pad_;
};
// gather: leaves -> flat (flatten); else flat -> leaves (rehydrate)
int launch_manifest(bool gather, void *flat, uint64_t flat_bytes, const ManifestLeaf *leaves,
                    uint32_t n_leaves, int n_cu, void *stream);
// Format v2/v3: per-item plans (code lengths) in the workspace after the
// WsLayout part, kHufPlanBytes each.
constexpr uint32_t kHufPlanBytes = 256;
inline uint64_t plans_offset(const WsLayout &L) { return (L.total + 255u) & ~255ull; }
// Format v2/v3 encode (full ship or index list): the code lengths, then one
// pass per chunk.
int launch_encode_v2(const void *state, const ChunkGeom &g, const uint32_t *idx,
                     const uint32_t *n_idx, const uint32_t *crc_in, uint32_t *crc_scratch,
                     uint32_t *global_crc, void *payload, uint64_t *payload_bytes, void *ws,
                     const WsLayout &L, int n_cu, void *stream);
// Format v2 records [r0, r1) (as launch_decode_records).
int launch_decode_records_v2(const void *payload, const ChunkGeom &g, void *staging,
                             uint32_t *rec_status, void *ws, const WsLayout &L, int n_cu,
                             uint32_t r0, uint32_t r1, void *stream);
int launch_decode_v2(const void *payload, uint64_t payload_cap, const ChunkGeom &g,
                     void *staging, uint64_t staging_cap, uint32_t *verdict,
                     uint32_t *rec_status, void *ws, const WsLayout &L, int n_cu,
                     void *stream);
int set_kernel_attributes();
// Device address and size of the built-in workspace (a file-scope device
// array) on the current device.
int scratch_address(void **ptr, uint64_t *bytes);

}  // namespace wm
