// wm_api.cpp -- the C ABI of libwm (declared in include/wm.h).
//
// Host side only: argument validation (before anything is enqueued),
// per-call geometry, workspace layout, and the launches.  Constant CRC tables
// are built once on the host and uploaded once per device.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <cstdint>
#include <map>
#include <mutex>
#include <vector>

#include "wm.h"
#include "wm_internal.h"

using namespace wm;

namespace {

constexpr int kMaxDevices = 64;
constexpr uint64_t kMaxBatches = 4096;  // record batches of one received payload
// Size of the built-in workspace (kScratchBytes of the device array): the
// layout of 65,536 chunks.
constexpr uint64_t kBuiltinWsBytes = 256 + 32ull * 65536;

struct DeviceState {
  bool ready = false;
  int n_cu = 0;
  void *scratch = nullptr;  // device address of the built-in workspace
  uint64_t scratch_bytes = 0;
};

std::mutex g_mu;
DeviceState g_dev[kMaxDevices];
CrcTables g_tables_host[2];
bool g_tables_built = false;

struct TailGeom {
  uint32_t k_tail;
  uint32_t mat[32];
};
std::map<uint64_t, TailGeom> g_tail_cache;

wm_status ensure_device(int *n_cu, void **scratch = nullptr, uint64_t *scratch_bytes = nullptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return WM_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_tables_built) {
    build_crc_tables(poly_of(0), &g_tables_host[0]);
    build_crc_tables(poly_of(1), &g_tables_host[1]);
    g_tables_built = true;
  }
  DeviceState &st = g_dev[dev];
  if (!st.ready) {
    if (upload_tables(dev, g_tables_host) != 0) return WM_ERR_HIP;
    if (set_kernel_attributes() != 0) return WM_ERR_HIP;
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cu <= 0)
      return WM_ERR_HIP;
    // the built-in workspace's address on this device (the current one)
    void *sp = nullptr;
    uint64_t sb = 0;
    if (scratch_address(&sp, &sb) != 0 || !sp) return WM_ERR_HIP;
    st.n_cu = cu;
    st.scratch = sp;
    st.scratch_bytes = sb;
    st.ready = true;
  }
  *n_cu = st.n_cu;
  if (scratch) *scratch = st.scratch;
  if (scratch_bytes) *scratch_bytes = st.scratch_bytes;
  return WM_OK;
}

wm_status check_params(const wm_params *p) {
  if (!p) return WM_ERR_INVALID_ARG;
  if (p->crc_kind > 1 ||
      (p->codec != WM_CODEC_EXPFOR && p->codec != WM_CODEC_EXPHUF &&
       p->codec != WM_CODEC_BYTEPLANE) ||
      p->flags != 0)
    return WM_ERR_INVALID_ARG;
  uint32_t c = p->chunk_bytes;
  bool pow2 = c >= 4096u && c <= (16u << 20) && (c & (c - 1)) == 0;
  if (!pow2) return WM_ERR_INVALID_ARG;
  if (c < kChunk) return WM_ERR_UNSUPPORTED;  // the kernels' unit is 64 KiB
  return WM_OK;
}

// cache_tail: keep the short last chunk's shift matrix in a host map for
// later calls (false: compute it in place, allocating nothing).
wm_status make_geom(uint64_t nbytes, const wm_params *p, ChunkGeom *g, bool cache_tail = true) {
  wm_status s = check_params(p);
  if (s != WM_OK) return s;
  uint64_t n = (nbytes + kChunk - 1) / kChunk;
  if (n >= (1ull << 24)) return WM_ERR_INVALID_ARG;  // look-back field width
  g->nbytes = nbytes;
  g->n_chunks = (uint32_t)n;
  g->tile_log2 = (uint32_t)__builtin_ctz(p->chunk_bytes) - 16u;
  g->hdr_n = (uint32_t)((nbytes + p->chunk_bytes - 1) / p->chunk_bytes);
  g->tail_len = n ? (uint32_t)(nbytes - (n - 1) * kChunk) : kChunk;
  g->crc_kind = p->crc_kind;
  g->codec = p->codec;
  g->k_tail = 0;
  for (int i = 0; i < 32; ++i) g->tail_mat[i] = 1u << i;
  if (g->tail_len != kChunk && !cache_tail) {
    const uint32_t poly = poly_of(p->crc_kind);
    g->k_tail = shift_apply(poly, g->tail_len, 0xFFFFFFFFu) ^ 0xFFFFFFFFu;
    shift_matrix(poly, -(int64_t)(kChunk - g->tail_len), g->tail_mat);
  } else if (g->tail_len != kChunk) {
    uint64_t key = ((uint64_t)p->crc_kind << 32) | g->tail_len;
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = g_tail_cache.find(key);
    if (it == g_tail_cache.end()) {
      uint32_t poly = poly_of(p->crc_kind);
      TailGeom t;
      t.k_tail = shift_apply(poly, g->tail_len, 0xFFFFFFFFu) ^ 0xFFFFFFFFu;
      shift_matrix(poly, -(int64_t)(kChunk - g->tail_len), t.mat);
      it = g_tail_cache.emplace(key, t).first;
    }
    g->k_tail = it->second.k_tail;
    for (int i = 0; i < 32; ++i) g->tail_mat[i] = it->second.mat[i];
  }
  return WM_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// CUs that launches on `stream` can use: the stream's CU mask when it has
// one (hipExtStreamCreateWithCUMask, e.g. one slice of the GPU per session),
// all of them otherwise.  The persistent kernels size their grids with it.
int stream_cus(void *stream, int n_cu) {
  if (!stream) return n_cu;
  uint32_t mask[32] = {0};  // up to 1024 CUs
  if (hipExtStreamGetCUMask(reinterpret_cast<hipStream_t>(stream), 32, mask) != hipSuccess)
    return n_cu;
  int c = 0;
  for (uint32_t m : mask) c += __builtin_popcount(m);
  return c > 0 && c < n_cu ? c : n_cu;
}

// Workspace: the WsLayout part, then (format v2) one plan per item and a
// dirty list with its length for a fused step whose caller passes no
// dirty_idx.
uint64_t list_offset(const WsLayout &L, uint32_t n_chunks) {
  return (plans_offset(L) + (uint64_t)kHufPlanBytes * n_chunks + 255u) & ~255ull;
}
uint64_t ws_base(const WsLayout &L, uint32_t n_chunks, uint32_t codec) {
  return codec != WM_CODEC_EXPFOR ? list_offset(L, n_chunks) + 4ull * n_chunks + 16u : L.total;
}
// Chunks above 64 KiB also keep, after that, the tile list of a chunk list
// with its length, and a chunk list with its length.
uint64_t tiles_offset(const WsLayout &L, uint32_t n_units, uint32_t codec) {
  return (ws_base(L, n_units, codec) + 255u) & ~255ull;
}
uint64_t ws_need(const ChunkGeom &g, const WsLayout &L) {
  if (!g.tile_log2) return ws_base(L, g.n_chunks, g.codec);
  return tiles_offset(L, g.n_chunks, g.codec) + 4ull * (g.n_chunks + g.hdr_n) + 32u;
}
struct TileLists {
  uint32_t *tiles, *n_tiles, *chunks, *n_chunks;
};
TileLists tile_lists(void *ws, const ChunkGeom &g, const WsLayout &L) {
  uint32_t *t = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(ws) +
                                             tiles_offset(L, g.n_chunks, g.codec));
  TileLists r;
  r.tiles = t;
  r.n_tiles = t + g.n_chunks;
  r.chunks = t + g.n_chunks + 4;
  r.n_chunks = r.chunks + g.hdr_n;
  return r;
}

wm_status hip_status(int e) { return e == 0 ? WM_OK : WM_ERR_HIP; }

// wm_encode for chunks above 64 KiB: the records are the listed chunks'
// tiles, so a chunk list is expanded to its tiles first.  Receipts are tile
// CRCs, which the caller's chunk CRCs cannot give: they are computed in the
// encoding pass (format v1) or by a checksum of every tile first (format v2,
// and format v1 with a list and no CRCs, whose global CRC covers unlisted
// chunks too).  With a list and the caller's CRCs, the global CRC combines
// those.
wm_status encode_tiles(const void *state, const ChunkGeom &g, const uint32_t *idx,
                       const uint32_t *n_idx, const uint32_t *crc, void *payload,
                       uint64_t *payload_bytes, void *ws, const WsLayout &L, int n_cu,
                       void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  uint32_t *unit_crc = reinterpret_cast<uint32_t *>(wsb + L.flags);
  const TileLists t = tile_lists(ws, g, L);
  if (idx && launch_expand_list(idx, n_idx, g, t.tiles, t.n_tiles, stream) != 0) return WM_ERR_HIP;
  const uint32_t *ul = idx ? t.tiles : nullptr, *un = idx ? t.n_tiles : nullptr;
  if (g.codec != WM_CODEC_EXPFOR)
    return hip_status(launch_encode_v2(state, g, ul, un, nullptr, unit_crc, nullptr, payload,
                                       payload_bytes, ws, L, n_cu, stream));
  if (!idx)
    return hip_status(launch_encode(1, state, nullptr, g, nullptr, nullptr, nullptr, unit_crc,
                                    nullptr, nullptr, nullptr, payload, payload_bytes, ws, L,
                                    n_cu, stream));
  if (!crc) {
    if (launch_checksum(state, g, unit_crc, nullptr, n_cu, stream, true) != 0) return WM_ERR_HIP;
    return hip_status(launch_encode(0, state, nullptr, g, ul, un, unit_crc, nullptr, nullptr,
                                    nullptr, nullptr, payload, payload_bytes, ws, L, n_cu,
                                    stream));
  }
  return hip_status(launch_encode(0, state, nullptr, g, ul, un, nullptr, unit_crc, nullptr,
                                  nullptr, nullptr, payload, payload_bytes, ws, L, n_cu, stream,
                                  crc));
}

// wm_encode_step for chunks above 64 KiB: dirtiness is the chunk's (any
// tile differs), so there is no single pass; the diff gives the dirty chunk
// list, every tile is checksummed (chunk CRCs fold from tile CRCs, and the
// global CRC covers every tile), and the list encoder ships the dirty
// chunks' tiles.  Without prev every chunk ships from one encoding pass.
wm_status encode_step_tiles(const void *cur, const void *prev, const ChunkGeom &g,
                            uint32_t *crc_out, uint32_t *global_crc, uint32_t *dirty_idx,
                            uint32_t *n_dirty, void *payload, uint64_t *payload_bytes, void *ws,
                            const WsLayout &L, int n_cu, void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  uint32_t *unit_crc = reinterpret_cast<uint32_t *>(wsb + L.flags);
  const TileLists t = tile_lists(ws, g, L);
  if (!prev) {
    int rc = g.codec != WM_CODEC_EXPFOR
                 ? launch_encode_v2(cur, g, nullptr, nullptr, nullptr, unit_crc, global_crc,
                                    payload, payload_bytes, ws, L, n_cu, stream)
                 : launch_encode(1, cur, nullptr, g, nullptr, nullptr, nullptr, unit_crc,
                                 global_crc, nullptr, nullptr, payload, payload_bytes, ws, L,
                                 n_cu, stream);
    if (rc == 0 && crc_out) rc = launch_fold_tiles(unit_crc, g, crc_out, stream);
    if (rc == 0 && (dirty_idx || n_dirty)) rc = launch_fill_all(dirty_idx, n_dirty, g.hdr_n, stream);
    return hip_status(rc);
  }
  uint32_t *list = dirty_idx ? dirty_idx : t.chunks;
  uint32_t *n_list = n_dirty ? n_dirty : t.n_chunks;
  if (launch_diff(cur, prev, g, list, n_list, ws, L, stream) != 0 ||
      launch_expand_list(list, n_list, g, t.tiles, t.n_tiles, stream) != 0 ||
      launch_checksum(cur, g, unit_crc, nullptr, n_cu, stream, true) != 0 ||
      (crc_out && launch_fold_tiles(unit_crc, g, crc_out, stream) != 0))
    return WM_ERR_HIP;
  if (g.codec != WM_CODEC_EXPFOR)
    return hip_status(launch_encode_v2(cur, g, t.tiles, t.n_tiles, unit_crc, nullptr, global_crc,
                                       payload, payload_bytes, ws, L, n_cu, stream));
  return hip_status(launch_encode(0, cur, nullptr, g, t.tiles, t.n_tiles, unit_crc, nullptr,
                                  global_crc, nullptr, nullptr, payload, payload_bytes, ws, L,
                                  n_cu, stream));
}

}  // namespace

extern "C" {

const char *wm_status_str(wm_status s) {
  switch (s) {
    case WM_OK: return "WM_OK";
    case WM_VERIFY_FAILED: return "WM_VERIFY_FAILED";
    case WM_ERR_INVALID_ARG: return "WM_ERR_INVALID_ARG";
    case WM_ERR_CAPACITY: return "WM_ERR_CAPACITY";
    case WM_ERR_HIP: return "WM_ERR_HIP";
    case WM_ERR_WORKSPACE: return "WM_ERR_WORKSPACE";
    case WM_ERR_UNSUPPORTED: return "WM_ERR_UNSUPPORTED";
    default: return "WM_UNKNOWN_STATUS";
  }
}

wm_status wm_init(int device) {
  if (device >= 0 && hipSetDevice(device) != hipSuccess) return WM_ERR_HIP;
  int n_cu = 0;
  return ensure_device(&n_cu);
}

uint64_t wm_workspace_bytes(uint64_t nbytes, const wm_params *p) {
  ChunkGeom g;
  if (make_geom(nbytes, p, &g, false) != WM_OK) return 0;
  return ws_need(g, ws_layout(g.n_chunks));
}

uint64_t wm_payload_bound(uint64_t nbytes, uint32_t n_records, const wm_params *p) {
  (void)nbytes;
  if (check_params(p) != WM_OK) return 0;
  // every record RAW: a chunk above 64 KiB ships as its 64 KiB tiles, one
  // record (16-byte header + body) and one table entry each
  const uint64_t units = (uint64_t)n_records * (p->chunk_bytes / kChunk);
  return 64u + units * (32u + kChunk);
}

wm_status wm_checksum_chunks(const void *data, uint64_t nbytes, const wm_params *p,
                             uint32_t *crc_out, uint32_t *global_crc, void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if ((nbytes && (!data || !crc_out)) || !aligned16(data)) return WM_ERR_INVALID_ARG;
  if (!nbytes && !global_crc) return WM_OK;
  if (!crc_out && global_crc) return WM_ERR_INVALID_ARG;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  return hip_status(launch_checksum(data, g, crc_out, global_crc, n_cu, stream));
}

wm_status wm_diff_dirty(const void *cur, const void *prev, uint64_t nbytes, const wm_params *p,
                        uint32_t *dirty_idx, uint32_t *n_dirty, void *ws, uint64_t ws_bytes,
                        void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if (!n_dirty || (nbytes && (!cur || !prev || !dirty_idx))) return WM_ERR_INVALID_ARG;
  if (!aligned16(cur) || !aligned16(prev)) return WM_ERR_INVALID_ARG;
  WsLayout L = ws_layout(g.n_chunks);
  if (!ws || ws_bytes < L.total || !aligned16(ws)) return WM_ERR_WORKSPACE;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  return hip_status(launch_diff(cur, prev, g, dirty_idx, n_dirty, ws, L, stream));
}

wm_status wm_encode(const void *state, uint64_t nbytes, const wm_params *p, const uint32_t *idx,
                    const uint32_t *n_idx, const uint32_t *crc, void *payload,
                    uint64_t payload_cap, uint64_t *payload_bytes, void *ws, uint64_t ws_bytes,
                    void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if (nbytes & 1u) return WM_ERR_INVALID_ARG;
  if ((nbytes && !state) || !aligned16(state)) return WM_ERR_INVALID_ARG;
  if ((idx == nullptr) != (n_idx == nullptr)) return WM_ERR_INVALID_ARG;
  if (!payload || !payload_bytes || !aligned16(payload)) return WM_ERR_INVALID_ARG;
  if (payload_cap < wm_payload_bound(nbytes, g.hdr_n, p)) return WM_ERR_CAPACITY;
  WsLayout L = ws_layout(g.n_chunks);
  if (!ws || ws_bytes < ws_need(g, L) || !aligned16(ws)) return WM_ERR_WORKSPACE;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  if (g.tile_log2) return encode_tiles(state, g, idx, n_idx, crc, payload, payload_bytes, ws, L,
                                       n_cu, stream);
  uint32_t *crc_scratch =
      crc ? nullptr : reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(ws) + L.flags);
  if (g.codec != WM_CODEC_EXPFOR)
    return hip_status(launch_encode_v2(state, g, idx, n_idx, crc, crc_scratch, nullptr, payload,
                                       payload_bytes, ws, L, n_cu, stream));
  if (idx && !crc) {
    // the header's global CRC covers every chunk, listed or not: checksum
    // the whole state first, then encode the list with those receipts
    const int rc = launch_checksum(state, g, crc_scratch, nullptr, n_cu, stream);
    if (rc) return WM_ERR_HIP;
    crc = crc_scratch;
    crc_scratch = nullptr;
  }
  int mode = idx ? 0 : 1;
  return hip_status(launch_encode(mode, state, nullptr, g, idx, n_idx, crc, crc_scratch, nullptr,
                                  nullptr, nullptr, payload, payload_bytes, ws, L, n_cu, stream));
}

}  // extern "C"

namespace {

// wm_encode_step on a caller's workspace, or (builtin) on the device's
// built-in one: then nothing is allocated on the way, host or device.
wm_status encode_step_call(const void *cur, const void *prev, uint64_t nbytes,
                           const wm_params *p, uint32_t *crc_out, uint32_t *global_crc,
                           uint32_t *dirty_idx, uint32_t *n_dirty, void *payload,
                           uint64_t payload_cap, uint64_t *payload_bytes, void *ws,
                           uint64_t ws_bytes, bool builtin, void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g, !builtin);
  if (s != WM_OK) return s;
  // the built-in workspace has the format v1, 64 KiB chunk layout only
  if (builtin && (g.codec != WM_CODEC_EXPFOR || g.tile_log2)) return WM_ERR_UNSUPPORTED;
  if (nbytes & 1u) return WM_ERR_INVALID_ARG;
  if ((nbytes && !cur) || !aligned16(cur) || !aligned16(prev)) return WM_ERR_INVALID_ARG;
  if (!payload || !payload_bytes || !aligned16(payload)) return WM_ERR_INVALID_ARG;
  if (payload_cap < wm_payload_bound(nbytes, g.hdr_n, p)) return WM_ERR_CAPACITY;
  WsLayout L = ws_layout(g.n_chunks);
  int n_cu = 0;
  if (builtin) {
    // the size limit is checked before the device is touched
    if (L.total > kBuiltinWsBytes) return WM_ERR_WORKSPACE;
    if ((s = ensure_device(&n_cu, &ws, &ws_bytes)) != WM_OK) return s;
    if (L.total > ws_bytes) return WM_ERR_WORKSPACE;
  } else {
    if (!ws || ws_bytes < ws_need(g, L) || !aligned16(ws)) return WM_ERR_WORKSPACE;
    if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  }
  n_cu = stream_cus(stream, n_cu);
  if (g.tile_log2)
    return encode_step_tiles(cur, prev, g, crc_out, global_crc, dirty_idx, n_dirty, payload,
                             payload_bytes, ws, L, n_cu, stream);
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  uint32_t *crcs = crc_out ? crc_out : reinterpret_cast<uint32_t *>(wsb + L.flags);
  if (g.codec != WM_CODEC_EXPFOR) {
    // format v2 has no single-pass encoder: the same outputs from the diff
    // (whose flags it consumes first), a checksum of every chunk and the
    // list encoder, each reading the state once
    uint32_t *list = dirty_idx ? dirty_idx : reinterpret_cast<uint32_t *>(wsb + list_offset(L, g.n_chunks));
    uint32_t *n_list = n_dirty ? n_dirty : list + g.n_chunks;
    if (prev && launch_diff(cur, prev, g, list, n_list, ws, L, stream) != 0) return WM_ERR_HIP;
    if (!prev && (dirty_idx || n_dirty) &&
        launch_fill_all(dirty_idx, n_dirty, g.n_chunks, stream) != 0)
      return WM_ERR_HIP;
    if (launch_checksum(cur, g, crcs, nullptr, n_cu, stream) != 0) return WM_ERR_HIP;
    return hip_status(launch_encode_v2(cur, g, prev ? list : nullptr, prev ? n_list : nullptr,
                                       crcs, nullptr, global_crc, payload, payload_bytes, ws, L,
                                       n_cu, stream));
  }
  return hip_status(launch_encode(2, cur, prev, g, nullptr, nullptr, nullptr, crcs, global_crc,
                                  dirty_idx, n_dirty, payload, payload_bytes, ws, L, n_cu,
                                  stream));
}

}  // namespace

extern "C" {

wm_status wm_encode_step(const void *cur, const void *prev, uint64_t nbytes, const wm_params *p,
                         uint32_t *crc_out, uint32_t *global_crc, uint32_t *dirty_idx,
                         uint32_t *n_dirty, void *payload, uint64_t payload_cap,
                         uint64_t *payload_bytes, void *ws, uint64_t ws_bytes, void *stream) {
  return encode_step_call(cur, prev, nbytes, p, crc_out, global_crc, dirty_idx, n_dirty, payload,
                          payload_cap, payload_bytes, ws, ws_bytes, false, stream);
}

wm_status wm_encode_step_static(const void *cur, const void *prev, uint64_t nbytes,
                                const wm_params *p, uint32_t *crc_out, uint32_t *global_crc,
                                uint32_t *dirty_idx, uint32_t *n_dirty, void *payload,
                                uint64_t payload_cap, uint64_t *payload_bytes, void *stream) {
  return encode_step_call(cur, prev, nbytes, p, crc_out, global_crc, dirty_idx, n_dirty, payload,
                          payload_cap, payload_bytes, nullptr, 0, true, stream);
}

wm_status wm_decode_verify(const void *payload, uint64_t payload_cap, uint64_t nbytes,
                           const wm_params *p, void *staging, uint64_t staging_cap,
                           uint32_t *verdict, uint32_t *rec_status, void *ws, uint64_t ws_bytes,
                           void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if (nbytes & 1u) return WM_ERR_INVALID_ARG;
  if (!payload || !verdict || !aligned16(payload)) return WM_ERR_INVALID_ARG;
  if ((staging_cap && !staging) || !aligned16(staging)) return WM_ERR_INVALID_ARG;
  WsLayout L = ws_layout(g.n_chunks);
  if (!ws || ws_bytes < L.total || !aligned16(ws)) return WM_ERR_WORKSPACE;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  if (g.codec != WM_CODEC_EXPFOR)
    return hip_status(launch_decode_v2(payload, payload_cap, g, staging, staging_cap, verdict,
                                       rec_status, ws, L, n_cu, stream));
  return hip_status(launch_decode(payload, payload_cap, g, staging, staging_cap, verdict,
                                  rec_status, ws, L, n_cu, stream));
}

wm_status wm_commit_or_abort(void *live, uint64_t nbytes, const wm_params *p, const void *staging,
                             const void *payload, const uint32_t *verdict, uint32_t mode,
                             void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if (!verdict || mode > WM_COMMIT_SCATTER) return WM_ERR_INVALID_ARG;
  if (mode == WM_COMMIT_SCATTER) {
    if ((nbytes && (!live || !staging || !payload)) || !aligned16(live) || !aligned16(staging) ||
        !aligned16(payload))
      return WM_ERR_INVALID_ARG;
  }
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (mode == WM_COMMIT_SCATTER) {
    if (launch_commit(live, g, staging, payload, verdict, n_cu, stream) != 0) return WM_ERR_HIP;
  }
  uint32_t v = 0xFFFFFFFFu;
  if (hipMemcpyAsync(&v, verdict, sizeof(v), hipMemcpyDeviceToHost, st) != hipSuccess)
    return WM_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return WM_ERR_HIP;
  return v == 0 ? WM_OK : WM_VERIFY_FAILED;
}

wm_status wm_commit_reverify(void *live, uint64_t nbytes, const wm_params *p,
                             const void *staging, const void *payload, uint32_t *verdict,
                             void *ws, uint64_t ws_bytes, void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if (!verdict || !payload || !aligned16(payload)) return WM_ERR_INVALID_ARG;
  if ((nbytes && (!live || !staging)) || !aligned16(live) || !aligned16(staging))
    return WM_ERR_INVALID_ARG;
  const WsLayout L = ws_layout(g.n_chunks);
  if (!ws || ws_bytes < L.total || !aligned16(ws)) return WM_ERR_WORKSPACE;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // a failed verification needs no further work: nothing is installed
  uint32_t v = 0xFFFFFFFFu;
  if (hipMemcpyAsync(&v, verdict, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return WM_ERR_HIP;
  if (v != 0) return WM_VERIFY_FAILED;
  // a zero verdict means the header and table passed their checks: the
  // staged records are chunks table[0..n_rec) in ascending order, each a
  // full chunk except possibly the last (the state's short last chunk)
  uint8_t head[64];
  uint8_t last[16] = {0};
  if (hipMemcpyAsync(head, payload, 64, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return WM_ERR_HIP;
  uint32_t n_rec = 0;
  uint64_t total = 0, state = 0;
  std::memcpy(&n_rec, head + 24, 4);
  std::memcpy(&total, head + 32, 8);
  std::memcpy(&state, head + 16, 8);
  // the payload a zero verdict was given for has these properties; another
  // payload is a caller error
  if (state != nbytes || n_rec > g.n_chunks || total < 64u + 16ull * n_rec)
    return WM_ERR_INVALID_ARG;
  uint64_t staged = 0;
  if (n_rec) {
    const uint8_t *entry = static_cast<const uint8_t *>(payload) + total - 16u;
    if (hipMemcpyAsync(last, entry, 16, hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
      return WM_ERR_HIP;
    uint32_t c_last = 0;
    std::memcpy(&c_last, last, 4);
    if (c_last >= g.n_chunks) return WM_ERR_INVALID_ARG;
    const uint64_t len_last = c_last + 1 == g.n_chunks ? g.tail_len : kChunk;
    staged = (uint64_t)(n_rec - 1) * kChunk + len_last;
  }
  ChunkGeom gs;
  if ((s = make_geom(staged, p, &gs)) != WM_OK) return s;
  if (launch_reverify(live, g, staging, gs, payload, verdict, ws, L, n_cu, stream) != 0)
    return WM_ERR_HIP;
  if (nbytes && launch_commit(live, g, staging, payload, verdict, n_cu, stream) != 0)
    return WM_ERR_HIP;
  if (hipMemcpyAsync(&v, verdict, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return WM_ERR_HIP;
  return v == 0 ? WM_OK : WM_VERIFY_FAILED;
}

uint64_t wm_flat_bytes(const wm_leaf *leaves, uint32_t n_leaves) {
  if (n_leaves && !leaves) return 0;
  uint64_t total = 0;
  for (uint32_t i = 0; i < n_leaves; ++i) {
    if (leaves[i].bytes > UINT64_MAX - 15u - total) return 0;
    total += (leaves[i].bytes + 15u) & ~15ull;
  }
  return total;
}

uint64_t wm_manifest_ws_bytes(uint32_t n_leaves) { return 32ull * n_leaves; }

}  // extern "C"

namespace {

// Checks the caller's table, writes the device copy (with offsets) into the
// workspace and launches the copy.
wm_status manifest_call(bool gather, const wm_leaf *leaves, uint32_t n_leaves, void *flat,
                        uint64_t flat_cap, void *ws, uint64_t ws_bytes, void *stream) {
  if (n_leaves && !leaves) return WM_ERR_INVALID_ARG;
  std::vector<ManifestLeaf> t(n_leaves);
  uint64_t total = 0;
  for (uint32_t i = 0; i < n_leaves; ++i) {
    const uint64_t b = leaves[i].bytes;
    if (b && (!leaves[i].ptr || !aligned16(leaves[i].ptr))) return WM_ERR_INVALID_ARG;
    if (b > UINT64_MAX - 15u - total) return WM_ERR_INVALID_ARG;
    t[i] = ManifestLeaf{reinterpret_cast<uint64_t>(leaves[i].ptr), total, b, 0};
    total += (b + 15u) & ~15ull;
  }
  if (total && (!flat || !aligned16(flat))) return WM_ERR_INVALID_ARG;
  if (flat_cap < total) return WM_ERR_CAPACITY;
  if (n_leaves && (!ws || !aligned16(ws) || ws_bytes < 32ull * n_leaves)) return WM_ERR_WORKSPACE;
  if (!total) return WM_OK;  // nothing to copy
  int n_cu = 0;
  wm_status s = ensure_device(&n_cu);
  if (s != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // an asynchronous copy from pageable host memory has read its source when
  // it returns, so the local table may go out of scope
  if (hipMemcpyAsync(ws, t.data(), 32ull * n_leaves, hipMemcpyHostToDevice, st) != hipSuccess)
    return WM_ERR_HIP;
  return hip_status(launch_manifest(gather, flat, total, static_cast<const ManifestLeaf *>(ws),
                                    n_leaves, n_cu, stream));
}

}  // namespace

extern "C" {

wm_status wm_flatten(const wm_leaf *leaves, uint32_t n_leaves, void *flat, uint64_t flat_cap,
                     void *ws, uint64_t ws_bytes, void *stream) {
  return manifest_call(true, leaves, n_leaves, flat, flat_cap, ws, ws_bytes, stream);
}

wm_status wm_rehydrate(const void *flat, uint64_t flat_cap, const wm_leaf *leaves,
                       uint32_t n_leaves, void *ws, uint64_t ws_bytes, void *stream) {
  return manifest_call(false, leaves, n_leaves, const_cast<void *>(flat), flat_cap, ws, ws_bytes,
                       stream);
}

}  // extern "C"

extern "C" {

wm_status wm_precopy_round(const void *cur, void *shipped, void *dest, uint64_t nbytes,
                           const wm_params *p, const wm_move_buffers *b, uint32_t crc_valid,
                           uint32_t *n_dirty_host, void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if ((nbytes & 1u) || crc_valid > 1) return WM_ERR_INVALID_ARG;
  if (!b || !n_dirty_host || !b->crc || !b->dirty_idx || !b->n_dirty) return WM_ERR_INVALID_ARG;
  if (nbytes && (!cur || !shipped || !dest)) return WM_ERR_INVALID_ARG;
  if (nbytes && (cur == shipped || cur == dest || shipped == dest)) return WM_ERR_INVALID_ARG;
  if (!aligned16(shipped) || !aligned16(dest)) return WM_ERR_INVALID_ARG;
  // the checks of every call the round makes come first, so that an
  // argument error leaves everything untouched
  if (!b->payload || !b->payload_bytes || !aligned16(b->payload) || !aligned16(cur))
    return WM_ERR_INVALID_ARG;
  if (b->payload_cap < wm_payload_bound(nbytes, g.hdr_n, p)) return WM_ERR_CAPACITY;
  if (!b->ws_src || !aligned16(b->ws_src) || b->ws_src_bytes < ws_need(g, ws_layout(g.n_chunks)))
    return WM_ERR_WORKSPACE;
  if (!b->verdict || (nbytes && !b->staging) || !aligned16(b->staging)) return WM_ERR_INVALID_ARG;
  if (b->staging_cap < (uint64_t)g.n_chunks * kChunk) return WM_ERR_CAPACITY;
  const uint64_t ws_need = ws_layout(g.n_chunks).total;
  if (!b->ws_dst || !aligned16(b->ws_dst) || b->ws_dst_bytes < ws_need || b->ws_src == b->ws_dst)
    return WM_ERR_WORKSPACE;
  if (!crc_valid || g.tile_log2) {
    // every chunk checksummed, the dirty ones encoded, in one pass (chunks
    // above 64 KiB: the kept CRCs are chunk CRCs, not the tile receipts the
    // records need, so every tile is checksummed)
    s = wm_encode_step(cur, shipped, nbytes, p, b->crc, b->global_crc, b->dirty_idx, b->n_dirty,
                       b->payload, b->payload_cap, b->payload_bytes, b->ws_src, b->ws_src_bytes,
                       stream);
    if (s != WM_OK) return s;
  } else {
    // the CRCs of clean chunks are those of shipped, kept from earlier
    // rounds: diff, then checksum and encode only the dirty chunks (each
    // CRC from the same read as its record)
    s = wm_diff_dirty(cur, shipped, nbytes, p, b->dirty_idx, b->n_dirty, b->ws_src,
                      b->ws_src_bytes, stream);
    if (s != WM_OK) return s;
    int n_cu0 = 0;
    if ((s = ensure_device(&n_cu0)) != WM_OK) return s;
    n_cu0 = stream_cus(stream, n_cu0);
    const WsLayout L = ws_layout(g.n_chunks);
    if (g.codec != WM_CODEC_EXPFOR) {
      // format v2 takes its receipts from a checksum of every chunk
      if (launch_checksum(cur, g, b->crc, nullptr, n_cu0, stream) != 0 ||
          launch_encode_v2(cur, g, b->dirty_idx, b->n_dirty, b->crc, nullptr, b->global_crc,
                           b->payload, b->payload_bytes, b->ws_src, L, n_cu0,
                           stream) != 0)
        return WM_ERR_HIP;
    } else if (launch_encode(0, cur, nullptr, g, b->dirty_idx, b->n_dirty, nullptr, b->crc,
                             b->global_crc, nullptr, nullptr, b->payload, b->payload_bytes,
                             b->ws_src, L, n_cu0, stream) != 0) {
      return WM_ERR_HIP;
    }
  }
  s = wm_decode_verify(b->payload, b->payload_cap, nbytes, p, b->staging, b->staging_cap,
                       b->verdict, b->rec_status, b->ws_dst, b->ws_dst_bytes, stream);
  if (s != WM_OK) return s;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  if (nbytes) {
    // both installs are conditional on the same device verdict word
    if (launch_commit(dest, g, b->staging, b->payload, b->verdict, n_cu, stream) != 0 ||
        launch_commit(shipped, g, b->staging, b->payload, b->verdict, n_cu, stream) != 0)
      return WM_ERR_HIP;
  }
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  uint32_t v[2] = {0xFFFFFFFFu, 0};
  if (hipMemcpyAsync(&v[0], b->verdict, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(&v[1], b->n_dirty, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return WM_ERR_HIP;
  *n_dirty_host = v[1];
  return v[0] == 0 ? WM_OK : WM_VERIFY_FAILED;
}

}  // extern "C"

namespace {

uint32_t host_u32(const uint8_t *p) {
  return (uint32_t)p[0] | (uint32_t)p[1] << 8 | (uint32_t)p[2] << 16 | (uint32_t)p[3] << 24;
}
uint64_t host_u64(const uint8_t *p) { return host_u32(p) | (uint64_t)host_u32(p + 4) << 32; }

// Two events (copy stream -> decode stream, and back) per thread and
// device, made on first use and kept for the process: one thread's calls
// are sequential, and a stream wait binds to the event's record at the time
// of the wait, so the same two serve every batch of every call.
hipEvent_t *order_events() {
  struct PerThread {
    hipEvent_t e[kMaxDevices][2];
    bool made[kMaxDevices];
  };
  thread_local PerThread t = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  if (!t.made[dev]) {
    for (int i = 0; i < 2; ++i)
      if (hipEventCreateWithFlags(&t.e[dev][i], hipEventDisableTiming) != hipSuccess)
        return nullptr;
    t.made[dev] = true;
  }
  return t.e[dev];
}

struct Batch {
  uint64_t b0, b1;  // payload bytes [b0, b1)
  uint32_t r0, r1;  // records [r0, r1)
};

// Copy schedule of a payload held in host memory: the header and the table
// first, then the records in batches of about batch_bytes.  Only the order
// of the copies depends on these host reads; whether the payload is valid is
// decided on the device.  A header or table that does not parse gives one
// batch of everything.
std::vector<Batch> receive_schedule(const uint8_t *h, uint64_t bytes, uint32_t n_chunks,
                                    uint64_t batch_bytes, uint64_t *table_off) {
  std::vector<Batch> out;
  uint32_t n_rec = 0;
  uint64_t total = 0;
  bool ok = bytes >= 64;
  if (ok) {
    n_rec = host_u32(h + 24);
    total = host_u64(h + 32);
    ok = n_rec <= n_chunks && total <= bytes && 64u + 16ull * n_rec <= total;
  }
  if (!ok) {
    *table_off = bytes;
    out.push_back(Batch{0, bytes, 0, n_chunks});
    return out;
  }
  const uint64_t toff = total - 16ull * n_rec;
  *table_off = toff;
  batch_bytes = std::max<uint64_t>(batch_bytes, (toff - 64u) / kMaxBatches + 1u);
  auto rec_off = [&](uint32_t r) {  // clamped into the record area
    const uint64_t o = host_u64(h + toff + 16ull * r + 8);
    return std::min(std::max<uint64_t>(o, 64u), toff);
  };
  uint64_t b0 = 64;
  uint32_t r0 = 0;
  while (r0 < n_rec) {
    uint32_t r1 = r0 + 1;
    uint64_t b1 = r1 < n_rec ? std::max(rec_off(r1), b0) : toff;
    while (r1 < n_rec && b1 - b0 < batch_bytes) {
      ++r1;
      b1 = r1 < n_rec ? std::max(rec_off(r1), b0) : toff;
    }
    out.push_back(Batch{b0, b1, r0, r1});
    b0 = b1;
    r0 = r1;
  }
  return out;
}

}  // namespace

extern "C" {

wm_status wm_receive_verify(const void *host_payload, uint64_t payload_bytes, void *payload,
                            uint64_t payload_cap, uint64_t nbytes, const wm_params *p,
                            void *staging, uint64_t staging_cap, uint32_t *verdict,
                            uint32_t *rec_status, void *ws, uint64_t ws_bytes,
                            uint64_t batch_bytes, void *copy_stream, void *stream) {
  ChunkGeom g;
  wm_status s = make_geom(nbytes, p, &g);
  if (s != WM_OK) return s;
  if (nbytes & 1u) return WM_ERR_INVALID_ARG;
  if (!payload || !verdict || !aligned16(payload)) return WM_ERR_INVALID_ARG;
  if (payload_bytes && !host_payload) return WM_ERR_INVALID_ARG;
  if ((staging_cap && !staging) || !aligned16(staging)) return WM_ERR_INVALID_ARG;
  if (payload_bytes > payload_cap) return WM_ERR_CAPACITY;
  WsLayout L = ws_layout(g.n_chunks);
  if (!ws || ws_bytes < L.total || !aligned16(ws)) return WM_ERR_WORKSPACE;
  int n_cu = 0;
  if ((s = ensure_device(&n_cu)) != WM_OK) return s;
  n_cu = stream_cus(stream, n_cu);
  const uint8_t *h = static_cast<const uint8_t *>(host_payload);
  uint8_t *d = static_cast<uint8_t *>(payload);
  uint64_t table_off = payload_bytes;
  const std::vector<Batch> batches =
      receive_schedule(h, payload_bytes, g.n_chunks, batch_bytes, &table_off);
  hipStream_t cs = reinterpret_cast<hipStream_t>(copy_stream);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  auto records = g.codec != WM_CODEC_EXPFOR ? launch_decode_records_v2 : launch_decode_records;
  hipEvent_t *ev = order_events();
  if (!ev) return WM_ERR_HIP;
  // `to` waits for the work enqueued on `from` so far (the wait binds to
  // the event's latest record, so the event is reused for every batch)
  auto order = [&](hipStream_t from, hipStream_t to) -> bool {
    hipEvent_t e = ev[from == cs ? 0 : 1];
    return hipEventRecord(e, from) == hipSuccess && hipStreamWaitEvent(to, e, 0) == hipSuccess;
  };
  // the decode stream waits for the copies enqueued so far
  auto arrived = [&]() { return cs == st || order(cs, st); };
  auto copy = [&](uint64_t b0, uint64_t b1) {
    return b1 <= b0 ||
           hipMemcpyAsync(d + b0, h + b0, b1 - b0, hipMemcpyHostToDevice, cs) == hipSuccess;
  };
  // the copies overwrite payload: they start after the work enqueued on
  // stream before this call (an earlier decode of the same buffer)
  bool ok = cs == st || order(st, cs);
  const bool parsed = !(batches.size() == 1 && batches[0].b0 == 0);
  if (parsed) {
    // the header and the table (which the checks and every batch read)
    // first, then the records batch by batch
    ok = copy(0, 64) && copy(table_off, payload_bytes) && arrived() &&
         launch_decode_begin(payload, payload_bytes, g, staging_cap, ws, L, stream) == 0;
    for (size_t i = 0; ok && i < batches.size(); ++i) {
      const Batch &b = batches[i];
      ok = copy(b.b0, b.b1) && arrived() &&
           records(payload, g, staging, rec_status, ws, L, n_cu, b.r0, b.r1, stream) == 0;
    }
  } else {
    ok = copy(0, payload_bytes) && arrived() &&
         launch_decode_begin(payload, payload_bytes, g, staging_cap, ws, L, stream) == 0 &&
         records(payload, g, staging, rec_status, ws, L, n_cu, 0u, g.n_chunks, stream) == 0;
  }
  ok = ok && launch_decode_end(g, verdict, ws, L, stream) == 0;
  return ok ? WM_OK : WM_ERR_HIP;
}

}  // extern "C"
