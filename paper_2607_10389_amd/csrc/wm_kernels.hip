// wm_kernels.hip -- CDNA4 (gfx950) kernels of the exact-state mover.
//
// Data layout.  A 64 KiB chunk is processed by one 512-thread workgroup with
// the chunk held in registers: wave w owns bytes [w*8K, (w+1)*8K); lane t of
// the wave owns 16 bytes of each 1 KiB row h (offset w*8K + h*1K + 16t), so
// every load and store is a coalesced 128-bit access.
//
// CRC (§4 "Sufficiency", §6.5: per-chunk zlib CRC, GF(2)-combined).  Each lane
// runs four independent dword "column" streams down its rows:
//     v <- F^1024(v ^ d)
// (the next dword of the column is 1 KiB further on).  A lane's four columns
// merge into one value, the 64 lane values of a wave merge through a 6-level
// shuffle tree of byte-table shifts, and the 8 wave values merge through one
// GF(2) matrix per wave.  The F^1024 tables are the hot ones: 16 copies in
// LDS, addressed as byte*256 + slot*64 + copy*4 with v_perm, where each group
// of 16 lanes starts at a different table slot so that one ds_read touches
// every bank once.  All other shift tables are read rarely and kept single.
#include <hip/hip_runtime.h>

#include "wm_internal.h"

namespace wm {

__device__ CrcTables g_tables[2];

// ------------------------------------------------------------ LDS layout --
constexpr uint32_t kLdsG = 0;                       // 64 KiB, replicated F^1024
constexpr uint32_t kLdsF4 = 65536;                  // 4 KiB
constexpr uint32_t kLdsF8 = kLdsF4 + 4096;          // 4 KiB
constexpr uint32_t kLdsTree = kLdsF8 + 4096;        // 6 x 4 KiB
constexpr uint32_t kLdsCrcEnd = kLdsTree + kTree * 4096;  // 98304
constexpr uint32_t kLdsMisc = kLdsCrcEnd;           // 8 KiB of small scratch
constexpr uint32_t kLdsMiscBytes = 8192;
constexpr uint32_t kLdsHist = kLdsMisc + kLdsMiscBytes;  // 16 KiB histogram
constexpr uint32_t kLdsCodes = kLdsHist + 16384;         // 28 KiB code staging
constexpr uint32_t kLdsCodesBytes = 7 * (kChunk / 2) / 8;
constexpr uint32_t kLdsEncode = kLdsCodes + kLdsCodesBytes;  // 147456
constexpr uint32_t kLdsBase = kLdsMisc + kLdsMiscBytes;      // 106496

// misc scratch (u32 index into kLdsMisc)
constexpr uint32_t M_PART = 0;      // [kWaves] wave CRC partials
constexpr uint32_t M_BCAST = 16;    // [32] broadcast words
constexpr uint32_t M_ESCW = 64;     // [kWaves] escapes per wave
constexpr uint32_t M_WKEY = 80;     // [4][8] window keys per wave
constexpr uint32_t M_WMISC = 120;   // [4][2] distinct / single per wave
constexpr uint32_t M_WSUM = 136;    // [4] wave sums of the histogram scan
constexpr uint32_t M_H = 256;       // [256] histogram
constexpr uint32_t M_P = 512;       // [257] prefix of the histogram
constexpr uint32_t M_QP = 1024;     // [4][128] quarter partials

static_assert(kLdsEncode <= 163840, "encoder LDS must fit one CU");

extern __shared__ __align__(16) uint8_t lds[];

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// 128-bit streaming load that does not allocate in the caches.
__device__ __forceinline__ uint4 ldg_nt(const void *p) {
  v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint32_t lds_u32(uint32_t off) {
  return *reinterpret_cast<const uint32_t *>(lds + off);
}
__device__ __forceinline__ uint32_t *misc() {
  return reinterpret_cast<uint32_t *>(lds + kLdsMisc);
}

// Byte-table application of a shift stored at LDS offset `off`.
__device__ __forceinline__ uint32_t tab4(uint32_t off, uint32_t x) {
  return lds_u32(off + ((x & 255u) << 2)) ^
         lds_u32(off + 1024u + (((x >> 8) & 255u) << 2)) ^
         lds_u32(off + 2048u + (((x >> 16) & 255u) << 2)) ^
         lds_u32(off + 3072u + ((x >> 24) << 2));
}

// Per-lane constants for the replicated F^1024 lookups.
struct GLane {
  uint32_t k[4], sel[4];
};

__device__ __forceinline__ GLane glane_make() {
  GLane gl;
  uint32_t lane = threadIdx.x & 63u;
  uint32_t grp = (lane >> 4) & 3u, copy = lane & 15u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t slot = (i + grp) & 3u;
    gl.k[i] = slot * 64u + copy * 4u;
    // result byte0 <- k byte0, byte1 <- x byte `slot`, bytes 2,3 <- 0
    gl.sel[i] = 0x0C0C0000u | ((4u + slot) << 8);
  }
  return gl;
}

__device__ __forceinline__ uint32_t g_step(uint32_t x, const GLane &gl) {
  uint32_t a0 = __builtin_amdgcn_perm(x, gl.k[0], gl.sel[0]);
  uint32_t a1 = __builtin_amdgcn_perm(x, gl.k[1], gl.sel[1]);
  uint32_t a2 = __builtin_amdgcn_perm(x, gl.k[2], gl.sel[2]);
  uint32_t a3 = __builtin_amdgcn_perm(x, gl.k[3], gl.sel[3]);
  return lds_u32(kLdsG + a0) ^ lds_u32(kLdsG + a1) ^ lds_u32(kLdsG + a2) ^
         lds_u32(kLdsG + a3);
}

__device__ void load_crc_tables(uint32_t kind) {
  const CrcTables &T = g_tables[kind];
  uint32_t *g = reinterpret_cast<uint32_t *>(lds + kLdsG);
  for (uint32_t i = threadIdx.x; i < 16384u; i += blockDim.x)
    g[i] = T.row[(i >> 4) & 3u][i >> 6];
  const uint32_t *src = &T.f4[0][0];  // f4, f8, tree are contiguous
  uint32_t *dst = reinterpret_cast<uint32_t *>(lds + kLdsF4);
  for (uint32_t i = threadIdx.x; i < (2u + kTree) * 1024u; i += blockDim.x)
    dst[i] = src[i];
}

// Columns applied to v (uniform matrix, scalar loads).
__device__ __forceinline__ uint32_t mat_apply(const uint32_t *__restrict__ m,
                                              uint32_t v) {
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 32; ++i) r ^= ((v >> i) & 1u) ? m[i] : 0u;
  return r;
}

// F^m(v) for any m >= 0, through the power-of-two shift matrices.
__device__ uint32_t shift_bytes(const CrcTables &T, uint64_t m, uint32_t v) {
  for (int i = 0; m; ++i, m >>= 1)
    if (m & 1) v = mat_apply(T.pow2[i], v);
  return v;
}

// Standard CRC (init/xorout ~0) of 4*nw bytes held as words, with F^4 tables
// in LDS.  One lane; used for headers and table entries.
__device__ __forceinline__ uint32_t crc_words(const uint32_t *w, int nw) {
  uint32_t s = 0xFFFFFFFFu;
  for (int i = 0; i < nw; ++i) s = tab4(kLdsF4, s ^ w[i]);
  return s ^ 0xFFFFFFFFu;
}

// -------------------------------------------------------- chunk movement --

struct Lane {
  uint32_t wave, lane, off0;  // off0: chunk offset of row 0
};
__device__ __forceinline__ Lane lane_info() {
  Lane l;
  l.wave = threadIdx.x >> 6;
  l.lane = threadIdx.x & 63u;
  l.off0 = l.wave * kSub + l.lane * 16u;
  return l;
}

__device__ __forceinline__ uint32_t chunk_len(const ChunkGeom &g, uint32_t c) {
  return c + 1 == g.n_chunks ? g.tail_len : kChunk;
}

__device__ __forceinline__ uint4 load16_partial(const uint8_t *p, uint32_t n) {
  uint32_t w[4] = {0, 0, 0, 0};
  for (uint32_t b = 0; b < n; ++b) w[b >> 2] |= (uint32_t)p[b] << (8 * (b & 3));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Load a chunk of `len` bytes into registers; bytes past len read as zero.
__device__ __forceinline__ void load_chunk(const uint8_t *__restrict__ base,
                                           uint32_t len, const Lane &l,
                                           uint4 (&d)[kRows]) {
  if (len == kChunk) {
#pragma unroll
    for (int h = 0; h < kRows; ++h)
      d[h] = ldg_nt(base + l.off0 + h * kRow);
  } else {
#pragma unroll
    for (int h = 0; h < kRows; ++h) {
      uint32_t off = l.off0 + h * kRow;
      if (off + 16u <= len)
        d[h] = *reinterpret_cast<const uint4 *>(base + off);
      else if (off < len)
        d[h] = load16_partial(base + off, len - off);
      else
        d[h] = make_uint4(0, 0, 0, 0);
    }
  }
}

// Store the first `len` bytes of a chunk held in registers (pieces that start
// below len are stored whole; their bytes past len are zero in registers).
__device__ __forceinline__ void store_chunk(uint8_t *__restrict__ base,
                                            uint32_t len, const Lane &l,
                                            const uint4 (&d)[kRows],
                                            bool pad_ok) {
#pragma unroll
  for (int h = 0; h < kRows; ++h) {
    uint32_t off = l.off0 + h * kRow;
    if (off + 16u <= len || (pad_ok && off < len)) {
      *reinterpret_cast<uint4 *>(base + off) = d[h];
    } else if (off < len) {
      const uint32_t w[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
      for (uint32_t b = 0; b < len - off; ++b)
        base[off + b] = (uint8_t)(w[b >> 2] >> (8 * (b & 3)));
    }
  }
}

// Wave-level CRC value Q of the wave's 8 KiB (valid in lane 0).
__device__ __forceinline__ uint32_t wave_q(const uint4 (&d)[kRows],
                                           const GLane &gl) {
  uint32_t v0 = 0, v1 = 0, v2 = 0, v3 = 0;
#pragma unroll
  for (int h = 0; h < kRows; ++h) {
    v0 = g_step(v0 ^ d[h].x, gl);
    v1 = g_step(v1 ^ d[h].y, gl);
    v2 = g_step(v2 ^ d[h].z, gl);
    v3 = g_step(v3 ^ d[h].w, gl);
  }
  // u = F^12 v0 ^ F^8 v1 ^ F^4 v2 ^ v3
  uint32_t u = tab4(kLdsF8, tab4(kLdsF4, v0) ^ v1) ^ tab4(kLdsF4, v2) ^ v3;
#pragma unroll
  for (int lv = 0; lv < kTree; ++lv) {
    uint32_t s = tab4(kLdsTree + lv * 4096u, u);
    uint32_t o = __shfl_down(u, 1u << lv, 64);
    u = s ^ o;
  }
  return u;
}

// Whole-workgroup chunk CRC.  Contains two barriers; the result is valid in
// thread 0 only.
__device__ __forceinline__ uint32_t chunk_crc(const uint4 (&d)[kRows],
                                              const GLane &gl, const Lane &l,
                                              uint32_t len, const ChunkGeom &g,
                                              const CrcTables &T) {
  uint32_t q = wave_q(d, gl);
  if (l.lane == 0) misc()[M_PART + l.wave] = mat_apply(T.wave_mat[l.wave], q);
  __syncthreads();
  uint32_t crc = 0;
  if (threadIdx.x == 0) {
    uint32_t raw = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) raw ^= misc()[M_PART + w];
    crc = (len == kChunk) ? raw ^ T.k_full
                          : mat_apply(g.tail_mat, raw) ^ g.k_tail;
  }
  __syncthreads();
  return crc;
}

// -------------------------------------------------------------- checksum --

__global__ __launch_bounds__(kThreads) void k_checksum(
    const uint8_t *__restrict__ data, ChunkGeom g,
    uint32_t *__restrict__ crc_out) {
  load_crc_tables(g.crc_kind);
  __syncthreads();
  const CrcTables &T = g_tables[g.crc_kind];
  const GLane gl = glane_make();
  const Lane l = lane_info();
  uint32_t c = blockIdx.x;
  uint4 d[kRows];
  if (c < g.n_chunks) load_chunk(data + (uint64_t)c * kChunk, chunk_len(g, c), l, d);
  while (c < g.n_chunks) {
    uint32_t cn = c + gridDim.x;
    uint4 dn[kRows];
    if (cn < g.n_chunks) load_chunk(data + (uint64_t)cn * kChunk, chunk_len(g, cn), l, dn);
    uint32_t crc = chunk_crc(d, gl, l, chunk_len(g, c), g, T);
    if (threadIdx.x == 0) crc_out[c] = crc;
#pragma unroll
    for (int h = 0; h < kRows; ++h) d[h] = dn[h];
    c = cn;
  }
}

// --------------------------------------------------------------- combine --
// CRC of a concatenation from the CRCs of its pieces: n pieces of 2^log2span
// bytes except the last, of last_len bytes.  One 1024-thread workgroup per
// job.

struct CombineJob {
  const uint32_t *vals;
  const uint32_t *n_dev;  // if non-null, n = *n_dev
  uint32_t n;
  uint32_t log2span;
  uint32_t last_len;
  uint32_t kind;
  uint32_t *out;
};

struct CombineJobs {
  CombineJob job[2];
};

__global__ __launch_bounds__(1024) void k_combine(CombineJobs jobs) {
  const CombineJob &J = jobs.job[blockIdx.x];
  const CrcTables &T = g_tables[J.kind];
  uint32_t n = J.n_dev ? *J.n_dev : J.n;
  __shared__ uint32_t tabF[1024];   // byte tables of F^span
  __shared__ uint32_t v[1024];
  uint32_t t = threadIdx.x;
  // build F^span tables: entry (j, b) = F^span(b << 8j)
  tabF[t] = mat_apply(T.pow2[J.log2span], (t & 255u) << (8 * (t >> 8)));
  __syncthreads();
  if (n == 0) {
    if (t == 0) *J.out = 0u;
    return;
  }
  uint32_t np = n - 1;  // all but the last piece, each exactly span bytes
  uint32_t m = 1, lm = 0;
  while (m * 1024u < np) {
    m <<= 1;
    ++lm;
  }
  // per-thread Horner over pieces [t*m, t*m + m) within [0, np)
  uint32_t lo = t * m, hi = min(lo + m, np);
  uint32_t acc = 0;
  for (uint32_t i = lo; i < hi; ++i) {
    uint32_t x = acc;
    acc = tabF[x & 255u] ^ tabF[256u + ((x >> 8) & 255u)] ^
          tabF[512u + ((x >> 16) & 255u)] ^ tabF[768u + (x >> 24)];
    acc ^= J.vals[i];
  }
  v[t] = acc;
  __syncthreads();
  uint32_t gc = np >> lm;           // complete groups (m pieces each)
  uint32_t rem = np - (gc << lm);   // pieces in the partial group (index gc)
  // perfect trees over aligned power-of-two blocks of complete groups
  for (uint32_t lv = 0; (1u << lv) < 1024u; ++lv) {
    uint32_t stride = 2u << lv;
    uint32_t i = t * stride;
    uint32_t x = 0;
    bool act = i + stride <= gc;
    if (act) x = mat_apply(T.pow2[lv + lm + J.log2span], v[i]) ^ v[i + (stride >> 1)];
    __syncthreads();
    if (act) v[i] = x;
    __syncthreads();
  }
  if (t == 0) {
    uint32_t r = 0;
    bool have = false;
    uint32_t pos = 0;
    for (int b = 10; b >= 0; --b) {
      if (!((gc >> b) & 1u)) continue;
      r = have ? mat_apply(T.pow2[b + lm + J.log2span], r) ^ v[pos] : v[pos];
      have = true;
      pos += 1u << b;
    }
    if (rem) {
      r = have ? shift_bytes(T, (uint64_t)rem << J.log2span, r) ^ v[gc] : v[gc];
      have = true;
    }
    uint32_t last = J.vals[n - 1];
    r = have ? shift_bytes(T, J.last_len, r) ^ last : last;
    *J.out = r;
  }
}

// ------------------------------------------------------------------ diff --

__global__ __launch_bounds__(256) void k_diff(const uint8_t *__restrict__ cur,
                                              const uint8_t *__restrict__ prev,
                                              ChunkGeom g,
                                              uint32_t *__restrict__ flags) {
  for (uint32_t c = blockIdx.x; c < g.n_chunks; c += gridDim.x) {
    uint32_t len = chunk_len(g, c);
    const uint8_t *a = cur + (uint64_t)c * kChunk;
    const uint8_t *b = prev + (uint64_t)c * kChunk;
    uint32_t diff = 0;
    if (len == kChunk) {
#pragma unroll 4
      for (uint32_t off = threadIdx.x * 16u; off < kChunk; off += 4096u) {
        uint4 x = ldg_nt(a + off);
        uint4 y = ldg_nt(b + off);
        diff |= (x.x ^ y.x) | (x.y ^ y.y) | (x.z ^ y.z) | (x.w ^ y.w);
      }
    } else {
      for (uint32_t off = threadIdx.x; off < len; off += 256u) diff |= a[off] ^ b[off];
    }
    int d = __syncthreads_or(diff != 0);
    if (threadIdx.x == 0) flags[c] = d ? 1u : 0u;
  }
}

// Single-workgroup stream compaction of flags into ascending indices.
__global__ __launch_bounds__(1024) void k_compact(const uint32_t *__restrict__ flags,
                                                  uint32_t n,
                                                  uint32_t *__restrict__ idx,
                                                  uint32_t *__restrict__ count) {
  __shared__ uint32_t wsum[16];
  __shared__ uint32_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  for (uint32_t base = 0; base < n; base += 1024u) {
    uint32_t i = base + threadIdx.x;
    bool f = i < n && flags[i];
    unsigned long long m = __ballot(f);
    uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                               __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (lane == 0) wsum[wave] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t before = carry;
    for (uint32_t w = 0; w < wave; ++w) before += wsum[w];
    if (f) idx[before + below] = i;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t s = 0;
      for (int w = 0; w < 16; ++w) s += wsum[w];
      carry += s;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *count = carry;
}

// ---------------------------------------------------------------- encode --

constexpr int kModeList = 0, kModeAll = 1, kModeStep = 2;
constexpr uint64_t kFlagAgg = 1, kFlagIncl = 2;

struct EncArgs {
  const uint8_t *cur;
  const uint8_t *prev;
  const uint32_t *idx;
  const uint32_t *n_idx;
  const uint32_t *crc_in;
  uint32_t *crc_out;
  uint32_t *dirty_idx;
  uint8_t *payload;
  uint8_t *ws;
  WsLayout L;
  int mode;
};

__device__ __forceinline__ uint64_t pad16(uint64_t x) { return (x + 15u) & ~15ull; }

// Chunk of a work item; a caller's list must be ascending and in range, a
// violation returns an out-of-range index (the item is then flagged).
__device__ __forceinline__ uint32_t item_chunk(const EncArgs &a, uint32_t item,
                                               const ChunkGeom &g) {
  if (a.mode != kModeList) return item;
  uint32_t c = a.idx[item];
  if (c >= g.n_chunks || (item > 0 && a.idx[item - 1] >= c)) return 0xFFFFFFFFu;
  return c;
}

__device__ __forceinline__ void status_store(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t status_load(const uint64_t *p) {
  return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t lanes_below(unsigned long long m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Exponent histogram of the chunk's valid words into H[256] (misc).  Uses the
// 32-copy packed histogram; contains barriers.
__device__ void chunk_histogram(const uint4 (&d)[kRows], const Lane &l,
                                uint32_t n_words) {
  uint32_t *hist = reinterpret_cast<uint32_t *>(lds + kLdsHist);
  uint4 *h4 = reinterpret_cast<uint4 *>(hist);
  for (uint32_t i = threadIdx.x; i < 1024u; i += kThreads) h4[i] = make_uint4(0, 0, 0, 0);
  __syncthreads();
  const uint32_t copy = threadIdx.x & 31u;
  const bool full = n_words == kChunk / 2;
#pragma unroll
  for (int h = 0; h < kRows; ++h) {
    const uint32_t w0 = (l.off0 + h * kRow) >> 1;  // first word of the piece
    const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        if (full || w0 + 2 * j + half < n_words) {
          uint32_t e = (x[j] >> (7 + 16 * half)) & 255u;
          atomicAdd(&hist[(e >> 1) * 32u + copy], 1u << ((e & 1u) * 16u));
        }
      }
    }
  }
  __syncthreads();
  // sum the 32 copies: thread (pair p, quarter q) sums 8 copies
  {
    uint32_t t = threadIdx.x;
    uint32_t p = t & 127u, q = t >> 7;
    uint32_t s = 0;
#pragma unroll
    for (uint32_t c = 8 * q; c < 8 * q + 8; ++c) s += hist[p * 32u + ((c + p) & 31u)];
    misc()[M_QP + q * 128u + p] = s;
  }
  __syncthreads();
  if (threadIdx.x < 128u) {
    uint32_t p = threadIdx.x;
    uint32_t s = misc()[M_QP + p] + misc()[M_QP + 128 + p] + misc()[M_QP + 256 + p] +
                 misc()[M_QP + 384 + p];
    misc()[M_H + 2 * p] = s & 0xFFFFu;
    misc()[M_H + 2 * p + 1] = s >> 16;
  }
  __syncthreads();
}

struct Plan {
  uint32_t mode, k, base, n_esc;
  uint64_t size;
};

// Mode choice from H (payload format v1 §3.3); result broadcast in misc.
__device__ Plan chunk_plan(uint32_t n_words) {
  uint32_t t = threadIdx.x, lane = t & 63u, wave = t >> 6;
  uint32_t *M = misc();
  if (t < 256u) {
    // inclusive scan of H over the 256 bins
    uint32_t h = M[M_H + t];
    uint32_t s = h;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      uint32_t y = __shfl_up(s, o, 64);
      if (lane >= (uint32_t)o) s += y;
    }
    if (lane == 63u) M[M_WSUM + wave] = s;
    unsigned long long nz = __ballot(h > 0);
    if (lane == 0) {
      M[M_WMISC + 2 * wave] = (uint32_t)__popcll(nz);
      M[M_WMISC + 2 * wave + 1] = nz ? wave * 64u + 63u - __clzll(nz) : 0u;
    }
    M[M_P + 1 + t] = s;
  }
  if (t == 0) M[M_P] = 0;
  __syncthreads();
  if (t < 256u) {
    uint32_t add = 0;
    for (uint32_t w = 0; w < wave; ++w) add += M[M_WSUM + w];
    M[M_P + 1 + t] += add;
  }
  __syncthreads();
  if (t < 256u) {
    uint32_t pb = M[M_P + t];
#pragma unroll
    for (int k = 1; k <= 7; ++k) {
      uint32_t end = min(t + (1u << k) - 1u, 256u);
      uint32_t key = ((M[M_P + end] - pb) << 8) | (255u - t);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) key = max(key, (uint32_t)__shfl_xor(key, o, 64));
      if (lane == 0) M[M_WKEY + wave * 8 + k] = key;
    }
  }
  __syncthreads();
  if (t == 0) {
    uint32_t distinct = 0, only = 0;
    for (int w = 0; w < 4; ++w) {
      distinct += M[M_WMISC + 2 * w];
      if (M[M_WMISC + 2 * w]) only = max(only, M[M_WMISC + 2 * w + 1]);
    }
    uint64_t n = n_words;
    Plan best = {0u, 0u, 0u, 0u, 16u + pad16(2 * n)};
    if (distinct == 1) {
      uint64_t s = 16u + pad16(n);
      if (s < best.size) best = Plan{1u, 0u, only, 0u, s};
    }
    for (uint32_t k = 1; k <= 7; ++k) {
      uint32_t key = 0;
      for (int w = 0; w < 4; ++w) key = max(key, M[M_WKEY + w * 8 + k]);
      uint32_t inside = key >> 8, base = 255u - (key & 255u);
      uint32_t esc = n_words - inside;
      uint64_t s = 16u + pad16((n * k + 7) / 8) + pad16(esc) + pad16(n);
      if (s < best.size) best = Plan{1u, k, base, esc, s};
    }
    M[M_BCAST + 0] = best.mode;
    M[M_BCAST + 1] = best.k;
    M[M_BCAST + 2] = best.base;
    M[M_BCAST + 3] = best.n_esc;
    M[M_BCAST + 4] = (uint32_t)best.size;
  }
  __syncthreads();
  Plan p;
  p.mode = M[M_BCAST + 0];
  p.k = M[M_BCAST + 1];
  p.base = M[M_BCAST + 2];
  p.n_esc = M[M_BCAST + 3];
  p.size = M[M_BCAST + 4];
  return p;
}

// Exclusive prefix (records, record bytes / 16) of `item` by decoupled
// look-back: wave 0 reads 64 predecessors per round trip and stops at the
// nearest inclusive one.  Every item publishes its aggregate before its own
// look-back, and tickets are taken in order by running workgroups, so every
// predecessor publishes eventually; the spin bound only guarantees
// termination if that were ever violated.
__device__ uint64_t lookback(const uint64_t *status, uint32_t item, WsCtl *ctl) {
  const uint32_t lane = threadIdx.x & 63u;
  uint64_t excl = 0;
  int64_t top = (int64_t)item - 1;
  uint32_t spins = 0;
  while (top >= 0) {
    const int64_t j = top - (int64_t)lane;
    const uint64_t s = j >= 0 ? status_load(&status[j]) : kFlagIncl;
    const uint32_t f = (uint32_t)(s & 3u);
    const unsigned long long incl = __ballot(f == kFlagIncl);
    const unsigned long long empty = __ballot(f == 0u);
    const uint32_t stop = incl ? (uint32_t)__ffsll((long long)incl) - 1u : 64u;
    const unsigned long long need = stop >= 63u ? ~0ull : ((2ull << stop) - 1ull);
    if (empty & need) {
      if (++spins > (1u << 22)) {
        if (lane == 0) atomicOr(&ctl->error, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      continue;
    }
    uint64_t v = lane <= stop ? (s >> 2) : 0ull;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    excl += v;
    if (stop < 64u) break;
    top -= 64;
  }
  return excl;
}

template <bool HAS_PREV>
__global__ __launch_bounds__(kThreads) void k_encode(EncArgs a, ChunkGeom g) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(a.ws + a.L.ctl);
  uint64_t *status = reinterpret_cast<uint64_t *>(a.ws + a.L.status);
  uint4 *tab_ws = reinterpret_cast<uint4 *>(a.ws + a.L.table);
  uint32_t *ecrc = reinterpret_cast<uint32_t *>(a.ws + a.L.entry_crc);
  const uint32_t n_items = a.mode == kModeList ? min(*a.n_idx, g.n_chunks) : g.n_chunks;
  const bool need_crc = a.crc_in == nullptr;
  constexpr bool has_prev = HAS_PREV;

  load_crc_tables(g.crc_kind);
  const CrcTables &T = g_tables[g.crc_kind];
  const GLane gl = glane_make();
  const Lane l = lane_info();
  uint32_t *M = misc();
  uint8_t *codes = lds + kLdsCodes;

  if (threadIdx.x == 0) {
    M[M_BCAST + 8] = atomicAdd(&ctl->ticket, 1u);
    M[M_BCAST + 13] = atomicAdd(&ctl->ticket, 1u);
  }
  __syncthreads();
  uint32_t item = M[M_BCAST + 8];
  uint32_t next = M[M_BCAST + 13];
  uint4 d[kRows], p[kRows];
  if (item < n_items) {
    uint32_t c = item_chunk(a, item, g);
    if (c < g.n_chunks) {
      load_chunk(a.cur + (uint64_t)c * kChunk, chunk_len(g, c), l, d);
      if (has_prev) load_chunk(a.prev + (uint64_t)c * kChunk, chunk_len(g, c), l, p);
    }
  }

  while (item < n_items) {
    uint4 dn[kRows], pn[kRows];
    if (next < n_items) {
      uint32_t cn = item_chunk(a, next, g);
      if (cn < g.n_chunks) {
        load_chunk(a.cur + (uint64_t)cn * kChunk, chunk_len(g, cn), l, dn);
        if (has_prev) load_chunk(a.prev + (uint64_t)cn * kChunk, chunk_len(g, cn), l, pn);
      }
    }

    // ---- one chunk (an invalid caller index is flagged and encoded as an
    // empty item so that the scan still completes)
    uint32_t c = item_chunk(a, item, g);
    const bool bad_index = c >= g.n_chunks;
    if (bad_index) {
      if (threadIdx.x == 0) atomicOr(&ctl->error, 2u);
      c = 0;
    }
    const uint32_t len = bad_index ? 0u : chunk_len(g, c);
    const uint32_t n_words = len / 2;
    uint32_t crc = 0;
    if (need_crc) crc = chunk_crc(d, gl, l, bad_index ? kChunk : len, g, T);
    else if (threadIdx.x == 0) crc = a.crc_in[c];

    bool dirty = !bad_index;
    if (has_prev && !bad_index) {
      uint32_t diff = 0;
#pragma unroll
      for (int h = 0; h < kRows; ++h)
        diff |= (d[h].x ^ p[h].x) | (d[h].y ^ p[h].y) | (d[h].z ^ p[h].z) | (d[h].w ^ p[h].w);
      dirty = __syncthreads_or(diff != 0) != 0;
    }

    Plan plan = {0u, 0u, 0u, 0u, 0u};
    if (dirty) {
      chunk_histogram(d, l, n_words);
      plan = chunk_plan(n_words);
    }
    // publish this item's aggregate (records, record bytes / 16)
    const uint64_t agg = ((uint64_t)(dirty ? 1u : 0u) << 2) |
                         ((uint64_t)(plan.size >> 4) << 26);
    if (threadIdx.x == 0 && item != 0) status_store(&status[item], agg | kFlagAgg);

    // codes into LDS staging, escape counts per row
    const uint32_t k = plan.k;
    const uint32_t esc_code = (1u << k) - 1u;
    const bool pack = dirty && plan.mode == 1 && k > 0;
    uint32_t row_rank[kRows];
    uint32_t wave_esc = 0;
    if (pack) {
      if (len != kChunk) {
        uint4 *c4 = reinterpret_cast<uint4 *>(codes);
        for (uint32_t i = threadIdx.x; i < kLdsCodesBytes / 16; i += kThreads)
          c4[i] = make_uint4(0, 0, 0, 0);
        __syncthreads();
      }
#pragma unroll
      for (int h = 0; h < kRows; ++h) {
        const uint32_t w0 = (l.off0 + h * kRow) >> 1;
        const uint32_t grp = w0 >> 3;
        const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
        uint64_t packed = 0;
        uint32_t lane_esc = 0;
        uint32_t before = 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          uint32_t e = (x[u >> 1] >> (7 + 16 * (u & 1))) & 255u;
          bool valid = w0 + u < n_words;
          uint32_t code = valid ? min(e - plan.base, esc_code) : 0u;
          packed |= (uint64_t)code << (u * k);
          bool esc = valid && code == esc_code;
          unsigned long long m = __ballot(esc);
          before += lanes_below(m);
          lane_esc += (uint32_t)__popcll(m);
        }
        row_rank[h] = wave_esc + before;
        wave_esc += lane_esc;
        if (w0 < n_words) {
          uint32_t at = grp * k;
          for (uint32_t b = 0; b < k; ++b) codes[at + b] = (uint8_t)(packed >> (8 * b));
        }
      }
      if (l.lane == 0) M[M_ESCW + l.wave] = wave_esc;
    }
    __syncthreads();

    // look-back for the exclusive prefix (records, bytes / 16); the next
    // ticket is taken here so its latency overlaps the look-back
    uint64_t excl = 0;
    uint32_t ticket = 0;
    if (threadIdx.x == 0) ticket = atomicAdd(&ctl->ticket, 1u);
    if (threadIdx.x < 64u) excl = lookback(status, item, ctl);
    if (threadIdx.x == 0) {
      M[M_BCAST + 13] = ticket;
      const uint64_t incl = excl + (agg >> 2);
      status_store(&status[item], (incl << 2) | kFlagIncl);
      if (item + 1 == n_items) {
        ctl->n_rec = (uint32_t)(incl & 0xFFFFFFu);
        ctl->payload_bytes = (incl >> 24) << 4;  // total record bytes
      }
      M[M_BCAST + 9] = (uint32_t)(excl & 0xFFFFFFu);      // record index
      M[M_BCAST + 10] = (uint32_t)(excl >> 24);           // bytes/16 low
      M[M_BCAST + 11] = (uint32_t)(excl >> 56);           // bytes/16 high
      M[M_BCAST + 12] = crc;
    }
    __syncthreads();
    const uint32_t rec_idx = M[M_BCAST + 9];
    const uint64_t rec_off =
        64u + (((uint64_t)M[M_BCAST + 10] | ((uint64_t)M[M_BCAST + 11] << 32)) << 4);
    crc = M[M_BCAST + 12];

    if (dirty) {
      uint8_t *rec = a.payload + rec_off;
      if (threadIdx.x == 0) {
        uint32_t hw[4];
        hw[0] = plan.mode | (k << 8) | (plan.base << 16);
        hw[1] = n_words;
        hw[2] = plan.n_esc;
        hw[3] = crc_words(hw, 3);
        *reinterpret_cast<uint4 *>(rec) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
        uint32_t ew[4] = {c, crc, (uint32_t)rec_off, (uint32_t)(rec_off >> 32)};
        tab_ws[rec_idx] = make_uint4(ew[0], ew[1], ew[2], ew[3]);
        ecrc[rec_idx] = crc_words(ew, 4);
        if (a.dirty_idx) a.dirty_idx[rec_idx] = c;
      }
      if (plan.mode == 0) {
        store_chunk(rec + 16, len, l, d, true);
      } else {
        const uint64_t code_bytes = ((uint64_t)n_words * k + 7) / 8;
        const uint64_t esc_off = 16 + pad16(code_bytes);
        const uint64_t sm_off = esc_off + pad16(plan.n_esc);
        // codes (whole 16-byte pieces, zero padding included)
        for (uint32_t i = threadIdx.x; i < pad16(code_bytes) / 16; i += kThreads)
          *reinterpret_cast<uint4 *>(rec + 16 + 16 * i) =
              *reinterpret_cast<const uint4 *>(codes + 16 * i);
        uint32_t esc_before = 0;
        for (uint32_t w = 0; w < l.wave; ++w) esc_before += pack ? M[M_ESCW + w] : 0u;
        // escapes and the sign/mantissa plane
#pragma unroll
        for (int h = 0; h < kRows; ++h) {
          const uint32_t w0 = (l.off0 + h * kRow) >> 1;
          const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
          uint32_t smw[2] = {0, 0};
          uint32_t rank = esc_before + (pack ? row_rank[h] : 0u);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            uint32_t w = (x[u >> 1] >> (16 * (u & 1))) & 0xFFFFu;
            uint32_t e = (w >> 7) & 255u;
            bool valid = w0 + u < n_words;
            uint32_t sm = ((w >> 8) & 0x80u) | (w & 0x7Fu);
            if (valid) smw[u >> 2] |= sm << (8 * (u & 3));
            if (pack && valid && min(e - plan.base, esc_code) == esc_code) {
              rec[esc_off + rank] = (uint8_t)e;
              ++rank;
            }
          }
          if (w0 < n_words)
            *reinterpret_cast<uint2 *>(rec + sm_off + w0) = make_uint2(smw[0], smw[1]);
        }
        if (threadIdx.x < 16u) {
          uint32_t t = threadIdx.x;
          if (plan.n_esc + t < pad16(plan.n_esc)) rec[esc_off + plan.n_esc + t] = 0;
          if (n_words + t < pad16(n_words)) rec[sm_off + n_words + t] = 0;
        }
      }
    }
    if (threadIdx.x == 0 && a.crc_out) a.crc_out[c] = crc;

#pragma unroll
    for (int h = 0; h < kRows; ++h) {
      d[h] = dn[h];
      if (HAS_PREV) p[h] = pn[h];
    }
    item = next;
    next = M[M_BCAST + 13];
    __syncthreads();  // everyone has read the ticket before it is rewritten
  }
}

// Zero the control block and the look-back words before an encode.
__global__ void k_encode_prepare(uint8_t *ws, WsLayout L, uint32_t n) {
  uint64_t *status = reinterpret_cast<uint64_t *>(ws + L.status);
  uint32_t *ctl = reinterpret_cast<uint32_t *>(ws + L.ctl);
  uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < 64u) ctl[i] = 0;
  for (; i < n; i += gridDim.x * blockDim.x) status[i] = 0;
}

// Table copy into the payload and the header.
__global__ __launch_bounds__(256) void k_encode_finish(
    uint8_t *__restrict__ payload, const uint8_t *__restrict__ ws, WsLayout L,
    ChunkGeom g, uint32_t full, const uint32_t *__restrict__ crcs,
    uint64_t *payload_bytes, uint32_t *n_dirty) {
  const WsCtl *ctl = reinterpret_cast<const WsCtl *>(ws + L.ctl);
  if (ctl->error) {  // invalid index list or an abandoned scan: no payload
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      *reinterpret_cast<uint4 *>(payload) = make_uint4(0, 0, 0, 0);
      if (payload_bytes) *payload_bytes = 0;
      if (n_dirty) *n_dirty = 0;
    }
    return;
  }
  const uint32_t n_rec = ctl->n_rec;
  const uint64_t table_off = 64u + ctl->payload_bytes;
  const uint4 *tab_ws = reinterpret_cast<const uint4 *>(ws + L.table);
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_rec;
       i += gridDim.x * blockDim.x)
    *reinterpret_cast<uint4 *>(payload + table_off + 16ull * i) = tab_ws[i];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const uint64_t total = table_off + 16ull * n_rec;
    uint32_t h[16];
    h[0] = 0x31564D57u;  // "WMV1"
    h[1] = 1u | (g.crc_kind << 16) | (1u << 24);
    h[2] = kChunk;
    h[3] = g.n_chunks;
    h[4] = (uint32_t)g.nbytes;
    h[5] = (uint32_t)(g.nbytes >> 32);
    h[6] = n_rec;
    h[7] = full;
    h[8] = (uint32_t)total;
    h[9] = (uint32_t)(total >> 32);
    h[10] = crcs[0];  // global CRC
    h[11] = crcs[1];  // table CRC
    h[12] = h[13] = h[14] = 0;
    // header CRC over bytes 0..59 with the byte-table step
    const uint32_t *t1 = g_tables[g.crc_kind].byte1;
    uint32_t s = 0xFFFFFFFFu;
    for (int i = 0; i < 60; ++i) {
      uint32_t b = (h[i >> 2] >> (8 * (i & 3))) & 255u;
      s = t1[(s ^ b) & 255u] ^ (s >> 8);
    }
    h[15] = s ^ 0xFFFFFFFFu;
    uint4 *out = reinterpret_cast<uint4 *>(payload);
    for (int i = 0; i < 4; ++i) out[i] = make_uint4(h[4 * i], h[4 * i + 1], h[4 * i + 2], h[4 * i + 3]);
    if (payload_bytes) *payload_bytes = total;
    if (n_dirty) *n_dirty = n_rec;
  }
}

// ---------------------------------------------------------------- decode --

__device__ __forceinline__ uint32_t ld_u32(const uint8_t *p) {
  return *reinterpret_cast<const uint32_t *>(p);
}
__device__ __forceinline__ uint64_t ld_u64(const uint8_t *p) {
  return (uint64_t)ld_u32(p) | ((uint64_t)ld_u32(p + 4) << 32);
}

// Header validation and control-block setup (one workgroup).
__global__ __launch_bounds__(256) void k_decode_prepare(
    const uint8_t *__restrict__ payload, uint64_t cap, ChunkGeom g,
    uint64_t staging_cap, uint8_t *ws, WsLayout L) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(ws + L.ctl);
  if (threadIdx.x != 0) return;
  ctl->ticket = 0;
  ctl->hdr_ok = 0;
  ctl->table_bad = 0;
  ctl->rec_bits = 0;
  ctl->n_rec = 0;
  ctl->payload_bytes = 0;
  ctl->table_off = 0;
  ctl->table_crc = 0;
  ctl->verdict_pre = 1u;  // header rejected unless every check passes
  if (cap < 64) return;
  const uint32_t *t1 = g_tables[g.crc_kind].byte1;
  uint32_t s = 0xFFFFFFFFu;
  for (int i = 0; i < 60; ++i) s = t1[(s ^ payload[i]) & 255u] ^ (s >> 8);
  if ((s ^ 0xFFFFFFFFu) != ld_u32(payload + 60)) return;
  if (ld_u32(payload) != 0x31564D57u) return;
  if (ld_u32(payload + 4) != (1u | (g.crc_kind << 16) | (1u << 24))) return;
  if (ld_u32(payload + 8) != kChunk || ld_u32(payload + 12) != g.n_chunks) return;
  if (ld_u64(payload + 16) != g.nbytes) return;
  uint32_t n_rec = ld_u32(payload + 24), flags = ld_u32(payload + 28);
  uint64_t total = ld_u64(payload + 32);
  if ((flags & ~1u) || ld_u32(payload + 48) || ld_u32(payload + 52) || ld_u32(payload + 56)) return;
  if (n_rec > g.n_chunks) return;
  if (64u + 16ull * n_rec > total || total > cap || (total & 15u)) return;
  if ((flags & 1u) && n_rec != g.n_chunks) return;
  if ((uint64_t)n_rec * kChunk > staging_cap) {
    ctl->verdict_pre = 16u;
    return;
  }
  ctl->n_rec = n_rec;
  ctl->payload_bytes = total;
  ctl->table_off = total - 16ull * n_rec;
  ctl->table_crc = ld_u32(payload + 44);
  ctl->verdict_pre = 0;
  ctl->hdr_ok = 1;
  if (n_rec == 0 && total != 64u) ctl->table_bad = 1;
}

// One wave decodes one record: no barriers, so the 16 waves of a workgroup
// overlap each other's memory latency.  Lane t of the wave owns bytes
// [16t, 16t+16) of every 1 KiB row of the chunk (rows processed in order);
// the CRC column streams run down the rows exactly as in the encoder.
constexpr int kDecWaves = 16;
constexpr uint32_t kLdsDecScratch = kLdsCrcEnd;  // per wave: 64 u32 row bases
constexpr uint32_t kLdsDecode = kLdsDecScratch + kDecWaves * 256;
constexpr int kChunkRows = kChunk / kRow;  // 64

// 8 codes of k bits for the 8 words of group `grp` (12-byte window load).
__device__ __forceinline__ uint64_t load_codes(const uint8_t *codes, uint32_t grp,
                                               uint32_t k) {
  uint64_t start = (uint64_t)grp * k;
  uint64_t a4 = start & ~3ull;
  const uint3 x = *reinterpret_cast<const uint3 *>(codes + a4);
  uint32_t sh = (uint32_t)(start - a4) * 8u;
  uint64_t lo = ((uint64_t)x.y << 32) | x.x;
  return sh ? (lo >> sh) | ((uint64_t)x.z << (64 - sh)) : lo;
}

// CRC of the wave's chunk from its four column states (valid in lane 0).
__device__ __forceinline__ uint32_t wave_chunk_crc(uint32_t v0, uint32_t v1, uint32_t v2,
                                                   uint32_t v3, uint32_t len,
                                                   const ChunkGeom &g, const CrcTables &T) {
  uint32_t u = tab4(kLdsF8, tab4(kLdsF4, v0) ^ v1) ^ tab4(kLdsF4, v2) ^ v3;
#pragma unroll
  for (int lv = 0; lv < kTree; ++lv) {
    uint32_t s = tab4(kLdsTree + lv * 4096u, u);
    uint32_t o = __shfl_down(u, 1u << lv, 64);
    u = s ^ o;
  }
  uint32_t raw = mat_apply(T.unrow_mat, u);
  return len == kChunk ? raw ^ T.k_full : mat_apply(g.tail_mat, raw) ^ g.k_tail;
}

__global__ __launch_bounds__(kDecWaves * 64) void k_decode(
    const uint8_t *__restrict__ payload, ChunkGeom g, uint8_t *__restrict__ staging,
    uint32_t *__restrict__ rec_status, uint8_t *ws, WsLayout L) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(ws + L.ctl);
  uint32_t *ecrc = reinterpret_cast<uint32_t *>(ws + L.entry_crc);
  if (!ctl->hdr_ok) return;
  const uint32_t n_rec = ctl->n_rec;
  const uint64_t table_off = ctl->table_off;
  load_crc_tables(g.crc_kind);
  __syncthreads();
  const CrcTables &T = g_tables[g.crc_kind];
  const GLane gl = glane_make();
  const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  uint32_t *rowbase = reinterpret_cast<uint32_t *>(lds + kLdsDecScratch + wave * 256u);
  const uint32_t stride = gridDim.x * kDecWaves;

  for (uint32_t r = blockIdx.x * kDecWaves + wave; r < n_rec; r += stride) {
    // ---- table entry, table-local rules (uniform across the wave)
    const uint8_t *e = payload + table_off + 16ull * r;
    const uint4 ent = *reinterpret_cast<const uint4 *>(e);
    const uint32_t c = ent.x, src_crc = ent.y;
    const uint64_t off = (uint64_t)ent.z | ((uint64_t)ent.w << 32);
    uint64_t end = table_off;
    bool tbad = false;
    if (r + 1 < n_rec) {
      const uint4 nx = *reinterpret_cast<const uint4 *>(e + 16);
      end = (uint64_t)nx.z | ((uint64_t)nx.w << 32);
      tbad = nx.x <= c;
    }
    {
      uint32_t ew[4] = {ent.x, ent.y, ent.z, ent.w};
      uint32_t ec = crc_words(ew, 4);
      if (lane == 0) ecrc[r] = ec;
    }
    tbad = tbad || c >= g.n_chunks || (r == 0 && off != 64u) || (off & 15u) || off >= end ||
           end > table_off;
    if (tbad) {
      if (lane == 0) atomicOr(&ctl->table_bad, 1u);
      continue;
    }
    // ---- record header
    const uint32_t len = chunk_len(g, c), n_words = len / 2;
    const uint64_t reclen = end - off;
    const uint8_t *rec = payload + off;
    uint32_t st = 0, mode = 0, k = 0, base = 0, n_esc = 0;
    if (reclen < 16) {
      st = 4;
    } else {
      const uint4 h4 = *reinterpret_cast<const uint4 *>(rec);
      uint32_t hw[4] = {h4.x, h4.y, h4.z, h4.w};
      mode = hw[0] & 255u;
      k = (hw[0] >> 8) & 255u;
      base = (hw[0] >> 16) & 255u;
      n_esc = hw[2];
      if (crc_words(hw, 3) != hw[3] || (hw[0] >> 24) || hw[1] != n_words || mode > 1) {
        st = 4;
      } else if (mode == 0) {
        if (k || base || n_esc || reclen != 16u + pad16(2ull * n_words)) st = 4;
      } else if (k > 7 || n_esc > n_words || (k == 0 && n_esc) ||
                 reclen != 16u + pad16(((uint64_t)n_words * k + 7) / 8) + pad16(n_esc) +
                               pad16(n_words)) {
        st = 4;
      }
    }
    if (st == 0) {
      uint8_t *dst = staging + (uint64_t)r * kChunk;
      uint32_t v0 = 0, v1 = 0, v2 = 0, v3 = 0;
      bool bad = false;
      if (mode == 0) {
        const uint8_t *body = rec + 16;
#pragma unroll 4
        for (int row = 0; row < kChunkRows; ++row) {
          const uint32_t o = row * kRow + lane * 16u;
          uint4 d;
          if (len == kChunk) d = ldg_nt(body + o);
          else if (o + 16u <= len) d = *reinterpret_cast<const uint4 *>(body + o);
          else if (o < len) d = load16_partial(body + o, len - o);
          else d = make_uint4(0, 0, 0, 0);
          v0 = g_step(v0 ^ d.x, gl);
          v1 = g_step(v1 ^ d.y, gl);
          v2 = g_step(v2 ^ d.z, gl);
          v3 = g_step(v3 ^ d.w, gl);
          if (o + 16u <= len) {
            *reinterpret_cast<uint4 *>(dst + o) = d;
          } else if (o < len) {
            const uint32_t w[4] = {d.x, d.y, d.z, d.w};
            for (uint32_t b = 0; b < len - o; ++b) dst[o + b] = (uint8_t)(w[b >> 2] >> (8 * (b & 3)));
          }
        }
        if (lane < 16u) {
          uint64_t at = 16u + 2ull * n_words + lane;
          if (at < 16u + pad16(2ull * n_words) && rec[at]) bad = true;
        }
      } else {
        const uint64_t code_bytes = ((uint64_t)n_words * k + 7) / 8;
        const uint64_t esc_off = 16 + pad16(code_bytes);
        const uint64_t sm_off = esc_off + pad16(n_esc);
        const uint32_t esc_code = (1u << k) - 1u;
        const uint8_t *codes = rec + 16;
        // pass 1: escapes per row (row bases into LDS), literal range check
        if (k) {
          uint32_t acc = 0;
#pragma unroll 4
          for (int row = 0; row < kChunkRows; ++row) {
            const uint32_t w0 = row * (kRow / 2) + lane * 8u;
            uint64_t v = 0;
            if (w0 < n_words) v = load_codes(codes, w0 >> 3, k);
            uint32_t s = 0;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              uint32_t code = (uint32_t)(v >> (u * k)) & esc_code;
              bool valid = w0 + u < n_words;
              if (valid && code != esc_code && base + code > 255u) bad = true;
              s += (uint32_t)__popcll(__ballot(valid && code == esc_code));
            }
            if (lane == 0) rowbase[row] = acc;
            acc += s;
          }
          if (acc != n_esc) bad = true;
        }
        // pass 2: rebuild words, CRC, store
#pragma unroll 2
        for (int row = 0; row < kChunkRows; ++row) {
          const uint32_t o = row * kRow + lane * 16u;
          const uint32_t w0 = o >> 1;
          uint32_t out[4] = {0, 0, 0, 0};
          uint64_t v = 0;
          if (k && w0 < n_words) v = load_codes(codes, w0 >> 3, k);
          uint32_t flags = 0;
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            uint32_t code = (uint32_t)(v >> (u * k)) & esc_code;
            if (k && w0 + u < n_words && code == esc_code) flags |= 1u << u;
          }
          // escapes in lower lanes of this row
          uint32_t below = 0;
#pragma unroll
          for (int u = 0; u < 8; ++u) below += lanes_below(__ballot((flags >> u) & 1u));
          if (w0 < n_words) {
            const uint2 smv = *reinterpret_cast<const uint2 *>(rec + sm_off + w0);
            const uint64_t sm8 = ((uint64_t)smv.y << 32) | smv.x;
            uint32_t rank = (k ? rowbase[row] : 0u) + below;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              if (w0 + u >= n_words) break;
              uint32_t code = (uint32_t)(v >> (u * k)) & esc_code;
              uint32_t ex;
              if ((flags >> u) & 1u) {
                ex = rank < n_esc ? rec[esc_off + rank] : 0u;
                ++rank;
              } else {
                ex = (base + code) & 255u;
              }
              uint32_t sm = (uint32_t)(sm8 >> (8 * u)) & 255u;
              uint32_t w = ((sm & 0x80u) << 8) | (ex << 7) | (sm & 0x7Fu);
              out[u >> 1] |= w << (16 * (u & 1));
            }
          }
          v0 = g_step(v0 ^ out[0], gl);
          v1 = g_step(v1 ^ out[1], gl);
          v2 = g_step(v2 ^ out[2], gl);
          v3 = g_step(v3 ^ out[3], gl);
          if (o + 16u <= len) {
            *reinterpret_cast<uint4 *>(dst + o) = make_uint4(out[0], out[1], out[2], out[3]);
          } else if (o < len) {
            for (uint32_t b = 0; b < len - o; ++b) dst[o + b] = (uint8_t)(out[b >> 2] >> (8 * (b & 3)));
          }
        }
        // padding: codes (whole bytes and unused bits), escapes, sm plane
        if (lane < 16u) {
          if (code_bytes + lane < pad16(code_bytes) && codes[code_bytes + lane]) bad = true;
          if (n_esc + lane < pad16(n_esc) && rec[esc_off + n_esc + lane]) bad = true;
          if (n_words + lane < pad16(n_words) && rec[sm_off + n_words + lane]) bad = true;
          uint64_t used = (uint64_t)n_words * k;
          if (lane == 0 && (used & 7u) && (codes[used / 8] >> (used & 7u))) bad = true;
        }
      }
      const uint32_t crc = wave_chunk_crc(v0, v1, v2, v3, len, g, T);
      if (__ballot(bad)) st = 4;
      else if (__shfl(crc, 0, 64) != src_crc) st = 8;
    }
    if (lane == 0) {
      if (rec_status) rec_status[r] = st;
      if (st) atomicOr(&ctl->rec_bits, st);
    }
  }
}

// Final verdict after the table CRC has been combined.
__global__ void k_decode_verdict(const uint8_t *ws, WsLayout L,
                                 const uint32_t *table_crc,
                                 uint32_t *verdict) {
  const WsCtl *ctl = reinterpret_cast<const WsCtl *>(ws + L.ctl);
  uint32_t v;
  if (!ctl->hdr_ok) v = ctl->verdict_pre;
  else if (ctl->table_bad || *table_crc != ctl->table_crc) v = 2u;
  else v = ctl->rec_bits;
  *verdict = v;
}

// ---------------------------------------------------------------- commit --

__global__ __launch_bounds__(256) void k_commit(uint8_t *__restrict__ live, ChunkGeom g,
                                                const uint8_t *__restrict__ staging,
                                                const uint8_t *__restrict__ payload,
                                                const uint32_t *__restrict__ verdict) {
  if (*verdict != 0u) return;
  const uint32_t n_rec = ld_u32(payload + 24);
  const uint64_t table_off = ld_u64(payload + 32) - 16ull * n_rec;
  for (uint32_t r = blockIdx.x; r < n_rec; r += gridDim.x) {
    uint32_t c = ld_u32(payload + table_off + 16ull * r);
    uint32_t len = chunk_len(g, c);
    const uint8_t *src = staging + (uint64_t)r * kChunk;
    uint8_t *dst = live + (uint64_t)c * kChunk;
    if (len == kChunk) {
#pragma unroll 4
      for (uint32_t off = threadIdx.x * 16u; off < kChunk; off += 4096u)
        *reinterpret_cast<uint4 *>(dst + off) = *reinterpret_cast<const uint4 *>(src + off);
    } else {
      for (uint32_t off = threadIdx.x; off < len; off += 256u) dst[off] = src[off];
    }
  }
}

// -------------------------------------------------------------- launchers --

static hipStream_t S(void *s) { return reinterpret_cast<hipStream_t>(s); }

int upload_tables(int device, const CrcTables tabs[2]) {
  (void)device;
  hipError_t e = hipMemcpyToSymbol(HIP_SYMBOL(g_tables), tabs, 2 * sizeof(CrcTables), 0,
                                   hipMemcpyHostToDevice);
  if (e != hipSuccess) return (int)e;
  return (int)hipDeviceSynchronize();
}

int set_kernel_attributes() {
  hipError_t e;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_checksum),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBase);
  if (e != hipSuccess) return (int)e;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_encode<false>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kLdsEncode);
  if (e != hipSuccess) return (int)e;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_encode<true>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kLdsEncode);
  if (e != hipSuccess) return (int)e;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_decode),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kLdsDecode);
  return (int)e;
}

static int launch_combine(const CombineJobs &jobs, int n_jobs, void *stream) {
  hipLaunchKernelGGL(k_combine, dim3(n_jobs), dim3(1024), 0, S(stream), jobs);
  return (int)hipGetLastError();
}

int launch_checksum(const void *data, const ChunkGeom &g, uint32_t *crc_out,
                    uint32_t *global_crc, int n_cu, void *stream) {
  if (g.n_chunks) {
    uint32_t grid = min((uint32_t)n_cu, g.n_chunks);
    hipLaunchKernelGGL(k_checksum, dim3(grid), dim3(kThreads), kLdsBase, S(stream),
                       static_cast<const uint8_t *>(data), g, crc_out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  if (global_crc) {
    CombineJobs jobs = {};
    jobs.job[0] = CombineJob{crc_out, nullptr, g.n_chunks, 16u, g.tail_len, g.crc_kind, global_crc};
    return launch_combine(jobs, 1, stream);
  }
  return 0;
}

int launch_diff(const void *cur, const void *prev, const ChunkGeom &g, uint32_t *dirty_idx,
                uint32_t *n_dirty, void *ws, const WsLayout &L, void *stream) {
  uint32_t *flags = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(ws) + L.flags);
  if (g.n_chunks) {
    uint32_t grid = min(g.n_chunks, 4096u);
    hipLaunchKernelGGL(k_diff, dim3(grid), dim3(256), 0, S(stream),
                       static_cast<const uint8_t *>(cur), static_cast<const uint8_t *>(prev), g,
                       flags);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, S(stream), flags, g.n_chunks, dirty_idx,
                     n_dirty);
  return (int)hipGetLastError();
}

int launch_encode(int mode, const void *cur, const void *prev, const ChunkGeom &g,
                  const uint32_t *idx, const uint32_t *n_idx, const uint32_t *crc_in,
                  uint32_t *crc_out, uint32_t *global_crc, uint32_t *dirty_idx,
                  uint32_t *n_dirty, void *payload, uint64_t *payload_bytes, void *ws,
                  const WsLayout &L, int n_cu, void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  hipLaunchKernelGGL(k_encode_prepare, dim3(64), dim3(256), 0, S(stream), wsb, L, g.n_chunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  EncArgs a;
  a.cur = static_cast<const uint8_t *>(cur);
  a.prev = static_cast<const uint8_t *>(prev);
  a.idx = idx;
  a.n_idx = n_idx;
  a.crc_in = crc_in;
  a.crc_out = crc_out;
  a.dirty_idx = dirty_idx;
  a.payload = static_cast<uint8_t *>(payload);
  a.ws = wsb;
  a.L = L;
  a.mode = mode;
  if (g.n_chunks) {
    uint32_t grid = min((uint32_t)n_cu, g.n_chunks);
    if (mode == kModeStep && prev != nullptr)
      hipLaunchKernelGGL(k_encode<true>, dim3(grid), dim3(kThreads), kLdsEncode, S(stream), a, g);
    else
      hipLaunchKernelGGL(k_encode<false>, dim3(grid), dim3(kThreads), kLdsEncode, S(stream), a, g);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  // global CRC over every chunk, table CRC over the staged entries
  uint32_t *ctl32 = reinterpret_cast<uint32_t *>(wsb + L.ctl);
  uint32_t *crcs = ctl32 + 60;  // two spare words of the control block
  const uint32_t *all_crc = crc_in ? crc_in : crc_out;
  CombineJobs jobs = {};
  jobs.job[0] = CombineJob{all_crc, nullptr, g.n_chunks, 16u, g.tail_len, g.crc_kind, crcs};
  jobs.job[1] = CombineJob{reinterpret_cast<const uint32_t *>(wsb + L.entry_crc),
                           &reinterpret_cast<WsCtl *>(wsb + L.ctl)->n_rec, 0u, 4u, 16u,
                           g.crc_kind, crcs + 1};
  int rc = launch_combine(jobs, 2, stream);
  if (rc) return rc;
  uint32_t full = mode == kModeAll || (mode == kModeStep && prev == nullptr) ? 1u : 0u;
  hipLaunchKernelGGL(k_encode_finish, dim3(64), dim3(256), 0, S(stream),
                     static_cast<uint8_t *>(payload), static_cast<const uint8_t *>(ws), L, g,
                     full, crcs, payload_bytes, n_dirty);
  e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  if (global_crc) {
    e = hipMemcpyAsync(global_crc, crcs, 4, hipMemcpyDeviceToDevice, S(stream));
    if (e != hipSuccess) return (int)e;
  }
  return 0;
}

int launch_decode(const void *payload, uint64_t payload_cap, const ChunkGeom &g, void *staging,
                  uint64_t staging_cap, uint32_t *verdict, uint32_t *rec_status, void *ws,
                  const WsLayout &L, int n_cu, void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  const uint8_t *pl = static_cast<const uint8_t *>(payload);
  hipLaunchKernelGGL(k_decode_prepare, dim3(1), dim3(64), 0, S(stream), pl, payload_cap, g,
                     staging_cap, wsb, L);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  if (g.n_chunks) {
    uint32_t grid = min((uint32_t)n_cu, g.n_chunks);
    uint32_t grid_d = min((uint32_t)n_cu, (g.n_chunks + kDecWaves - 1) / kDecWaves);
    hipLaunchKernelGGL(k_decode, dim3(grid_d), dim3(kDecWaves * 64), kLdsDecode, S(stream), pl,
                       g, static_cast<uint8_t *>(staging), rec_status, wsb, L);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  WsCtl *ctl = reinterpret_cast<WsCtl *>(wsb + L.ctl);
  uint32_t *computed = reinterpret_cast<uint32_t *>(wsb + L.ctl) + 60;
  CombineJobs jobs = {};
  jobs.job[0] = CombineJob{reinterpret_cast<const uint32_t *>(wsb + L.entry_crc), &ctl->n_rec,
                           0u, 4u, 16u, g.crc_kind, computed};
  int rc = launch_combine(jobs, 1, stream);
  if (rc) return rc;
  hipLaunchKernelGGL(k_decode_verdict, dim3(1), dim3(1), 0, S(stream), wsb, L, computed,
                     verdict);
  return (int)hipGetLastError();
}

int launch_commit(void *live, const ChunkGeom &g, const void *staging, const void *payload,
                  const uint32_t *verdict, int n_cu, void *stream) {
  if (!g.n_chunks) return 0;
  uint32_t grid = min((uint32_t)n_cu * 4u, g.n_chunks);
  hipLaunchKernelGGL(k_commit, dim3(grid), dim3(256), 0, S(stream),
                     static_cast<uint8_t *>(live), g, static_cast<const uint8_t *>(staging),
                     static_cast<const uint8_t *>(payload), verdict);
  return (int)hipGetLastError();
}

}  // namespace wm
