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
constexpr uint32_t kLookbackWindow = 256;  // predecessors read per round trip

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

// Encoder LDS beyond the CRC tables.
struct EncShared {
  uint32_t part[kWaves];     // wave CRC partials
  uint32_t dirty_w[kWaves];  // per-wave "differs from prev"
  uint32_t esc_w[kWaves];    // escapes per wave
  uint32_t mode, k, base, n_esc, size, crc, dirty, pad0;
  uint32_t rec_idx, off_lo, off_hi, ticket;
  uint32_t H[256];           // histogram
  uint32_t P[260];           // exclusive prefix of H (P[256] = n)
};
static_assert(sizeof(EncShared) <= kLdsMiscBytes, "encoder scratch fits");
constexpr uint32_t kLdsHistE = kLdsMisc + kLdsMiscBytes;  // 256 bins x 16 copies
constexpr uint32_t kLdsStage = kLdsHistE + 16384;         // code staging
constexpr uint32_t kLdsStageBytes = 7 * (kChunk / 2) / 8;
constexpr uint32_t kLdsEncode = kLdsStage + kLdsStageBytes;
static_assert(kLdsEncode <= 163840, "encoder LDS fits one CU");

__device__ __forceinline__ EncShared &enc_shared() {
  return *reinterpret_cast<EncShared *>(lds + kLdsMisc);
}

__device__ __forceinline__ uint64_t pad16(uint64_t x) { return (x + 15u) & ~15ull; }

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

// Inclusive prefix sum over the 64 lanes of a wave (DPP row shifts and row
// broadcasts).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
  return v;
}
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, 64));
  return v;
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_sub_min(uint32_t ex, uint32_t base2, uint32_t esc2) {
  u16x2 a = __builtin_bit_cast(u16x2, ex), b = __builtin_bit_cast(u16x2, base2);
  u16x2 e = __builtin_bit_cast(u16x2, esc2);
  u16x2 d = a - b;
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(d, e));
}

// The 8 sign/mantissa bytes of a 16-byte piece: byte u = (w_u >> 8 & 0x80) |
// (w_u & 0x7F).
__device__ __forceinline__ uint2 sm_bytes(const uint4 &x) {
  uint32_t s0 = (x.x & 0x007F007Fu) | ((x.x >> 8) & 0x00800080u);
  uint32_t s1 = (x.y & 0x007F007Fu) | ((x.y >> 8) & 0x00800080u);
  uint32_t s2 = (x.z & 0x007F007Fu) | ((x.z >> 8) & 0x00800080u);
  uint32_t s3 = (x.w & 0x007F007Fu) | ((x.w >> 8) & 0x00800080u);
  // gather bytes 0 and 2 of each word pair
  uint32_t lo = __builtin_amdgcn_perm(s1, s0, 0x06040200u);
  uint32_t hi = __builtin_amdgcn_perm(s3, s2, 0x06040200u);
  return make_uint2(lo, hi);
}

// Chunk of a work item; a caller's list must be ascending and in range, a
// violation returns an out-of-range index (the item is then flagged).
__device__ __forceinline__ uint32_t item_chunk(const EncArgs &a, uint32_t item,
                                               const ChunkGeom &g) {
  if (a.mode != kModeList) return item;
  uint32_t c = a.idx[item];
  if (c >= g.n_chunks || (item > 0 && a.idx[item - 1] >= c)) return 0xFFFFFFFFu;
  return c;
}

// Look-back (wave 0).  The first window is loaded by lookback_issue before
// other work; lookback_finish consumes it and reads further windows only if
// needed.  Every item publishes its aggregate before its own look-back and
// tickets are handed out in order to running workgroups, so each
// predecessor publishes eventually; the spin bound only guarantees that the
// kernel terminates if that were ever violated (the call then reports an
// empty payload).
struct Window {
  uint64_t s[kLookbackWindow / 64];
};

__device__ __forceinline__ Window lookback_issue(const uint64_t *status, int64_t top) {
  Window w;
  const uint32_t lane = threadIdx.x & 63u;
#pragma unroll
  for (int q = 0; q < (int)(kLookbackWindow / 64); ++q) {
    int64_t j = top - (int64_t)(lane * (kLookbackWindow / 64) + q);
    w.s[q] = j >= 0 ? status_load(&status[j]) : kFlagIncl;
  }
  return w;
}

__device__ uint64_t lookback_finish(const uint64_t *status, int64_t top, Window w,
                                    WsCtl *ctl) {
  constexpr int Q = kLookbackWindow / 64;
  const uint32_t lane = threadIdx.x & 63u;
  uint64_t excl = 0;
  uint32_t spins = 0;
  while (top >= 0) {
    // distance of an entry from `top` is lane*Q + q
    uint32_t first = 0xFFFFFFFFu;  // nearest inclusive distance held by this lane
#pragma unroll
    for (int q = Q - 1; q >= 0; --q)
      if ((w.s[q] & 3u) == kFlagIncl) first = lane * Q + q;
    uint32_t stop = first;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) stop = min(stop, (uint32_t)__shfl_xor((int)stop, o, 64));
    bool missing = false;
    uint64_t v = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      uint32_t dist = lane * Q + q;
      if (dist <= stop) {
        if ((w.s[q] & 3u) == 0) missing = true;
        v += w.s[q] >> 2;
      }
    }
    if (__ballot(missing)) {
      if (++spins > (1u << 22)) {
        if (lane == 0) atomicOr(&ctl->error, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      w = lookback_issue(status, top);
      continue;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    excl += v;
    if (stop != 0xFFFFFFFFu) break;
    top -= kLookbackWindow;
    w = lookback_issue(status, top);
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

  load_crc_tables(g.crc_kind);
  const CrcTables &T = g_tables[g.crc_kind];
  const GLane gl = glane_make();
  const Lane l = lane_info();
  EncShared &sh = enc_shared();
  uint8_t *stage = lds + kLdsStage;
  uint32_t *hist = reinterpret_cast<uint32_t *>(lds + kLdsHistE);
  const uint32_t copy4 = (threadIdx.x & 15u) * 4u;
  {
    uint4 *h4 = reinterpret_cast<uint4 *>(hist);
    for (uint32_t i = threadIdx.x; i < 1024u; i += kThreads) h4[i] = make_uint4(0, 0, 0, 0);
  }
  if (threadIdx.x == 0) {
    sh.rec_idx = atomicAdd(&ctl->ticket, 1u);
    sh.ticket = atomicAdd(&ctl->ticket, 1u);
  }
  __syncthreads();
  uint32_t item = sh.rec_idx;
  uint32_t next = sh.ticket;
  uint4 d[kRows];
  if (item < n_items) {
    uint32_t c = item_chunk(a, item, g);
    if (c < g.n_chunks) load_chunk(a.cur + (uint64_t)c * kChunk, chunk_len(g, c), l, d);
  }
  __syncthreads();

  while (item < n_items) {
    // ---- 1. prefetch the next chunk; prev of this chunk; next ticket
    uint4 dn[kRows];
    if (next < n_items) {
      uint32_t cn = item_chunk(a, next, g);
      if (cn < g.n_chunks) load_chunk(a.cur + (uint64_t)cn * kChunk, chunk_len(g, cn), l, dn);
    }
    uint32_t c = item_chunk(a, item, g);
    const bool bad_index = c >= g.n_chunks;
    if (bad_index) c = 0;
    const uint32_t len = bad_index ? 0u : chunk_len(g, c);
    const uint32_t n_words = len / 2;
    uint4 p[kRows];
    if (HAS_PREV && !bad_index) load_chunk(a.prev + (uint64_t)c * kChunk, len, l, p);
    uint32_t ticket = 0;
    if (threadIdx.x == 0) ticket = atomicAdd(&ctl->ticket, 1u);

    // ---- 2. CRC (and the diff against prev)
    if (need_crc) {
      uint32_t q = wave_q(d, gl);
      if (l.lane == 0) sh.part[l.wave] = mat_apply(T.wave_mat[l.wave], q);
    }
    bool dirty = !bad_index;
    if (HAS_PREV) {
      uint32_t diff = 0;
#pragma unroll
      for (int h = 0; h < kRows; ++h)
        diff |= (d[h].x ^ p[h].x) | (d[h].y ^ p[h].y) | (d[h].z ^ p[h].z) | (d[h].w ^ p[h].w);
      unsigned long long any = __ballot(diff != 0);
      if (l.lane == 0) sh.dirty_w[l.wave] = any ? 1u : 0u;
      __syncthreads();
      uint32_t dw = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) dw |= sh.dirty_w[w];
      dirty = dirty && dw != 0;
    }

    // ---- 3. exponent histogram (16 copies x 256 bins)
    const bool full = len == kChunk;
    if (dirty) {
#pragma unroll
      for (int h = 0; h < kRows; ++h) {
        const uint32_t w0 = (l.off0 + h * kRow) >> 1;
        const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (full || w0 + 2 * j < n_words)
            atomicAdd(reinterpret_cast<uint32_t *>(lds + kLdsHistE + (((x[j] >> 1) & 0x3FC0u) | copy4)), 1u);
          if (full || w0 + 2 * j + 1 < n_words)
            atomicAdd(reinterpret_cast<uint32_t *>(lds + kLdsHistE + (((x[j] >> 17) & 0x3FC0u) | copy4)), 1u);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();  // B1: histogram and CRC partials complete

    // ---- 4. histogram reduce (all waves, 32 bins each)
    if (dirty) {
      const uint32_t bin = l.wave * 32u + (l.lane >> 1), half = l.lane & 1u;
      uint32_t s = 0;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        uint32_t cp = (half * 8u + ((cc + (l.lane >> 1)) & 7u));
        s += hist[bin * 16u + cp];
      }
      s += __shfl_xor((int)s, 1, 64);
      if (half == 0) sh.H[bin] = s;
    }
    __syncthreads();  // B2: H complete; the histogram copies are free

    // ---- 5. wave 0: chunk CRC, plan, aggregate, first look-back window
    Window win;
    if (l.wave == 0) {
      uint32_t crc = 0;
      if (need_crc) {
        uint32_t raw = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) raw ^= sh.part[w];
        crc = bad_index ? 0u : (full ? raw ^ T.k_full : mat_apply(g.tail_mat, raw) ^ g.k_tail);
      } else {
        crc = a.crc_in[c];
      }
      uint32_t mode = 0, k = 0, base = 0, n_esc = 0;
      uint64_t size = 0;
      if (dirty) {
        // exclusive prefix P over the 256 bins (4 per lane)
        const uint32_t b0 = l.lane * 4u;
        const uint32_t h0 = sh.H[b0], h1 = sh.H[b0 + 1], h2 = sh.H[b0 + 2], h3 = sh.H[b0 + 3];
        const uint32_t t4 = h0 + h1 + h2 + h3;
        const uint32_t ex = wave_incl_scan(t4) - t4;
        sh.P[b0] = ex;
        sh.P[b0 + 1] = ex + h0;
        sh.P[b0 + 2] = ex + h0 + h1;
        sh.P[b0 + 3] = ex + h0 + h1 + h2;
        if (l.lane == 63u) sh.P[256] = ex + t4;
        const uint32_t nzmask = (h0 ? 1u : 0u) | (h1 ? 2u : 0u) | (h2 ? 4u : 0u) | (h3 ? 8u : 0u);
        const uint32_t distinct = wave_incl_scan(__popc(nzmask));
        const uint32_t n_distinct = __builtin_amdgcn_readlane(distinct, 63);
        const uint32_t only = wave_max(nzmask ? b0 + 31u - __clz(nzmask) : 0u);
        const uint64_t n = n_words;
        // candidates: lane 0 RAW, lane 1 k=0, lanes 2..8 k = lane-1
        uint64_t cand = ~0ull;
        uint32_t c_base = 0, c_esc = 0;
#pragma unroll
        for (uint32_t kk = 1; kk <= 7; ++kk) {
          const uint32_t win_w = (1u << kk) - 1u;
          uint32_t key = 0;
#pragma unroll
          for (uint32_t j = 0; j < 4; ++j) {
            uint32_t b = b0 + j;
            uint32_t end = min(b + win_w, 256u);
            uint32_t inside = sh.P[end] - sh.P[b];
            key = max(key, (inside << 8) | (255u - b));
          }
          key = wave_max(key);
          if (l.lane == kk + 1) {
            uint32_t inside = key >> 8;
            c_base = 255u - (key & 255u);
            c_esc = n_words - inside;
            cand = 16u + pad16((n * kk + 7) / 8) + pad16(2 * ((n + 511) / 512)) + pad16(c_esc) +
                   pad16(n);
          }
        }
        if (l.lane == 0) cand = 16u + pad16(2 * n);
        if (l.lane == 1 && n_distinct == 1) {
          cand = 16u + pad16(n);
          c_base = only;
        }
        // smallest size, then lowest lane
        uint64_t key = (cand << 8) | l.lane;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
          uint64_t y = __shfl_xor(key, o, 64);
          key = y < key ? y : key;
        }
        const uint32_t win_lane = (uint32_t)(key & 255u);
        size = key >> 8;
        mode = win_lane == 0 ? 0u : 1u;
        k = win_lane <= 1 ? 0u : win_lane - 1u;
        base = __shfl((int)c_base, (int)win_lane, 64);
        n_esc = __shfl((int)c_esc, (int)win_lane, 64);
      }
      const uint64_t agg = ((uint64_t)(dirty ? 1u : 0u) << 2) | ((size >> 4) << 26);
      if (l.lane == 0) {
        if (item != 0) status_store(&status[item], agg | kFlagAgg);
        sh.mode = mode;
        sh.k = k;
        sh.base = base;
        sh.n_esc = n_esc;
        sh.size = (uint32_t)size;
        sh.crc = crc;
        sh.dirty = dirty ? 1u : 0u;
      }
      win = lookback_issue(status, (int64_t)item - 1);
    }
    __syncthreads();  // B3: plan known

    // ---- 6. codes into staging, escape counts, sign/mantissa bytes
    const uint32_t mode = sh.mode, k = sh.k, base = sh.base, n_esc = sh.n_esc;
    dirty = sh.dirty != 0;
    const bool pack = dirty && mode == 1u && k > 0u;
    const uint32_t esc_code = (1u << k) - 1u;
    const uint32_t base2 = base | (base << 16), esc2 = esc_code | (esc_code << 16);
    uint32_t escm[2] = {0, 0};      // escape flags, 8 bits per row
    uint32_t row_base[kRows];      // escapes in earlier rows of this wave
    uint32_t wave_esc = 0;
    if (pack) {
      if (!full) {
        uint4 *s4 = reinterpret_cast<uint4 *>(stage);
        for (uint32_t i = threadIdx.x; i < kLdsStageBytes / 16; i += kThreads)
          s4[i] = make_uint4(0, 0, 0, 0);
        __syncthreads();
      }
#pragma unroll
      for (int h = 0; h < kRows; ++h) {
        const uint32_t w0 = (l.off0 + h * kRow) >> 1;
        const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
        uint32_t cp[4];
        uint32_t flags = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          cp[j] = pk_sub_min((x[j] >> 7) & 0x00FF00FFu, base2, esc2);
          if (!full) {  // words past the chunk code as 0, never escape
            if (w0 + 2 * j >= n_words) cp[j] &= 0xFFFF0000u;
            if (w0 + 2 * j + 1 >= n_words) cp[j] &= 0x0000FFFFu;
          }
          uint32_t lo = cp[j] & 0xFFFFu, hi = cp[j] >> 16;
          bool vlo = full || w0 + 2 * j < n_words, vhi = full || w0 + 2 * j + 1 < n_words;
          flags |= ((vlo && lo == esc_code) ? 1u : 0u) << (2 * j);
          flags |= ((vhi && hi == esc_code) ? 1u : 0u) << (2 * j + 1);
        }
        // 8 codes of k bits
        uint64_t packed = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          uint64_t pair = (uint64_t)(cp[j] & 0xFFFFu) | ((uint64_t)(cp[j] >> 16) << k);
          packed |= pair << (2 * j * k);
        }
        if (w0 < n_words) {
          const uint32_t at = (w0 >> 3) * k;
          if (k == 4u) {
            *reinterpret_cast<uint32_t *>(stage + at) = (uint32_t)packed;
          } else if (k == 2u) {
            *reinterpret_cast<uint16_t *>(stage + at) = (uint16_t)packed;
          } else if (k == 1u) {
            stage[at] = (uint8_t)packed;
          } else {
            for (uint32_t b = 0; b < k; ++b) stage[at + b] = (uint8_t)(packed >> (8 * b));
          }
        }
        const uint32_t cnt = __popc(flags);
        const uint32_t incl = wave_incl_scan(cnt);
        row_base[h] = wave_esc;
        wave_esc += __builtin_amdgcn_readlane(incl, 63);
        escm[h >> 2] |= flags << (8 * (h & 3));
        __builtin_amdgcn_sched_barrier(0);
      }
      if (l.lane == 0) sh.esc_w[l.wave] = wave_esc;
    }
    // zero the histogram copies for the next chunk
    {
      uint4 *h4 = reinterpret_cast<uint4 *>(hist);
      for (uint32_t i = threadIdx.x; i < 1024u; i += kThreads) h4[i] = make_uint4(0, 0, 0, 0);
    }
    // wave 0: finish the look-back, publish the inclusive prefix
    if (l.wave == 0) {
      const uint64_t excl = lookback_finish(status, (int64_t)item - 1, win, ctl);
      if (l.lane == 0) {
        const uint64_t agg = ((uint64_t)(dirty ? 1u : 0u) << 2) | ((uint64_t)(sh.size >> 4) << 26);
        const uint64_t incl = excl + (agg >> 2);
        status_store(&status[item], (incl << 2) | kFlagIncl);
        if (item + 1 == n_items) {
          ctl->n_rec = (uint32_t)(incl & 0xFFFFFFu);
          ctl->payload_bytes = (incl >> 24) << 4;  // total record bytes
        }
        sh.rec_idx = (uint32_t)(excl & 0xFFFFFFu);
        const uint64_t off = 64u + ((excl >> 24) << 4);
        sh.off_lo = (uint32_t)off;
        sh.off_hi = (uint32_t)(off >> 32);
        sh.ticket = ticket;
        if (bad_index) atomicOr(&ctl->error, 2u);
      }
    }
    __syncthreads();  // B4: offset known, codes staged, escape totals known

    // ---- 7. write the record
    const uint32_t rec_idx = sh.rec_idx;
    const uint64_t rec_off = (uint64_t)sh.off_lo | ((uint64_t)sh.off_hi << 32);
    const uint32_t crc = sh.crc;
    if (dirty) {
      uint8_t *rec = a.payload + rec_off;
      if (threadIdx.x == 0) {
        uint32_t hw[4];
        hw[0] = mode | (k << 8) | (base << 16);
        hw[1] = n_words;
        hw[2] = n_esc;
        hw[3] = crc_words(hw, 3);
        *reinterpret_cast<uint4 *>(rec) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
        uint32_t ew[4] = {c, crc, (uint32_t)rec_off, (uint32_t)(rec_off >> 32)};
        tab_ws[rec_idx] = make_uint4(ew[0], ew[1], ew[2], ew[3]);
        ecrc[rec_idx] = crc_words(ew, 4);
        if (a.dirty_idx) a.dirty_idx[rec_idx] = c;
      }
      if (mode == 0) {
        store_chunk(rec + 16, len, l, d, true);
      } else {
        const uint64_t n = n_words;
        const uint64_t code_bytes = (n * k + 7) / 8;
        const uint64_t n_blocks = k ? (n + 511) / 512 : 0;
        const uint64_t idx_off = 16 + pad16(code_bytes);
        const uint64_t esc_off = idx_off + pad16(2 * n_blocks);
        const uint64_t sm_off = esc_off + pad16(n_esc);
        for (uint32_t i = threadIdx.x; i < pad16(code_bytes) / 16; i += kThreads)
          *reinterpret_cast<uint4 *>(rec + 16 + 16 * i) =
              *reinterpret_cast<const uint4 *>(stage + 16 * i);
        uint32_t wave_base = 0;
        if (pack) {
          for (uint32_t w = 0; w < l.wave; ++w) wave_base += sh.esc_w[w];
        }
#pragma unroll
        for (int h = 0; h < kRows; ++h) {
          const uint32_t w0 = (l.off0 + h * kRow) >> 1;
          if (w0 < n_words) *reinterpret_cast<uint2 *>(rec + sm_off + w0) = sm_bytes(d[h]);
          if (pack) {
            // escape index entry of this row's 512-word block
            if (l.lane == 0 && (w0 >> 9) < n_blocks)
              *reinterpret_cast<uint16_t *>(rec + idx_off + 2 * (w0 >> 9)) =
                  (uint16_t)(wave_base + row_base[h]);
            const uint32_t flags = (escm[h >> 2] >> (8 * (h & 3))) & 255u;
            const uint32_t cnt = __popc(flags);
            const uint32_t lane_before = wave_incl_scan(cnt) - cnt;
            if (flags) {
              const uint32_t xx[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
              uint32_t rank = wave_base + row_base[h] + lane_before;
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                if ((flags >> u) & 1u) {
                  rec[esc_off + rank] = (uint8_t)((xx[u >> 1] >> (7 + 16 * (u & 1))) & 255u);
                  ++rank;
                }
              }
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        if (threadIdx.x < 16u) {
          const uint32_t t = threadIdx.x;
          if (2 * n_blocks + t < pad16(2 * n_blocks)) rec[idx_off + 2 * n_blocks + t] = 0;
          if (n_esc + t < pad16(n_esc)) rec[esc_off + n_esc + t] = 0;
          if (n + t < pad16(n)) rec[sm_off + n + t] = 0;
        }
      }
    }
    if (threadIdx.x == 0 && a.crc_out && !bad_index) a.crc_out[c] = crc;

#pragma unroll
    for (int h = 0; h < kRows; ++h) d[h] = dn[h];
    item = next;
    next = sh.ticket;
    __syncthreads();  // B5: scratch may be rewritten
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

// One wave decodes one record with no barriers, so the 16 waves of a
// workgroup overlap each other's memory latency.  Lane t owns bytes
// [16t, 16t+16) of every 1 KiB row (one 512-word escape-index block); rows are
// decoded in batches of 2 while the next batch's codes, sign/mantissa bytes
// and escape bytes are already being fetched.
constexpr int kDecWaves = 12;
constexpr int kBatch = 2;                       // rows per batch
constexpr uint32_t kEscPieces = 2;              // 16-byte escape pieces per lane
constexpr uint32_t kEscStage = 64 * 16 * kEscPieces;  // escape staging per wave
constexpr uint32_t kLdsDecStage = kLdsCrcEnd;
constexpr uint32_t kLdsDecode = kLdsDecStage + kDecWaves * kEscStage;
constexpr int kChunkRows = kChunk / kRow;       // 64
static_assert(kLdsDecode <= 163840, "decoder LDS fits one CU");

__device__ __forceinline__ uint64_t load_codes(const uint8_t *codes, uint32_t grp, uint32_t k) {
  uint64_t start = (uint64_t)grp * k;
  uint64_t a4 = start & ~3ull;
  const uint3 x = *reinterpret_cast<const uint3 *>(codes + a4);
  uint32_t sh = (uint32_t)(start - a4) * 8u;
  uint64_t lo = ((uint64_t)x.y << 32) | x.x;
  return sh ? (lo >> sh) | ((uint64_t)x.z << (64 - sh)) : lo;
}

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

struct PackRec {
  const uint8_t *rec;
  uint64_t code_off, idx_off, esc_off, sm_off;
  uint32_t k, base, n_esc, n_words, n_blocks, esc_code;
  uint32_t blk;  // lane b holds escape-index entry b (lane n_blocks: n_esc)
};

struct DecBatch {
  uint3 code[kBatch];
  uint2 sm[kBatch];
  uint4 esc[kEscPieces];
  uint32_t lo, lo_al, hi;
};

__device__ __forceinline__ uint32_t blk_at(const PackRec &R, uint32_t b) {
  if (b >= R.n_blocks) return R.n_esc;
  return (uint32_t)__shfl((int)R.blk, (int)b, 64);
}

__device__ __forceinline__ void dec_load(DecBatch &B, const PackRec &R, int j, uint32_t lane,
                                         uint64_t reclen) {
#pragma unroll
  for (int q = 0; q < kBatch; ++q) {
    const uint32_t row = j * kBatch + q;
    const uint32_t w0 = row * (kRow / 2) + lane * 8u;
    B.code[q] = make_uint3(0, 0, 0);
    B.sm[q] = make_uint2(0, 0);
    if (w0 < R.n_words) {
      if (R.k) {
        uint64_t a4 = ((uint64_t)(w0 >> 3) * R.k) & ~3ull;
        B.code[q] = *reinterpret_cast<const uint3 *>(R.rec + R.code_off + a4);
      }
      B.sm[q] = *reinterpret_cast<const uint2 *>(R.rec + R.sm_off + w0);
    }
  }
  // escape bytes of the batch: [index[4j], index[4j+4]) from the index
  B.lo = B.lo_al = B.hi = 0;
  if (R.k) {
    uint32_t lo = blk_at(R, j * kBatch), hi = blk_at(R, j * kBatch + kBatch);
    lo = min(lo, R.n_esc);
    hi = min(max(hi, lo), R.n_esc);
    if (hi - lo > kBatch * (kRow / 2)) hi = lo;  // inconsistent index: rejected later
    B.lo = lo;
    B.hi = hi;
    B.lo_al = lo & ~15u;
#pragma unroll
    for (int p = 0; p < (int)kEscPieces; ++p) {
      const uint32_t piece = lane + 64u * p;
      B.esc[p] = make_uint4(0, 0, 0, 0);
      const uint64_t at = R.esc_off + B.lo_al + 16u * piece;
      if (B.lo_al + 16u * piece < hi && at + 16 <= reclen)
        B.esc[p] = *reinterpret_cast<const uint4 *>(R.rec + at);
    }
  }
}

// Decode one batch; returns whether any structure rule failed.
__device__ __forceinline__ bool dec_process(const DecBatch &B, const PackRec &R, int j,
                                            uint32_t lane, uint8_t *stage, uint32_t &acc,
                                            uint32_t &v0, uint32_t &v1, uint32_t &v2,
                                            uint32_t &v3, const GLane &gl, uint8_t *dst,
                                            uint32_t len) {
  bool bad = false;
  if (R.k) {
#pragma unroll
    for (int p = 0; p < (int)kEscPieces; ++p)
      *reinterpret_cast<uint4 *>(stage + 16u * (lane + 64u * p)) = B.esc[p];
  }
#pragma unroll
  for (int q = 0; q < kBatch; ++q) {
    const uint32_t row = j * kBatch + q;
    const uint32_t w0 = row * (kRow / 2) + lane * 8u;
    const uint32_t o = w0 * 2u;
    uint32_t out[4] = {0, 0, 0, 0};
    if (row * (kRow / 2) < R.n_words) {
      uint64_t v = 0;
      if (R.k) {
        const uint64_t start = (uint64_t)(w0 >> 3) * R.k;
        const uint32_t sh = (uint32_t)(start & 3u) * 8u;
        const uint64_t lo = ((uint64_t)B.code[q].y << 32) | B.code[q].x;
        v = sh ? (lo >> sh) | ((uint64_t)B.code[q].z << (64 - sh)) : lo;
      }
      uint32_t flags = 0;
      uint32_t codes[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        codes[u] = (uint32_t)(v >> (u * R.k)) & R.esc_code;
        bool valid = w0 + u < R.n_words;
        if (R.k && valid && codes[u] == R.esc_code) flags |= 1u << u;
        if (R.k && valid && codes[u] != R.esc_code && R.base + codes[u] > 255u) bad = true;
      }
      const uint32_t cnt = __popc(flags);
      const uint32_t incl = wave_incl_scan(cnt);
      // the index entry of this block must equal the escapes decoded so far
      if (R.k && blk_at(R, row) != acc) bad = true;
      uint32_t rank = acc + incl - cnt;
      acc += __builtin_amdgcn_readlane(incl, 63);
      const uint64_t sm8 = ((uint64_t)B.sm[q].y << 32) | B.sm[q].x;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        uint32_t ex = (R.base + codes[u]) & 255u;
        if ((flags >> u) & 1u) {
          uint32_t at = rank - B.lo_al;
          ex = (rank >= B.lo && rank < B.hi && at < kEscStage) ? stage[at] : 0u;
          if (!(rank >= B.lo && rank < B.hi)) bad = true;
          ++rank;
        }
        const uint32_t sm = (uint32_t)(sm8 >> (8 * u)) & 255u;
        const uint32_t w = ((sm & 0x80u) << 8) | (ex << 7) | (sm & 0x7Fu);
        if (w0 + u < R.n_words) out[u >> 1] |= w << (16 * (u & 1));
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
    __builtin_amdgcn_sched_barrier(0);
  }
  return bad;
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
  uint8_t *stage = lds + kLdsDecStage + wave * kEscStage;
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
    uint64_t code_bytes = 0, n_blocks = 0;
    if (reclen < 16) {
      st = 4;
    } else {
      const uint4 h4 = *reinterpret_cast<const uint4 *>(rec);
      uint32_t hw[4] = {h4.x, h4.y, h4.z, h4.w};
      mode = hw[0] & 255u;
      k = (hw[0] >> 8) & 255u;
      base = (hw[0] >> 16) & 255u;
      n_esc = hw[2];
      code_bytes = ((uint64_t)n_words * k + 7) / 8;
      n_blocks = k ? ((uint64_t)n_words + 511) / 512 : 0;
      if (crc_words(hw, 3) != hw[3] || (hw[0] >> 24) || hw[1] != n_words || mode > 1) {
        st = 4;
      } else if (mode == 0) {
        if (k || base || n_esc || reclen != 16u + pad16(2ull * n_words)) st = 4;
      } else if (k > 7 || n_esc > n_words || (k == 0 && n_esc) ||
                 reclen != 16u + pad16(code_bytes) + pad16(2 * n_blocks) + pad16(n_esc) +
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
#pragma unroll 8
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
        PackRec R;
        R.rec = rec;
        R.k = k;
        R.base = base;
        R.n_esc = n_esc;
        R.n_words = n_words;
        R.n_blocks = (uint32_t)n_blocks;
        R.esc_code = (1u << k) - 1u;
        R.code_off = 16;
        R.idx_off = 16 + pad16(code_bytes);
        R.esc_off = R.idx_off + pad16(2 * n_blocks);
        R.sm_off = R.esc_off + pad16(n_esc);
        R.blk = (k && lane < n_blocks)
                    ? (uint32_t)(*reinterpret_cast<const uint16_t *>(rec + R.idx_off + 2 * lane))
                    : n_esc;
        const int n_batches = (int)((n_words + kBatch * (kRow / 2) - 1) / (kBatch * (kRow / 2)));
        uint32_t acc = 0;
        DecBatch A, B2;
        dec_load(A, R, 0, lane, reclen);
        for (int j = 0; j < n_batches; j += 2) {
          if (j + 1 < n_batches) dec_load(B2, R, j + 1, lane, reclen);
          bad |= dec_process(A, R, j, lane, stage, acc, v0, v1, v2, v3, gl, dst, len);
          if (j + 1 >= n_batches) break;
          if (j + 2 < n_batches) dec_load(A, R, j + 2, lane, reclen);
          bad |= dec_process(B2, R, j + 1, lane, stage, acc, v0, v1, v2, v3, gl, dst, len);
        }
        // rows past the chunk: zero data, as in the zero-padded CRC layout
        for (int row = n_batches * kBatch; row < kChunkRows; ++row) {
          v0 = g_step(v0, gl);
          v1 = g_step(v1, gl);
          v2 = g_step(v2, gl);
          v3 = g_step(v3, gl);
        }
        if (acc != n_esc) bad = true;
        // padding: codes (whole bytes and unused bits), index, escapes, sm
        if (lane < 16u) {
          const uint8_t *codes = rec + R.code_off;
          if (code_bytes + lane < pad16(code_bytes) && codes[code_bytes + lane]) bad = true;
          if (2 * n_blocks + lane < pad16(2 * n_blocks) && rec[R.idx_off + 2 * n_blocks + lane]) bad = true;
          if (n_esc + lane < pad16(n_esc) && rec[R.esc_off + n_esc + lane]) bad = true;
          if (n_words + lane < pad16(n_words) && rec[R.sm_off + n_words + lane]) bad = true;
          uint64_t used = (uint64_t)n_words * k;
          if (lane == 0 && (used & 7u) && (codes[used / 8] >> (used & 7u))) bad = true;
        }
      }
      const uint32_t crc = wave_chunk_crc(v0, v1, v2, v3, len, g, T);
      if (__ballot(bad)) st = 4;
      else if ((uint32_t)__shfl((int)crc, 0, 64) != src_crc) st = 8;
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
