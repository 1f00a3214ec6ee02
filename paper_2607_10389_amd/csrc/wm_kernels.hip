// wm_kernels.hip -- CDNA4 (gfx950) kernels of the exact-state mover.
//
// Data layout.  A 64 KiB chunk is split into 64 rows of 1 KiB; lane t of a
// wave owns bytes [16t, 16t+16) of each row it handles, so every load and
// store is a coalesced 128-bit access.  The encoder gives each of 8 data
// waves 8 consecutive rows of a chunk; the decoder gives one wave a whole
// record.
//
// CRC (§4 "Sufficiency", §6.5: per-chunk zlib CRC, GF(2)-combined).  Each lane
// runs four independent dword "column" streams down its rows:
//     v <- F^1024(v ^ d)
// (the next dword of the column is 1 KiB further on).  A lane's four columns
// merge into one value, the lane values of the eight waves fold together
// through one byte-table shift per wave, and each lane's fold enters the chunk
// value through a GF(2) matrix of its own (its distance from the chunk end),
// the 64 results XORed across the wave.  The F^1024 tables are the hot ones: 16 copies in LDS,
// addressed as byte*256 + slot*64 + copy*4 with v_perm, where each group of
// 16 lanes starts at a different table slot so that one ds_read touches every
// bank once.  All other shift tables are read rarely and kept single.
//
// Memory ordering rule followed by the streaming loops: a wave that has
// issued its prefetch of the next rows issues no other vector-memory load
// until it consumes that prefetch (vector-memory loads retire in order, so
// any later load would wait for the whole prefetch).  Uniform data (tables,
// matrices) therefore comes through scalar loads.
#include <hip/hip_runtime.h>

#include "wm_internal.h"

namespace wm {

__device__ CrcTables g_tables[2];

// ------------------------------------------------------------ LDS layout --
// The first 32 KiB are kernel-specific (encoder histogram, decoder escape
// windows): below 64 KiB, so their base folds into an instruction's offset.
constexpr uint32_t kLdsLow = 0;
constexpr uint32_t kLdsLowBytes = 32768;
constexpr uint32_t kLdsG = kLdsLow + kLdsLowBytes;  // 64 KiB, replicated F^1024
constexpr uint32_t kLdsF4 = kLdsG + 65536;          // 4 KiB each: F^4, F^8, F^12
constexpr uint32_t kLdsF8 = kLdsF4 + 4096;
constexpr uint32_t kLdsF12 = kLdsF8 + 4096;
constexpr uint32_t kLdsLaneMat = kLdsF12 + 4096;    // 64 lanes x 32 columns (8 KiB)
constexpr uint32_t kLdsWaveStep = kLdsLaneMat + 8192;  // 4 KiB, F^kSub
constexpr uint32_t kLdsCrcEnd = kLdsWaveStep + 4096;        // 122880
constexpr uint32_t kLdsMisc = kLdsCrcEnd;           // 4 KiB of small scratch
constexpr uint32_t kLdsMiscBytes = 4096;
constexpr uint32_t kLdsBase = kLdsMisc + kLdsMiscBytes;  // 126976


// Dynamic LDS of the kernels below.  They declare no static LDS (checked at
// set-up, set_kernel_attributes), so it begins at LDS address 0: addresses
// are plain numbers, and their constant parts stay in the LDS instructions'
// offset fields instead of an extern array's base (a link-time value) being
// added to every address.
__device__ __forceinline__ uint8_t *lds_at(uint32_t off) {
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  return (uint8_t *)(lds_u8 *)(uintptr_t)off;  // C-style: address-space cast
}

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// 128-bit streaming load that does not allocate in the caches.
__device__ __forceinline__ uint4 ldg_nt(const void *p) {
  v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Buffer loads through a descriptor that covers [base, base + bytes): reads
// past the range return zero instead of touching memory, so a loop can issue
// the same loads whatever the length (a zero range turns them into no-ops).
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kNt = 2;  // buffer-load cache policy: non-temporal
__device__ __forceinline__ Rsrc rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, 0x00020000);
}
template <int AUX = 0>
__device__ __forceinline__ uint4 buf16(Rsrc r, uint32_t off) {
  const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 buf8(Rsrc r, uint32_t off) {
  typedef uint32_t v2u __attribute__((ext_vector_type(2)));
  const v2u v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint3 buf12(Rsrc r, uint32_t off) {
  typedef uint32_t v3u __attribute__((ext_vector_type(3)));
  const v3u v = __builtin_amdgcn_raw_buffer_load_b96(r, off, 0, 0);
  return make_uint3(v.x, v.y, v.z);
}

// Uniform read-only kernel inputs through the constant address space, which
// the compiler serves with scalar loads (no vector-memory wait).
__device__ __forceinline__ uint32_t ld_const(const uint32_t *p) {
  typedef const __attribute__((address_space(4))) uint32_t cu32;
  return *(cu32 *)(uintptr_t)p;
}

__device__ __forceinline__ uint32_t lds_u32(uint32_t off) {
  return *reinterpret_cast<const uint32_t *>(lds_at(off));
}
__device__ __forceinline__ uint32_t uniform(uint32_t v) {
  return __builtin_amdgcn_readfirstlane(v);
}

// a ^ b ^ c in one instruction (three-input logic op, truth table 0x96).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// Byte-table application of a shift stored at LDS offset `off`, XORed with y.
__device__ __forceinline__ uint32_t tab4x(uint32_t off, uint32_t x, uint32_t y) {
  return xor3(xor3(lds_u32(off + ((x & 255u) << 2)), lds_u32(off + 1024u + (((x >> 8) & 255u) << 2)),
                   lds_u32(off + 2048u + (((x >> 16) & 255u) << 2))),
              lds_u32(off + 3072u + ((x >> 24) << 2)), y);
}
__device__ __forceinline__ uint32_t tab4(uint32_t off, uint32_t x) {
  return xor3(lds_u32(off + ((x & 255u) << 2)), lds_u32(off + 1024u + (((x >> 8) & 255u) << 2)),
              lds_u32(off + 2048u + (((x >> 16) & 255u) << 2))) ^
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

// F^kRow(x) ^ y.
__device__ __forceinline__ uint32_t g_step(uint32_t x, uint32_t y, const GLane &gl) {
  uint32_t a0 = __builtin_amdgcn_perm(x, gl.k[0], gl.sel[0]);
  uint32_t a1 = __builtin_amdgcn_perm(x, gl.k[1], gl.sel[1]);
  uint32_t a2 = __builtin_amdgcn_perm(x, gl.k[2], gl.sel[2]);
  uint32_t a3 = __builtin_amdgcn_perm(x, gl.k[3], gl.sel[3]);
  return xor3(xor3(lds_u32(kLdsG + a0), lds_u32(kLdsG + a1), lds_u32(kLdsG + a2)),
              lds_u32(kLdsG + a3), y);
}

__device__ void load_crc_tables(uint32_t kind) {
  const CrcTables &T = g_tables[kind];
  uint32_t *g = reinterpret_cast<uint32_t *>(lds_at(kLdsG));
  for (uint32_t i = threadIdx.x; i < 16384u; i += blockDim.x)
    g[i] = T.row[(i >> 4) & 3u][i >> 6];
  const uint32_t *src = &T.f4[0][0];  // f4, f8, f12, lane_mat, wave_step
  uint32_t *dst = reinterpret_cast<uint32_t *>(lds_at(kLdsF4));
  static_assert(offsetof(CrcTables, wave_step) - offsetof(CrcTables, f4) == 5 * 4096u &&
                    kLdsWaveStep - kLdsF4 == 5 * 4096u,
                "f4 .. wave_step copied as one block");
  for (uint32_t i = threadIdx.x; i < 6u * 1024u; i += blockDim.x) dst[i] = src[i];
}

// Columns applied to v; `m` must be wave-uniform (the columns then arrive
// through scalar loads).
__device__ __forceinline__ uint32_t mat_apply(const uint32_t *__restrict__ m,
                                              uint32_t v) {
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 32; ++i) r ^= m[i] & (0u - ((v >> i) & 1u));  // no load under a branch
  return r;
}

// mat_apply with the 32 columns in LDS (four per read, the same address in
// every lane).
__device__ __forceinline__ uint32_t mat_apply_lds(const uint4 *m, uint32_t v) {
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint4 c = m[i];
    r ^= (c.x & (0u - ((v >> (4 * i)) & 1u))) ^ (c.y & (0u - ((v >> (4 * i + 1)) & 1u))) ^
         (c.z & (0u - ((v >> (4 * i + 2)) & 1u))) ^ (c.w & (0u - ((v >> (4 * i + 3)) & 1u)));
  }
  return r;
}

// F^m(v) for any m >= 0, through the power-of-two shift matrices.
__device__ uint32_t shift_bytes(const CrcTables &T, uint64_t m, uint32_t v) {
  for (int i = 0; m; ++i, m >>= 1)
    if (m & 1) v = mat_apply(T.pow2[i], v);
  return v;
}

// Standard CRC (init/xorout ~0) of 4*nw bytes held as words, with F^4 tables
// in LDS.  Used for headers and table entries.  crc_feed continues a
// register state s (start from ~0, finish with ^ ~0).
__device__ __forceinline__ uint32_t crc_feed(uint32_t s, const uint32_t *w, int nw) {
  for (int i = 0; i < nw; ++i) s = tab4(kLdsF4, s ^ w[i]);
  return s;
}
__device__ __forceinline__ uint32_t crc_words(const uint32_t *w, int nw) {
  return crc_feed(0xFFFFFFFFu, w, nw) ^ 0xFFFFFFFFu;
}

__device__ __forceinline__ uint64_t pad16(uint64_t x) { return (x + 15u) & ~15ull; }

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

// -------------------------------------------------------- chunk movement --

struct Lane {
  uint32_t wave, lane, off0;  // off0: chunk offset of the lane's first row
};
__device__ __forceinline__ Lane lane_info() {
  Lane l;
  l.wave = uniform(threadIdx.x >> 6);
  l.lane = threadIdx.x & 63u;
  l.off0 = l.wave * kSub + l.lane * 16u;
  return l;
}

// The same lane offsets, hidden from loop-invariant code motion: per-row
// addresses derived from them are then recomputed in each iteration of a
// chunk loop instead of being hoisted out of it and held in registers for its
// whole duration (dozens of them with the k-specialised paths).
__device__ __forceinline__ Lane lane_fresh(Lane l) {
  asm volatile("" : "+v"(l.lane), "+v"(l.off0));
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

// Load a wave's 8 rows of a chunk of `len` bytes (0 for none: the loads are
// still issued, so every path has the same number in flight); bytes past len
// read 0.  Only a tail chunk's 16-byte piece that straddles len is refetched
// bytewise.
__device__ __forceinline__ void load_chunk(const uint8_t *__restrict__ base,
                                           uint32_t len, const Lane &l,
                                           uint4 (&d)[kRows]) {
  const Rsrc r = rsrc(base, len);
#pragma unroll
  for (int h = 0; h < kRows; ++h) d[h] = buf16<kNt>(r, l.off0 + h * kRow);
  if (len & 15u) {
#pragma unroll
    for (int h = 0; h < kRows; ++h) {
      const uint32_t off = l.off0 + h * kRow;
      if (off < len && off + 16u > len) d[h] = load16_partial(base + off, len - off);
    }
  }
}

// How a wave's 8 KiB enter the chunk CRC.  The word at chunk offset o
// contributes F^(kChunk - o) of itself to the zero-init register R (see
// wm_internal.h), and for lane l, row h, column j of wave w
//     kChunk - o = kSub (7 - w) + kRow (7 - h) + 16 (63 - l) + 4 (3 - j) + 4.
// The four factors are applied in stages: column streams over the rows
// (w_j = sum_h F^(kRow (7 - h)) word_hj), the lane merge over the columns,
// a per-lane shift matrix over the lanes, and a per-wave shift F^(kSub (7 - w)).

// Lane merge of the four column streams: F^12 w0 ^ F^8 w1 ^ F^4 w2 ^ w3.
__device__ __forceinline__ uint32_t lane_merge(uint32_t v0, uint32_t v1, uint32_t v2,
                                               uint32_t v3) {
  return tab4x(kLdsF12, v0, tab4x(kLdsF8, v1, tab4x(kLdsF4, v2, v3)));
}

// Lane shift: lane l's merged value covers bytes that lie 16 (63 - l) + 4
// bytes before the end of its wave's share (see lane_value), so it enters the
// wave's value shifted by F^(16 (63 - l) + 4): a GF(2) matrix of its own,
// applied from its 32 columns in LDS (eight 16-byte reads issued together;
// columns 4q..4q+3 of lane l at kLdsLaneMat + 1024 q + 16 l).
// lane_fold XORs the shifted values of the 64 lanes: the wave's contribution,
// the common F^4 included, as a uniform value.
__device__ __forceinline__ uint32_t lane_shift(uint32_t u) {
  const uint4 *m = reinterpret_cast<const uint4 *>(lds_at(kLdsLaneMat + (threadIdx.x & 63u) * 16u));
  uint4 c[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) c[i] = m[64 * i];
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    // (column & -bit) ^ r, one three-input logic op per column
    r = __builtin_amdgcn_bitop3_b32(c[i].x, (uint32_t)__builtin_amdgcn_sbfe((int)u, 4 * i, 1), r, 0x6A);
    r = __builtin_amdgcn_bitop3_b32(c[i].y, (uint32_t)__builtin_amdgcn_sbfe((int)u, 4 * i + 1, 1), r, 0x6A);
    r = __builtin_amdgcn_bitop3_b32(c[i].z, (uint32_t)__builtin_amdgcn_sbfe((int)u, 4 * i + 2, 1), r, 0x6A);
    r = __builtin_amdgcn_bitop3_b32(c[i].w, (uint32_t)__builtin_amdgcn_sbfe((int)u, 4 * i + 3, 1), r, 0x6A);
  }
  return r;
}
// XOR over the wave's lanes (DPP row shifts and broadcasts), as a uniform value.
__device__ __forceinline__ uint32_t wave_xor(uint32_t v) {
  v ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);
  v ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);
  v ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);
  v ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);
  v ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
  v ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
  return uniform(__builtin_amdgcn_readlane(v, 63));
}
__device__ __forceinline__ uint32_t lane_fold(uint32_t u) { return wave_xor(lane_shift(u)); }

// The lane's merged value of the wave's 8 rows (before its lane shift).
__device__ __forceinline__ uint32_t lane_value(const uint4 (&d)[kRows], const GLane &gl) {
  uint32_t v0 = d[0].x, v1 = d[0].y, v2 = d[0].z, v3 = d[0].w;
#pragma unroll
  for (int h = 1; h < kRows; ++h) {
    v0 = g_step(v0, d[h].x, gl);
    v1 = g_step(v1, d[h].y, gl);
    v2 = g_step(v2, d[h].z, gl);
    v3 = g_step(v3, d[h].w, gl);
  }
  return lane_merge(v0, v1, v2, v3);
}

// lane_value of d while the next chunk's rows load into dn (one load per
// row step, so the memory pipe takes them between the LDS rounds); a short
// chunk's straddling piece is refetched as in load_chunk.
__device__ __forceinline__ uint32_t lane_value_load(const uint4 (&d)[kRows], const GLane &gl,
                                                    const uint8_t *__restrict__ nbase,
                                                    uint32_t nlen, const Lane &l,
                                                    uint4 (&dn)[kRows]) {
  const Rsrc r = rsrc(nbase, nlen);
  dn[0] = buf16<kNt>(r, l.off0);
  uint32_t v0 = d[0].x, v1 = d[0].y, v2 = d[0].z, v3 = d[0].w;
#pragma unroll
  for (int h = 1; h < kRows; ++h) {
    if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);  // (see k_encode)
    dn[h] = buf16<kNt>(r, l.off0 + h * kRow);
    v0 = g_step(v0, d[h].x, gl);
    v1 = g_step(v1, d[h].y, gl);
    v2 = g_step(v2, d[h].z, gl);
    v3 = g_step(v3, d[h].w, gl);
  }
  if (nlen & 15u) {
#pragma unroll
    for (int h = 0; h < kRows; ++h) {
      const uint32_t off = l.off0 + h * kRow;
      if (off < nlen && off + 16u > nlen) dn[h] = load16_partial(nbase + off, nlen - off);
    }
  }
  return lane_merge(v0, v1, v2, v3);
}

// Chunk CRC from the raw (zero-init, padded) value of the whole chunk.
__device__ __forceinline__ uint32_t finish_crc(uint32_t raw, uint32_t len,
                                               const ChunkGeom &g, const CrcTables &T) {
  return len == kChunk ? raw ^ T.k_full : mat_apply(g.tail_mat, raw) ^ g.k_tail;
}

// -------------------------------------------------------------- checksum --

// Lane CRC values of a chunk, double-buffered by chunk step (low region).
__device__ __forceinline__ uint32_t *chk_u(uint32_t b) {
  return reinterpret_cast<uint32_t *>(lds_at(kLdsLow + b * (kThreads * 4u)));
}

// Chunk CRCs: the eight data waves take chunk i's lane values while chunk
// i+1 loads; the ninth wave folds chunk i-1's values into its CRC (the
// Horner step over waves, then the lane shifts and their XOR).
// With `per_chunk` and chunks above 64 KiB, each tile's CRC is shifted past
// the rest of its chunk and XORed into its chunk's entry (zeroed before the
// launch): CRC(A|B) = F^|B|(CRC(A)) ^ CRC(B) is linear in the pieces' CRCs.
__global__ __launch_bounds__(kThreads + 64) void k_checksum(
    const uint8_t *__restrict__ data, ChunkGeom g,
    uint32_t *__restrict__ crc_out, uint32_t per_chunk) {
  load_crc_tables(g.crc_kind);
  __syncthreads();
  const CrcTables &T = g_tables[g.crc_kind];
  const bool is_fold = threadIdx.x >= (uint32_t)kThreads;
  const GLane gl = glane_make();
  const Lane l0 = lane_info();
  const uint32_t G = gridDim.x;
  const uint32_t my_n = blockIdx.x < g.n_chunks ? (g.n_chunks - 1 - blockIdx.x) / G + 1 : 0;
  uint4 d[kRows];
  if (!is_fold)
    load_chunk(data + (uint64_t)blockIdx.x * kChunk, my_n ? chunk_len(g, blockIdx.x) : 0u, l0, d);
  for (uint32_t i = 0; i <= my_n; ++i) {
    const Lane l = lane_fresh(l0);
    if (!is_fold) {
      if (i < my_n) {
        const uint32_t cn = blockIdx.x + (i + 1) * G;
        const bool nv = i + 1 < my_n;
        uint4 dn[kRows];
        chk_u(i & 1)[l.wave * 64u + l.lane] =
            lane_value_load(d, gl, data + (uint64_t)(nv ? cn : 0u) * kChunk,
                            nv ? chunk_len(g, cn) : 0u, l, dn);
#pragma unroll
        for (int h = 0; h < kRows; ++h) d[h] = dn[h];
      }
    } else if (i >= 1) {
      const uint32_t c = blockIdx.x + (i - 1) * G;
      const uint32_t *u = chk_u((i - 1) & 1);
      uint32_t acc = u[l.lane];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) acc = tab4x(kLdsWaveStep, acc, u[w * 64 + l.lane]);
      const uint32_t crc = finish_crc(lane_fold(acc), chunk_len(g, c), g, T);
      if (per_chunk && g.tile_log2) {
        const uint32_t big = c >> g.tile_log2;
        const uint64_t big_end = min((uint64_t)(big + 1) << (16 + g.tile_log2), g.nbytes);
        const uint64_t tile_end = min((uint64_t)(c + 1) * kChunk, g.nbytes);
        const uint32_t part = shift_bytes(T, big_end - tile_end, crc);
        if (l.lane == 0) atomicXor(&crc_out[big], part);
      } else if (l.lane == 0) {
        crc_out[c] = crc;
      }
    }
    __syncthreads();
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
  // decoder: the table CRC just combined settles the verdict (null: none)
  const WsCtl *vctl;
  uint32_t *verdict;
};

struct CombineJobs {
  CombineJob job[2];
};

// The decoder's verdict word once the table CRC is known: the header's
// verdict if the header was rejected, 2 for a bad table, else the records'
// bits.
__device__ __forceinline__ uint32_t decode_verdict(const WsCtl *ctl, uint32_t table_crc) {
  if (!ctl->hdr_ok) return ctl->verdict_pre;
  if (ctl->table_bad || table_crc != ctl->table_crc) return 2u;
  return ctl->rec_bits;
}

// XOR of x over lanes 0..31, valid in every lane (DPP row steps, then the
// two rows' totals through lane 15 and lane 31).
__device__ __forceinline__ uint32_t xor_lanes32(uint32_t x) {
  x ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x ^= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  return __builtin_amdgcn_readlane(x, 15) ^ __builtin_amdgcn_readlane(x, 31);
}

// The pieces' CRCs v_0 .. v_{n-2} (span bytes each) fold to
//     R = sum_i A^(n-2-i) v_i,   A = F^span,
// and the result is F^last_len(R) ^ v_{n-1}.  Zeros put in front of the
// pieces change no term, so the count is padded to N = 4096 K and thread t
// takes the runs of four consecutive (padded) pieces that start at
// 4 (t + 1024 k), k < K: every load instruction of a wave then reads 1 KiB
// of consecutive values.  Its Horner steps by A inside a run and by
// B = A^4096 from run to run, and the threads' results fold as 1024 blocks of
// four pieces (a perfect tree, shifts A^(4 * 2^level)).
__global__ __launch_bounds__(1024) void k_combine(CombineJobs jobs) {
  const CombineJob &J = jobs.job[blockIdx.x];
  const CrcTables &T = g_tables[J.kind];
  const uint32_t n = J.n_dev ? *J.n_dev : J.n;
  // byte tables of A = F^span and B = F^(4096 span), four copies: entry
  // (j, b) of copy c at ((j*256 + b) * 4 + c), a lane reading copy lane % 4,
  // so the random lookups of the steps below spread over more banks
  __shared__ __attribute__((aligned(16))) uint32_t tabA[4096];
  __shared__ __attribute__((aligned(16))) uint32_t tabB[4096];
  __shared__ uint32_t v[1024];
  // F^(2^i), columns: every matrix the steps below take (the index stays
  // below 2 + 10 + 16 + 1)
  __shared__ uint4 pw[48 * 8];
  const uint32_t t = threadIdx.x;
  if (t < 48u * 8u) pw[t] = reinterpret_cast<const uint4 *>(&T.pow2[0][0])[t];
  {  // entry (j, b) = F^k(b << 8j)
    const uint32_t x = (t & 255u) << (8 * (t >> 8));
    const uint32_t a = mat_apply(T.pow2[J.log2span], x);
    const uint32_t b = mat_apply(T.pow2[J.log2span + 12u], x);
    reinterpret_cast<uint4 *>(tabA)[t] = make_uint4(a, a, a, a);
    reinterpret_cast<uint4 *>(tabB)[t] = make_uint4(b, b, b, b);
  }
  __syncthreads();
  if (n == 0) {
    if (t == 0) {
      *J.out = 0u;
      if (J.verdict) *J.verdict = decode_verdict(J.vctl, 0u);
    }
    return;
  }
  const uint32_t *tA = tabA + (t & 3u), *tB = tabB + (t & 3u);
  auto step = [](const uint32_t *tb, uint32_t x) {
    return tb[(x & 255u) * 4u] ^ tb[(256u + ((x >> 8) & 255u)) * 4u] ^
           tb[(512u + ((x >> 16) & 255u)) * 4u] ^ tb[(768u + (x >> 24)) * 4u];
  };
  const uint32_t np = n - 1;                  // the pieces of span bytes
  const uint32_t K = (np + 4095u) >> 12;      // runs per thread
  const uint32_t pad = (K << 12) - np;        // zeros in front
  uint32_t acc = 0;
  for (uint32_t k0 = 0; k0 < K; k0 += 4u) {  // four runs' loads in flight at once
    uint32_t x[16];
#pragma unroll
    for (uint32_t r = 0; r < 4u; ++r) {
#pragma unroll
      for (uint32_t q = 0; q < 4u; ++q) {
        // padded index j, piece j - pad (none in front of the pieces or
        // past the last run)
        const uint32_t jp = 4u * (t + 1024u * (k0 + r)) + q;
        const bool in = k0 + r < K && jp >= pad;
        x[4 * r + q] = J.vals[in ? jp - pad : 0u];
        x[4 * r + q] = in ? x[4 * r + q] : 0u;
      }
    }
#pragma unroll
    for (uint32_t r = 0; r < 4u; ++r) {
      if (k0 + r < K) {
        uint32_t run = x[4 * r];
#pragma unroll
        for (uint32_t q = 1; q < 4u; ++q) run = step(tA, run) ^ x[4 * r + q];
        acc = step(tB, acc) ^ run;
      }
    }
  }
  v[t] = acc;
  __syncthreads();
  // thread t's result precedes 4 (1023 - t) pieces: a perfect tree, whose
  // level-lv pairs go to the lowest threads (whole waves drop out)
  for (uint32_t lv = 0; lv < 10u; ++lv) {
    const uint32_t stride = 2u << lv, i = t * stride;
    const bool act = i < 1024u;
    uint32_t y = 0;
    if (act) y = mat_apply_lds(pw + 8u * (lv + 2u + J.log2span), v[i]) ^ v[i + (stride >> 1)];
    __syncthreads();
    if (act) v[i] = y;
    __syncthreads();
  }
  if (t < 64u) {
    // the first wave shifts the result past the last piece; each matrix
    // product takes the whole wave (lane i < 32 the term of column i)
    const uint32_t lane = t;
    const uint32_t *pcol = reinterpret_cast<const uint32_t *>(pw) + (lane & 31u);
    uint32_t r = v[0];
    for (uint32_t i = 0, k = J.last_len; k; ++i, k >>= 1)
      if (k & 1u) r = xor_lanes32(lane < 32u && ((r >> lane) & 1u) ? pcol[32u * i] : 0u);
    r ^= J.vals[n - 1];
    if (lane == 0) {
      *J.out = r;
      if (J.verdict) *J.verdict = decode_verdict(J.vctl, r);
    }
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

// Single-workgroup stream compaction of flags into ascending indices.  Item
// i is set when any of flags[i << log2per .. (i + 1) << log2per) (below
// n_flags) is: chunks above 64 KiB from their tiles' flags.
__global__ __launch_bounds__(1024) void k_compact(const uint32_t *__restrict__ flags,
                                                  uint32_t n, uint32_t log2per,
                                                  uint32_t n_flags,
                                                  uint32_t *__restrict__ idx,
                                                  uint32_t *__restrict__ count) {
  __shared__ uint32_t wsum[16];
  __shared__ uint32_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  for (uint32_t base = 0; base < n; base += 1024u) {
    uint32_t i = base + threadIdx.x;
    bool f = false;
    if (i < n) {
      const uint32_t t0 = i << log2per, t1 = min((i + 1) << log2per, n_flags);
      for (uint32_t t = t0; t < t1 && !f; ++t) f = flags[t] != 0;
    }
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
//
// One 576-thread workgroup per CU: 8 data waves hold a chunk in registers
// (8 rows each) and a dedicated control wave owns everything that waits on
// global memory other than the data itself (tickets, the decoupled
// look-back of record offsets, headers, table entries) and folds the chunk
// CRC from the data waves' lane values.  The per-phase schedule is given
// above k_encode.

constexpr int kModeList = 0, kModeAll = 1, kModeStep = 2;
constexpr uint64_t kFlagAgg = 1, kFlagIncl = 2;
constexpr uint32_t kLookbackWindow = 256;  // predecessors read per round trip
constexpr int kEncThreads = kThreads + 64;

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
  const uint8_t *plans;  // format v2/v3: the items' code lengths (k_huf_lengths)
};

struct EncShared {
  uint32_t u[kThreads];      // lane values of the chunk's CRC (lane_value)
  uint32_t dirty_w[kWaves];  // per-wave "differs from prev"
  alignas(16) uint32_t esc_w[kWaves];  // escapes per wave
  uint32_t crc;               // the chunk's CRC
  uint32_t first, next;      // tickets before the loop
  uint32_t ticket[2];        // in the loop, by iteration parity
  uint32_t off_lo, off_hi;   // record offset
  alignas(16) uint4 cand[9];    // plan candidates: size, base | k << 8 | mode << 16, n_esc
  alignas(16) uint32_t H[256];  // histogram
  int64_t my_last;              // control: this workgroup's last finished item
  uint64_t my_last_incl;        //          and its inclusive prefix
  uint32_t p4_done;             // format v2/v3: data waves through phase 4
};
static_assert(sizeof(EncShared) <= kLdsMiscBytes, "encoder scratch fits");
constexpr uint32_t kLdsHistE = kLdsLow;   // 256 bins x 32 copies of 2 x u16 (32 KiB)
constexpr uint32_t kLdsStage = kLdsBase;  // record body staging
// codes + escape index + escapes of a chosen packed record: the plan only
// packs when the record is smaller than RAW, so they stay below half a chunk
constexpr uint32_t kLdsStageBytes = kChunk / 2;
// 256 x 8 bytes: for an 8-bit set of escaped words, the v_perm selectors
// that gather their exponent bytes, in word order, from the row's eight
// exponent bytes (0x0C, a zero byte, past the last one)
constexpr uint32_t kLdsEscLut = kLdsStage + kLdsStageBytes;
constexpr uint32_t kLdsEncode = kLdsEscLut + 256 * 8;
static_assert(kLdsEncode <= 163840, "encoder LDS fits one CU");

__device__ __forceinline__ EncShared &enc_shared() {
  return *reinterpret_cast<EncShared *>(lds_at(kLdsMisc));
}

__device__ __forceinline__ void status_store(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t status_load(const uint64_t *p) {
  return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
// Per 16-bit half: min((e - base) mod 2^16, esc).
__device__ __forceinline__ uint32_t pk_sub_min(uint32_t ex, uint32_t base2, uint32_t esc2) {
  u16x2 a = __builtin_bit_cast(u16x2, ex), b = __builtin_bit_cast(u16x2, base2);
  u16x2 e = __builtin_bit_cast(u16x2, esc2);
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(a - b, e));
}

// The 8 sign/mantissa bytes of a 16-byte piece: byte u = (w_u >> 8 & 0x80) |
// (w_u & 0x7F), from the gathered low and high bytes of the words.
__device__ __forceinline__ uint2 sm_bytes(const uint4 &x) {
  const uint32_t lo0 = __builtin_amdgcn_perm(x.y, x.x, 0x06040200u);
  const uint32_t hi0 = __builtin_amdgcn_perm(x.y, x.x, 0x07050301u);
  const uint32_t lo1 = __builtin_amdgcn_perm(x.w, x.z, 0x06040200u);
  const uint32_t hi1 = __builtin_amdgcn_perm(x.w, x.z, 0x07050301u);
  return make_uint2((lo0 & 0x7F7F7F7Fu) | (hi0 & 0x80808080u),
                    (lo1 & 0x7F7F7F7Fu) | (hi1 & 0x80808080u));
}

// Maximum over the wave (DPP row shifts and broadcasts), as a uniform value.
__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));
  return __builtin_amdgcn_readlane(v, 63);
}

// Chunk of a work item; a caller's list must be ascending and in range, a
// violation returns an out-of-range index (the item is then flagged).
__device__ __forceinline__ uint32_t item_chunk(const EncArgs &a, uint32_t item,
                                               const ChunkGeom &g) {
  if (a.mode != kModeList) return item;
  const uint32_t c = ld_const(a.idx + item);
  if (c >= g.n_chunks || (item > 0 && ld_const(a.idx + item - 1) >= c)) return 0xFFFFFFFFu;
  return c;
}

// Look-back (control wave).  lookback_issue reads a window of predecessors
// before other work; lookback_finish consumes it and reads further windows
// only if needed.  The workgroup's own previous item (`known`, whose
// inclusive prefix it computed itself) ends the walk, so a look-back never
// reads further back than the items handed out since that one.  Every item
// publishes its aggregate before its own look-back and tickets go to running
// workgroups in order, so each predecessor publishes eventually; the spin
// bound only guarantees that the kernel terminates if that were ever
// violated (the call then reports an empty payload).
struct Window {
  uint64_t s[kLookbackWindow / 64];
};

__device__ __forceinline__ Window lookback_issue(const uint64_t *status, int64_t top,
                                                 int64_t known, uint64_t known_incl) {
  Window w;
  const uint32_t lane = threadIdx.x & 63u;
#pragma unroll
  for (int q = 0; q < (int)(kLookbackWindow / 64); ++q) {
    const int64_t j = top - (int64_t)(lane * (kLookbackWindow / 64) + q);
    w.s[q] = j > known ? status_load(&status[j])
                       : (j == known ? (known_incl << 2) | kFlagIncl : kFlagIncl);
  }
  return w;
}

__device__ uint64_t lookback_finish(const uint64_t *status, int64_t top, Window w,
                                    int64_t known, uint64_t known_incl, WsCtl *ctl) {
  constexpr int Q = kLookbackWindow / 64;
  const uint32_t lane = threadIdx.x & 63u;
  uint64_t excl = 0;
  uint32_t spins = 0;
  while (top >= 0) {
    // distance of an entry from `top` is lane*Q + q
    uint32_t first = 0xFFFFFFFFu;
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
      w = lookback_issue(status, top, known, known_incl);
      continue;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    excl += v;
    if (stop != 0xFFFFFFFFu) break;
    top -= kLookbackWindow;
    w = lookback_issue(status, top, known, known_incl);
  }
  return excl;
}

// K-bit codes of the data wave's 8 rows into LDS staging.  Codes are formed
// two words at a time in 16-bit lanes: c = min((e - base) mod 2^16, esc), and
// c + 1 carries into bit K exactly for escapes (K = 3: escapes are found on
// the row's packed codes instead).  Per row: escm holds the
// lane's escape flags (bit u = word u, 8 bits per row), lane_r the number of
// the wave's escapes before the lane's first one in this row; lane h of
// row_base receives the wave's escapes before row h (its index entry).  FULL: the
// chunk has kChunk bytes (no word needs a bounds check).
template <uint32_t K, bool FULL>
__device__ __forceinline__ void pack_codes(const uint4 (&d)[kRows], const Lane &l,
                                           uint32_t n_words, uint32_t base,
                                           uint8_t *stage, uint32_t (&escm)[2],
                                           uint32_t (&lane_r)[kRows], uint32_t &wave_esc,
                                           uint32_t &row_base) {
  if constexpr (K == 8) {  // RAW: the exponent plane, one byte per word
#pragma unroll
    for (int h = 0; h < kRows; ++h) {
      if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);  // (see k_encode)
      const uint32_t w0 = (l.off0 + h * kRow) >> 1;
      const uint4 x = d[h];
      // a dword rotated left by one bit holds its low word's exponent in
      // byte 1 and its high word's in byte 3
      const uint32_t r0 = __builtin_amdgcn_alignbit(x.x, x.x, 31), r1 = __builtin_amdgcn_alignbit(x.y, x.y, 31);
      const uint32_t r2 = __builtin_amdgcn_alignbit(x.z, x.z, 31), r3 = __builtin_amdgcn_alignbit(x.w, x.w, 31);
      uint2 e = make_uint2(__builtin_amdgcn_perm(r1, r0, 0x07050301u),
                           __builtin_amdgcn_perm(r3, r2, 0x07050301u));
      if (FULL || w0 < n_words) *reinterpret_cast<uint2 *>(stage + w0) = e;
      lane_r[h] = 0;
    }
    return;
  }
  constexpr uint32_t esc = (1u << K) - 1u;
  constexpr uint32_t esc2 = esc * 0x00010001u;
  const uint32_t base2 = base * 0x00010001u;
  uint32_t cnt3[(kRows + 2) / 3] = {};  // the lane's escapes per row, three rows a word
#pragma unroll
  for (int h = 0; h < kRows; ++h) {
    if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);  // (see k_encode)
    const uint32_t w0 = (l.off0 + h * kRow) >> 1;
    const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
    uint32_t pair[4], m = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t c2 = pk_sub_min((x[j] >> 7) & 0x00FF00FFu, base2, esc2);
      if constexpr (K != 3) m |= (((c2 + 0x00010001u) >> K) & 0x00010001u) << (2 * j);
      pair[j] = (c2 & 0xFFFFu) | (c2 >> (16 - K));  // lo | hi << K
    }
    uint32_t m8 = (m | (m >> 15)) & 0xFFu;
    if constexpr (!FULL) {  // words past the chunk code as 0 and never escape
      const uint32_t vw = w0 >= n_words ? 0u : min(n_words - w0, 8u);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        pair[j] &= vw >= 2u * j + 2u ? ~0u : (vw == 2u * j + 1u ? esc : 0u);
      m8 &= (1u << vw) - 1u;
    }
    if constexpr (K == 3) {
      // escapes are the all-ones codes of the row's 24 code bits: flag u
      // at bit 3u, then gathered to bit u in three shift-or-mask steps
      const uint32_t p3 = pair[0] | (pair[1] << 6) | (pair[2] << 12) | (pair[3] << 18);
      const uint32_t t = p3 & (p3 >> 1) & (p3 >> 2) & 0x00249249u;
      const uint32_t s1 = (t | (t >> 2)) & 0x000C30C3u;
      const uint32_t s2 = (s1 | (s1 >> 4)) & 0x0000F00Fu;
      m8 = (s2 | (s2 >> 8)) & 0xFFu;
    }
    if (FULL || w0 < n_words) {
      uint8_t *at = stage + (w0 >> 3) * K;
      if constexpr (K * 8 <= 32) {
        const uint32_t p = pair[0] | (pair[1] << (2 * K)) | (pair[2] << (4 * K)) |
                           (pair[3] << (6 * K));
        if constexpr (K == 4) *reinterpret_cast<uint32_t *>(at) = p;
        else if constexpr (K == 2) *reinterpret_cast<uint16_t *>(at) = (uint16_t)p;
        else if constexpr (K == 1) *at = (uint8_t)p;
        else {
#pragma unroll
          for (uint32_t b = 0; b < K; ++b) at[b] = (uint8_t)(p >> (8 * b));
        }
      } else {
        const uint64_t p = (uint64_t)pair[0] | ((uint64_t)pair[1] << (2 * K)) |
                           ((uint64_t)pair[2] << (4 * K)) | ((uint64_t)pair[3] << (6 * K));
        if constexpr (K == 6) {
#pragma unroll
          for (uint32_t b = 0; b < 3; ++b)
            reinterpret_cast<uint16_t *>(at)[b] = (uint16_t)(p >> (16 * b));
        } else {
#pragma unroll
          for (uint32_t b = 0; b < K; ++b) at[b] = (uint8_t)(p >> (8 * b));
        }
      }
    }
    escm[h >> 2] |= m8 << (8 * (h & 3));
    cnt3[h / 3] |= __popc(m8) << (10 * (h % 3));
  }
  // escape ranks from the packed counts: one scan per three rows (a wave's
  // row holds at most 512 escapes, so 10-bit fields never carry)
#pragma unroll
  for (int q = 0; q < (kRows + 2) / 3; ++q) {
    const uint32_t incl = wave_incl_scan(cnt3[q]);
    const uint32_t excl = incl - cnt3[q];
    const uint32_t tot = uniform(__builtin_amdgcn_readlane(incl, 63));
#pragma unroll
    for (int j = 0; j < 3 && 3 * q + j < kRows; ++j) {
      const int h = 3 * q + j;
      lane_r[h] = wave_esc + ((excl >> (10 * j)) & 1023u);
      row_base = l.lane == (uint32_t)h ? wave_esc : row_base;
      wave_esc += (tot >> (10 * j)) & 1023u;
    }
  }
}

// A data wave's share of a chunk's exponent histogram in the low LDS
// region: all 32768 words, the words past a short chunk loaded as zero (the
// reduce takes their count off bin 0).  Bin e is 32 dwords at e * 128, one
// per copy (copy = lane mod 32, so the 32 lanes an LDS cycle serves never
// touch the same bank nor the same counter); the low 16 bits of a dword count
// the low words of the lanes' dwords, the high 16 bits their high words.  The
// low word's exponent sits at bits 7..14 already, so its counter's address is
// one three-input logic op, (x & 0x7F80) | copy4, and both increments are
// constants.  A counter counts at most 16 lanes x 32 words.
__device__ __forceinline__ void hist_add(const uint4 (&d)[kRows], uint32_t copy4) {
  static_assert(kLdsHistE == 0, "bin address = e << 7 | copy4");
  uint32_t one = 1u, one_hi = 0x10000u;
  asm volatile("" : "+v"(one), "+v"(one_hi));  // kept in registers across the loop
#pragma unroll
  for (int h = 0; h < kRows; ++h) {
    const uint32_t x[4] = {d[h].x, d[h].y, d[h].z, d[h].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      atomicAdd(reinterpret_cast<uint32_t *>(lds_at(__builtin_amdgcn_bitop3_b32(x[j], 0x7F80u, copy4, 0xEA))),
                one);
      atomicAdd(reinterpret_cast<uint32_t *>(
                    lds_at(__builtin_amdgcn_bitop3_b32(x[j] >> 16, 0x7F80u, copy4, 0xEA))),
                one_hi);
    }
  }
}

// A chunk's record fields as the control wave holds them (uniform).
struct RecFields {
  uint32_t item, c, n_words, mode, k, base, n_esc, size, crc;
  bool dirty, bad;
  uint32_t hcrc;   // CRC of the record header's first 12 bytes
  uint32_t epart;  // CRC register after the table entry's first 8 bytes
};

// Control wave: the record's payload offset (finishing the look-back window
// `win` issued for item - 1), then the item's inclusive prefix, the record
// header and the table entry; the offset goes to the data waves through LDS.
__device__ __forceinline__ void ctl_emit(const EncArgs &a, const RecFields &r, const Window &win,
                                         uint32_t n_items, uint64_t *status, WsCtl *ctl,
                                         uint4 *tab_ws, uint32_t *ecrc, EncShared &sh,
                                         int64_t &my_last, uint64_t &my_last_incl) {
  const uint64_t excl =
      lookback_finish(status, (int64_t)r.item - 1, win, my_last, my_last_incl, ctl);
  const uint64_t agg = ((uint64_t)(r.dirty ? 1u : 0u) << 2) | ((uint64_t)(r.size >> 4) << 26);
  const uint64_t incl = excl + (agg >> 2);
  my_last = r.item;
  my_last_incl = incl;
  const uint32_t rec_idx = (uint32_t)(excl & 0xFFFFFFu);
  const uint64_t rec_off = 64u + ((excl >> 24) << 4);
  const uint32_t hw[4] = {r.mode | (r.k << 8) | (r.base << 16), r.n_words, r.n_esc, r.hcrc};
  const uint32_t ew[4] = {r.c, r.crc, (uint32_t)rec_off, (uint32_t)(rec_off >> 32)};
  const uint32_t eck = crc_feed(r.epart, ew + 2, 2) ^ 0xFFFFFFFFu;
  if ((threadIdx.x & 63u) == 0) {
    status_store(&status[r.item], (incl << 2) | kFlagIncl);
    if (r.item + 1 == n_items) {
      ctl->n_rec = (uint32_t)(incl & 0xFFFFFFu);
      ctl->payload_bytes = (incl >> 24) << 4;  // total record bytes
    }
    if (r.bad) atomicOr(&ctl->error, 2u);
    sh.off_lo = (uint32_t)rec_off;
    sh.off_hi = (uint32_t)(rec_off >> 32);
    if (r.dirty) {
      *reinterpret_cast<uint4 *>(a.payload + rec_off) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
      tab_ws[rec_idx] = make_uint4(ew[0], ew[1], ew[2], ew[3]);
      ecrc[rec_idx] = eck;
      if (a.dirty_idx) a.dirty_idx[rec_idx] = r.c;
    }
    if (a.crc_out && !r.bad) a.crc_out[r.c] = r.crc;
  }
}

// The encoder runs one chunk behind on output: iteration i computes chunk
// X_i (CRC, histogram, plan, codes staged in LDS, sign/mantissa bytes kept
// in registers) and writes the record of X_{i-1}, whose payload offset the
// control wave resolved by look-back: for a full ship at the end of
// iteration i-1, right after X_{i-1}'s size was published (its predecessors
// run alongside and have published theirs by then); for a step, whose clean
// chunks finish early and let workgroups drift apart, in phases 1-2 of
// iteration i, issued before B0 and finished after it (nothing waits for it
// before B2).
//   phase 1:        data: prefetch X_{i+1}, lane CRC values of X_i (step:
//                   diff flags, then B0); control: next ticket
//   phase 2 (..B2): data: reduce X_i's histogram (accumulated in phase 4 of
//                   iteration i-1, or before the loop for the first chunk)
//   phase 3 (..B3): data: write X_{i-1} (staging + sign/mantissa bytes),
//                   score the plan candidates of X_i; control: first step
//                   of X_i's CRC
//   phase 4 (..B4): all: pick X_i's plan; control: publish its size, finish
//                   its CRC; data: X_{i+1}'s histogram, X_i's codes into
//                   staging, escape counts, sign/mantissa bytes
//   phase 5:        control (full ship): look-back of X_i, its prefix,
//                   header and table entry; data: escape index and escapes
//                   into staging
// Each SIMD holds two data waves, and the older one wins issue slots: left
// alone, the younger one finishes each phase last and runs its tail by
// itself.  In the row loops of phases 1 (full ship), 4 and 5 the younger
// one (waves 4..7) takes priority for the first half of its rows, so that
// the two finish together.
template <bool HAS_PREV>
__global__ __launch_bounds__(kEncThreads) void k_encode(EncArgs a, ChunkGeom g) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(a.ws + a.L.ctl);
  uint64_t *status = reinterpret_cast<uint64_t *>(a.ws + a.L.status);
  uint4 *tab_ws = reinterpret_cast<uint4 *>(a.ws + a.L.table);
  uint32_t *ecrc = reinterpret_cast<uint32_t *>(a.ws + a.L.entry_crc);
  // a list longer than the chunk count is invalid (k_encode_prepare flagged
  // it): nothing is encoded
  const uint32_t n_list = a.mode == kModeList ? ld_const(a.n_idx) : 0u;
  const uint32_t n_items =
      uniform(a.mode == kModeList ? (n_list > g.n_chunks ? 0u : n_list) : g.n_chunks);
  const bool need_crc = a.crc_in == nullptr;
  const bool is_ctl = threadIdx.x >= (uint32_t)kThreads;

  load_crc_tables(g.crc_kind);
  const CrcTables &T = g_tables[g.crc_kind];
  EncShared &sh = enc_shared();
  uint8_t *stage = lds_at(kLdsStage);
  uint32_t *hist = reinterpret_cast<uint32_t *>(lds_at(kLdsHistE));
  {
    uint4 *h4 = reinterpret_cast<uint4 *>(hist);
    for (uint32_t i = threadIdx.x; i < 2048u; i += kEncThreads) h4[i] = make_uint4(0, 0, 0, 0);
    if (threadIdx.x < 256u) {
      uint32_t f = threadIdx.x, sel[2] = {0x0C0C0C0Cu, 0x0C0C0C0Cu};
      for (uint32_t j = 0; f; ++j, f &= f - 1u)
        sel[j >> 2] = (sel[j >> 2] & ~(0xFFu << (8 * (j & 3)))) | ((uint32_t)__builtin_ctz(f) << (8 * (j & 3)));
      *reinterpret_cast<uint2 *>(lds_at(kLdsEscLut + 8 * threadIdx.x)) = make_uint2(sel[0], sel[1]);
    }
  }
  if (threadIdx.x == (uint32_t)kThreads) {
    sh.first = atomicAdd(&ctl->ticket, 1u);
    sh.next = atomicAdd(&ctl->ticket, 1u);
    // full ship: the control wave takes each further ticket after B4, an
    // iteration before it is read; the first one is taken here
    if (!HAS_PREV) sh.ticket[0] = atomicAdd(&ctl->ticket, 1u);
    sh.my_last = -1;
    sh.my_last_incl = 0;
  }
  __syncthreads();
  uint32_t item = uniform(sh.first);
  uint32_t next = uniform(sh.next);

  const GLane gl = glane_make();
  const Lane l0 = lane_info();
  uint4 d[kRows];
  if (!is_ctl) {
    const uint32_t c = item < n_items ? uniform(item_chunk(a, item, g)) : 0xFFFFFFFFu;
    load_chunk(a.cur + (uint64_t)(c < g.n_chunks ? c : 0u) * kChunk,
               c < g.n_chunks ? chunk_len(g, c) : 0u, l0, d);
    if (c < g.n_chunks) hist_add(d, (l0.lane & 31u) * 4u);  // copies zeroed before the barrier
  }
  // Every path has its first rows in registers before the loop.  Otherwise
  // the compiler, which merges this entry with the loop's back edge, keeps
  // them pending and inserts counter waits before each read of d inside the
  // loop, and those waits also drain the record stores issued after them.
#pragma unroll
  for (int h = 0; h < kRows; ++h) asm volatile("" ::"v"(d[h].x), "v"(d[h].y), "v"(d[h].z), "v"(d[h].w));
  __syncthreads();  // the first chunk's histogram is complete (the loop has no B1)

  // the chunk whose record is still to be written (uniform), and its
  // sign/mantissa bytes (data waves)
  bool pend = false, p_dirty = false;
  uint32_t p_nw = 0, p_send = 0;
  RecFields pr = {};  // control, step variant: X_{i-1}'s record fields
  // (the step variant keeps them in LDS: only the control wave uses them,
  // and as registers they would stay allocated through the data waves'
  // phases, where that variant has none to spare)
  int64_t my_last_r = -1;
  uint64_t my_last_incl_r = 0;
  int64_t &my_last = HAS_PREV ? sh.my_last : my_last_r;
  uint64_t &my_last_incl = HAS_PREV ? sh.my_last_incl : my_last_incl_r;
  uint2 smp[kRows];
#pragma unroll
  for (int h = 0; h < kRows; ++h) smp[h] = make_uint2(0, 0);

  for (uint32_t it = 0; item < n_items || pend; ++it) {
    const bool cur = item < n_items;
    const Lane l = lane_fresh(l0);
    const uint32_t copy4 = (l.lane & 31u) * 4u;
    uint32_t c = cur ? uniform(item_chunk(a, item, g)) : 0u;
    const bool bad_index = cur && c >= g.n_chunks;
    if (!cur || bad_index) c = 0;
    const uint32_t len = (cur && !bad_index) ? chunk_len(g, c) : 0u;
    const uint32_t n_words = len / 2;
    const bool full = len == kChunk;
    uint4 dn[kRows];
    uint32_t ticket = 0;
    bool next_valid = false;  // X_{i+1} exists and its index is valid

    // ---- phase 1
    if (!is_ctl) {
      const uint32_t cn =
          !HAS_PREV && next < n_items ? uniform(item_chunk(a, next, g)) : 0xFFFFFFFFu;
      if (!HAS_PREV) next_valid = cn < g.n_chunks;
      const uint8_t *nbase = a.cur + (uint64_t)(next_valid ? cn : 0u) * kChunk;
      const uint32_t nlen = next_valid ? chunk_len(g, cn) : 0u;
      if (HAS_PREV) {
        // prev's rows land four at a time while X_i's lane CRC values are
        // taken (rows 0..3 under the first half of the column steps, rows
        // 4..7 under the second), each half compared once the steps are done;
        // X_{i+1}'s loads wait for phase 2, so no more than a chunk and a half
        // of rows are ever live
        const uint8_t *pbase = a.prev + (uint64_t)c * kChunk;
        const Rsrc rp = rsrc(pbase, len);
        auto prev_rows = [&](int h0, uint4 (&p)[4]) {
#pragma unroll
          for (int i = 0; i < 4; ++i) p[i] = buf16<kNt>(rp, l.off0 + (h0 + i) * kRow);
          if (len & 15u) {  // a tail chunk's straddling piece, as in load_chunk
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const uint32_t off = l.off0 + (h0 + i) * kRow;
              if (off < len && off + 16u > len) p[i] = load16_partial(pbase + off, len - off);
            }
          }
        };
        auto diff_rows = [&](int h0, const uint4 (&p)[4]) {
          uint32_t df = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            df |= (d[h0 + i].x ^ p[i].x) | (d[h0 + i].y ^ p[i].y) | (d[h0 + i].z ^ p[i].z) |
                  (d[h0 + i].w ^ p[i].w);
          return df;
        };
        const bool crc_now = need_crc && cur;
        uint32_t v0 = d[0].x, v1 = d[0].y, v2 = d[0].z, v3 = d[0].w;
        auto steps = [&](int h0, int h1) {
#pragma unroll
          for (int h = h0; h < h1; ++h) {
            v0 = g_step(v0, d[h].x, gl);
            v1 = g_step(v1, d[h].y, gl);
            v2 = g_step(v2, d[h].z, gl);
            v3 = g_step(v3, d[h].w, gl);
          }
        };
        uint4 p[4];
        prev_rows(0, p);
        if (crc_now) steps(1, 4);
        uint32_t diff = diff_rows(0, p);
        prev_rows(4, p);
        if (crc_now) {
          steps(4, kRows);
          sh.u[l.wave * 64u + l.lane] = lane_merge(v0, v1, v2, v3);
        }
        diff |= diff_rows(4, p);
        const unsigned long long any = __ballot(diff != 0);
        if (l.lane == 0) sh.dirty_w[l.wave] = any ? 1u : 0u;
      } else if (need_crc && cur) {  // X_i's lane CRC values while X_{i+1} loads
        if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);  // (see above)
        sh.u[l.wave * 64u + l.lane] = lane_value_load(d, gl, nbase, nlen, l, dn);
      } else {
        load_chunk(nbase, nlen, l, dn);
      }
    } else {
      if (HAS_PREV && cur && l.lane == 0) ticket = atomicAdd(&ctl->ticket, 1u);
    }
    bool dirty = cur && !bad_index;
    if (HAS_PREV) {
      __syncthreads();  // B0: per-wave diff flags
      uint32_t dw = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) dw |= sh.dirty_w[w];
      dirty = dirty && uniform(dw) != 0;
      if (is_ctl && pend)  // ---- control: X_{i-1}'s offset, header and table entry
        ctl_emit(a, pr, lookback_issue(status, (int64_t)pr.item - 1, my_last, my_last_incl),
                 n_items, status, ctl, tab_ws, ecrc, sh, my_last, my_last_incl);
    }
    // No barrier here: the histogram reduced below was completed before the
    // last B4, the lane values and X_{i-1}'s offset (step: emitted after B0,
    // possibly still being resolved) are read after B2, and the ticket slot
    // alternates so the control cannot overwrite one still unread.

    // ---- phase 2
    if (HAS_PREV && !is_ctl) {  // X_{i+1}'s loads (its histogram is taken in phase 4)
      const uint32_t cn = next < n_items ? uniform(item_chunk(a, next, g)) : 0xFFFFFFFFu;
      next_valid = cn < g.n_chunks;
      load_chunk(a.cur + (uint64_t)(next_valid ? cn : 0u) * kChunk, next_valid ? chunk_len(g, cn) : 0u,
                 l, dn);
    }
    uint32_t crc = 0;
    if (is_ctl) {
      if (cur) {
        if (!need_crc) crc = bad_index ? 0u : ld_const(a.crc_in + c);
        if (HAS_PREV && l.lane == 0) sh.ticket[it & 1] = ticket;
      }
    } else if (dirty) {
      // reduce the copies: wave w sums bins 32w..32w+31 (its own 4 KiB of
      // them); two lanes share a bin, 16 copies each (four 16-byte reads),
      // the packed halves adding without carry (each half at most 16384)
      const uint32_t bin = l.wave * 32u + (l.lane >> 1);
      const uint4 *src = reinterpret_cast<const uint4 *>(hist + bin * 32u + (l.lane & 1u) * 16u);
      const uint4 q0 = src[0], q1 = src[1], q2 = src[2], q3 = src[3];
      uint32_t s = (q0.x + q0.y + q0.z + q0.w) + (q1.x + q1.y + q1.z + q1.w) +
                   (q2.x + q2.y + q2.z + q2.w) + (q3.x + q3.y + q3.z + q3.w);
      s += (uint32_t)__shfl_xor((int)s, 1, 64);
      if ((l.lane & 1u) == 0)
        sh.H[bin] = (s & 0xFFFFu) + (s >> 16) - (bin == 0 ? kChunk / 2 - n_words : 0u);
    }
    __syncthreads();  // B2: H complete

    // ---- phase 3
    uint32_t crc_acc = 0, hcrc = 0, epart = 0;
    if (is_ctl) {
      if (cur && need_crc) {
        // the chunk CRC from the data waves' lane values, first step: lane l
        // folds lane l of the eight waves (F^kSub per wave)
        crc_acc = sh.u[l.lane];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) crc_acc = tab4x(kLdsWaveStep, crc_acc, sh.u[w * 64 + l.lane]);
        crc_acc = lane_shift(crc_acc);
      }
    } else {
      if (pend && p_dirty) {
        // write X_{i-1}: staged section, then its sign/mantissa plane
        const uint64_t rec_off = (uint64_t)uniform(sh.off_lo) | ((uint64_t)uniform(sh.off_hi) << 32);
        uint8_t *rec = a.payload + rec_off;
        // two staged pieces per thread and step, both read before either is
        // stored (one LDS round trip per pair); the thread's first address
        // is formed here each time rather than held across the loop (a held
        // one is spilled, and its reload would wait for the next chunk's
        // loads)
        const uint32_t n16 = p_send / 16u;
        uint32_t tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        for (uint32_t i = tid; i < n16; i += 2u * kThreads) {
          const uint32_t i2 = i + kThreads;
          const uint4 q0 = *reinterpret_cast<const uint4 *>(stage + 16 * i);
          const uint4 q1 = *reinterpret_cast<const uint4 *>(stage + 16 * min(i2, n16 - 1u));
          *reinterpret_cast<uint4 *>(rec + 16 + 16 * i) = q0;
          if (i2 < n16) *reinterpret_cast<uint4 *>(rec + 16 + 16 * i2) = q1;
        }
        uint8_t *sm_at = rec + 16 + p_send;
#pragma unroll
        for (int h = 0; h < kRows; ++h) {
          const uint32_t w0 = (l.off0 + h * kRow) >> 1;
          if (w0 < p_nw) *reinterpret_cast<uint2 *>(sm_at + w0) = smp[h];
        }
        if (threadIdx.x < 16u && p_nw + threadIdx.x < pad16(p_nw)) sm_at[p_nw + threadIdx.x] = 0;
      }
      if (dirty) {
        // score the plan candidates, one per wave: waves 0..6 place a window
        // of 2^k - 1 exponents (k = wave + 1) where it covers the most words
        // (lowest base on ties), wave 7 prices RAW and a constant exponent;
        // each wave's prefix scratch lives in its own, already reduced, 4 KiB
        // of the histogram copies, which it clears afterwards
        const uint32_t lane = l.lane, b0 = lane * 4u;
        const uint4 hv = *reinterpret_cast<const uint4 *>(&sh.H[b0]);
        const uint64_t n = n_words;
        uint32_t *slice = hist + l.wave * 1024u;
        if (l.wave < 7u) {
          const uint32_t t4 = hv.x + hv.y + hv.z + hv.w;
          const uint32_t ex = wave_incl_scan(t4) - t4;
          const uint32_t pv[4] = {ex, ex + hv.x, ex + hv.x + hv.y, ex + hv.x + hv.y + hv.z};
          uint32_t *P = slice;
          *reinterpret_cast<uint4 *>(P + b0) = make_uint4(pv[0], pv[1], pv[2], pv[3]);
          if (lane == 63u) P[256] = ex + t4;
          const uint32_t kk = l.wave + 1u, width = (1u << kk) - 1u;
          uint32_t key = 0;
#pragma unroll
          for (uint32_t j = 0; j < 4; ++j) {
            const uint32_t inside = P[min(b0 + j + width, 256u)] - pv[j];
            key = max(key, (inside << 8) | (255u - (b0 + j)));
          }
          key = wave_max_u(key);
          const uint32_t c_esc = n_words - (key >> 8);
          const uint64_t sz = pad16((n * kk + 7) / 8) + pad16(2 * ((n + 511) / 512)) +
                              pad16(c_esc) + pad16(n) + 16u;
          if (lane == 0)
            sh.cand[2 + l.wave] =
                make_uint4((uint32_t)sz, (255u - (key & 255u)) | (kk << 8) | (1u << 16), c_esc, 0);
        } else {
          const uint32_t nz = (hv.x ? 1u : 0u) | (hv.y ? 2u : 0u) | (hv.z ? 4u : 0u) | (hv.w ? 8u : 0u);
          const uint32_t n_distinct = __builtin_amdgcn_readlane(wave_incl_scan(__popc(nz)), 63);
          const uint32_t only = wave_max_u(nz ? b0 + 31u - __clz(nz) : 0u);
          if (lane == 0) {
            sh.cand[0] = make_uint4((uint32_t)(16u + 2 * pad16(n)), 0, 0, 0);  // RAW
            sh.cand[1] = make_uint4(n_distinct == 1 ? (uint32_t)(16u + pad16(n)) : ~0u,
                                    only | (1u << 16), 0, 0);
          }
        }
        uint4 *s4 = reinterpret_cast<uint4 *>(slice);
#pragma unroll
        for (uint32_t i = 0; i < 4u; ++i) s4[l.lane + 64u * i] = make_uint4(0, 0, 0, 0);
      } else if (HAS_PREV && cur) {  // a clean chunk's histogram, unused
        uint4 *s4 = reinterpret_cast<uint4 *>(hist + l.wave * 1024u);
#pragma unroll
        for (uint32_t i = 0; i < 4u; ++i) s4[l.lane + 64u * i] = make_uint4(0, 0, 0, 0);
      }
    }
    __syncthreads();  // B3: candidates scored, X_{i-1}'s staging read

    // ---- phase 4: every wave picks the plan, the smallest candidate (the
    // first in the order RAW, constant, k = 1..7 on ties)
    uint32_t mode = 0, k = 0, base = 0, n_esc = 0, size = 0;
    if (dirty) {
      uint4 best = sh.cand[0];
#pragma unroll
      for (int i = 1; i < 9; ++i) {
        const uint4 cc = sh.cand[i];
        if (cc.x < best.x) best = cc;
      }
      size = uniform(best.x);
      base = uniform(best.y) & 255u;
      k = (uniform(best.y) >> 8) & 255u;
      mode = uniform(best.y) >> 16;
      n_esc = uniform(best.z);
    }
    // staged: the exponent-derived section of the record (RAW exponent
    // plane, or codes + escape index + escapes); the sign/mantissa plane
    // follows it
    const uint32_t kbits = mode == 0 ? 8u : k;
    const bool pack = dirty && kbits > 0u;
    const bool has_esc = mode == 1u && k > 0u;
    const uint64_t n = n_words;
    const uint32_t code_bytes = (uint32_t)((n * kbits + 7) / 8);
    const uint32_t n_blocks = has_esc ? (n_words + 511u) / 512u : 0u;
    const uint32_t s_idx = (uint32_t)pad16(code_bytes);  // staging offsets
    const uint32_t s_esc = s_idx + (uint32_t)pad16(2 * n_blocks);
    const uint32_t s_end = s_esc + (uint32_t)pad16(n_esc);
    uint32_t escm[2] = {0, 0};
    uint32_t lane_r[kRows];
    uint32_t row_base = 0;
    if (is_ctl) {
      if (cur && item != 0 && l.lane == 0) {
        const uint64_t agg = ((uint64_t)(dirty ? 1u : 0u) << 2) | ((uint64_t)(size >> 4) << 26);
        status_store(&status[item], agg | kFlagAgg);
      }
      if (cur && need_crc) {
        // second step: the XOR of the shifted lane values (F^4 included)
        crc = bad_index ? 0u : finish_crc(wave_xor(crc_acc), len, g, T);
      }
      if (!HAS_PREV && cur) {
        // full ship: the record header's CRC and the table entry's CRC
        // prefix, here where the control wave is idle rather than after B4
        const uint32_t hw[3] = {mode | (k << 8) | (base << 16), n_words, n_esc};
        hcrc = crc_words(hw, 3);
        const uint32_t ew[2] = {c, crc};
        epart = crc_feed(0xFFFFFFFFu, ew, 2);
      }
    } else {
      // ---- data: X_{i+1}'s histogram (its loads were issued an iteration
      // ago); the atomics drain while the codes below keep the VALUs busy
      if (next_valid) hist_add(dn, copy4);
    }
    if (!is_ctl && dirty) {
      if (pack) {
        // ---- data: codes into staging, escape flags and counts
        if (!full) {  // the wave's own code bytes; lanes past the chunk write none
          uint4 *s4 = reinterpret_cast<uint4 *>(stage + l.wave * 512u * kbits);
          for (uint32_t i = l.lane; i < 32u * kbits; i += 64u) s4[i] = make_uint4(0, 0, 0, 0);
        }
        uint32_t wave_esc = 0;
        if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);  // (see above)
#define WM_PACK(K)                                                                        \
  (full ? pack_codes<K, true>(d, l, n_words, base, stage, escm, lane_r, wave_esc, row_base) \
        : pack_codes<K, false>(d, l, n_words, base, stage, escm, lane_r, wave_esc, row_base))
        switch (kbits) {
          case 1: WM_PACK(1); break;
          case 2: WM_PACK(2); break;
          case 3: WM_PACK(3); break;
          case 4: WM_PACK(4); break;
          case 5: WM_PACK(5); break;
          case 6: WM_PACK(6); break;
          case 7: WM_PACK(7); break;
          default: WM_PACK(8); break;
        }
#undef WM_PACK
        if (l.lane == 0) sh.esc_w[l.wave] = wave_esc;
        // the escape section (with its padding) starts as zeros: phase 5
        // ORs the escaped exponents in
        for (uint32_t i = s_esc + 16u * threadIdx.x; i < s_end; i += 16u * kThreads)
          *reinterpret_cast<uint4 *>(stage + i) = make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int h = 0; h < kRows; ++h) smp[h] = sm_bytes(d[h]);
    }
    __syncthreads();  // B4: codes staged, escape totals known

    if (is_ctl && cur) {
      // ---- control: X_i's offset, prefix, header and table entry.  Its size
      // was published before B4, and the vector-memory pipe is idle here (the
      // data waves' next loads come after the loop top).  The header CRC and
      // the entry's CRC prefix are computed while the look-back loads fly.
      if (!HAS_PREV) {
        // full ship: the ticket for the end of the next iteration (its slot
        // was last read at the end of the previous one), issued with the
        // look-back window so that their latencies overlap; the address
        // goes through a register the compiler cannot see into, so the
        // uniform-address atomic combining (which reads the result back at
        // once, waiting for it) is not applied
        uint32_t zero = 0;
        asm volatile("" : "+v"(zero));
        if (l.lane == 0) ticket = atomicAdd(&ctl->ticket + zero, 1u);
        const Window win = lookback_issue(status, (int64_t)item - 1, my_last, my_last_incl);
        const RecFields r = {item, c, n_words, mode, k, base, n_esc, size, crc, dirty, bad_index,
                             hcrc, epart};
        ctl_emit(a, r, win, n_items, status, ctl, tab_ws, ecrc, sh, my_last, my_last_incl);
        if (l.lane == 0) sh.ticket[(it + 1) & 1] = ticket;
      } else {
        const uint32_t hw[3] = {mode | (k << 8) | (base << 16), n_words, n_esc};
        hcrc = crc_words(hw, 3);
        const uint32_t ew[2] = {c, crc};
        epart = crc_feed(0xFFFFFFFFu, ew, 2);
      }
    }

    // ---- phase 5
    if (!is_ctl && pack && has_esc) {
      // escapes of the waves before this one: two reads, no dependent chain
      const uint4 ea = *reinterpret_cast<const uint4 *>(&sh.esc_w[0]);
      const uint4 eb = *reinterpret_cast<const uint4 *>(&sh.esc_w[4]);
      const uint32_t ew[kWaves] = {ea.x, ea.y, ea.z, ea.w, eb.x, eb.y, eb.z, eb.w};
      uint32_t wave_base = 0;
#pragma unroll
      for (uint32_t w = 0; w < (uint32_t)kWaves - 1u; ++w) wave_base += w < l.wave ? ew[w] : 0u;
      wave_base = uniform(wave_base);
      {  // lane h writes the escape-index entry of the wave's row h (block
         // wave * 8 + h, present when its first word is in the chunk)
        const uint32_t blk = l.wave * kRows + l.lane;
        if (l.lane < (uint32_t)kRows && blk * (kRow / 2) < n_words)
          *reinterpret_cast<uint16_t *>(stage + s_idx + 2 * blk) = (uint16_t)(wave_base + row_base);
      }
      // the lane's escaped exponents of each row, in word order, at byte
      // `at` of the zeroed escape section: gathered by one table lookup and
      // two byte permutes, shifted to at's byte within its dword and ORed in
      // by the lanes that have any
      if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);  // (see above)
#pragma unroll
      for (int h = 0; h < kRows; ++h) {
        if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);
        const uint32_t flags = (escm[h >> 2] >> (8 * (h & 3))) & 255u;
        const uint2 sel = *reinterpret_cast<const uint2 *>(lds_at(kLdsEscLut + 8u * flags));
        // each dword rotated left by one bit puts the low word's exponent in
        // byte 1 and the high word's in byte 3
        const uint4 x = d[h];
        const uint32_t r0 = __builtin_amdgcn_alignbit(x.x, x.x, 31), r1 = __builtin_amdgcn_alignbit(x.y, x.y, 31);
        const uint32_t r2 = __builtin_amdgcn_alignbit(x.z, x.z, 31), r3 = __builtin_amdgcn_alignbit(x.w, x.w, 31);
        const uint32_t ex = __builtin_amdgcn_perm(r1, r0, 0x07050301u);  // words 0..3
        const uint32_t ey = __builtin_amdgcn_perm(r3, r2, 0x07050301u);  // words 4..7
        const uint64_t cb = (uint64_t)__builtin_amdgcn_perm(ey, ex, sel.x) |
                            ((uint64_t)__builtin_amdgcn_perm(ey, ex, sel.y) << 32);
        const uint32_t at = s_esc + wave_base + lane_r[h];
        const uint32_t shb = (at & 3u) * 8u;
        const uint64_t lo = cb << shb;
        const uint32_t hi = (uint32_t)(((cb >> 32) << shb) >> 32);
        uint32_t *w = reinterpret_cast<uint32_t *>(stage + (at & ~3u));
        const uint32_t span = (at & 3u) + __popc(flags);  // bytes from w to the last escape
        if (flags) {
          atomicOr(w, (uint32_t)lo);
          if (span > 4u) atomicOr(w + 1, (uint32_t)(lo >> 32));
          if (span > 8u) atomicOr(w + 2, hi);
        }
      }
      if (threadIdx.x < 16u) {  // zero padding of the index
        const uint32_t t = threadIdx.x;
        if (2 * n_blocks + t < s_esc - s_idx) stage[s_idx + 2 * n_blocks + t] = 0;
      }
    }

    // ---- X_i becomes the pending record
    if (HAS_PREV)
      pr = RecFields{item, c, n_words, mode, k, base, n_esc, size, crc, dirty, bad_index, hcrc, epart};
    pend = cur;
    p_nw = n_words;
    p_dirty = dirty;
    p_send = s_end;
    if (!is_ctl) {
#pragma unroll
      for (int h = 0; h < kRows; ++h) d[h] = dn[h];
    }
    item = next;
    if (cur) next = uniform(sh.ticket[it & 1]);
  }
}

// Zero the control block and the look-back words before an encode.  An
// index list of more than n entries is rejected here (error 2: the payload
// comes out empty).
__global__ void k_encode_prepare(uint8_t *ws, WsLayout L, uint32_t n,
                                 const uint32_t *__restrict__ n_idx) {
  uint64_t *status = reinterpret_cast<uint64_t *>(ws + L.status);
  uint32_t *ctl = reinterpret_cast<uint32_t *>(ws + L.ctl);
  uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  static_assert(offsetof(WsCtl, error) == 4, "error is word 1 of the control block");
  if (i < 64u) ctl[i] = (i == 1u && n_idx && *n_idx > n) ? 2u : 0u;
  for (; i < n; i += gridDim.x * blockDim.x) status[i] = 0;
}

// CRC of a 60-byte payload header held as 15 little-endian words, with the
// byte table in LDS (a chain of 60 dependent lookups: LDS keeps each one
// short).
__device__ __forceinline__ uint32_t header_crc60(const uint32_t (&h)[15], const uint32_t *t1) {
  uint32_t s = 0xFFFFFFFFu;
#pragma unroll
  for (int i = 0; i < 15; ++i) {
#pragma unroll
    for (int b = 0; b < 4; ++b) s = t1[(s ^ (h[i] >> (8 * b))) & 255u] ^ (s >> 8);
  }
  return s ^ 0xFFFFFFFFu;
}
__device__ __forceinline__ void byte_table_to_lds(uint32_t *t1, uint32_t kind) {
  for (uint32_t i = threadIdx.x; i < 256u; i += blockDim.x) t1[i] = g_tables[kind].byte1[i];
}

// Table copy into the payload and the header.
__global__ __launch_bounds__(256) void k_encode_finish(
    uint8_t *__restrict__ payload, const uint8_t *__restrict__ ws, WsLayout L,
    ChunkGeom g, uint32_t full, const uint32_t *__restrict__ crcs,
    uint64_t *payload_bytes, uint32_t *n_dirty, uint32_t *global_crc) {
  const WsCtl *ctl = reinterpret_cast<const WsCtl *>(ws + L.ctl);
  __shared__ uint32_t t1[256];
  if (blockIdx.x == 0) byte_table_to_lds(t1, g.crc_kind);
  __syncthreads();
  if (global_crc && blockIdx.x == 0 && threadIdx.x == 0) *global_crc = crcs[0];
  if (ctl->error) {  // invalid index list or an abandoned scan: no payload
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      for (int i = 0; i < 4; ++i) reinterpret_cast<uint4 *>(payload)[i] = make_uint4(0, 0, 0, 0);
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
    h[0] = 0x30564D57u + (g.codec << 24);  // "WMV1", "WMV2", "WMV3"
    h[1] = g.codec | (g.crc_kind << 16) | (g.codec << 24);
    h[2] = kChunk << g.tile_log2;  // the caller's chunk size and count
    h[3] = g.hdr_n;
    h[4] = (uint32_t)g.nbytes;
    h[5] = (uint32_t)(g.nbytes >> 32);
    h[6] = n_rec;
    h[7] = full;
    h[8] = (uint32_t)total;
    h[9] = (uint32_t)(total >> 32);
    h[10] = crcs[0];  // global CRC
    h[11] = crcs[1];  // table CRC
    h[12] = h[13] = h[14] = 0;
    h[15] = header_crc60(reinterpret_cast<const uint32_t(&)[15]>(h), t1);
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
__global__ __launch_bounds__(64) void k_decode_prepare(
    const uint8_t *__restrict__ payload, uint64_t cap, ChunkGeom g,
    uint64_t staging_cap, uint8_t *ws, WsLayout L) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(ws + L.ctl);
  __shared__ uint32_t t1[256];
  byte_table_to_lds(t1, g.crc_kind);
  __syncthreads();
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
  uint32_t hw[15];
#pragma unroll
  for (int i = 0; i < 15; ++i) hw[i] = ld_u32(payload + 4 * i);
  if (header_crc60(hw, t1) != ld_u32(payload + 60)) return;
  if (ld_u32(payload) != 0x30564D57u + (g.codec << 24)) return;  // "WMV" + codec digit
  if (ld_u32(payload + 4) != (g.codec | (g.crc_kind << 16) | (g.codec << 24))) return;
  if (ld_u32(payload + 8) != (kChunk << g.tile_log2) || ld_u32(payload + 12) != g.hdr_n) return;
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

// One 576-thread workgroup per CU, laid out like the encoder: 8 data waves
// decode one record (wave w: rows 8w..8w+7, which are escape-index blocks
// 8w..8w+7, so each wave finds its escapes from the index alone) while the
// control wave validates the table entry, header, padding and index of the
// record two steps ahead and publishes its layout in LDS.  Data waves hold
// the current record in registers and have the next one's loads in flight
// while they decode; the control wave also settles the previous record
// (chunk CRC from the wave partials, status).
// 8 data waves, the record-check wave and the settle wave (CRC of the
// decoded record against its receipt)
constexpr int kDecThreads = kThreads + 128;
constexpr uint32_t kDecEscBytes = 1024;  // escape window prefetched per data wave
constexpr uint32_t kMetaSkip = 0xFFu;    // table entry rejected: no record status

struct DecMeta {
  uint32_t st;  // 0 decode, kMetaSkip, else the record's status
  uint32_t mode, k, base, n_words, n_esc, c, src_crc, r;
  uint32_t off_lo, off_hi, rlen, esc_off, sm_off;
  uint32_t pad_[2];
  uint32_t ent[68];  // escape index; entries from n_blocks on read n_esc
};
struct CtlRec {  // one record in the control pipeline (LDS, written by lane 0)
  uint32_t valid;  // record exists and its table entry passed its checks
  uint32_t r, c, src_crc;
  uint64_t off, end;
  uint4 ent;       // the entry as read (for the table CRC)
  uint4 hdr;       // record header (step 2)
};

struct DecShared {
  DecMeta meta[4];  // slot = record step & 3
  CtlRec cr[4];  // control pipeline, slot = record step & 3
  uint32_t bad[2][kWaves];   // wave structure failures
};
static_assert(sizeof(DecShared) <= kLdsMiscBytes, "decoder scratch fits");
constexpr uint32_t kLdsDecEsc = kLdsLow;  // + 16 B of read slack, inside the region
// lane CRC values of a record (lane_value), double-buffered by record step
constexpr uint32_t kLdsDecU = kLdsDecEsc + kWaves * kDecEscBytes + 256;
static_assert(kLdsDecU + 2 * kThreads * 4 <= kLdsLow + kLdsLowBytes, "decoder low region fits");
__device__ __forceinline__ uint32_t *dec_u(uint32_t b) {
  return reinterpret_cast<uint32_t *>(lds_at(kLdsDecU + b * (kThreads * 4u)));
}
constexpr uint32_t kLdsDecode = kLdsBase;
static_assert(kLdsDecode <= 163840, "decoder LDS fits one CU");

__device__ __forceinline__ DecShared &dec_shared() {
  return *reinterpret_cast<DecShared *>(lds_at(kLdsMisc));
}

// Control wave: record checks in three steps, each a memory round trip that
// depends on the previous one (table entry, record header, padding and
// escape index).  The decoder runs them for three different records in each
// iteration, so the control wave waits for one round trip per record.

// Steps 1 and 2 are split into issue and record halves: the loads go out
// as vector loads (which complete in order), step 3 of an older record runs
// while they are in flight, and only then are the results recorded in R.
struct CtlLoads {
  uint4 ent, nx, hdr;
};

// Chunks above 64 KiB ship whole: a table of tiles lists, for each chunk it
// ships, every tile of it in order.  Per entry (tile c, whether it is the
// first entry, the next entry's tile if there is one): the first entry
// starts a chunk, a tile that does not end its chunk (nor the state) is
// followed by the next tile, and the next entry, unless it starts a chunk,
// is the next tile.  Over all entries these are exactly the rules that no
// tile lacks the tile before or after it in its chunk.
__device__ __forceinline__ bool tile_order_bad(const ChunkGeom &g, uint32_t c, bool first,
                                               bool has_next, uint32_t next) {
  if (!g.tile_log2) return false;
  const uint32_t m = (1u << g.tile_log2) - 1u;
  bool bad = first && (c & m) != 0u;
  if (((c + 1u) & m) != 0u && c + 1u < g.n_chunks) bad = bad || !has_next || next != c + 1u;
  if (has_next && (next & m) != 0u) bad = bad || next != c + 1u;
  return bad;
}

// Step 1: table entry r and the next one.
__device__ __forceinline__ void ctl_entry_issue(const uint8_t *__restrict__ payload,
                                                uint64_t table_off, uint32_t n_rec, uint32_t r,
                                                bool exists, CtlLoads &L) {
  const uint32_t bytes = !exists ? 0u : (r + 1 < n_rec ? 32u : 16u);
  const Rsrc rs = rsrc(payload + table_off + 16ull * r, bytes);
  L.ent = buf16(rs, 0);
  L.nx = buf16(rs, 16);
}

__device__ __forceinline__ void ctl_entry_record(uint64_t table_off, uint32_t n_rec, uint32_t r,
                                                 bool exists, const ChunkGeom &g,
                                                 const CtlLoads &L, CtlRec &R) {
  uint32_t valid = 0, c = 0, src = 0;
  uint64_t off = 0, end = 0;
  uint4 ent = make_uint4(0, 0, 0, 0);
  if (exists) {
    ent = make_uint4(uniform(L.ent.x), uniform(L.ent.y), uniform(L.ent.z), uniform(L.ent.w));
    c = ent.x;
    src = ent.y;
    off = (uint64_t)ent.z | ((uint64_t)ent.w << 32);
    end = table_off;
    bool tbad = false;
    const uint32_t nxc = uniform(L.nx.x);
    if (r + 1 < n_rec) {
      end = (uint64_t)uniform(L.nx.z) | ((uint64_t)uniform(L.nx.w) << 32);
      tbad = nxc <= c;
    }
    tbad = tbad || tile_order_bad(g, c, r == 0, r + 1 < n_rec, nxc);
    tbad = tbad || c >= g.n_chunks || (r == 0 && off != 64u) || (off & 15u) || off >= end ||
           end > table_off;
    valid = tbad ? 2u : 1u;  // 2: entry rejected
  }
  if ((threadIdx.x & 63u) == 0) {
    R.valid = valid;
    R.r = r;
    R.c = c;
    R.src_crc = src;
    R.off = off;
    R.end = end;
    R.ent = ent;
  }
}

// Step 2: the record header of R.
__device__ __forceinline__ void ctl_header_issue(const uint8_t *__restrict__ payload,
                                                 const CtlRec &R, CtlLoads &L) {
  const uint32_t valid = uniform(R.valid);
  const uint64_t off = ((uint64_t)uniform((uint32_t)(R.off >> 32)) << 32) | uniform((uint32_t)R.off);
  const uint64_t end = ((uint64_t)uniform((uint32_t)(R.end >> 32)) << 32) | uniform((uint32_t)R.end);
  L.hdr = buf16(rsrc(payload + off, valid == 1u && end - off >= 16u ? 16u : 0u), 0);
}

__device__ __forceinline__ void ctl_header_record(const CtlLoads &L, CtlRec &R) {
  const uint4 h = make_uint4(uniform(L.hdr.x), uniform(L.hdr.y), uniform(L.hdr.z), uniform(L.hdr.w));
  if ((threadIdx.x & 63u) == 0) R.hdr = h;
}

// Step 3: header rules, padding, escape index; the layout goes to M.
__device__ __forceinline__ void ctl_body(const uint8_t *__restrict__ payload, const CtlRec &RL,
                                         const ChunkGeom &g, uint32_t *__restrict__ ecrc,
                                         WsCtl *ctl, DecMeta &M) {
  const uint32_t lane = threadIdx.x & 63u;
  CtlRec R;  // uniform copy
  R.valid = uniform(RL.valid);
  if (R.valid == 0u) return;  // no such record
  R.r = uniform(RL.r);
  R.c = uniform(RL.c);
  R.src_crc = uniform(RL.src_crc);
  R.off = ((uint64_t)uniform((uint32_t)(RL.off >> 32)) << 32) | uniform((uint32_t)RL.off);
  R.end = ((uint64_t)uniform((uint32_t)(RL.end >> 32)) << 32) | uniform((uint32_t)RL.end);
  R.ent = make_uint4(uniform(RL.ent.x), uniform(RL.ent.y), uniform(RL.ent.z), uniform(RL.ent.w));
  R.hdr = make_uint4(uniform(RL.hdr.x), uniform(RL.hdr.y), uniform(RL.hdr.z), uniform(RL.hdr.w));
  {
    uint32_t ew[4] = {R.ent.x, R.ent.y, R.ent.z, R.ent.w};
    const uint32_t ec = crc_words(ew, 4);
    if (lane == 0) ecrc[R.r] = ec;
  }
  if (R.valid == 2u) {
    if (lane == 0) {
      atomicOr(&ctl->table_bad, 1u);
      M.st = kMetaSkip;
    }
    return;
  }
  const uint32_t len = chunk_len(g, R.c), n_words = len / 2;
  const uint64_t reclen = R.end - R.off;
  const uint8_t *rec = payload + R.off;
  uint32_t st = 0, mode = 0, k = 0, base = 0, n_esc = 0;
  uint64_t code_bytes = 0, n_blocks = 0, idx_off = 16, esc_off = 16, sm_off = 16;
  if (reclen < 16) {
    st = 4;
  } else {
    uint32_t hw[4] = {R.hdr.x, R.hdr.y, R.hdr.z, R.hdr.w};
    mode = hw[0] & 255u;
    k = (hw[0] >> 8) & 255u;
    base = (hw[0] >> 16) & 255u;
    n_esc = hw[2];
    // RAW keeps one exponent byte per word where codes would be
    const uint32_t kbits = mode == 0 ? 8u : k;
    code_bytes = ((uint64_t)n_words * kbits + 7) / 8;
    n_blocks = (mode == 1 && k) ? ((uint64_t)n_words + 511) / 512 : 0;
    idx_off = 16 + pad16(code_bytes);
    esc_off = idx_off + pad16(2 * n_blocks);
    sm_off = esc_off + pad16(n_esc);
    if (crc_words(hw, 3) != hw[3] || (hw[0] >> 24) || hw[1] != n_words || mode > 1) {
      st = 4;
    } else if (mode == 0) {
      if (k || base || n_esc || reclen != 16u + 2 * pad16(n_words)) st = 4;
    } else if (k > 7 || n_esc > n_words || (k == 0 && n_esc) ||
               reclen != sm_off + pad16(n_words)) {
      st = 4;
    }
  }
  uint32_t entry = n_esc;
  if (st == 0) {
    bool bad = false;
    if (mode == 0) {  // padding of both planes
      if (lane < 16u && n_words + lane < pad16(n_words) &&
          (rec[16 + n_words + lane] | rec[sm_off + n_words + lane]))
        bad = true;
    } else {
      // padding: whole bytes after each section, code bits past n*k
      if (lane < 16u) {
        if (code_bytes + lane < pad16(code_bytes) && rec[16 + code_bytes + lane]) bad = true;
        if (2 * n_blocks + lane < pad16(2 * n_blocks) && rec[idx_off + 2 * n_blocks + lane])
          bad = true;
        if (n_esc + lane < pad16(n_esc) && rec[esc_off + n_esc + lane]) bad = true;
        if (n_words + lane < pad16(n_words) && rec[sm_off + n_words + lane]) bad = true;
        const uint64_t used = (uint64_t)n_words * k;
        if (lane == 0 && (used & 7u) && (rec[16 + used / 8] >> (used & 7u))) bad = true;
      }
      if (lane < n_blocks) entry = *reinterpret_cast<const uint16_t *>(rec + idx_off + 2 * lane);
      if (lane == 0 && n_blocks && entry != 0) bad = true;  // the first block starts at 0
    }
    if (__ballot(bad)) st = 4;
  }
  M.ent[lane] = entry;
  if (lane == 0) {
    M.ent[64] = n_esc;
    M.st = st;
    M.mode = mode;
    M.k = mode == 0 ? 8u : k;  // code bits per word
    M.base = base;
    M.n_words = n_words;
    M.n_esc = n_esc;
    M.c = R.c;
    M.src_crc = R.src_crc;
    M.r = R.r;
    M.off_lo = (uint32_t)R.off;
    M.off_hi = (uint32_t)(R.off >> 32);
    M.rlen = st == 0 ? (uint32_t)reclen : 0u;
    M.esc_off = (uint32_t)esc_off;
    M.sm_off = (uint32_t)sm_off;
  }
}

// A data wave's share of a record: RAW rows in a[], or codes (a[].xyz) and
// sign/mantissa bytes (b[]) plus the head of the wave's escape range (e).
struct DecBuf {
  uint4 a[kRows];
  uint2 b[kRows];
  uint4 e;
};

struct DecView {  // uniform fields of a record as a data wave needs them
  const uint8_t *rec;
  uint32_t rlen;    // bytes of the record the loads may touch (0: none)
  uint32_t mode, k, base, n_words, n_esc, len;
  uint32_t E0, Ee;  // the wave's escape range from the index
  uint32_t al;      // 16-byte aligned start of the prefetched escape window
  uint32_t esc_off, sm_off, r;
};

__device__ __forceinline__ DecView dec_view(const uint8_t *payload, const DecMeta &M,
                                            const Lane &l, const ChunkGeom &g) {
  DecView v;
  const uint64_t off = (uint64_t)uniform(M.off_lo) | ((uint64_t)uniform(M.off_hi) << 32);
  v.rec = payload + off;
  v.rlen = uniform(M.rlen);
  v.mode = uniform(M.mode);
  v.k = uniform(M.k);
  v.base = uniform(M.base);
  v.n_words = uniform(M.n_words);
  v.n_esc = uniform(M.n_esc);
  v.len = chunk_len(g, uniform(M.c));
  v.E0 = uniform(M.ent[l.wave * kRows]);
  v.Ee = uniform(M.ent[l.wave * kRows + kRows]);
  const uint32_t e0c = min(v.E0, v.n_esc);
  v.al = e0c & ~15u;
  v.esc_off = uniform(M.esc_off);
  v.sm_off = uniform(M.sm_off);
  v.r = uniform(M.r);
  return v;
}

// The same 17 loads for every record (codes or RAW exponent bytes, sign /
// mantissa bytes, the head of the wave's escape range) through a descriptor
// that covers the record, so the compiler can count them on every path.
__device__ __forceinline__ void dec_load_row(DecBuf &B, const DecView &v, const Lane &l, Rsrc r,
                                             int h) {
  const uint32_t w0 = (l.off0 + h * kRow) >> 1;
  B.a[h] = buf16(r, 16u + (((w0 >> 3) * v.k) & ~3u));
  B.b[h] = buf8(r, v.sm_off + w0);
}
__device__ __forceinline__ void dec_load_esc(DecBuf &B, const DecView &v, const Lane &l, Rsrc r) {
  B.e = buf16(r, v.esc_off + v.al + 16u * l.lane);
}
__device__ __forceinline__ void dec_load(DecBuf &B, const DecView &v, const Lane &l) {
  const Rsrc r = rsrc(v.rec, v.rlen);
#pragma unroll
  for (int h = 0; h < kRows; ++h) dec_load_row(B, v, l, r, h);
  dec_load_esc(B, v, l, r);
}

__device__ __forceinline__ void dec_store(uint8_t *dst, uint32_t o, uint32_t len,
                                          const uint32_t (&out)[4]) {
  if (o + 16u <= len) {
    *reinterpret_cast<uint4 *>(dst + o) = make_uint4(out[0], out[1], out[2], out[3]);
  } else if (o < len) {
    for (uint32_t b = 0; b < len - o; ++b) dst[o + b] = (uint8_t)(out[b >> 2] >> (8 * (b & 3)));
  }
}

__device__ __forceinline__ uint32_t bfi(uint32_t m, uint32_t a, uint32_t b) {
  return (a & m) | (b & ~m);
}

// The lane's 8 K-bit codes, which start at bit `sh` of a.x, one per byte
// (codes 0..3 in .x, 4..7 in .y).
template <uint32_t K>
__device__ __forceinline__ uint2 unpack_codes(const uint4 &a, uint32_t sh) {
  uint2 c = make_uint2(0, 0);
  if constexpr (K == 0) {
    return c;
  } else {
    const uint32_t v0 = __builtin_amdgcn_alignbit(a.y, a.x, sh);
    if constexpr (K == 8) {
      c = make_uint2(a.x, a.y);  // byte aligned: sh is 0
    } else if constexpr (K == 3) {
      // each 12-bit half (four codes) spreads in two shift-or-mask steps:
      // codes 2, 3 up by 10 bits, then the odd codes up by 5
      const uint32_t g0 = v0 & 0xFFFu, g1 = __builtin_amdgcn_ubfe(v0, 12, 12);
      const uint32_t t0 = ((g0 << 10) | g0) & 0x003F003Fu, t1 = ((g1 << 10) | g1) & 0x003F003Fu;
      c.x = ((t0 << 5) | t0) & 0x07070707u;
      c.y = ((t1 << 5) | t1) & 0x07070707u;
    } else if constexpr (K == 4) {
      const uint32_t t0 = __builtin_amdgcn_perm(0u, v0, 0x01010000u);  // b0 b0 b1 b1
      const uint32_t t1 = __builtin_amdgcn_perm(0u, v0, 0x03030202u);  // b2 b2 b3 b3
      c.x = (t0 & 0x000F000Fu) | ((t0 >> 4) & 0x0F000F00u);
      c.y = (t1 & 0x000F000Fu) | ((t1 >> 4) & 0x0F000F00u);
    } else {
      const uint32_t v1 = K > 4 ? __builtin_amdgcn_alignbit(a.z, a.y, sh) : 0u;
      constexpr uint32_t m = (1u << K) - 1u;
#pragma unroll
      for (uint32_t u = 0; u < 8; ++u) {
        const uint32_t lo = u * K;
        uint32_t f;
        if (lo + K <= 32) f = (v0 >> lo) & m;
        else if (lo >= 32) f = (v1 >> (lo - 32)) & m;
        else f = __builtin_amdgcn_alignbit(v1, v0, lo) & m;
        if (u < 4) c.x |= f << (8 * u);
        else c.y |= f << (8 * (u - 4));
      }
    }
    return c;
  }
}

// Four words from their exponent bytes e and sign/mantissa bytes s:
// word i = (s_i & 0x80) << 8 | e_i << 7 | (s_i & 0x7F).
__device__ __forceinline__ uint2 assemble4(uint32_t e, uint32_t s) {
  const uint32_t b0 = bfi(0x7F7F7F7Fu, s, e << 7);   // low bytes
  const uint32_t b1 = bfi(0x80808080u, s, e >> 1);   // high bytes
  return make_uint2(__builtin_amdgcn_perm(b1, b0, 0x05010400u),
                    __builtin_amdgcn_perm(b1, b0, 0x07030602u));
}

// Decode a packed share with K-bit codes; returns whether a structure rule
// failed.  Works on four words per instruction (one byte each); escapes,
// codes that can overflow the exponent byte and the chunk tail take uniform
// branches.  CRC column streams are advanced over all 8 rows.
template <uint32_t K>
__device__ __forceinline__ bool dec_packed(const DecBuf &B, const DecView &v, const DecMeta &M,
                                           const Lane &l, uint8_t *stage, uint8_t *dst,
                                           uint32_t (&cv)[4], const GLane &gl, DecBuf &N,
                                           const DecView &vn) {
  // the next record's loads go out one row at a time, between the rows of
  // this one, so the memory pipe takes them while the VALUs decode
  const Rsrc rn = rsrc(vn.rec, vn.rlen);
  dec_load_esc(N, vn, l, rn);
  constexpr bool kEsc = K > 0 && K < 8;  // K = 8: RAW exponent bytes, no escapes
  constexpr uint32_t esc = K < 8 ? (1u << K) - 1u : 255u;
  bool bad = false;
  uint32_t acc = v.E0;
  const uint32_t e0c = min(v.E0, v.n_esc), eec = min(max(v.Ee, e0c), v.n_esc);
  const uint32_t sh = ((l.lane * K) & 3u) * 8u;
  const uint32_t base4 = v.base * 0x01010101u;
  const bool wrap = kEsc && v.base + esc > 255u;  // a code can carry out of its byte
  const bool full = v.n_words == kChunk / 2;
  if (kEsc) *reinterpret_cast<uint4 *>(stage + 16u * l.lane) = B.e;
#pragma unroll
  for (int h = 0; h < kRows; ++h) {
    if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);  // (see k_decode)
    dec_load_row(N, vn, l, rn, h);
    const uint32_t row = l.wave * kRows + h;
    const uint32_t w0 = (l.off0 + h * kRow) >> 1;
    uint32_t out[4] = {0, 0, 0, 0};
    if (row * (kRow / 2) < v.n_words) {
      uint2 c = unpack_codes<K>(B.a[h], sh);
      uint32_t vm0 = ~0u, vm1 = ~0u;  // valid code bytes
      if (!full) {
        const uint32_t vw = w0 >= v.n_words ? 0u : min(v.n_words - w0, 8u);
        vm0 = vw >= 4 ? ~0u : (1u << (8 * vw)) - 1u;
        vm1 = vw >= 8 ? ~0u : (vw <= 4 ? 0u : (1u << (8 * (vw - 4))) - 1u);
        c.x &= vm0;
        c.y &= vm1;
      }
      uint2 f = make_uint2(0, 0);  // escape flags at bit 8u+K
      if (kEsc) {
        f.x = (c.x + 0x01010101u) & (0x01010101u << K);
        f.y = (c.y + 0x01010101u) & (0x01010101u << K);
      }
      uint2 e;
      if (!wrap) {
        e = make_uint2(c.x + base4, c.y + base4);
      } else {  // bytewise sum; a non-escape code past 255 is invalid
        const uint32_t s0 = ((c.x & 0x7F7F7F7Fu) + (base4 & 0x7F7F7F7Fu)) ^ ((c.x ^ base4) & 0x80808080u);
        const uint32_t s1 = ((c.y & 0x7F7F7F7Fu) + (base4 & 0x7F7F7F7Fu)) ^ ((c.y ^ base4) & 0x80808080u);
        const uint32_t k0 = ((c.x & base4) | ((c.x | base4) & ~s0)) & 0x80808080u;
        const uint32_t k1 = ((c.y & base4) | ((c.y | base4) & ~s1)) & 0x80808080u;
        if ((k0 & ~(f.x << (7 - (K & 7))) & vm0) | (k1 & ~(f.y << (7 - (K & 7))) & vm1)) bad = true;
        e = make_uint2(s0, s1);
      }
      if (kEsc) {
        // the index entry of this block equals the escapes before it
        if (uniform(M.ent[row]) != acc) bad = true;
        // The lane's escapes are cnt consecutive bytes from rank r0 on; byte
        // u of the lane takes escape number (flagged bytes before u).  No
        // branch on the flags: a lane without escapes merges nothing.
        const uint32_t bx = f.x >> K, by = f.y >> K;  // 0x01 per flagged byte
        const uint32_t cx = __popc(bx), cnt = cx + __popc(by);
        const uint32_t incl = wave_incl_scan(cnt);
        const uint32_t r0 = acc + incl - cnt;
        acc += __builtin_amdgcn_readlane(incl, 63);
        if (r0 + cnt > eec) bad = true;
        const uint32_t at = r0 - v.al;
        const bool in_win = at + cnt <= kDecEscBytes;
        const uint32_t atw = in_win ? at : 0u;  // an address inside the window
        const uint32_t *w = reinterpret_cast<const uint32_t *>(stage + (atw & ~3u));
        const uint32_t sa = (atw & 3u) * 8u;
        uint2 ev = make_uint2(__builtin_amdgcn_alignbit(w[1], w[0], sa),
                              __builtin_amdgcn_alignbit(w[2], w[1], sa));
        if (__ballot(!in_win && cnt != 0)) {  // rare: past the prefetched window
          if (!in_win && cnt != 0) {
            uint32_t t[2] = {0, 0};
            for (uint32_t j = 0; j < cnt; ++j)
              if (r0 + j < eec) t[j >> 2] |= (uint32_t)v.rec[v.esc_off + r0 + j] << (8 * (j & 3));
            ev = make_uint2(t[0], t[1]);
          }
        }
        const uint32_t px = (bx << 8) + (bx << 16) + (bx << 24);  // exclusive prefix
        const uint32_t py = (by << 8) + (by << 16) + (by << 24) + cx * 0x01010101u;
        e.x = bfi((bx << 8) - bx, __builtin_amdgcn_perm(ev.y, ev.x, px), e.x);
        e.y = bfi((by << 8) - by, __builtin_amdgcn_perm(ev.y, ev.x, py), e.y);
      }
      const uint2 lo = assemble4(e.x, B.b[h].x), hi = assemble4(e.y, B.b[h].y);
      out[0] = lo.x;
      out[1] = lo.y;
      out[2] = hi.x;
      out[3] = hi.y;
      if (!full) {  // words past the chunk are zero
        const uint32_t vw = w0 >= v.n_words ? 0u : min(v.n_words - w0, 8u);
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j)
          out[j] &= vw >= 2 * j + 2 ? ~0u : (vw == 2 * j + 1 ? 0xFFFFu : 0u);
      }
    }
    if (h == 0) {
      cv[0] = out[0], cv[1] = out[1], cv[2] = out[2], cv[3] = out[3];
    } else {
      cv[0] = g_step(cv[0], out[0], gl);
      cv[1] = g_step(cv[1], out[1], gl);
      cv[2] = g_step(cv[2], out[2], gl);
      cv[3] = g_step(cv[3], out[3], gl);
    }
    dec_store(dst, l.off0 + h * kRow, v.len, out);
  }
  if (kEsc && acc != v.Ee) bad = true;  // the wave's escapes end where the next block's begin
  return bad;
}

// Decodes records [r0, r1) of the table (clamped to its length), so that a
// payload arriving in batches can be decoded batch by batch.
__global__ __launch_bounds__(kDecThreads) void k_decode(
    const uint8_t *__restrict__ payload, ChunkGeom g, uint8_t *__restrict__ staging,
    uint32_t *__restrict__ rec_status, uint8_t *ws, WsLayout L, uint32_t r0, uint32_t r1) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(ws + L.ctl);
  uint32_t *ecrc = reinterpret_cast<uint32_t *>(ws + L.entry_crc);
  if (!uniform(ctl->hdr_ok)) return;
  const uint32_t n_rec = uniform(ctl->n_rec);
  const uint64_t table_off = ctl->table_off;
  load_crc_tables(g.crc_kind);
  __syncthreads();
  const CrcTables &T = g_tables[g.crc_kind];
  DecShared &sh = dec_shared();
  const bool is_ctl = threadIdx.x >= (uint32_t)kThreads;  // either control wave
  const bool is_settle = threadIdx.x >= (uint32_t)kThreads + 64u;
  const GLane gl = glane_make();
  const Lane l0 = lane_info();
  uint8_t *stage = lds_at(kLdsDecEsc + l0.wave * kDecEscBytes);
  const uint32_t G = gridDim.x;
  const uint32_t lo = min(r0, n_rec), n_in = min(r1, n_rec) - lo;
  const uint32_t my_n = blockIdx.x < n_in ? (n_in - 1 - blockIdx.x) / G + 1 : 0;
  auto rec_of = [&](uint32_t i) { return lo + blockIdx.x + i * G; };

  // control pipeline: in step i, records i+2 (body), i+3 (header) and i+4
  // (entry)
  if (is_ctl && !is_settle) {
    CtlLoads L;
    for (uint32_t j = 0; j < 4; ++j) {
      ctl_entry_issue(payload, table_off, n_rec, rec_of(j), j < my_n, L);
      ctl_entry_record(table_off, n_rec, rec_of(j), j < my_n, g, L, sh.cr[j]);
    }
    for (uint32_t j = 0; j < 3; ++j) {
      ctl_header_issue(payload, sh.cr[j], L);
      ctl_header_record(L, sh.cr[j]);
    }
    for (uint32_t j = 0; j < 2; ++j) ctl_body(payload, sh.cr[j], g, ecrc, ctl, sh.meta[j]);
  }
  __syncthreads();
  DecBuf cur, nxt;
  if (!is_ctl) {
    DecView v0 = dec_view(payload, sh.meta[0], l0, g);
    if (my_n == 0 || uniform(sh.meta[0].st) != 0) v0.rlen = 0;
    dec_load(cur, v0, l0);
  }

  for (uint32_t i = 0; i <= my_n; ++i) {
    const Lane l = lane_fresh(l0);
    if (!is_ctl) {
      const DecMeta &Mn = sh.meta[(i + 1) & 3];
      DecView vn = dec_view(payload, Mn, l, g);
      if (i + 1 >= my_n || uniform(Mn.st) != 0) vn.rlen = 0;  // loads become no-ops
      const DecMeta &M = sh.meta[i & 3];
      if (i >= my_n || uniform(M.st) != 0) {
        dec_load(nxt, vn, l);  // nothing to decode in this step
      } else {
        // Each SIMD holds two data waves, and the older one wins issue
        // slots; left alone the younger one finishes its record last and
        // runs its tail by itself.  The younger one takes priority for the
        // first half of its rows, so that the two finish together.
        if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);
        {
          const DecView v = dec_view(payload, M, l, g);
          uint8_t *dst = staging + (uint64_t)v.r * kChunk;
          uint32_t cv[4] = {0, 0, 0, 0};
          bool bad = false;
          switch (v.k) {  // 8: RAW exponent plane
            case 0: bad = dec_packed<0>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 1: bad = dec_packed<1>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 2: bad = dec_packed<2>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 3: bad = dec_packed<3>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 4: bad = dec_packed<4>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 5: bad = dec_packed<5>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 6: bad = dec_packed<6>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            case 7: bad = dec_packed<7>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
            default: bad = dec_packed<8>(cur, v, M, l, stage, dst, cv, gl, nxt, vn); break;
          }
          dec_u(i & 1)[l.wave * 64u + l.lane] = lane_merge(cv[0], cv[1], cv[2], cv[3]);
          const bool any_bad = __ballot(bad) != 0;
          if (l.lane == 0) sh.bad[i & 1][l.wave] = any_bad ? 1u : 0u;
        }
      }
    } else if (is_settle) {
      if (i >= 1) {  // settle the previous record
        const DecMeta &M = sh.meta[(i - 1) & 3];
        uint32_t st = uniform(M.st);
        if (st != kMetaSkip) {
          if (st == 0) {
            uint32_t bad = 0;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) bad |= sh.bad[(i - 1) & 1][w];
            // the record's CRC from the data waves' lane values: lane l folds
            // lane l of the eight waves (F^kSub per wave), then the lane
            // shifts (F^4 included) and their XOR (see lane_value)
            const uint32_t *u = dec_u((i - 1) & 1);
            uint32_t acc = u[l.lane];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) acc = tab4x(kLdsWaveStep, acc, u[w * 64 + l.lane]);
            const uint32_t c = uniform(M.c);
            const uint32_t crc = finish_crc(lane_fold(acc), chunk_len(g, c), g, T);
            st = bad ? 4u : (crc != uniform(M.src_crc) ? 8u : 0u);
          }
          if (l.lane == 0) {
            if (rec_status) rec_status[uniform(M.r)] = st;
            if (st) atomicOr(&ctl->rec_bits, st);
          }
        }
      }
    } else {
      CtlLoads L;
      ctl_header_issue(payload, sh.cr[(i + 3) & 3], L);
      ctl_entry_issue(payload, table_off, n_rec, rec_of(i + 4), i + 4 < my_n, L);
      ctl_body(payload, sh.cr[(i + 2) & 3], g, ecrc, ctl, sh.meta[(i + 2) & 3]);
      ctl_header_record(L, sh.cr[(i + 3) & 3]);
      ctl_entry_record(table_off, n_rec, rec_of(i + 4), i + 4 < my_n, g, L, sh.cr[(i + 4) & 3]);
    }
    __syncthreads();
    if (!is_ctl) cur = nxt;
  }
}

// ---------------------------------------------------------------- commit --

// 512 threads per workgroup with eight 16-byte pieces each in flight copy
// at about 0.73 of HBM peak on this part, 256 threads with sixteen at about
// 0.66 (measured over grid sizes of 1 to 16 workgroups per CU).
constexpr uint32_t kCopyThreads = 512;
constexpr uint32_t kCopyPieces = kChunk / (16u * kCopyThreads);

__global__ __launch_bounds__(kCopyThreads) void k_commit(uint8_t *__restrict__ live, ChunkGeom g,
                                                const uint8_t *__restrict__ staging,
                                                const uint8_t *__restrict__ payload,
                                                const uint32_t *__restrict__ verdict) {
  if (*verdict != 0u) return;
  const uint32_t n_rec = ld_u32(payload + 24);
  const uint64_t table_off = ld_u64(payload + 32) - 16ull * n_rec;
  // the next record's chunk index is read while the current one copies
  uint32_t c_next = blockIdx.x < n_rec ? ld_u32(payload + table_off + 16ull * blockIdx.x) : 0u;
  for (uint32_t r = blockIdx.x; r < n_rec; r += gridDim.x) {
    const uint32_t c = c_next;
    const uint32_t rn = r + gridDim.x;
    c_next = rn < n_rec ? ld_u32(payload + table_off + 16ull * rn) : 0u;
    uint32_t len = chunk_len(g, c);
    const uint8_t *src = staging + (uint64_t)r * kChunk;
    uint8_t *dst = live + (uint64_t)c * kChunk;
    if (len == kChunk) {
      // all the thread's 16-byte pieces in flight at once, streamed past the
      // caches (neither side is read again here)
      v4u v[kCopyPieces];
#pragma unroll
      for (uint32_t i = 0; i < kCopyPieces; ++i)
        v[i] = __builtin_nontemporal_load(
            reinterpret_cast<const v4u *>(src + threadIdx.x * 16u + i * 16u * kCopyThreads));
#pragma unroll
      for (uint32_t i = 0; i < kCopyPieces; ++i)
        __builtin_nontemporal_store(
            v[i], reinterpret_cast<v4u *>(dst + threadIdx.x * 16u + i * 16u * kCopyThreads));
    } else {
      for (uint32_t off = threadIdx.x; off < len; off += kCopyThreads) dst[off] = src[off];
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

// Dynamic LDS limits, and the premise of lds_at: the kernels that address
// dynamic LDS from 0 have no static LDS.
// -------------------------------------------------------------- format v2 --
// Records are RAW (as in format v1) or HUF: the chunk's exponents in the
// chunk's own canonical Huffman code, lengths at most kHufMaxLen, in 512
// streams.  Stream s holds the words of wave s / 64, lane s % 64 of the
// kernels' row layout (the lane's 8 words of each of its wave's 8 rows, row
// by row), each stream padded to a byte; a code goes into its stream most
// significant bit first, stream bit j being bit j % 8 of byte j / 8.  HUF
// body with k >= 1: code-length nibbles (128 B) | stream byte counts (512 B)
// | streams, padded to 16 | sign/mantissa plane, padded to 16.  With k = 0
// (a single exponent, `base`): the sign/mantissa plane only.  A HUF record
// must be shorter than the RAW one.  The encoder codes each chunk in one
// pass, in the v1 encoder's pipeline (k_huf_encode); the decoder takes a
// record per wave and decodes each stream through a table of the code's
// first kHufMaxLen bits (k_huf_decode_w).

constexpr uint32_t kHufMaxLen = 11;
constexpr uint32_t kHufStreams = 512;
constexpr uint32_t kHufHead = 16 + 128 + kHufStreams;  // record header and the two tables

__device__ __forceinline__ uint64_t huf_rec_size(uint32_t n, uint32_t k, uint32_t sb) {
  return k == 0 ? 16u + pad16(n) : kHufHead + pad16(sb) + pad16(n);
}
__device__ __forceinline__ uint64_t raw_rec_size(uint32_t n) { return 16u + 2 * pad16(n); }

// CRC of whole words with the byte table in device memory (kernels without
// the LDS tables).
__device__ uint32_t crc_words_g(uint32_t kind, const uint32_t *w, int nw) {
  const uint32_t *t1 = g_tables[kind].byte1;
  uint32_t s = 0xFFFFFFFFu;
  for (int i = 0; i < 4 * nw; ++i) s = t1[(s ^ (w[i >> 2] >> (8 * (i & 3)))) & 255u] ^ (s >> 8);
  return s ^ 0xFFFFFFFFu;
}

// Word j (0..7) of a 16-byte row piece, its exponent and sign/mantissa byte.
__device__ __forceinline__ uint32_t word_of(const uint4 &x, int j) {
  const uint32_t v = j < 2 ? x.x : (j < 4 ? x.y : (j < 6 ? x.z : x.w));
  return (v >> (16 * (j & 1))) & 0xFFFFu;
}
// Plane A (Huffman-coded) and plane B (kept raw) of a word, and the word
// from its planes: format v2 codes the exponent and keeps the sign/mantissa
// byte; format v3, the bf16 byte-plane split, codes the high byte (sign and
// the exponent's upper seven bits) and keeps the low byte.
__device__ __forceinline__ uint32_t pa_of(bool v3, uint32_t w) {
  return v3 ? w >> 8 : (w >> 7) & 255u;
}
__device__ __forceinline__ uint32_t pb_of(bool v3, uint32_t w) {
  return v3 ? w & 255u : ((w >> 8) & 0x80u) | (w & 0x7Fu);
}
__device__ __forceinline__ uint32_t word_from(bool v3, uint32_t a, uint32_t b) {
  return v3 ? (a << 8) | b : ((b & 0x80u) << 8) | (a << 7) | (b & 0x7Fu);
}

// Ordering of LDS accesses between the lanes of one wave.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The v2 encoder kernels take one chunk per wave, kHufWaves waves per
// workgroup, each with this scratch (static LDS).
constexpr int kHufWaves = 8;
constexpr uint32_t kHufCopies = 8;  // histogram copies while counting
struct HufWave {
  union {
    struct {
      uint32_t hist[256];
      uint32_t wt[256];     // weights of the length construction
      uint32_t nw[512];     // node weights; canonical codes in the write kernel
      uint32_t key[256];    // weight << 8 | symbol of the nonzero symbols
      uint16_t sym[256];    // nonzero symbols
      uint16_t order[256];  // nonzero symbols by (weight, symbol)
      uint16_t parent[512];
      uint8_t depth[512];
      uint8_t lens[256];
    };
    uint32_t copies[256 * kHufCopies];  // the count's copies, folded into hist
  };
};
static_assert(sizeof(HufWave) * kHufWaves <= 65536, "v2 encoder scratch");

// Code lengths of the counts in W.hist (the oracle's construction: leaves
// sorted by (count, symbol), the two lightest nodes merged with a leaf taken
// before an internal node of equal weight, a symbol's length its depth;
// counts halved while the longest exceeds kHufMaxLen).  Returns the longest
// length (0 for a single symbol, which is then W.order[0]).
// The same construction for 2..64 distinct symbols with every pass in
// registers: lane l holds the weights of symbols l, 64 + l, 128 + l and
// 192 + l (wq), the keys (weight << 8 | symbol) are gathered into lanes
// 0..m-1 through LDS, each lane ranks its key against the m keys read from
// the other lanes, the sorted keys give the leaves in order, and a pass that
// needs capping halves wq in place.
__device__ uint32_t huf_lengths_small(HufWave &W, uint32_t lane, uint32_t (&wq)[4], uint32_t m) {
  constexpr uint32_t kInf = 0xFFFFFFFFu;
  for (int q = 0; q < 4; ++q) W.lens[q * 64 + lane] = 0;
  for (;;) {
    uint32_t i0 = 0;
    for (int q = 0; q < 4; ++q) {
      const unsigned long long msk = __ballot(wq[q] != 0u);
      if (wq[q]) W.key[i0 + lanes_below(msk)] = (wq[q] << 8) | (q * 64 + lane);
      i0 += (uint32_t)__popcll(msk);
    }
    wave_sync();
    const uint32_t key = lane < m ? W.key[lane] : kInf;
    uint32_t rank = 0;  // keys are distinct: ranks 0..m-1 are a permutation
    for (uint32_t j = 0; j < m; ++j)
      rank += (uint32_t)__builtin_amdgcn_readlane((int)key, (int)j) < key ? 1u : 0u;
    if (lane < m) W.nw[rank] = key;
    wave_sync();
    const uint32_t skey = lane < m ? W.nw[lane] : kInf;  // lane r: the key of rank r
    wave_sync();  // (W.key and W.nw are written again by the next pass)
    // leaf i in lane i, internal node j (node m + j) in lane j; picks read
    // lanes at uniform indices
    const uint32_t leafw = lane < m ? skey >> 8 : kInf;
    uint32_t intw = kInf, par_leaf = 0, par_int = 0;
    uint32_t li = 0, ii = 0, n_int = 0;
    for (uint32_t s2 = 0; s2 + 1 < m; ++s2) {
      uint32_t wsum = 0;
      for (int q = 0; q < 2; ++q) {
        const uint32_t wl = li < m ? (uint32_t)__builtin_amdgcn_readlane((int)leafw, (int)li) : kInf;
        const uint32_t wi = ii < n_int ? (uint32_t)__builtin_amdgcn_readlane((int)intw, (int)ii) : kInf;
        if (li < m && (ii >= n_int || wl <= wi)) {
          par_leaf = lane == li ? n_int : par_leaf;
          wsum += wl;
          ++li;
        } else {
          par_int = lane == ii ? n_int : par_int;
          wsum += wi;
          ++ii;
        }
      }
      intw = lane == n_int ? wsum : intw;
      ++n_int;
    }
    uint32_t dint = 0;  // depth of internal node j; the root (last) is 0
    for (int32_t j = (int32_t)n_int - 2; j >= 0; --j) {
      const uint32_t p = (uint32_t)__builtin_amdgcn_readlane((int)par_int, j);
      const uint32_t dp = (uint32_t)__builtin_amdgcn_readlane((int)dint, (int)p);
      dint = lane == (uint32_t)j ? dp + 1u : dint;
    }
    const uint32_t dleaf = (uint32_t)__shfl((int)dint, (int)(lane < m ? par_leaf : 0u), 64) + 1u;
    const uint32_t longest = uniform(wave_max(lane < m ? dleaf : 0u));
    if (longest <= kHufMaxLen) {
      if (lane < m) W.lens[skey & 255u] = (uint8_t)dleaf;
      wave_sync();
      return longest;
    }
    for (int q = 0; q < 4; ++q) wq[q] = wq[q] ? (wq[q] + 1u) >> 1 : 0u;
  }
}

__device__ uint32_t huf_lengths_wave(HufWave &W, uint32_t lane) {
  {
    uint32_t wq[4], m = 0;
    for (int q = 0; q < 4; ++q) {
      wq[q] = W.hist[q * 64 + lane];
      m += (uint32_t)__popcll(__ballot(wq[q] != 0u));
    }
    if (m >= 2u && m <= 64u) return huf_lengths_small(W, lane, wq, m);
  }
  for (int q = 0; q < 4; ++q) W.wt[q * 64 + lane] = W.hist[q * 64 + lane];
  for (;;) {
    wave_sync();
    uint32_t m = 0;
    for (int q = 0; q < 4; ++q) {
      const uint32_t s = q * 64 + lane, w = W.wt[s];
      const unsigned long long msk = __ballot(w != 0u);
      if (w) {
        const uint32_t i = m + lanes_below(msk);
        W.sym[i] = (uint16_t)s;
        W.key[i] = (w << 8) | s;
      }
      m += (uint32_t)__popcll(msk);
      W.lens[s] = 0;
    }
    wave_sync();
    for (uint32_t i = lane; i < m; i += 64u) {  // rank by (weight, symbol)
      const uint32_t ki = W.key[i];
      uint32_t rank = 0;
      for (uint32_t j = 0; j < m; ++j) rank += W.key[j] < ki ? 1u : 0u;
      W.order[rank] = W.sym[i];
    }
    wave_sync();
    uint32_t longest = 0;
    if (m >= 2 && m <= 64) {
      // the same construction in registers: leaf i in lane i, internal node
      // j (node m + j) in lane j; picks read lanes at uniform indices
      const uint32_t kInf = 0xFFFFFFFFu;
      const uint32_t leafw = lane < m ? W.wt[W.order[lane]] : kInf;
      uint32_t intw = kInf, par_leaf = 0, par_int = 0;
      uint32_t li = 0, ii = 0, n_int = 0;
      for (uint32_t s2 = 0; s2 + 1 < m; ++s2) {
        uint32_t wsum = 0;
        for (int q = 0; q < 2; ++q) {
          const uint32_t wl = li < m ? (uint32_t)__builtin_amdgcn_readlane((int)leafw, (int)li) : kInf;
          const uint32_t wi = ii < n_int ? (uint32_t)__builtin_amdgcn_readlane((int)intw, (int)ii) : kInf;
          if (li < m && (ii >= n_int || wl <= wi)) {
            par_leaf = lane == li ? n_int : par_leaf;
            wsum += wl;
            ++li;
          } else {
            par_int = lane == ii ? n_int : par_int;
            wsum += wi;
            ++ii;
          }
        }
        intw = lane == n_int ? wsum : intw;
        ++n_int;
      }
      uint32_t dint = 0;  // depth of internal node j; the root (last) is 0
      for (int32_t j = (int32_t)n_int - 2; j >= 0; --j) {
        const uint32_t p = (uint32_t)__builtin_amdgcn_readlane((int)par_int, j);
        const uint32_t dp = (uint32_t)__builtin_amdgcn_readlane((int)dint, (int)p);
        dint = lane == (uint32_t)j ? dp + 1u : dint;
      }
      const uint32_t dleaf = (uint32_t)__shfl((int)dint, (int)(lane < m ? par_leaf : 0u), 64) + 1u;
      if (lane < m) W.lens[W.order[lane]] = (uint8_t)dleaf;
      longest = wave_max(lane < m ? dleaf : 0u);
    } else if (lane == 0 && m >= 2) {
      for (uint32_t i = 0; i < m; ++i) W.nw[i] = W.wt[W.order[i]];
      uint32_t li = 0, ii = m, n_int = m;
      for (uint32_t s2 = 0; s2 + 1 < m; ++s2) {
        uint32_t pick[2];
        for (int q = 0; q < 2; ++q) {
          if (li < m && (ii >= n_int || W.nw[li] <= W.nw[ii])) pick[q] = li++;
          else pick[q] = ii++;
        }
        W.nw[n_int] = W.nw[pick[0]] + W.nw[pick[1]];
        W.parent[pick[0]] = W.parent[pick[1]] = (uint16_t)n_int;
        ++n_int;
      }
      W.depth[n_int - 1] = 0;
      for (int32_t i = (int32_t)n_int - 2; i >= 0; --i) W.depth[i] = (uint8_t)(W.depth[W.parent[i]] + 1);
      for (uint32_t i = 0; i < m; ++i) {
        W.lens[W.order[i]] = W.depth[i];
        longest = max(longest, (uint32_t)W.depth[i]);
      }
    }
    longest = uniform(__builtin_amdgcn_readfirstlane(longest));
    wave_sync();
    if (longest <= kHufMaxLen) return longest;
    for (int q = 0; q < 4; ++q) {
      const uint32_t s = q * 64 + lane;
      if (W.wt[s]) W.wt[s] = (W.wt[s] + 1u) >> 1;
    }
  }
}

// ------------------------------------------------ format v2/v3, fused encoder --
// The records, from one read of each chunk once k_huf_lengths (below) has
// found its code lengths, in the v1 encoder's pipeline (one workgroup per
// CU, 8 data waves holding a chunk in registers, a control wave, tickets and
// the decoupled look-back; iteration i computes X_i and writes X_{i-1}):
//   phase 1: data: X_i's lane CRC values while X_{i+1} loads; control:
//            X_{i-1}'s look-back, header and table entry, the next ticket
//   phase 2: control: X_i's plan (code lengths) loads
//   phase 3: data: write X_{i-1} (staged section, then plane B from
//            registers); control: first CRC step, X_i's canonical codes into
//            LDS from the code lengths k_huf_lengths found (the construction's
//            serial merges run there, a chunk per wave, so that they overlap)
//   phase 4: data: X_i's plane-B bytes, each lane's stream byte count;
//            control: X_i's CRC
//   phase 5: all: the record's mode and size from the stream totals;
//            control: publish X_i's size, its header CRC and the entry's
//            CRC prefix; data: the code-length nibbles, stream byte counts
//            and streams (HUF) or plane A (RAW) into staging
// Stream s = wave * 64 + lane holds the lane's 8 words of each of its wave's
// 8 rows, which are in its registers.
constexpr uint32_t kLdsHufCode = kLdsStage + kLdsStageBytes;  // 256 x u32: reversed code | len << 24
constexpr uint32_t kLdsHufPend = kLdsHufCode + 1024;  // the control wave's RecFields of X_{i-1}
constexpr uint32_t kLdsHufEncode = kLdsHufPend + 64;
static_assert(kLdsHufEncode <= 163840, "fused format v2 encoder LDS fits one CU");

// Byte offset of the counter of plane A of the low (HI = 0) or high word of
// dword x, copy cp4 / 4: (symbol * kHufCopies + copy) * 4, from the word's
// bits with one shift and one mask (the symbol is bits 7..14 of the word in
// format v2, bits 8..15 in format v3).
template <bool V3, int HI>
__device__ __forceinline__ uint32_t huf_bin_off(uint32_t x, uint32_t cp4) {
  static_assert(kHufCopies == 8, "symbol * 32 bytes");
  constexpr int sh = (V3 ? 3 : 2) + 16 * HI;
  return ((x >> sh) & 0x1FE0u) | cp4;
}

// Code lengths of format v2/v3, one chunk per wave (kHufWaves per
// workgroup): the plane-A histogram (eight interleaved copies, bin b of copy
// c at 8b + c, copy = lane mod 8, so equal symbols of neighbouring lanes hit
// different banks and each address is shared by at most 8 lanes), then the
// format's construction.  Plan of item i at
// plans + kHufPlanBytes i: the longest length k, the single symbol (k = 0),
// and from byte 16 the record's 128 code-length nibble bytes.
template <bool V3>
__global__ __launch_bounds__(64 * kHufWaves) void k_huf_lengths(
    const uint8_t *__restrict__ state, ChunkGeom g, const uint32_t *__restrict__ idx,
    const uint32_t *__restrict__ n_idx, uint8_t *__restrict__ plans) {
  __shared__ HufWave sw[kHufWaves];
  const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63u;
  HufWave &W = sw[wave];
  const uint32_t n_items = idx ? (*n_idx > g.n_chunks ? 0u : *n_idx) : g.n_chunks;
  for (uint32_t item = blockIdx.x * kHufWaves + wave; item < n_items;
       item += gridDim.x * kHufWaves) {
    const uint32_t c = idx ? idx[item] : item;
    if (c >= g.n_chunks) continue;  // (the encoder rejects the list)
    const uint32_t len = chunk_len(g, c), n = len / 2;
    const uint8_t *base = state + (uint64_t)c * kChunk;
    const Rsrc rs = rsrc(base, len);
    uint32_t *H8 = W.copies;
    constexpr uint32_t kQ = 256u * kHufCopies / 256u;  // 16-byte pieces per lane
#pragma unroll
    for (uint32_t q = 0; q < kQ; ++q) reinterpret_cast<uint4 *>(H8)[q * 64 + lane] = make_uint4(0, 0, 0, 0);
    wave_sync();
    const uint32_t cp = lane & (kHufCopies - 1u);
    for (uint32_t q = 0; q < 8u; ++q) {
      uint4 x[8];
#pragma unroll
      for (int h = 0; h < 8; ++h) x[h] = buf16<kNt>(rs, 16u * (512u * q + lane + 64u * h));
      if (len & 15u) {
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const uint32_t o = 16u * (512u * q + lane + 64u * h);
          if (o < len && o + 16u > len) x[h] = load16_partial(base + o, len - o);
        }
      }
      if (len == kChunk) {  // a full chunk: every word counts, no per-word test
        uint8_t *H8b = reinterpret_cast<uint8_t *>(H8);
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const uint32_t xs[4] = {x[h].x, x[h].y, x[h].z, x[h].w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            atomicAdd(reinterpret_cast<uint32_t *>(H8b + huf_bin_off<V3, 0>(xs[j], 4u * cp)), 1u);
            atomicAdd(reinterpret_cast<uint32_t *>(H8b + huf_bin_off<V3, 1>(xs[j], 4u * cp)), 1u);
          }
        }
      } else {
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const uint32_t i0 = 8u * (512u * q + lane + 64u * h);
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (i0 + j < n) atomicAdd(&H8[kHufCopies * pa_of(V3, word_of(x[h], j)) + cp], 1u);
        }
      }
    }
    wave_sync();
    {  // fold the copies into hist: lane l sums bins 4l..4l+3 (every read is
       // issued before any write)
      static_assert(kHufCopies == 8, "two 16-byte reads per bin");
      uint4 cs[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) cs[q] = reinterpret_cast<const uint4 *>(H8)[8 * lane + q];
#pragma unroll
      for (int b = 0; b < 4; ++b)
        W.hist[4 * lane + b] = cs[2 * b].x + cs[2 * b].y + cs[2 * b].z + cs[2 * b].w +
                               cs[2 * b + 1].x + cs[2 * b + 1].y + cs[2 * b + 1].z + cs[2 * b + 1].w;
    }
    wave_sync();
    const uint32_t k = huf_lengths_wave(W, lane);
    uint8_t *P = plans + (uint64_t)item * kHufPlanBytes;
    const uint32_t s0 = 4u * lane;
    *reinterpret_cast<uint16_t *>(P + 16 + 2 * lane) =
        (uint16_t)(W.lens[s0] | (W.lens[s0 + 1] << 4) | (W.lens[s0 + 2] << 8) | (W.lens[s0 + 3] << 12));
    if (lane == 0)
      *reinterpret_cast<uint4 *>(P) = make_uint4(k, k == 0 ? (uint32_t)W.order[0] : 0u, 0u, 0u);
    wave_sync();
  }
}

// Plane A (bytes 0..3: words 0..3 of x) and plane B of a 16-byte row piece.
template <bool V3>
__device__ __forceinline__ uint2 plane_a8(const uint4 &x) {
  if constexpr (V3) {
    return make_uint2(__builtin_amdgcn_perm(x.y, x.x, 0x07050301u),
                      __builtin_amdgcn_perm(x.w, x.z, 0x07050301u));
  } else {  // a dword rotated left by one bit: the exponents in bytes 1 and 3
    const uint32_t r0 = __builtin_amdgcn_alignbit(x.x, x.x, 31), r1 = __builtin_amdgcn_alignbit(x.y, x.y, 31);
    const uint32_t r2 = __builtin_amdgcn_alignbit(x.z, x.z, 31), r3 = __builtin_amdgcn_alignbit(x.w, x.w, 31);
    return make_uint2(__builtin_amdgcn_perm(r1, r0, 0x07050301u),
                      __builtin_amdgcn_perm(r3, r2, 0x07050301u));
  }
}
template <bool V3>
__device__ __forceinline__ uint2 plane_b8(const uint4 &x) {
  if constexpr (V3) {
    return make_uint2(__builtin_amdgcn_perm(x.y, x.x, 0x06040200u),
                      __builtin_amdgcn_perm(x.w, x.z, 0x06040200u));
  } else {
    return sm_bytes(x);
  }
}

// A bool as a type, to pick an instance of a generic lambda.
template <bool B>
struct BoolC {
  static constexpr bool value = B;
};

template <bool V3>
__global__ __launch_bounds__(kEncThreads) void k_huf_encode(EncArgs a, ChunkGeom g) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(a.ws + a.L.ctl);
  uint64_t *status = reinterpret_cast<uint64_t *>(a.ws + a.L.status);
  uint4 *tab_ws = reinterpret_cast<uint4 *>(a.ws + a.L.table);
  uint32_t *ecrc = reinterpret_cast<uint32_t *>(a.ws + a.L.entry_crc);
  const uint32_t n_list = a.mode == kModeList ? ld_const(a.n_idx) : 0u;
  const uint32_t n_items =
      uniform(a.mode == kModeList ? (n_list > g.n_chunks ? 0u : n_list) : g.n_chunks);
  const bool need_crc = a.crc_in == nullptr;
  const bool is_ctl = threadIdx.x >= (uint32_t)kThreads;

  load_crc_tables(g.crc_kind);
  const CrcTables &T = g_tables[g.crc_kind];
  EncShared &sh = enc_shared();
  uint8_t *stage = lds_at(kLdsStage);
  const uint32_t *code = reinterpret_cast<const uint32_t *>(lds_at(kLdsHufCode));
  if (threadIdx.x == (uint32_t)kThreads) {
    sh.first = atomicAdd(&ctl->ticket, 1u);
    sh.next = atomicAdd(&ctl->ticket, 1u);
    sh.p4_done = 0;
  }
  __syncthreads();
  uint32_t item = uniform(sh.first);
  uint32_t next = uniform(sh.next);

  const GLane gl = glane_make();
  const Lane l0 = lane_info();
  uint4 d[kRows];
  if (!is_ctl) {
    const uint32_t c = item < n_items ? uniform(item_chunk(a, item, g)) : 0xFFFFFFFFu;
    load_chunk(a.cur + (uint64_t)(c < g.n_chunks ? c : 0u) * kChunk,
               c < g.n_chunks ? chunk_len(g, c) : 0u, l0, d);
  }
  // the first rows are in registers before the loop (as in k_encode)
#pragma unroll
  for (int h = 0; h < kRows; ++h) asm volatile("" ::"v"(d[h].x), "v"(d[h].y), "v"(d[h].z), "v"(d[h].w));

  bool pend = false, p_dirty = false;
  uint32_t p_nw = 0, p_send = 0;
  int64_t my_last = -1;
  uint64_t my_last_incl = 0;
  // control: X_{i-1}'s record fields, emitted in phase 1 (in LDS: as
  // registers they would stay allocated through the data waves' phases)
  static_assert(sizeof(RecFields) <= 64, "pending record fields fit");
  RecFields &pr = *reinterpret_cast<RecFields *>(lds_at(kLdsHufPend));
  uint2 smp[kRows];
#pragma unroll
  for (int h = 0; h < kRows; ++h) smp[h] = make_uint2(0, 0);

  for (uint32_t it = 0; item < n_items || pend; ++it) {
    const bool cur = item < n_items;
    const Lane l = lane_fresh(l0);
    uint32_t c = cur ? uniform(item_chunk(a, item, g)) : 0u;
    const bool bad_index = cur && c >= g.n_chunks;
    if (!cur || bad_index) c = 0;
    const uint32_t len = (cur && !bad_index) ? chunk_len(g, c) : 0u;
    const uint32_t n_words = len / 2;
    const bool dirty = cur && !bad_index;
    uint4 dn[kRows];
    uint32_t ticket = 0;
    uint32_t pk_v = 0, pbase_v = 0, nib = 0;  // control: X_i's plan as loaded

    // ---- phase 1
    if (!is_ctl) {
      const uint32_t cn = next < n_items ? uniform(item_chunk(a, next, g)) : 0xFFFFFFFFu;
      const bool next_valid = cn < g.n_chunks;
      const uint8_t *nbase = a.cur + (uint64_t)(next_valid ? cn : 0u) * kChunk;
      const uint32_t nlen = next_valid ? chunk_len(g, cn) : 0u;
      // the younger data wave of each SIMD takes issue priority for the
      // first half of the rows of each row loop (as in k_encode)
      if (need_crc && cur) {
        if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);
        sh.u[l.wave * 64u + l.lane] = lane_value_load(d, gl, nbase, nlen, l, dn);
      } else {
        load_chunk(nbase, nlen, l, dn);
      }
    } else {
      // control: X_{i-1}'s look-back and emission, deferred from the end of
      // iteration i-1.  Its aggregate went out then, as did those of the
      // items just before it in the other workgroups, so the walk rarely
      // waits; the next ticket is taken in the same round trip, its address
      // through a register the compiler cannot see into (no uniform-address
      // atomic combining, which would wait for the result at once).  The
      // offset reaches the data waves before B2, where they first use it.
      // X_i's plan loads go out first, with the ticket and the window, so
      // that the round trips overlap (read in phase 2)
      if (dirty) {
        const uint8_t *P = a.plans + (uint64_t)item * kHufPlanBytes;
        pk_v = ld_u32(P);
        pbase_v = ld_u32(P + 4);
        nib = *reinterpret_cast<const uint16_t *>(P + 16 + 2 * l.lane);
      }
      uint32_t zero = 0;
      asm volatile("" : "+v"(zero));
      if (cur && l.lane == 0) ticket = atomicAdd(&ctl->ticket + zero, 1u);
      if (pend) {
        const RecFields r = pr;
        ctl_emit(a, r, lookback_issue(status, (int64_t)r.item - 1, my_last, my_last_incl),
                 n_items, status, ctl, tab_ws, ecrc, sh, my_last, my_last_incl);
      }
    }

    // ---- phase 2
    uint32_t crc = 0;
    uint32_t pk = 0, pbase = 0;  // control: X_i's plan (k_huf_lengths)
    if (is_ctl) {
      if (cur) {
        if (!need_crc) crc = bad_index ? 0u : ld_const(a.crc_in + c);
        if (l.lane == 0) sh.ticket[it & 1] = ticket;
      }
      if (dirty) {
        pk = uniform(pk_v);
        pbase = uniform(pbase_v);
      }
    }
    __syncthreads();  // B2: lane values and X_{i-1}'s offset

    // ---- phase 3
    uint32_t crc_acc = 0;
    if (is_ctl) {
      if (cur && need_crc) {
        crc_acc = sh.u[l.lane];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) crc_acc = tab4x(kLdsWaveStep, crc_acc, sh.u[w * 64 + l.lane]);
        crc_acc = lane_shift(crc_acc);
      }
      if (dirty) {
        // canonical codes from the lengths: per length, consecutive values
        // in symbol order (lane l holds symbols 4l..4l+3)
        const uint32_t ln[4] = {nib & 15u, (nib >> 4) & 15u, (nib >> 8) & 15u, nib >> 12};
        const unsigned long long below = (1ull << l.lane) - 1ull;
        uint32_t ent[4] = {0, 0, 0, 0};
        uint32_t first = 0, prev_cnt = 0;
        for (uint32_t b = 1; b <= pk; ++b) {
          first = (first + prev_cnt) << 1;
          uint32_t before = 0, cnt = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const unsigned long long m = __ballot(ln[j] == b);
            before += (uint32_t)__popcll(m & below);
            cnt += (uint32_t)__popcll(m);
          }
          uint32_t r = first + before;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (ln[j] == b) {
              ent[j] = (__builtin_bitreverse32(r) >> (32u - b)) | (b << 24);
              ++r;
            }
          }
          prev_cnt = cnt;
        }
        *reinterpret_cast<uint4 *>(lds_at(kLdsHufCode + 16u * l.lane)) =
            make_uint4(ent[0], ent[1], ent[2], ent[3]);
        if (l.lane == 0) sh.cand[0] = make_uint4(pk, pbase, 0u, 0u);
        sh.u[l.lane] = nib;  // the record's nibbles, for wave 0 in phase 5
      }
    } else {
      if (pend && p_dirty) {
        // write X_{i-1}: staged section, then its plane B
        const uint64_t rec_off = (uint64_t)uniform(sh.off_lo) | ((uint64_t)uniform(sh.off_hi) << 32);
        uint8_t *rec = a.payload + rec_off;
        const uint32_t n16 = p_send / 16u;
        for (uint32_t i = threadIdx.x; i < n16; i += 2u * kThreads) {
          const uint32_t i2 = i + kThreads;
          const uint4 q0 = *reinterpret_cast<const uint4 *>(stage + 16 * i);
          const uint4 q1 = *reinterpret_cast<const uint4 *>(stage + 16 * min(i2, n16 - 1u));
          *reinterpret_cast<uint4 *>(rec + 16 + 16 * i) = q0;
          if (i2 < n16) *reinterpret_cast<uint4 *>(rec + 16 + 16 * i2) = q1;
        }
        uint8_t *pb_at = rec + 16 + p_send;
#pragma unroll
        for (int h = 0; h < kRows; ++h) {
          const uint32_t w0 = (l.off0 + h * kRow) >> 1;
          if (w0 < p_nw) *reinterpret_cast<uint2 *>(pb_at + w0) = smp[h];
        }
        if (threadIdx.x < 16u && p_nw + threadIdx.x < pad16(p_nw)) pb_at[p_nw + threadIdx.x] = 0;
      }
    }
    __syncthreads();  // B3: the code is in LDS, X_{i-1}'s staging read

    // ---- phase 4
    const uint32_t k = dirty ? uniform(sh.cand[0].x) : 0u;
    uint32_t sb_lane = 0, lane_excl = 0;
    if (is_ctl) {
      if (cur && need_crc) crc = bad_index ? 0u : finish_crc(wave_xor(crc_acc), len, g, T);
    } else {
      if (dirty) {
        // the streams' section of the staging starts as zeros (phase 5 ORs
        // the streams in; X_{i-1}'s staging was read before B3)
        for (uint32_t i = (kHufHead - 16u) / 16u + threadIdx.x; i < kLdsStageBytes / 16u; i += kThreads)
          reinterpret_cast<uint4 *>(stage)[i] = make_uint4(0, 0, 0, 0);
        if (k) {  // the lane's stream: its words' code lengths
          // (a full chunk takes an instance without the per-word test, so
          // that a row's eight table reads go out together instead of one
          // branch and round trip per word)
          auto lengths = [&](auto full_c) {
            constexpr bool kFull = decltype(full_c)::value;
            uint32_t bits = 0;
            if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int h = 0; h < kRows; ++h) {
              if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);
              const uint2 pa = plane_a8<V3>(d[h]);
              const uint32_t w0 = (l.off0 + h * kRow) >> 1;
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const uint32_t e = ((j < 4 ? pa.x : pa.y) >> (8 * (j & 3))) & 255u;
                if (kFull || w0 + j < n_words) bits += code[e] >> 24;
              }
            }
            return bits;
          };
          const uint32_t bits =
              n_words == kChunk / 2 ? lengths(BoolC<true>{}) : lengths(BoolC<false>{});
          sb_lane = (bits + 7u) >> 3;
          const uint32_t incl = wave_incl_scan(sb_lane);
          lane_excl = incl - sb_lane;
          if (l.lane == 63u) sh.esc_w[l.wave] = incl;
        }
#pragma unroll
        for (int h = 0; h < kRows; ++h) smp[h] = plane_b8<V3>(d[h]);
      }
      if (cur && item != 0u) {
        // The last data wave through phase 4 publishes X_i's size (every
        // wave's stream total is in LDS by then), a phase before the
        // control wave could: the next items' look-backs, a phase later,
        // then find it in place instead of waiting for it.
        __threadfence_block();
        uint32_t done = 0;
        if (l.lane == 0) done = atomicAdd(&sh.p4_done, 1u);
        if (__builtin_amdgcn_readfirstlane(done) == (uint32_t)kWaves - 1u) {
          __threadfence_block();
          uint32_t sbt = 0;
          if (dirty && k) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w) sbt += uniform(sh.esc_w[w]);
          }
          const uint64_t raw = raw_rec_size(n_words), hs = huf_rec_size(n_words, k, sbt);
          const uint32_t sz = dirty ? (uint32_t)(hs < raw ? hs : raw) : 0u;
          const uint64_t agg = ((uint64_t)(dirty ? 1u : 0u) << 2) | ((uint64_t)(sz >> 4) << 26);
          if (l.lane == 0) status_store(&status[item], agg | kFlagAgg);
        }
      }
    }
    __syncthreads();  // B4: stream totals known

    // ---- phase 5: the plan (every wave computes it), then the record
    uint32_t mode = 0, base = 0, sb = 0, size = 0, s_send = 0;
    uint32_t wave_base = 0;
    if (dirty) {
      const uint4 ea = *reinterpret_cast<const uint4 *>(&sh.esc_w[0]);
      const uint4 eb = *reinterpret_cast<const uint4 *>(&sh.esc_w[4]);
      const uint32_t ew[kWaves] = {ea.x, ea.y, ea.z, ea.w, eb.x, eb.y, eb.z, eb.w};
      if (k) {
#pragma unroll
        for (uint32_t w = 0; w < (uint32_t)kWaves; ++w) {
          if (w < l.wave) wave_base += ew[w];
          sb += ew[w];
        }
        sb = uniform(sb);
        wave_base = uniform(wave_base);
      }
      const uint64_t raw = raw_rec_size(n_words), hs = huf_rec_size(n_words, k, sb);
      const bool huf = hs < raw;
      mode = huf ? 2u : 0u;
      base = huf && k == 0 ? uniform(sh.cand[0].y) : 0u;
      if (!huf) sb = 0;
      size = (uint32_t)(huf ? hs : raw);
      s_send = huf ? (k ? kHufHead - 16u + (uint32_t)pad16(sb) : 0u) : (uint32_t)pad16(n_words);
    }
    const uint32_t kr = mode == 2u ? k : 0u;
    if (is_ctl && cur) {
      // X_i's size went out in phase 4; the look-back and emission wait for
      // the next iteration's phase 1
      if (l.lane == 0) sh.p4_done = 0;
      const uint32_t hw[3] = {mode | (kr << 8) | (base << 16), n_words, sb};
      const uint32_t hcrc = crc_words(hw, 3);
      const uint32_t ew2[2] = {c, crc};
      const uint32_t epart = crc_feed(0xFFFFFFFFu, ew2, 2);
      if (l.lane == 0)
        pr = RecFields{item, c, n_words, mode, kr, base, sb, size, crc, dirty, bad_index, hcrc, epart};
    }
    if (!is_ctl && dirty) {
      if (mode == 2u && k) {
        // code-length nibbles (wave 0) and stream byte counts, then the
        // lane's stream, ORed into the zeroed section 32 bits at a time at
        // any bit offset (the streams are packed end to end)
        if (l.wave == 0) *reinterpret_cast<uint16_t *>(stage + 2u * l.lane) = (uint16_t)sh.u[l.lane];
        stage[128u + l.wave * 64u + l.lane] = (uint8_t)sb_lane;
        uint32_t *sw = reinterpret_cast<uint32_t *>(stage);
        uint32_t P = 8u * (kHufHead - 16u + wave_base + lane_excl);  // next bit to place
        uint64_t acc = 0;
        uint32_t nb = 0;
        auto emit = [&](bool whole) {  // the low 32 bits if held (all at the end)
          const bool e32 = whole || nb >= 32u;
          const uint64_t v = (uint64_t)(e32 ? (uint32_t)acc : 0u) << (P & 31u);
          atomicOr(&sw[P >> 5], (uint32_t)v);
          atomicOr(&sw[(P >> 5) + 1u], (uint32_t)(v >> 32));
          P += e32 ? 32u : 0u;
          acc = e32 ? acc >> 32 : acc;
          nb -= e32 && !whole ? 32u : 0u;
        };
        // (a full chunk takes an instance without the per-word test, as
        // above)
        auto pack = [&](auto full_c) {
          constexpr bool kFull = decltype(full_c)::value;
          if (l.wave >= kWaves / 2) __builtin_amdgcn_s_setprio(1);
#pragma unroll
          for (int h = 0; h < kRows; ++h) {
            if (h == kRows / 2) __builtin_amdgcn_s_setprio(0);
            const uint2 pa = plane_a8<V3>(d[h]);
            const uint32_t w0 = (l.off0 + h * kRow) >> 1;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const uint32_t e = ((j < 4 ? pa.x : pa.y) >> (8 * (j & 3))) & 255u;
              const uint32_t cw = kFull || w0 + j < n_words ? code[e] : 0u;
              acc |= (uint64_t)(cw & 0xFFFFFFu) << nb;
              nb += cw >> 24;
              if (j & 1) emit(false);  // at most 22 bits since the last emission
            }
          }
        };
        if (n_words == kChunk / 2) pack(BoolC<true>{});
        else pack(BoolC<false>{});
        emit(true);  // fewer than 32 bits are left
      } else if (mode == 0u) {  // RAW: plane A, one byte per word
#pragma unroll
        for (int h = 0; h < kRows; ++h) {
          const uint32_t w0 = (l.off0 + h * kRow) >> 1;
          if (w0 < n_words) *reinterpret_cast<uint2 *>(stage + w0) = plane_a8<V3>(d[h]);
        }
        if (threadIdx.x < 16u && n_words + threadIdx.x < pad16(n_words)) stage[n_words + threadIdx.x] = 0;
      }
    }

    // ---- X_i becomes the pending record
    pend = cur;
    p_nw = n_words;
    p_dirty = dirty;
    p_send = s_send;
    if (!is_ctl) {
#pragma unroll
      for (int h = 0; h < kRows; ++h) d[h] = dn[h];
    }
    item = next;
    if (cur) next = uniform(sh.ticket[it & 1]);
  }
}

// ---------------------------------------------- format v2/v3, one record per wave --
// The Huffman-format decoder with a record per wave: kHwWaves records in
// flight per workgroup, each wave checking, decoding and verifying its own
// record with no workgroup barrier, so that one record's dependent steps
// (table checks, code construction, the symbol-by-symbol decode of each
// stream) overlap the other waves' work.  Lane l decodes streams q * 64 + l
// (q = 0..7), which are its 16 bytes of rows 8q..8q+7 in the row layout: a
// lane's output runs down rows 0..63 in order, so its four CRC column
// streams take all 64 rows and the lane shifts and the XOR over the wave give
// the record's CRC without a per-wave step.
// The 64 streams of group q are contiguous in the record; the wave copies
// them into an LDS stage with coalesced loads issued one group ahead, and
// each lane refills its bit buffer from the stage, so the decode waits on
// LDS only (a refill from device memory would wait behind every store and
// load issued before it).  A group whose streams overflow the stage, and the
// last, short record, take a per-symbol path.  Checks and verdict bits are
// the same as the per-workgroup decoders'.
constexpr int kHwWaves = 8;
constexpr uint32_t kHwTab = 4096;    // per wave: decode table, 2^11 u16 entries
constexpr uint32_t kHwStage = 4096;  // per wave: a group's streams (code order first)
constexpr uint32_t kHwScratch = kHwTab + kHwStage;
constexpr uint32_t kHwOverrun = 64u * 11u / 8u + 8u;  // bytes a stream's reads may pass its end
// waves 0..3 in the low region, waves 4..7 after the CRC tables; tables at
// multiples of 4096, so an entry's address is the table's base ORed with it
__device__ __forceinline__ uint32_t hw_scratch(uint32_t wave) {
  return wave < 4u ? kLdsLow + wave * kHwScratch : kLdsBase + (wave - 4u) * kHwScratch;
}
constexpr uint32_t kLdsHufDecodeW = kLdsBase + 4u * kHwScratch;
static_assert(4u * kHwScratch <= kLdsLowBytes && kLdsHufDecodeW <= 163840 &&
                  kLdsBase % 4096u == 0 && kHwScratch % 4096u == 0,
              "record-per-wave decoder LDS fits one CU");

__device__ __forceinline__ uint32_t buf4(Rsrc r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
// The low `take` bytes (0..4) of d.
__device__ __forceinline__ uint32_t low_bytes(uint32_t d, uint32_t take) {
  return take >= 4u ? d : d & ((1u << (8u * take)) - 1u);
}

// (m & a) | (~m & b) in one three-input logic op (truth table 0xCA).
__device__ __forceinline__ uint32_t bitsel(uint32_t m, uint32_t a, uint32_t b) {
  return __builtin_amdgcn_bitop3_b32(m, a, b, 0xCA);
}

// Eight words from their plane bytes: byte j of a and b makes word j
// (words 0..3 from .x, 4..7 from .y), two words per output dword.
template <bool V3>
__device__ __forceinline__ void words_from_planes(const uint2 &a, const uint2 &b,
                                                  uint32_t (&out)[4]) {
#pragma unroll
  for (int qq = 0; qq < 4; ++qq) {
    // bytes b_j, a_j, b_j+1, a_j+1: the v3 words as they are
    const uint32_t p = __builtin_amdgcn_perm(qq < 2 ? a.x : a.y, qq < 2 ? b.x : b.y,
                                             (qq & 1) ? 0x07030602u : 0x05010400u);
    // v2: sign bit 7 of b to bit 15, the exponent a to bits 7..14, b's low
    // seven bits stay (both halves at once)
    if constexpr (V3) out[qq] = p;
    else out[qq] = bitsel(0x80008000u, p << 8, bitsel(0x007F007Fu, p, p >> 1));
  }
}

// One row's words, CRC column steps and store, for rows that may pass the
// chunk's end.
template <bool V3>
__device__ __forceinline__ void hw_row_out(const uint2 &pa, const uint2 &pb, uint32_t w0,
                                           uint32_t n, bool full, uint32_t len, uint8_t *dst,
                                           uint32_t (&cv)[4], const GLane &gl) {
  uint32_t out[4];
  words_from_planes<V3>(pa, pb, out);
  if (!full && w0 + 8u > n) {  // words past the chunk's end are zero
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (w0 + j >= n) out[j >> 1] &= (j & 1) ? 0x0000FFFFu : 0xFFFF0000u;
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) cv[c] = g_step(cv[c], out[c], gl);
  dec_store(dst, 2u * w0, len, out);
}

template <bool V3>
__global__ __launch_bounds__(64 * kHwWaves) void k_huf_decode_w(
    const uint8_t *__restrict__ payload, ChunkGeom g, uint8_t *__restrict__ staging,
    uint32_t *__restrict__ rec_status, uint8_t *ws, WsLayout L, uint32_t r0, uint32_t r1) {
  WsCtl *ctl = reinterpret_cast<WsCtl *>(ws + L.ctl);
  uint32_t *ecrc = reinterpret_cast<uint32_t *>(ws + L.entry_crc);
  if (!uniform(ctl->hdr_ok)) return;
  const uint32_t n_rec = uniform(ctl->n_rec);
  const uint32_t r_hi = min(r1, n_rec), r_lo = min(r0, r_hi);
  const uint64_t table_off = ((uint64_t)uniform((uint32_t)(ctl->table_off >> 32)) << 32) |
                             uniform((uint32_t)ctl->table_off);
  load_crc_tables(g.crc_kind);
  __syncthreads();  // the only barrier: the tables are in LDS
  const CrcTables &T = g_tables[g.crc_kind];
  const uint32_t wave = uniform(threadIdx.x >> 6), lane = threadIdx.x & 63u;
  const uint32_t tbase = hw_scratch(wave), sbase = tbase + kHwTab;
  uint16_t *tab = reinterpret_cast<uint16_t *>(lds_at(tbase));
  uint8_t *sorted = lds_at(sbase);  // symbols in code order, while the table is built
  const GLane gl = glane_make();
  const unsigned long long below = (1ull << lane) - 1ull;
  for (uint32_t r = r_lo + blockIdx.x * kHwWaves + wave; r < r_hi; r += gridDim.x * kHwWaves) {
    // ---- table entry (and its neighbours' chunk and offset) and header
    const uint8_t *e = payload + table_off + 16ull * r;
    uint32_t ew[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ew[i] = uniform(ld_u32(e + 4 * i));
    const uint32_t prevc = r > 0 ? uniform(ld_u32(e - 16)) : 0u;
    const bool has_next = r + 1 < n_rec;
    const uint32_t nextc = has_next ? uniform(ld_u32(e + 16)) : 0u;
    const uint64_t end = has_next ? ((uint64_t)uniform(ld_u32(e + 28)) << 32) | uniform(ld_u32(e + 24))
                                  : table_off;
    const uint32_t c = ew[0];
    const uint64_t off = ew[2] | ((uint64_t)ew[3] << 32);
    const bool tbad = c >= g.n_chunks || (r > 0 && prevc >= c) || (r == 0 && off != 64u) ||
                      (off & 15u) || off >= end || end > table_off ||
                      tile_order_bad(g, c, r == 0, has_next, nextc);
    const uint32_t ec = crc_words(ew, 4);
    if (lane == 0) ecrc[r] = ec;
    if (tbad) {
      if (lane == 0) atomicOr(&ctl->table_bad, 1u);
      continue;  // no record status for a rejected entry
    }
    const uint32_t len = chunk_len(g, c), n = len / 2;
    const uint64_t rl = end - off;
    const uint8_t *rec = payload + off;
    uint32_t st = 0, mode = 0, k = 0, base = 0, sb = 0;
    if (rl < 16) {
      st = 4;
    } else {
      uint32_t hw[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) hw[i] = uniform(ld_u32(rec + 4 * i));
      mode = hw[0] & 255u;
      k = (hw[0] >> 8) & 255u;
      base = (hw[0] >> 16) & 255u;
      sb = hw[2];
      if (crc_words(hw, 3) != hw[3] || (hw[0] >> 24) || hw[1] != n) {
        st = 4;
      } else if (mode == 0) {
        if (k || base || sb || rl != raw_rec_size(n)) st = 4;
      } else if (mode == 2) {
        if (k > kHufMaxLen || (k == 0 && sb) || (k && base)) st = 4;
        else if (huf_rec_size(n, k, sb) >= raw_rec_size(n) || rl != huf_rec_size(n, k, sb)) st = 4;
      } else {
        st = 4;
      }
    }
    if (st) {
      if (lane == 0) {
        if (rec_status) rec_status[r] = st;
        atomicOr(&ctl->rec_bits, st);
      }
      continue;
    }
    const bool hufk = mode == 2 && k > 0;
    const uint64_t smo = mode == 0 ? 16u + pad16(n) : (hufk ? kHufHead + pad16(sb) : 16u);
    bool bad = false;
    // ---- code lengths, their checks and the decode table (HUF, k >= 1):
    // lane l holds symbols 2l, 2l+1 (nibble byte l) and 128+2l, 129+2l
    // (nibble byte 64 + l)
    uint32_t so[8] = {0, 0, 0, 0, 0, 0, 0, 0}, sbq[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    // the streams section (whole, with its padding: no load straddles its
    // end) and the first group's stage loads, in flight while the table is
    // built
    const Rsrc rs = rsrc(rec + kHufHead, hufk ? (uint32_t)pad16(sb) : 0u);
    uint4 sq0[4] = {};
    if (hufk) {
      const uint32_t nb0 = rec[16 + lane], nb1 = rec[16 + 64 + lane];
      const uint32_t ln[4] = {nb0 & 15u, nb0 >> 4, nb1 & 15u, nb1 >> 4};
      const uint32_t sym[4] = {2u * lane, 2u * lane + 1u, 128u + 2u * lane, 129u + 2u * lane};
      uint32_t kr = 0, mx = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (ln[j] > k) bad = true;
        if (ln[j]) kr += 1u << (kHufMaxLen - min(ln[j], kHufMaxLen));
        mx = max(mx, ln[j]);
      }
      const uint32_t kraft = uniform(__builtin_amdgcn_readlane(wave_incl_scan(kr), 63));
      const uint32_t longest = uniform(wave_max(mx));
      // stream byte counts and offsets: stream q * 64 + lane follows the
      // streams before it
      uint32_t tot = 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        sbq[q] = rec[16 + 128 + q * 64 + lane];
        const uint32_t incl = wave_incl_scan(sbq[q]);
        so[q] = tot + incl - sbq[q];
        tot += uniform(__builtin_amdgcn_readlane(incl, 63));
      }
      bool hufbad = uniform(__ballot(bad) != 0) || kraft != (1u << kHufMaxLen) || longest != k ||
                    tot != sb;
#pragma unroll
      for (int i = 0; i < 4; ++i) sq0[i] = buf16(rs, 1024u * i + 16u * lane);
      if (!hufbad) {
        // canonical codes: per length, consecutive values in symbol order;
        // the left-aligned 11-bit values of length b fill [lb[b], lb[b+1])
        uint32_t first = 0, prev = 0, start = 0;
        uint32_t lb[kHufMaxLen + 1], stb[kHufMaxLen + 1], cnb[kHufMaxLen + 1];
#pragma unroll
        for (uint32_t b = 1; b <= kHufMaxLen; ++b) {
          const unsigned long long m0 = __ballot(ln[0] == b), m1 = __ballot(ln[1] == b);
          const unsigned long long m2 = __ballot(ln[2] == b), m3 = __ballot(ln[3] == b);
          const uint32_t half = (uint32_t)(__popcll(m0) + __popcll(m1));
          const uint32_t cnt = half + (uint32_t)(__popcll(m2) + __popcll(m3));
          first = (first + prev) << 1;
          const uint32_t rk0 = (uint32_t)(__popcll(m0 & below) + __popcll(m1 & below));
          const uint32_t rk2 = half + (uint32_t)(__popcll(m2 & below) + __popcll(m3 & below));
          if (ln[0] == b) sorted[start + rk0] = (uint8_t)sym[0];
          if (ln[1] == b) sorted[start + rk0 + (ln[0] == b ? 1u : 0u)] = (uint8_t)sym[1];
          if (ln[2] == b) sorted[start + rk2] = (uint8_t)sym[2];
          if (ln[3] == b) sorted[start + rk2 + (ln[2] == b ? 1u : 0u)] = (uint8_t)sym[3];
          lb[b] = first << (kHufMaxLen - b);
          stb[b] = start;
          cnb[b] = cnt;
          start += cnt;
          prev = cnt;
        }
        wave_sync();
        // table entry v (code length | symbol << 8): the code whose bits,
        // first bit as the most significant of 11, begin v (the left-aligned
        // order: length-b codes take 2^(11-b) consecutive entries each, so
        // lanes reading the entries of one short code spread over the LDS
        // banks)
#pragma unroll
        for (uint32_t b = 1; b <= kHufMaxLen; ++b) {
          const uint32_t run = uniform(cnb[b] << (kHufMaxLen - b));
          for (uint32_t t = lane; t < run; t += 64u) {
            const uint32_t v = lb[b] + t;
            tab[v] = (uint16_t)(b | ((uint32_t)sorted[stb[b] + (t >> (kHufMaxLen - b))] << 8));
          }
        }
        wave_sync();
      }
      if (hufbad) bad = true;
    }
    const bool hok = !hufk || uniform(__ballot(bad) == 0);
    // plane ranges cover whole sections with their padding (part of the
    // record), so no piece straddles a range end; padding bytes are checked
    // below
    const Rsrc rb = rsrc(rec + smo, (uint32_t)pad16(n));                       // plane B
    const Rsrc ra = rsrc(rec + 16, mode == 0 ? (uint32_t)pad16(n) : 0u);       // RAW plane A
    uint8_t *dst = staging + (uint64_t)r * kChunk;
    uint32_t cv[4] = {0, 0, 0, 0};
    const bool dec = hufk && hok;
    const bool full = n == kChunk / 2;
    if (!dec) {
      // ---- RAW (plane A stored) or a single exponent / high byte
#pragma unroll 1
      for (uint32_t q = 0; q < 8u; ++q) {
        uint2 pa[8], pb[8];
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const uint32_t w0 = (8u * q + h) * 512u + 8u * lane;
          pb[h] = buf8(rb, w0);
          pa[h] = mode == 0 ? buf8(ra, w0) : make_uint2(base * 0x01010101u, base * 0x01010101u);
        }
#pragma unroll
        for (int h = 0; h < 8; ++h)
          hw_row_out<V3>(pa[h], pb[h], (8u * q + h) * 512u + 8u * lane, n, full, len, dst, cv, gl);
      }
    } else {
      // ---- Huffman streams: group q's bytes [A, A + 4096) staged as 4 KiB
      // (lane l's 16 bytes of each KiB); the next group's loads are in
      // flight while this one decodes and enter the stage after it
      const uint32_t s4 = k <= 8u ? 1u : 0u;  // 4 symbols per refill check, else 2
      const uint32_t *stg = reinterpret_cast<const uint32_t *>(lds_at(sbase));
      uint32_t A = 0;  // group 0 starts the section
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<uint4 *>(lds_at(sbase + 1024u * i + 16u * lane)) = sq0[i];
      wave_sync();
#pragma unroll 1
      for (uint32_t q = 0; q < 8u; ++q) {
        const uint32_t soq = so[q], sbl = sbq[q];
        // in the stage, with room for the reads of a stream that overruns
        // its bytes (64 codes of at most 11 bits and a dword ahead)
        const bool fits =
            uniform(__builtin_amdgcn_readlane(soq + sbl, 63)) - A <= kHwStage - kHwOverrun;
        const bool more = q < 7u;
        uint2 pb[8];
#pragma unroll
        for (int h = 0; h < 8; ++h) pb[h] = buf8(rb, (8u * q + h) * 512u + 8u * lane);
        uint4 sq[4];
        uint32_t an = 0;
        if (more) {
          an = uniform(__builtin_amdgcn_readlane(so[q + 1u], 0)) & ~15u;
#pragma unroll
          for (int i = 0; i < 4; ++i) sq[i] = buf16(rs, an + 1024u * i + 16u * lane);
        }
        // the lane's stream: bits in acc (next bit the most significant, nb
        // of them), whole dwords taken, bit-reversed (a stream's first bit
        // is bit 0 of its first byte), while fewer than 32 bits are held;
        // bytes after the stream's end may enter acc but are never decoded
        // from a well-formed stream: the bits used, 8 (pos - pos0) - nb,
        // must fill exactly the stream's bytes
        uint64_t acc;
        int32_t nb;
        uint32_t pos = soq - A;
        const uint32_t pos0 = pos;
        if (fits && full) {
          // one block without branches per group: each row's symbols, its
          // words, CRC steps and store, so that the table lookups' latency is
          // filled with the rows around them.  The stage is read at the LDS
          // address `ra` of the next whole dword (inside the stage: `fits`).
          const uint32_t tb = tbase;
          uint32_t ra = sbase + (pos & ~3u);
          acc = (uint64_t)__builtin_bitreverse32(lds_u32(ra) >> (8u * (pos & 3u))) << 32;
          nb = (int32_t)(32u - 8u * (pos & 3u));
          ra += 4u;
          uint32_t nxt = lds_u32(ra);
          // nb is kept in the low byte of nbx, from which whole entries
          // (length | symbol << 8) are subtracted; the next dword enters below
          // the nb bits held when fewer than 32 are
          int32_t nbx = nb;
          auto refill = [&]() {
            const int32_t nbv = nbx & 255;
            nbx = nbv;
            if (nbv < 32) {
              const uint32_t x = __builtin_bitreverse32(nxt);
              acc |= ((uint64_t)(x >> nbv) << 32) | __builtin_amdgcn_alignbit(x, 0u, (uint32_t)nbv);
              nbx += 32;
              ra += 4u;
              nxt = lds_u32(ra);
            }
          };
          // one code: its entry, the length in the low bits (a 64-bit shift
          // takes the low six bits of its count)
          auto symbol = [&]() -> uint32_t {
            const uint32_t ent = *reinterpret_cast<const uint16_t *>(
                lds_at(tb + 2u * ((uint32_t)(acc >> 32) >> (32 - kHufMaxLen))));
            acc <<= (ent & 63u);
            nbx -= (int32_t)ent;
            return ent;
          };
          // symbols (byte 1 of four entries) into one dword
          auto pack4 = [](uint32_t e0, uint32_t e1, uint32_t e2, uint32_t e3) -> uint32_t {
            return __builtin_amdgcn_perm(e1, e0, 0x0C0C0501u) |
                   (__builtin_amdgcn_perm(e3, e2, 0x0C0C0501u) << 16);
          };
          auto row = [&](int h, const uint32_t (&a8)[2]) {
            uint32_t out[4];
            words_from_planes<V3>(make_uint2(a8[0], a8[1]), pb[h], out);
#pragma unroll
            for (int c = 0; c < 4; ++c) cv[c] = g_step(cv[c], out[c], gl);
            *reinterpret_cast<uint4 *>(dst + 2u * ((8u * q + h) * 512u + 8u * lane)) =
                make_uint4(out[0], out[1], out[2], out[3]);
          };
          if (s4) {
#pragma unroll
            for (int h = 0; h < 8; ++h) {
              uint32_t a8[2];
#pragma unroll
              for (int j = 0; j < 2; ++j) {
                refill();
                const uint32_t x0 = symbol(), x1 = symbol(), x2 = symbol(), x3 = symbol();
                a8[j] = pack4(x0, x1, x2, x3);
              }
              row(h, a8);
            }
          } else {
#pragma unroll
            for (int h = 0; h < 8; ++h) {
              uint32_t a8[2];
#pragma unroll
              for (int j = 0; j < 2; ++j) {
                refill();
                const uint32_t x0 = symbol(), x1 = symbol();
                refill();
                const uint32_t x2 = symbol(), x3 = symbol();
                a8[j] = pack4(x0, x1, x2, x3);
              }
              row(h, a8);
            }
          }
          pos = ra - sbase;
          nb = nbx & 255;
        } else {
          // per symbol: words past the chunk's end have none; bytes from the
          // stage, or from the record where the group overflows it
          auto rd = [&](uint32_t p) -> uint32_t {
            return fits ? stg[min(p, kHwStage - 4u) >> 2] : buf4(rs, A + (p & ~3u));
          };
          acc = (uint64_t)__builtin_bitreverse32(rd(pos) >> (8u * (pos & 3u))) << 32;
          nb = (int32_t)(32u - 8u * (pos & 3u));
          pos = (pos & ~3u) + 4u;
#pragma unroll
          for (int h = 0; h < 8; ++h) {
            const uint32_t w0 = (8u * q + h) * 512u + 8u * lane;
            uint32_t a8[2] = {0, 0};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              if (w0 + j < n) {
                if (nb < 32) {
                  acc |= (uint64_t)__builtin_bitreverse32(rd(pos)) << (32 - nb);
                  nb += 32;
                  pos += 4u;
                }
                const uint32_t ent = tab[(uint32_t)(acc >> (64 - kHufMaxLen))];
                const uint32_t ln = ent & 15u;
                acc <<= ln;
                nb -= (int32_t)ln;
                a8[j >> 2] |= (ent >> 8) << (8 * (j & 3));
              }
            }
            hw_row_out<V3>(make_uint2(a8[0], a8[1]), pb[h], w0, n, full, len, dst, cv, gl);
          }
        }
        // exactly the stream's bytes, the last one's unused bits zero
        const uint32_t used = 8u * (pos - pos0) - (uint32_t)nb;
        if ((used + 7u) / 8u != sbl) bad = true;
        if ((used & 7u) && (uint32_t)(acc >> (56u + (used & 7u)))) bad = true;
        if (more) {  // the next group enters the stage once this one is read
          wave_sync();
#pragma unroll
          for (int i = 0; i < 4; ++i)
            *reinterpret_cast<uint4 *>(lds_at(sbase + 1024u * i + 16u * lane)) = sq[i];
          wave_sync();
          A = an;
        }
      }
    }
    // ---- zero padding after each section
    if (lane < 16u && n + lane < pad16(n) && rec[smo + n + lane]) bad = true;
    if (mode == 0 && lane >= 16u && lane < 32u && n + lane - 16u < pad16(n) &&
        rec[16 + n + lane - 16u])
      bad = true;
    if (hufk && lane >= 32u && lane < 48u && sb + lane - 32u < pad16(sb) &&
        rec[kHufHead + sb + lane - 32u])
      bad = true;
    // ---- the record's CRC against its receipt
    const uint32_t crc = finish_crc(lane_fold(lane_merge(cv[0], cv[1], cv[2], cv[3])), len, g, T);
    const uint32_t stf = __ballot(bad) ? 4u : (crc != ew[1] ? 8u : 0u);
    if (lane == 0) {
      if (rec_status) rec_status[r] = stf;
      if (stf) atomicOr(&ctl->rec_bits, stf);
    }
  }
}

int set_kernel_attributes() {
  const void *kern[8] = {reinterpret_cast<const void *>(&k_checksum),
                         reinterpret_cast<const void *>(&k_encode<false>),
                         reinterpret_cast<const void *>(&k_encode<true>),
                         reinterpret_cast<const void *>(&k_decode),
                         reinterpret_cast<const void *>(&k_huf_encode<false>),
                         reinterpret_cast<const void *>(&k_huf_encode<true>),
                         reinterpret_cast<const void *>(&k_huf_decode_w<false>),
                         reinterpret_cast<const void *>(&k_huf_decode_w<true>)};
  const uint32_t bytes[8] = {kLdsBase,      kLdsEncode,     kLdsEncode,     kLdsDecode,
                             kLdsHufEncode, kLdsHufEncode, kLdsHufDecodeW, kLdsHufDecodeW};
  for (int i = 0; i < 8; ++i) {
    hipError_t e = hipFuncSetAttribute(kern[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)bytes[i]);
    if (e != hipSuccess) return (int)e;
    hipFuncAttributes fa;
    e = hipFuncGetAttributes(&fa, kern[i]);
    if (e != hipSuccess) return (int)e;
    if (fa.sharedSizeBytes != 0) return (int)hipErrorInvalidConfiguration;
  }
  return 0;
}

// Built-in workspace of wm_encode_step_static, for callers that cannot
// allocate: the workspace layout of 65,536 chunks (a 4 GiB state in 64 KiB
// chunks).  Each device holds its own copy at its own address, shared by
// every call on that device.  Host code must never pass `scratch` itself to
// a kernel (on the host it is only a stand-in for the symbol): launches take
// the device address that scratch_address returns.
constexpr uint64_t kScratchBytes = 256 + 32ull * 65536;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

int scratch_address(void **ptr, uint64_t *bytes) {
  *bytes = kScratchBytes;
  return (int)hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch));
}

static int launch_combine(const CombineJobs &jobs, int n_jobs, void *stream) {
  hipLaunchKernelGGL(k_combine, dim3(n_jobs), dim3(1024), 0, S(stream), jobs);
  return (int)hipGetLastError();
}

__global__ void k_zero_u32(uint32_t *__restrict__ p, uint32_t n) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    p[i] = 0;
}

// The combine job of the global CRC from per-chunk CRCs (the caller's
// chunks) or per-unit CRCs.
static CombineJob global_job(const ChunkGeom &g, const uint32_t *vals, bool units, uint32_t *out) {
  if (units || !g.tile_log2)
    return CombineJob{vals, nullptr, g.n_chunks, 16u, g.tail_len, g.crc_kind, out};
  const uint64_t last = g.hdr_n ? g.nbytes - ((uint64_t)(g.hdr_n - 1) << (16 + g.tile_log2)) : 0;
  return CombineJob{vals, nullptr, g.hdr_n, 16u + g.tile_log2, (uint32_t)last, g.crc_kind, out};
}

int launch_checksum(const void *data, const ChunkGeom &g, uint32_t *crc_out,
                    uint32_t *global_crc, int n_cu, void *stream, bool units) {
  const bool per_chunk = !units && g.tile_log2;
  if (per_chunk && g.hdr_n) {
    hipLaunchKernelGGL(k_zero_u32, dim3(min((g.hdr_n + 255u) / 256u, 64u)), dim3(256), 0,
                       S(stream), crc_out, g.hdr_n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  if (g.n_chunks) {
    uint32_t grid = min((uint32_t)n_cu, g.n_chunks);
    hipLaunchKernelGGL(k_checksum, dim3(grid), dim3(kThreads + 64), kLdsBase, S(stream),
                       static_cast<const uint8_t *>(data), g, crc_out, per_chunk ? 1u : 0u);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  if (global_crc) {
    CombineJobs jobs = {};
    jobs.job[0] = global_job(g, crc_out, units, global_crc);
    return launch_combine(jobs, 1, stream);
  }
  return 0;
}

// A caller's list of chunks above 64 KiB as the list of their tiles (each
// chunk's tiles in order; the state's last chunk may have fewer).  A list
// that is longer than the chunk count, not strictly ascending or out of
// range becomes a tile list longer than the tile count, which the encoder
// rejects (an empty payload).  One workgroup.
__global__ __launch_bounds__(1024) void k_expand_list(const uint32_t *__restrict__ idx,
                                                      const uint32_t *__restrict__ n_idx,
                                                      ChunkGeom g, uint32_t *__restrict__ out,
                                                      uint32_t *__restrict__ n_out) {
  const uint32_t n = *n_idx, per = 1u << g.tile_log2;
  bool bad = n > g.hdr_n;
  const uint32_t m = bad ? 0u : n;
  for (uint32_t r = threadIdx.x; r < m; r += blockDim.x) {
    const uint32_t c = idx[r];
    bad = bad || c >= g.hdr_n || (r > 0 && idx[r - 1] >= c);
    // (a valid list writes slots below its tile count, hence below n_chunks)
    if (c < g.hdr_n)
      for (uint32_t j = 0; j < per; ++j)
        if ((c << g.tile_log2) + j < g.n_chunks && r * per + j < g.n_chunks)
          out[r * per + j] = (c << g.tile_log2) + j;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) {
    uint32_t tiles = m * per;
    // only the last entry can be the state's last chunk, with fewer tiles
    if (m && idx[m - 1] + 1u == g.hdr_n) tiles -= (g.hdr_n << g.tile_log2) - g.n_chunks;
    *n_out = bad ? g.n_chunks + 1u : tiles;
  }
}

int launch_expand_list(const uint32_t *idx, const uint32_t *n_idx, const ChunkGeom &g,
                       uint32_t *out, uint32_t *n_out, void *stream) {
  hipLaunchKernelGGL(k_expand_list, dim3(1), dim3(1024), 0, S(stream), idx, n_idx, g, out, n_out);
  return (int)hipGetLastError();
}

// Chunk CRCs from their tiles' CRCs, CRC(A|B) = F^|B|(CRC(A)) ^ CRC(B) tile by
// tile; one thread per chunk.
__global__ void k_fold_tiles(const uint32_t *__restrict__ tile_crc, ChunkGeom g,
                             uint32_t *__restrict__ out) {
  const CrcTables &T = g_tables[g.crc_kind];
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < g.hdr_n;
       i += gridDim.x * blockDim.x) {
    const uint32_t t0 = i << g.tile_log2, t1 = min((i + 1) << g.tile_log2, g.n_chunks);
    uint32_t acc = tile_crc[t0];
    for (uint32_t t = t0 + 1; t < t1; ++t)
      acc = shift_bytes(T, t + 1 == g.n_chunks ? g.tail_len : kChunk, acc) ^ tile_crc[t];
    out[i] = acc;
  }
}

int launch_fold_tiles(const uint32_t *tile_crc, const ChunkGeom &g, uint32_t *out, void *stream) {
  if (!g.hdr_n) return 0;
  hipLaunchKernelGGL(k_fold_tiles, dim3(min((g.hdr_n + 63u) / 64u, 1024u)), dim3(64), 0,
                     S(stream), tile_crc, g, out);
  return (int)hipGetLastError();
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
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, S(stream), flags, g.hdr_n, g.tile_log2,
                     g.n_chunks, dirty_idx, n_dirty);
  return (int)hipGetLastError();
}

int launch_encode(int mode, const void *cur, const void *prev, const ChunkGeom &g,
                  const uint32_t *idx, const uint32_t *n_idx, const uint32_t *crc_in,
                  uint32_t *crc_out, uint32_t *global_crc, uint32_t *dirty_idx,
                  uint32_t *n_dirty, void *payload, uint64_t *payload_bytes, void *ws,
                  const WsLayout &L, int n_cu, void *stream, const uint32_t *global_from) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  hipLaunchKernelGGL(k_encode_prepare, dim3(64), dim3(256), 0, S(stream), wsb, L, g.n_chunks,
                     mode == kModeList ? n_idx : nullptr);
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
  a.plans = nullptr;
  if (g.n_chunks) {
    uint32_t grid = min((uint32_t)n_cu, g.n_chunks);
    if (mode == kModeStep && prev != nullptr)
      hipLaunchKernelGGL(k_encode<true>, dim3(grid), dim3(kEncThreads), kLdsEncode, S(stream), a, g);
    else
      hipLaunchKernelGGL(k_encode<false>, dim3(grid), dim3(kEncThreads), kLdsEncode, S(stream), a, g);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  // global CRC over every chunk, table CRC over the staged entries
  uint32_t *ctl32 = reinterpret_cast<uint32_t *>(wsb + L.ctl);
  uint32_t *crcs = ctl32 + 60;  // two spare words of the control block
  const uint32_t *all_crc = crc_in ? crc_in : crc_out;
  CombineJobs jobs = {};
  jobs.job[0] = global_from ? global_job(g, global_from, false, crcs)
                            : global_job(g, all_crc, true, crcs);
  jobs.job[1] = CombineJob{reinterpret_cast<const uint32_t *>(wsb + L.entry_crc),
                           &reinterpret_cast<WsCtl *>(wsb + L.ctl)->n_rec, 0u, 4u, 16u,
                           g.crc_kind, crcs + 1};
  int rc = launch_combine(jobs, 2, stream);
  if (rc) return rc;
  uint32_t full = mode == kModeAll || (mode == kModeStep && prev == nullptr) ? 1u : 0u;
  hipLaunchKernelGGL(k_encode_finish, dim3(64), dim3(256), 0, S(stream),
                     static_cast<uint8_t *>(payload), static_cast<const uint8_t *>(ws), L, g,
                     full, crcs, payload_bytes, n_dirty, global_crc);
  return (int)hipGetLastError();
}

int launch_decode_begin(const void *payload, uint64_t payload_cap, const ChunkGeom &g,
                        uint64_t staging_cap, void *ws, const WsLayout &L, void *stream) {
  hipLaunchKernelGGL(k_decode_prepare, dim3(1), dim3(64), 0, S(stream),
                     static_cast<const uint8_t *>(payload), payload_cap, g, staging_cap,
                     static_cast<uint8_t *>(ws), L);
  return (int)hipGetLastError();
}

int launch_decode_records(const void *payload, const ChunkGeom &g, void *staging,
                          uint32_t *rec_status, void *ws, const WsLayout &L, int n_cu,
                          uint32_t r0, uint32_t r1, void *stream) {
  if (r1 <= r0 || !g.n_chunks) return 0;
  const uint32_t grid_d = min((uint32_t)n_cu, min(r1 - r0, g.n_chunks));
  hipLaunchKernelGGL(k_decode, dim3(grid_d), dim3(kDecThreads), kLdsDecode, S(stream),
                     static_cast<const uint8_t *>(payload), g, static_cast<uint8_t *>(staging),
                     rec_status, static_cast<uint8_t *>(ws), L, r0, r1);
  return (int)hipGetLastError();
}

int launch_decode(const void *payload, uint64_t payload_cap, const ChunkGeom &g, void *staging,
                  uint64_t staging_cap, uint32_t *verdict, uint32_t *rec_status, void *ws,
                  const WsLayout &L, int n_cu, void *stream) {
  int rc = launch_decode_begin(payload, payload_cap, g, staging_cap, ws, L, stream);
  if (rc) return rc;
  rc = launch_decode_records(payload, g, staging, rec_status, ws, L, n_cu, 0u, g.n_chunks, stream);
  if (rc) return rc;
  return launch_decode_end(g, verdict, ws, L, stream);
}

int launch_decode_end(const ChunkGeom &g, uint32_t *verdict, void *ws, const WsLayout &L,
                      void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  WsCtl *ctl = reinterpret_cast<WsCtl *>(wsb + L.ctl);
  uint32_t *computed = reinterpret_cast<uint32_t *>(wsb + L.ctl) + 60;
  CombineJobs jobs = {};
  jobs.job[0] = CombineJob{reinterpret_cast<const uint32_t *>(wsb + L.entry_crc), &ctl->n_rec,
                           0u, 4u, 16u, g.crc_kind, computed, ctl, verdict};
  return launch_combine(jobs, 1, stream);
}

// ------------------------------------------------------------- manifest --
// Flatten (gather the leaves into the flat state) and rehydrate (scatter it
// back).  Each workgroup takes 64 KiB windows of the flat buffer, so the
// work is balanced whatever the leaf sizes; a window finds its first leaf by
// binary search over the leaf offsets (uniform, scalar loads) and copies the
// pieces of the leaves it overlaps.  Leaf i occupies flat[off_i, off_i +
// bytes_i), off_i a multiple of 16; on flatten the bytes up to the next leaf
// are written as zeros.
template <bool GATHER>
__global__ __launch_bounds__(kCopyThreads) void k_manifest(uint8_t *__restrict__ flat, uint64_t flat_bytes,
                                                  const ManifestLeaf *__restrict__ leaves,
                                                  uint32_t n_leaves) {
  typedef const __attribute__((address_space(4))) ManifestLeaf cleaf;
  const cleaf *L = (cleaf *)(uintptr_t)leaves;
  const uint64_t n_win = (flat_bytes + kChunk - 1) / kChunk;
  for (uint64_t w = blockIdx.x; w < n_win; w += gridDim.x) {
    const uint64_t w0 = w * kChunk, w1 = min(w0 + kChunk, flat_bytes);
    // first leaf whose padded extent reaches past w0: the last with off <= w0
    uint32_t lo = 0, hi = n_leaves;
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (L[mid].off <= w0) lo = mid; else hi = mid;
    }
    for (uint32_t i = lo; i < n_leaves; ++i) {
      const uint64_t off = L[i].off;
      if (off >= w1) break;
      const uint64_t bytes = L[i].bytes;
      const uint64_t end = i + 1 < n_leaves ? L[i + 1].off : flat_bytes;  // padded end
      const uint64_t s0 = max(off, w0), s1 = min(end, w1);
      if (s0 >= s1) continue;
      uint8_t *leaf = reinterpret_cast<uint8_t *>(L[i].ptr);
      const uint64_t data_end = off + bytes;
      if (s0 == w0 && s1 == w0 + kChunk && data_end >= s1) {
        // the whole window inside one leaf's data: the thread's eight
        // 16-byte pieces all in flight
        const uint8_t *src = GATHER ? leaf + (w0 - off) : flat + w0;
        uint8_t *dst = GATHER ? flat + w0 : leaf + (w0 - off);
        v4u v[kCopyPieces];
#pragma unroll
        for (uint32_t j = 0; j < kCopyPieces; ++j)
          v[j] = __builtin_nontemporal_load(
              reinterpret_cast<const v4u *>(src + threadIdx.x * 16u + j * 16u * kCopyThreads));
#pragma unroll
        for (uint32_t j = 0; j < kCopyPieces; ++j)
          __builtin_nontemporal_store(
              v[j], reinterpret_cast<v4u *>(dst + threadIdx.x * 16u + j * 16u * kCopyThreads));
        continue;
      }
      // general piece [s0, s1): 16-byte units; the unit holding the leaf's
      // last bytes is copied bytewise (flatten zero-fills the rest of it)
      for (uint64_t a = s0 + threadIdx.x * 16u; a < s1; a += kCopyThreads * 16u) {
        if (a + 16u <= data_end) {
          if (GATHER)
            *reinterpret_cast<uint4 *>(flat + a) = *reinterpret_cast<const uint4 *>(leaf + (a - off));
          else
            *reinterpret_cast<uint4 *>(leaf + (a - off)) = *reinterpret_cast<const uint4 *>(flat + a);
        } else if (GATHER) {
          uint32_t t[4] = {0, 0, 0, 0};
          for (uint32_t b = 0; a + b < data_end && b < 16u; ++b)
            t[b >> 2] |= (uint32_t)leaf[a - off + b] << (8 * (b & 3));
          *reinterpret_cast<uint4 *>(flat + a) = make_uint4(t[0], t[1], t[2], t[3]);
        } else {
          for (uint32_t b = 0; a + b < data_end && b < 16u; ++b) leaf[a - off + b] = flat[a + b];
        }
      }
    }
  }
}

int launch_manifest(bool gather, void *flat, uint64_t flat_bytes, const ManifestLeaf *leaves,
                    uint32_t n_leaves, int n_cu, void *stream) {
  const uint64_t n_win = (flat_bytes + kChunk - 1) / kChunk;
  if (!n_win) return 0;
  const uint32_t grid = (uint32_t)min((uint64_t)n_cu * 2u, n_win);
  if (gather)
    hipLaunchKernelGGL(k_manifest<true>, dim3(grid), dim3(kCopyThreads), 0, S(stream),
                       static_cast<uint8_t *>(flat), flat_bytes, leaves, n_leaves);
  else
    hipLaunchKernelGGL(k_manifest<false>, dim3(grid), dim3(kCopyThreads), 0, S(stream),
                       static_cast<uint8_t *>(flat), flat_bytes, leaves, n_leaves);
  return (int)hipGetLastError();
}

int launch_commit(void *live, const ChunkGeom &g, const void *staging, const void *payload,
                  const uint32_t *verdict, int n_cu, void *stream) {
  if (!g.n_chunks) return 0;
  uint32_t grid = min((uint32_t)n_cu * 2u, g.n_chunks);
  hipLaunchKernelGGL(k_commit, dim3(grid), dim3(kCopyThreads), 0, S(stream),
                     static_cast<uint8_t *>(live), g, static_cast<const uint8_t *>(staging),
                     static_cast<const uint8_t *>(payload), verdict);
  return (int)hipGetLastError();
}

// A full ship's dirty list: every chunk, in order.
__global__ void k_fill_all(uint32_t *__restrict__ idx, uint32_t *__restrict__ n_out, uint32_t n) {
  if (idx)
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
      idx[i] = i;
  if (n_out && blockIdx.x == 0 && threadIdx.x == 0) *n_out = n;
}

int launch_fill_all(uint32_t *idx, uint32_t *n_out, uint32_t n, void *stream) {
  hipLaunchKernelGGL(k_fill_all, dim3(64), dim3(256), 0, S(stream), idx, n_out, n);
  return (int)hipGetLastError();
}

// ------------------------------------------------------------- reverify --
// Re-verifying install (Table 1: commit re-verifies, then swaps).  live_crc
// holds the CRC of every chunk of live, staged_crc that of every staged
// record.  One workgroup walks the payload's table: a staged record whose
// CRC differs from its receipt sets the flag, and the record's receipt
// replaces the CRC of the chunk it will overwrite, so that live_crc becomes
// the chunk CRCs of the state the install would produce.
__global__ __launch_bounds__(1024) void k_reverify_records(const uint8_t *__restrict__ payload,
                                                           uint32_t *__restrict__ live_crc,
                                                           const uint32_t *__restrict__ staged_crc,
                                                           uint32_t *__restrict__ flag,
                                                           uint32_t n_chunks) {
  __shared__ uint32_t any;
  if (threadIdx.x == 0) any = 0;
  __syncthreads();
  const uint32_t n_rec = ld_u32(payload + 24);
  const uint64_t table_off = ld_u64(payload + 32) - 16ull * n_rec;
  uint32_t bad = 0;
  for (uint32_t r = threadIdx.x; r < n_rec; r += blockDim.x) {
    const uint2 e = *reinterpret_cast<const uint2 *>(payload + table_off + 16ull * r);
    bad |= staged_crc[r] != e.y || e.x >= n_chunks ? 1u : 0u;
    if (e.x < n_chunks) live_crc[e.x] = e.y;
  }
  if (bad) atomicOr(&any, 1u);
  __syncthreads();
  if (threadIdx.x == 0) *flag = any;
}

// The resulting state's global CRC (combined from live_crc) against the
// header's: any disagreement, or a flagged record, adds WM_V_REVERIFY to the
// verdict, so that the install that follows copies nothing.
__global__ void k_reverify_end(const uint8_t *__restrict__ payload, const uint32_t *flag,
                               const uint32_t *global, uint32_t *verdict) {
  if (threadIdx.x == 0 && (*flag != 0u || *global != ld_u32(payload + 40))) *verdict |= 32u;
}

int launch_reverify(const void *live, const ChunkGeom &g, const void *staging,
                    const ChunkGeom &gs, const void *payload, uint32_t *verdict, void *ws,
                    const WsLayout &L, int n_cu, void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  uint32_t *live_crc = reinterpret_cast<uint32_t *>(wsb + L.flags);
  uint32_t *staged_crc = reinterpret_cast<uint32_t *>(wsb + L.entry_crc);
  uint32_t *words = reinterpret_cast<uint32_t *>(wsb + L.ctl);  // [0] flag, [1] global
  int rc = launch_checksum(live, g, live_crc, nullptr, n_cu, stream, true);
  if (rc) return rc;
  rc = launch_checksum(staging, gs, staged_crc, nullptr, n_cu, stream, true);
  if (rc) return rc;
  hipLaunchKernelGGL(k_reverify_records, dim3(1), dim3(1024), 0, S(stream),
                     static_cast<const uint8_t *>(payload), live_crc,
                     static_cast<const uint32_t *>(staged_crc), words, g.n_chunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  CombineJobs jobs = {};
  jobs.job[0] = CombineJob{live_crc, nullptr, g.n_chunks, 16u, g.tail_len, g.crc_kind, words + 1};
  rc = launch_combine(jobs, 1, stream);
  if (rc) return rc;
  hipLaunchKernelGGL(k_reverify_end, dim3(1), dim3(64), 0, S(stream),
                     static_cast<const uint8_t *>(payload), words, words + 1, verdict);
  return (int)hipGetLastError();
}

int launch_encode_v2(const void *state, const ChunkGeom &g, const uint32_t *idx,
                     const uint32_t *n_idx, const uint32_t *crc_in, uint32_t *crc_scratch,
                     uint32_t *global_crc, void *payload, uint64_t *payload_bytes, void *ws,
                     const WsLayout &L, int n_cu, void *stream) {
  uint8_t *wsb = static_cast<uint8_t *>(ws);
  WsCtl *ctl = reinterpret_cast<WsCtl *>(wsb + L.ctl);
  hipLaunchKernelGGL(k_encode_prepare, dim3(64), dim3(256), 0, S(stream), wsb, L, g.n_chunks,
                     idx ? n_idx : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  // receipts: given, computed in the pass (every chunk is encoded), or for a
  // list checksummed first (the global CRC covers every chunk)
  const uint32_t *crcs = crc_in;
  uint32_t *crc_out = nullptr;
  if (!crcs && idx) {
    const int rc = launch_checksum(state, g, crc_scratch, nullptr, n_cu, stream, true);
    if (rc) return rc;
    crcs = crc_scratch;
  } else if (!crcs) {
    crc_out = crc_scratch;
  }
  EncArgs a;
  a.cur = static_cast<const uint8_t *>(state);
  a.prev = nullptr;
  a.idx = idx;
  a.n_idx = n_idx;
  a.crc_in = crcs;
  a.crc_out = crc_out;
  a.dirty_idx = nullptr;
  a.payload = static_cast<uint8_t *>(payload);
  a.ws = wsb;
  a.L = L;
  a.mode = idx ? kModeList : kModeAll;
  uint8_t *plans = wsb + plans_offset(L);
  a.plans = plans;
  if (g.n_chunks) {
    const uint32_t lgrid = min((uint32_t)n_cu * 2u, (g.n_chunks + kHufWaves - 1) / kHufWaves);
    if (g.codec == 3)
      hipLaunchKernelGGL(k_huf_lengths<true>, dim3(lgrid), dim3(64 * kHufWaves), 0, S(stream),
                         static_cast<const uint8_t *>(state), g, idx, n_idx, plans);
    else
      hipLaunchKernelGGL(k_huf_lengths<false>, dim3(lgrid), dim3(64 * kHufWaves), 0, S(stream),
                         static_cast<const uint8_t *>(state), g, idx, n_idx, plans);
    const uint32_t grid = min((uint32_t)n_cu, g.n_chunks);
    if (g.codec == 3)
      hipLaunchKernelGGL(k_huf_encode<true>, dim3(grid), dim3(kEncThreads), kLdsHufEncode,
                         S(stream), a, g);
    else
      hipLaunchKernelGGL(k_huf_encode<false>, dim3(grid), dim3(kEncThreads), kLdsHufEncode,
                         S(stream), a, g);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  uint32_t *sums = reinterpret_cast<uint32_t *>(wsb + L.ctl) + 60;  // global and table CRC
  CombineJobs jobs = {};
  jobs.job[0] = CombineJob{crcs ? crcs : crc_out, nullptr, g.n_chunks, 16u, g.tail_len,
                           g.crc_kind, sums};
  jobs.job[1] = CombineJob{reinterpret_cast<const uint32_t *>(wsb + L.entry_crc), &ctl->n_rec,
                           0u, 4u, 16u, g.crc_kind, sums + 1};
  const int rc = launch_combine(jobs, 2, stream);
  if (rc) return rc;
  hipLaunchKernelGGL(k_encode_finish, dim3(64), dim3(256), 0, S(stream),
                     static_cast<uint8_t *>(payload), static_cast<const uint8_t *>(ws), L, g,
                     idx ? 0u : 1u, sums, payload_bytes, nullptr, global_crc);
  return (int)hipGetLastError();
}

int launch_decode_records_v2(const void *payload, const ChunkGeom &g, void *staging,
                             uint32_t *rec_status, void *ws, const WsLayout &L, int n_cu,
                             uint32_t r0, uint32_t r1, void *stream) {
  if (r1 <= r0 || !g.n_chunks) return 0;
  const uint32_t recs = min(r1 - r0, g.n_chunks);
  const uint32_t grid = min((uint32_t)n_cu, (recs + kHwWaves - 1u) / kHwWaves);
  if (g.codec == 3)
    hipLaunchKernelGGL(k_huf_decode_w<true>, dim3(grid), dim3(64 * kHwWaves), kLdsHufDecodeW,
                       S(stream), static_cast<const uint8_t *>(payload), g,
                       static_cast<uint8_t *>(staging), rec_status, static_cast<uint8_t *>(ws), L, r0,
                       r1);
  else
    hipLaunchKernelGGL(k_huf_decode_w<false>, dim3(grid), dim3(64 * kHwWaves), kLdsHufDecodeW,
                       S(stream), static_cast<const uint8_t *>(payload), g,
                       static_cast<uint8_t *>(staging), rec_status, static_cast<uint8_t *>(ws), L, r0,
                       r1);
  return (int)hipGetLastError();
}

int launch_decode_v2(const void *payload, uint64_t payload_cap, const ChunkGeom &g,
                     void *staging, uint64_t staging_cap, uint32_t *verdict,
                     uint32_t *rec_status, void *ws, const WsLayout &L, int n_cu,
                     void *stream) {
  int rc = launch_decode_begin(payload, payload_cap, g, staging_cap, ws, L, stream);
  if (rc) return rc;
  rc = launch_decode_records_v2(payload, g, staging, rec_status, ws, L, n_cu, 0u, g.n_chunks,
                                stream);
  if (rc) return rc;
  return launch_decode_end(g, verdict, ws, L, stream);
}

}  // namespace wm
