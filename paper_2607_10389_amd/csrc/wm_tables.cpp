// wm_tables.cpp -- host construction of the GF(2) shift tables.
//
// Everything here is derived from the polynomial: the one-bit register step
// Z (and its inverse), composed into byte shifts F^m by square-and-multiply
// over 32x32 GF(2) matrices stored as columns.
#include <cstring>

#include "wm_internal.h"

namespace wm {

namespace {

struct Mat {
  uint32_t c[32];
};

uint32_t apply(const Mat &m, uint32_t v) {
  uint32_t r = 0;
  for (int i = 0; i < 32; ++i)
    if ((v >> i) & 1u) r ^= m.c[i];
  return r;
}

// a after b
Mat compose(const Mat &a, const Mat &b) {
  Mat r;
  for (int i = 0; i < 32; ++i) r.c[i] = apply(a, b.c[i]);
  return r;
}

Mat identity() {
  Mat r;
  for (int i = 0; i < 32; ++i) r.c[i] = 1u << i;
  return r;
}

// One zero bit: Z(c) = (c >> 1) ^ (P & -(c & 1)).
Mat zero_bit(uint32_t poly) {
  Mat r;
  for (int i = 0; i < 32; ++i) {
    uint32_t c = 1u << i;
    r.c[i] = (c >> 1) ^ (poly & (0u - (c & 1u)));
  }
  return r;
}

// Inverse of Z.  Bit 31 of Z(c) equals bit 0 of c (P has bit 31 set and
// c >> 1 has it clear), so c = ((z ^ (P if bit) ) << 1) | bit.
Mat zero_bit_inverse(uint32_t poly) {
  Mat r;
  for (int i = 0; i < 32; ++i) {
    uint32_t z = 1u << i;
    uint32_t b0 = z >> 31;
    r.c[i] = ((z ^ (poly & (0u - b0))) << 1) | b0;
  }
  return r;
}

Mat power(Mat base, uint64_t e) {
  Mat r = identity();
  while (e) {
    if (e & 1) r = compose(base, r);
    base = compose(base, base);
    e >>= 1;
  }
  return r;
}

Mat byte_shift(uint32_t poly, int64_t m) {
  if (m >= 0) return power(power(zero_bit(poly), 8), (uint64_t)m);
  return power(power(zero_bit_inverse(poly), 8), (uint64_t)(-m));
}

void byte_tables(const Mat &m, uint32_t out[4][256]) {
  for (int j = 0; j < 4; ++j)
    for (uint32_t b = 0; b < 256; ++b) out[j][b] = apply(m, b << (8 * j));
}

}  // namespace

uint32_t poly_of(uint32_t crc_kind) {
  return crc_kind == 1 ? 0x82F63B78u : 0xEDB88320u;
}

void shift_matrix(uint32_t poly, int64_t m, uint32_t cols[32]) {
  Mat s = byte_shift(poly, m);
  std::memcpy(cols, s.c, sizeof(s.c));
}

uint32_t shift_apply(uint32_t poly, int64_t m, uint32_t v) {
  return apply(byte_shift(poly, m), v);
}

void build_crc_tables(uint32_t poly, CrcTables *t) {
  std::memset(t, 0, sizeof(*t));
  byte_tables(byte_shift(poly, kRow), t->row);
  byte_tables(byte_shift(poly, 4), t->f4);
  byte_tables(byte_shift(poly, 8), t->f8);
  byte_tables(byte_shift(poly, 12), t->f12);
  for (int l = 0; l < 64; ++l) {
    const Mat m = byte_shift(poly, 16 * (63 - l) + 4);
    for (int i = 0; i < 32; ++i) t->lane_mat[i / 4][l][i % 4] = m.c[i];
  }
  byte_tables(byte_shift(poly, kSub), t->wave_step);
  Mat one = byte_shift(poly, 1);
  for (uint32_t b = 0; b < 256; ++b) t->byte1[b] = apply(one, b);
  Mat p = byte_shift(poly, 1);
  for (int i = 0; i < 48; ++i) {
    std::memcpy(t->pow2[i], p.c, sizeof(p.c));
    p = compose(p, p);
  }
  t->k_full = apply(byte_shift(poly, kChunk), 0xFFFFFFFFu) ^ 0xFFFFFFFFu;
}

WsLayout ws_layout(uint32_t n_chunks) {
  WsLayout L;
  uint64_t n = n_chunks ? n_chunks : 1;
  L.ctl = 0;
  L.status = 256;
  L.table = L.status + ((8 * n + 255) & ~255ull);
  L.entry_crc = L.table + ((16 * n + 255) & ~255ull);
  L.flags = L.entry_crc + ((4 * n + 255) & ~255ull);
  L.total = L.flags + ((4 * n + 255) & ~255ull);
  return L;
}

}  // namespace wm
