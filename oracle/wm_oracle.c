/*
 * wm_oracle.c -- plain CPU oracle for the exact-state mover's data path.
 *
 * TEST INFRASTRUCTURE ONLY (see wm_oracle.h).  Slow on purpose: every step is
 * written the way its definition reads.  Threads only split the loop over
 * independent chunks; outputs do not depend on the thread count.
 *
 * Payload format v1 (this project's own definition; the paper names a lossless
 * codec but fixes no byte layout, §6.4 codec paragraph).  All integers are
 * little-endian, all sections are padded with zero bytes to a multiple of 16.
 *
 *   header (64 B)
 *     0 u32 magic 'W','M','V','1'     4 u16 version = 1
 *     6 u8  crc kind                  7 u8  codec = 1
 *     8 u32 chunk_bytes              12 u32 n_chunks = ceil(state_bytes/chunk)
 *    16 u64 state_bytes              24 u32 n_records
 *    28 u32 flags (bit0 FULL)        32 u64 payload_bytes
 *    40 u32 global_crc (CRC of the whole source state)
 *    44 u32 table_crc  (CRC of the 16*n_records table bytes)
 *    48..59 zero                     60 u32 header_crc = CRC(bytes 0..59)
 *   records, contiguous from offset 64, in ascending unit order
 *   table (16 B per record, after the last record, ending at payload_bytes):
 *     u32 unit_idx, u32 src_crc, u64 record_offset
 *   The record unit is the chunk for chunks of at most 64 KiB.  A larger
 *   chunk is shipped as its 64 KiB tiles (unit i = bytes [64Ki*i, 64Ki*(i+1))
 *   of the state), one record and one receipt each, and a table lists every
 *   tile of each chunk it ships; n_records counts units.  This keeps a
 *   record's escape counts within 16 bits and its words within one
 *   decoder's reach whatever the chunk size.
 *   Record:
 *     0 u8 mode (0 RAW, 1 PACK)  1 u8 k  2 u8 base  3 u8 0
 *     4 u32 n_words  8 u32 n_esc  12 u32 rec_crc = CRC(record bytes 0..11)
 *     RAW : exponent plane (n B, e of every word) | sign/mantissa plane (n B)
 *     PACK: codes (ceil(n*k/8) B, LSB-first k-bit codes) | escape index
 *           (ceil(n/512) u16: escaped words before each 512-word block)
 *           | escapes (n_esc B) | sign/mantissa plane (n B); k = 0 has only
 *           the sign/mantissa plane
 *   A bf16 word w splits into sign w>>15, exponent e = (w>>7)&255 and
 *   mantissa w&127; sm = sign<<7 | mantissa.  PACK with k >= 1 codes e as
 *   e - base when 0 <= e - base < 2^k - 1, else as ESC = 2^k - 1 with e
 *   appended to the escapes; PACK with k = 0 means every e equals base.
 *
 * Formats v2 (codec 2, magic 'WMV2') and v3 (codec 3, 'WMV3') share this
 * header, table and tiling, with RAW or Huffman records (below).
 */
#include "wm_oracle.h"

#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ CRC -- */

static uint32_t poly_of(int kind) {
  return kind == ORC_CRC32C ? 0x82F63B78u : 0xEDB88320u;
}

/* The reflected CRC-32 register update, one message bit at a time. */
uint32_t orc_crc_bitwise(int kind, const uint8_t *p, uint64_t n) {
  uint32_t poly = poly_of(kind);
  uint32_t c = 0xFFFFFFFFu;
  for (uint64_t i = 0; i < n; i++) {
    c ^= p[i];
    for (int b = 0; b < 8; b++) c = (c >> 1) ^ (poly & (0u - (c & 1u)));
  }
  return c ^ 0xFFFFFFFFu;
}

static uint32_t byte_table[2][256];
static pthread_once_t table_once = PTHREAD_ONCE_INIT;

/* Entry v is the register after feeding byte v into a zero register through
 * the bitwise step; a byte step is then c = table[(c ^ b) & 255] ^ (c >> 8). */
static void build_tables(void) {
  for (int kind = 0; kind < 2; kind++) {
    uint32_t poly = poly_of(kind);
    for (uint32_t v = 0; v < 256; v++) {
      uint32_t c = v;
      for (int b = 0; b < 8; b++) c = (c >> 1) ^ (poly & (0u - (c & 1u)));
      byte_table[kind][v] = c;
    }
  }
}

uint32_t orc_crc(int kind, const uint8_t *p, uint64_t n) {
  pthread_once(&table_once, build_tables);
  const uint32_t *t = byte_table[kind == ORC_CRC32C ? 1 : 0];
  uint32_t c = 0xFFFFFFFFu;
  for (uint64_t i = 0; i < n; i++) c = t[(c ^ p[i]) & 255u] ^ (c >> 8);
  return c ^ 0xFFFFFFFFu;
}

/* -------------------------------------------------------------- threads -- */

typedef void (*range_fn)(void *ctx, uint64_t lo, uint64_t hi);
typedef struct {
  range_fn fn;
  void *ctx;
  uint64_t lo, hi;
} range_job;

static void *range_thread(void *arg) {
  range_job *j = (range_job *)arg;
  j->fn(j->ctx, j->lo, j->hi);
  return NULL;
}

/* Run fn over [0, n) split into `threads` contiguous ranges. */
static void parallel_for(uint64_t n, int threads, range_fn fn, void *ctx) {
  if (threads < 1) threads = 1;
  if (threads > 256) threads = 256;
  if ((uint64_t)threads > n) threads = n ? (int)n : 1;
  if (threads == 1) {
    fn(ctx, 0, n);
    return;
  }
  pthread_t tid[256];
  range_job job[256];
  for (int t = 0; t < threads; t++) {
    job[t].fn = fn;
    job[t].ctx = ctx;
    job[t].lo = n * (uint64_t)t / (uint64_t)threads;
    job[t].hi = n * (uint64_t)(t + 1) / (uint64_t)threads;
    pthread_create(&tid[t], NULL, range_thread, &job[t]);
  }
  for (int t = 0; t < threads; t++) pthread_join(tid[t], NULL);
}

/* ------------------------------------------------------------- chunking -- */

static uint64_t n_chunks_of(uint64_t nbytes, uint32_t chunk) {
  return (nbytes + chunk - 1) / chunk;
}
static uint32_t chunk_len(uint64_t nbytes, uint32_t chunk, uint64_t c) {
  uint64_t start = c * (uint64_t)chunk;
  uint64_t left = nbytes - start;
  return left < chunk ? (uint32_t)left : chunk;
}
static int chunk_ok(uint32_t chunk) {
  /* a power of two between 4 KiB and 16 MiB */
  return chunk >= 4096u && chunk <= (16u << 20) && (chunk & (chunk - 1)) == 0;
}
static uint64_t pad16(uint64_t x) { return (x + 15u) & ~(uint64_t)15u; }
/* the record unit of a chunk size: the chunk itself up to 64 KiB, else a
 * 64 KiB tile */
#define ORC_TILE 65536u
static uint32_t unit_of(uint32_t chunk) { return chunk < ORC_TILE ? chunk : ORC_TILE; }

/* --------------------------------------------------------- checksumming -- */

typedef struct {
  int kind;
  const uint8_t *data;
  uint64_t nbytes;
  uint32_t chunk;
  uint32_t *crc;
} ck_ctx;

static void ck_range(void *vp, uint64_t lo, uint64_t hi) {
  ck_ctx *x = (ck_ctx *)vp;
  for (uint64_t c = lo; c < hi; c++)
    x->crc[c] = orc_crc(x->kind, x->data + c * (uint64_t)x->chunk,
                        chunk_len(x->nbytes, x->chunk, c));
}

int orc_checksum_chunks(int kind, const uint8_t *data, uint64_t nbytes,
                        uint32_t chunk_bytes, uint32_t *crc_out,
                        uint32_t *global_out, int threads) {
  if (!chunk_ok(chunk_bytes) || (kind != 0 && kind != 1)) return -1;
  ck_ctx x = {kind, data, nbytes, chunk_bytes, crc_out};
  parallel_for(n_chunks_of(nbytes, chunk_bytes), threads, ck_range, &x);
  /* the global CRC is the plain CRC of the whole buffer, read again */
  if (global_out) *global_out = orc_crc(kind, data, nbytes);
  return 0;
}

/* ----------------------------------------------------------------- diff -- */

typedef struct {
  const uint8_t *cur, *prev;
  uint64_t nbytes;
  uint32_t chunk;
  uint8_t *dirty;
} df_ctx;

static void df_range(void *vp, uint64_t lo, uint64_t hi) {
  df_ctx *x = (df_ctx *)vp;
  for (uint64_t c = lo; c < hi; c++) {
    uint64_t off = c * (uint64_t)x->chunk;
    x->dirty[c] = memcmp(x->cur + off, x->prev + off,
                         chunk_len(x->nbytes, x->chunk, c)) != 0;
  }
}

uint32_t orc_diff_dirty(const uint8_t *cur, const uint8_t *prev,
                        uint64_t nbytes, uint32_t chunk_bytes,
                        uint32_t *idx_out, int threads) {
  if (!chunk_ok(chunk_bytes)) return 0;
  uint64_t n = n_chunks_of(nbytes, chunk_bytes);
  uint8_t *dirty = (uint8_t *)calloc(n ? n : 1, 1);
  df_ctx x = {cur, prev, nbytes, chunk_bytes, dirty};
  parallel_for(n, threads, df_range, &x);
  uint32_t m = 0;
  for (uint64_t c = 0; c < n; c++)
    if (dirty[c]) idx_out[m++] = (uint32_t)c;
  free(dirty);
  return m;
}

/* ---------------------------------------------------------------- codec -- */

static uint16_t word_at(const uint8_t *p, uint32_t i) {
  return (uint16_t)(p[2 * i] | (p[2 * i + 1] << 8));
}
static uint32_t exponent_of(uint16_t w) { return (w >> 7) & 255u; }
static uint8_t sm_of(uint16_t w) {
  return (uint8_t)(((w >> 15) << 7) | (w & 127u));
}

static uint64_t raw_size(uint32_t n) { return 16 + 2 * pad16(n); }
static int all_zero(const uint8_t *p, uint64_t n) {
  for (uint64_t i = 0; i < n; i++)
    if (p[i]) return 0;
  return 1;
}
/* escape-index entries: one per block of 512 words (k >= 1 only) */
static uint64_t index_bytes(uint32_t n, uint32_t k) {
  return k ? 2 * (((uint64_t)n + 511) / 512) : 0;
}
static uint64_t pack_size(uint32_t n, uint32_t k, uint32_t n_esc) {
  return 16 + pad16(((uint64_t)n * k + 7) / 8) + pad16(index_bytes(n, k)) +
         pad16(n_esc) + pad16(n);
}

/* Mode choice for one chunk of len bytes (len even).  Candidates, in the
 * order that also breaks ties: RAW, PACK k=0 (only when every exponent is the
 * same), PACK k=1..7 with the base that puts the most words inside the
 * window [base, base + 2^k - 2] (smallest base on ties).  The smallest
 * record wins. */
int orc_plan_chunk(const uint8_t *chunk, uint32_t len, uint32_t *mode,
                   uint32_t *k, uint32_t *base, uint32_t *n_esc,
                   uint64_t *size) {
  uint32_t n = len / 2;
  uint64_t hist[256];
  memset(hist, 0, sizeof(hist));
  for (uint32_t i = 0; i < n; i++) hist[exponent_of(word_at(chunk, i))]++;

  uint32_t distinct = 0, only = 0;
  for (uint32_t e = 0; e < 256; e++)
    if (hist[e]) {
      distinct++;
      only = e;
    }

  uint32_t best_mode = 0, best_k = 0, best_base = 0, best_esc = 0;
  uint64_t best = raw_size(n);

  if (distinct == 1) {
    uint64_t s = pack_size(n, 0, 0);
    if (s < best) {
      best = s;
      best_mode = 1;
      best_k = 0;
      best_base = only;
      best_esc = 0;
    }
  }
  for (uint32_t kk = 1; kk <= 7; kk++) {
    uint32_t window = (1u << kk) - 1u;
    uint64_t top = 0;
    uint32_t top_base = 0;
    for (uint32_t b = 0; b < 256; b++) {
      uint64_t inside = 0;
      for (uint32_t e = b; e < b + window && e < 256; e++) inside += hist[e];
      if (inside > top) {
        top = inside;
        top_base = b;
      }
    }
    uint32_t esc = n - (uint32_t)top;
    uint64_t s = pack_size(n, kk, esc);
    if (s < best) {
      best = s;
      best_mode = 1;
      best_k = kk;
      best_base = top_base;
      best_esc = esc;
    }
  }
  *mode = best_mode;
  *k = best_k;
  *base = best_base;
  *n_esc = best_esc;
  *size = best;
  return 0;
}

static void put_u16(uint8_t *p, uint16_t v) {
  p[0] = (uint8_t)v;
  p[1] = (uint8_t)(v >> 8);
}
static void put_u32(uint8_t *p, uint32_t v) {
  for (int i = 0; i < 4; i++) p[i] = (uint8_t)(v >> (8 * i));
}
static void put_u64(uint8_t *p, uint64_t v) {
  for (int i = 0; i < 8; i++) p[i] = (uint8_t)(v >> (8 * i));
}
static uint32_t get_u32(const uint8_t *p) {
  return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) |
         ((uint32_t)p[3] << 24);
}
static uint64_t get_u64(const uint8_t *p) {
  return (uint64_t)get_u32(p) | ((uint64_t)get_u32(p + 4) << 32);
}

/* Write one record (size bytes, already zeroed by the caller). */
static void write_record(int kind, const uint8_t *chunk, uint32_t len,
                         uint32_t mode, uint32_t k, uint32_t base,
                         uint32_t n_esc, uint8_t *out) {
  uint32_t n = len / 2;
  out[0] = (uint8_t)mode;
  out[1] = (uint8_t)k;
  out[2] = (uint8_t)base;
  out[3] = 0;
  put_u32(out + 4, n);
  put_u32(out + 8, n_esc);
  put_u32(out + 12, orc_crc(kind, out, 12));
  uint8_t *body = out + 16;
  if (mode == 0) {
    for (uint32_t i = 0; i < n; i++) {
      uint16_t w = word_at(chunk, i);
      body[i] = (uint8_t)exponent_of(w);
      body[pad16(n) + i] = sm_of(w);
    }
    return;
  }
  uint8_t *codes = body;
  uint8_t *index = codes + pad16(((uint64_t)n * k + 7) / 8);
  uint8_t *escapes = index + pad16(index_bytes(n, k));
  uint8_t *sm = escapes + pad16(n_esc);
  uint32_t esc_code = (1u << k) - 1u;
  uint32_t esc_written = 0;
  for (uint32_t i = 0; i < n; i++) {
    uint16_t w = word_at(chunk, i);
    uint32_t e = exponent_of(w);
    sm[i] = sm_of(w);
    if (k == 0) continue; /* every exponent equals base */
    if (i % 512 == 0) put_u16(index + 2 * (i / 512), (uint16_t)esc_written);
    uint32_t code;
    if (e >= base && e - base < esc_code) {
      code = e - base;
    } else {
      code = esc_code;
      escapes[esc_written++] = (uint8_t)e;
    }
    /* stream bit i*k + b is bit b of code i; stream bit j lives in bit
     * j % 8 of byte j / 8 */
    for (uint32_t b = 0; b < k; b++) {
      uint64_t j = (uint64_t)i * k + b;
      if ((code >> b) & 1u) codes[j / 8] |= (uint8_t)(1u << (j % 8));
    }
  }
}


static uint32_t decode_record(int kind, const uint8_t *rec, uint64_t L,
                              uint32_t len, uint32_t src_crc, uint8_t *out);

/* ------------------------------------------------------ codec 2 (v2) -- */
/* The paper's codec is an entropy coder over the bf16 words, whose
 * redundancy sits in the exponent plane (§6.4).  Format v2 codes each
 * chunk's exponents with that chunk's own canonical Huffman code (lengths at
 * most ORC_HUF_MAX_LEN) in 512 streams, so that 512 decoders can run side
 * by side; sign/mantissa bytes stay raw.  Records are RAW (as v1) or HUF. */

#define HUF_STREAMS 512u

/* The two byte planes of a word in the Huffman formats: plane A is coded,
 * plane B kept raw.  Codec 2 (v2): A is the exponent, B the sign/mantissa
 * byte.  Codec 3 (v3, the paper's bf16 byte-plane split, §6.4 codec
 * paragraph): A is the high byte (sign and the exponent's upper seven bits),
 * B the low byte (the exponent's lowest bit and the mantissa), which is close
 * to 8 bits of entropy and stays raw. */
static uint32_t plane_a(int codec, uint16_t w) {
  return codec == 3 ? (uint32_t)(w >> 8) : exponent_of(w);
}
static uint8_t plane_b(int codec, uint16_t w) {
  return codec == 3 ? (uint8_t)(w & 255u) : sm_of(w);
}
static uint16_t from_planes(int codec, uint32_t a, uint32_t b) {
  if (codec == 3) return (uint16_t)((a << 8) | b);
  return (uint16_t)(((b >> 7) << 15) | (a << 7) | (b & 127u));
}

/* Word i of stream s (s < 512, i < 64): row 8*(s/64) + i/8 of 512 words,
 * word 8*(s%64) + i%8 of the row. */
static uint32_t stream_word(uint32_t s, uint32_t i) {
  return (8u * (s / 64u) + i / 8u) * 512u + 8u * (s % 64u) + i % 8u;
}

/* Huffman code lengths for the symbols with nonzero count: leaves sorted by
 * (count, symbol); the two lightest nodes are merged repeatedly, a leaf
 * taken before an internal node of equal weight; a symbol's length is its
 * depth.  While the longest exceeds ORC_HUF_MAX_LEN every nonzero count c
 * becomes (c + 1) / 2 and the code is rebuilt.  One symbol: length 0.
 * Returns the longest length. */
uint32_t orc_huffman_lengths(const uint32_t *count, uint8_t *len) {
  uint64_t w[256];
  for (int i = 0; i < 256; i++) w[i] = count[i];
  for (;;) {
    uint32_t sym[256], m = 0;
    for (uint32_t i = 0; i < 256; i++) {
      len[i] = 0;
      if (w[i]) sym[m++] = i;
    }
    if (m <= 1) return 0;
    /* insertion sort by (weight, symbol) */
    for (uint32_t a = 1; a < m; a++) {
      uint32_t v = sym[a], b = a;
      while (b > 0 && (w[sym[b - 1]] > w[v] ||
                       (w[sym[b - 1]] == w[v] && sym[b - 1] > v))) {
        sym[b] = sym[b - 1];
        b--;
      }
      sym[b] = v;
    }
    /* nodes 0..m-1 are the sorted leaves, m..2m-2 the merges in order */
    uint64_t nw[511];
    int32_t parent[511];
    for (uint32_t i = 0; i < m; i++) nw[i] = w[sym[i]];
    uint32_t li = 0, ii = m, n_int = m;
    for (uint32_t t = 0; t < m - 1; t++) {
      uint32_t pick[2];
      for (int q = 0; q < 2; q++) {
        if (li < m && (ii >= n_int || nw[li] <= nw[ii]))
          pick[q] = li++;
        else
          pick[q] = ii++;
      }
      nw[n_int] = nw[pick[0]] + nw[pick[1]];
      parent[pick[0]] = parent[pick[1]] = (int32_t)n_int;
      n_int++;
    }
    uint32_t depth[511];
    depth[n_int - 1] = 0;
    for (int32_t i = (int32_t)n_int - 2; i >= 0; i--)
      depth[i] = depth[parent[i]] + 1;
    uint32_t longest = 0;
    for (uint32_t i = 0; i < m; i++) {
      len[sym[i]] = (uint8_t)depth[i];
      if (depth[i] > longest) longest = depth[i];
    }
    if (longest <= ORC_HUF_MAX_LEN) return longest;
    for (int i = 0; i < 256; i++)
      if (w[i]) w[i] = (w[i] + 1) / 2;
  }
}

/* Canonical codes (symbols ordered by (length, symbol) take consecutive
 * values): code[s] for every symbol with len[s] > 0. */
static void canonical_codes(const uint8_t *len, uint32_t *code) {
  uint32_t bl[ORC_HUF_MAX_LEN + 2] = {0}, next[ORC_HUF_MAX_LEN + 2] = {0};
  for (int s = 0; s < 256; s++) bl[len[s]]++;
  bl[0] = 0;
  uint32_t c = 0;
  for (uint32_t b = 1; b <= ORC_HUF_MAX_LEN; b++) {
    c = (c + bl[b - 1]) << 1;
    next[b] = c;
  }
  for (int s = 0; s < 256; s++) code[s] = len[s] ? next[len[s]]++ : 0;
}

static uint64_t huf_size(uint32_t n, uint32_t k, uint64_t stream_bytes) {
  if (k == 0) return 16 + pad16(n);
  return 16 + 128 + HUF_STREAMS + pad16(stream_bytes) + pad16(n);
}

/* Bits of each stream for the given lengths; returns the total bytes. */
static uint64_t stream_bytes_of(int codec, const uint8_t *chunk, uint32_t n,
                                const uint8_t *len, uint8_t *sbytes) {
  uint64_t total = 0;
  for (uint32_t s = 0; s < HUF_STREAMS; s++) {
    uint64_t bits = 0;
    for (uint32_t i = 0; i < 64; i++) {
      uint32_t wi = stream_word(s, i);
      if (wi < n) bits += len[plane_a(codec, word_at(chunk, wi))];
    }
    sbytes[s] = (uint8_t)((bits + 7) / 8);
    total += sbytes[s];
  }
  return total;
}

/* Mode choice of formats v2 and v3: RAW, or HUF when strictly smaller.  HUF
 * with a single plane-A symbol has k = 0 and base = that symbol; otherwise k
 * is the longest code length, base 0, and n_esc carries the stream bytes. */
int orc_plan_chunk_huf(int codec, const uint8_t *chunk, uint32_t len,
                       uint32_t *mode, uint32_t *k, uint32_t *base,
                       uint32_t *n_sb, uint64_t *size) {
  uint32_t n = len / 2;
  uint32_t count[256] = {0};
  uint8_t lens[256], sbytes[HUF_STREAMS];
  for (uint32_t i = 0; i < n; i++) count[plane_a(codec, word_at(chunk, i))]++;
  uint32_t longest = orc_huffman_lengths(count, lens);
  uint32_t only = 0, distinct = 0;
  for (uint32_t e = 0; e < 256; e++)
    if (count[e]) {
      distinct++;
      only = e;
    }
  uint64_t sb = longest ? stream_bytes_of(codec, chunk, n, lens, sbytes) : 0;
  uint64_t hs = huf_size(n, longest, sb);
  *mode = 0;
  *k = *base = *n_sb = 0;
  *size = raw_size(n);
  if (n && hs < *size) {
    *mode = 2;
    *k = longest;
    *base = distinct == 1 ? only : 0;
    *n_sb = (uint32_t)sb;
    *size = hs;
  }
  return 0;
}

int orc_plan_chunk_v2(const uint8_t *chunk, uint32_t len, uint32_t *mode,
                      uint32_t *k, uint32_t *base, uint32_t *n_sb,
                      uint64_t *size) {
  return orc_plan_chunk_huf(2, chunk, len, mode, k, base, n_sb, size);
}

/* Write one v2/v3 record (size bytes, already zeroed by the caller).  RAW is
 * plane A (n B) then plane B (n B), each padded: for codec 2 exactly the
 * RAW record of format v1. */
static void write_record_v2(int kind, int codec, const uint8_t *chunk, uint32_t len,
                            uint32_t mode, uint32_t k, uint32_t base,
                            uint32_t n_sb, uint8_t *out) {
  uint32_t n = len / 2;
  if (mode == 0) {
    put_u32(out + 4, n);
    put_u32(out + 12, orc_crc(kind, out, 12));
    for (uint32_t i = 0; i < n; i++) {
      uint16_t w = word_at(chunk, i);
      out[16 + i] = (uint8_t)plane_a(codec, w);
      out[16 + pad16(n) + i] = plane_b(codec, w);
    }
    return;
  }
  out[0] = 2;
  out[1] = (uint8_t)k;
  out[2] = (uint8_t)base;
  out[3] = 0;
  put_u32(out + 4, n);
  put_u32(out + 8, n_sb);
  put_u32(out + 12, orc_crc(kind, out, 12));
  uint8_t *body = out + 16;
  uint8_t *sm;
  if (k == 0) {
    sm = body;
  } else {
    uint32_t count[256] = {0}, code[256];
    uint8_t lens[256];
    for (uint32_t i = 0; i < n; i++) count[plane_a(codec, word_at(chunk, i))]++;
    orc_huffman_lengths(count, lens);
    canonical_codes(lens, code);
    uint8_t *ltab = body, *sbytes = body + 128, *streams = body + 128 + HUF_STREAMS;
    for (uint32_t e = 0; e < 256; e++) ltab[e / 2] |= (uint8_t)(lens[e] << (4 * (e % 2)));
    stream_bytes_of(codec, chunk, n, lens, sbytes);
    uint64_t at = 0;
    for (uint32_t s = 0; s < HUF_STREAMS; s++) {
      uint64_t bit = 0;
      for (uint32_t i = 0; i < 64; i++) {
        uint32_t wi = stream_word(s, i);
        if (wi >= n) continue;
        uint32_t e = plane_a(codec, word_at(chunk, wi));
        /* the code's bits, most significant first, go to the stream in
         * order; stream bit j is bit j % 8 of byte j / 8 */
        for (int b = lens[e] - 1; b >= 0; b--, bit++)
          if ((code[e] >> b) & 1u) streams[at + bit / 8] |= (uint8_t)(1u << (bit % 8));
      }
      at += sbytes[s];
    }
    sm = streams + pad16(at);
  }
  for (uint32_t i = 0; i < n; i++) sm[i] = plane_b(codec, word_at(chunk, i));
}

/* Structure checks and decode of one v2/v3 record (see decode_record). */
static uint32_t decode_record_v2(int kind, int codec, const uint8_t *rec, uint64_t L,
                                 uint32_t len, uint32_t src_crc, uint8_t *out) {
  uint32_t n = len / 2;
  if (L < 16) return ORC_V_RECORD;
  if (orc_crc(kind, rec, 12) != get_u32(rec + 12)) return ORC_V_RECORD;
  uint32_t mode = rec[0], k = rec[1], base = rec[2];
  uint32_t n_words = get_u32(rec + 4), n_sb = get_u32(rec + 8);
  if (rec[3] != 0 || n_words != n || (mode != 0 && mode != 2))
    return ORC_V_RECORD;
  const uint8_t *body = rec + 16, *sm;
  if (mode == 0) {
    if (k != 0 || base != 0 || n_sb != 0 || L != raw_size(n)) return ORC_V_RECORD;
    const uint8_t *pa = body, *pb = body + pad16(n);
    if (!all_zero(pa + n, pad16(n) - n) || !all_zero(pb + n, pad16(n) - n))
      return ORC_V_RECORD;
    for (uint32_t i = 0; i < n; i++)
      put_u16(out + 2 * (uint64_t)i, from_planes(codec, pa[i], pb[i]));
    return orc_crc(kind, out, len) == src_crc ? 0u : ORC_V_DATA;
  }
  uint8_t e_of[32768];
  if (k > ORC_HUF_MAX_LEN) return ORC_V_RECORD;
  /* the encoder codes a chunk only when that beats RAW: a longer HUF record
   * is malformed (this also bounds the stream section a decoder stages) */
  if (huf_size(n, k, n_sb) >= raw_size(n)) return ORC_V_RECORD;
  if (k == 0) {
    if (n_sb != 0 || L != huf_size(n, 0, 0)) return ORC_V_RECORD;
    sm = body;
    for (uint32_t i = 0; i < n; i++) e_of[i] = (uint8_t)base;
  } else {
    if (base != 0 || L != huf_size(n, k, n_sb)) return ORC_V_RECORD;
    const uint8_t *ltab = body, *sbytes = body + 128, *streams = body + 128 + HUF_STREAMS;
    uint8_t lens[256];
    uint32_t longest = 0;
    uint64_t kraft = 0; /* sum of 2^(MAX - len): a complete code fills 2^MAX */
    for (uint32_t e = 0; e < 256; e++) {
      lens[e] = (uint8_t)((ltab[e / 2] >> (4 * (e % 2))) & 15u);
      if (lens[e] > k) return ORC_V_RECORD;
      if (lens[e] > longest) longest = lens[e];
      if (lens[e]) kraft += 1u << (ORC_HUF_MAX_LEN - lens[e]);
    }
    if (longest != k || kraft != (1u << ORC_HUF_MAX_LEN)) return ORC_V_RECORD;
    uint32_t code[256];
    canonical_codes(lens, code);
    /* canonical decoding: per length, the first code and the symbols in
     * code order */
    uint32_t first[ORC_HUF_MAX_LEN + 1], cnt[ORC_HUF_MAX_LEN + 1];
    uint32_t start[ORC_HUF_MAX_LEN + 1], order[256], m = 0;
    for (uint32_t b = 1; b <= ORC_HUF_MAX_LEN; b++) {
      first[b] = 0;
      cnt[b] = 0;
      start[b] = m;
      for (uint32_t e = 0; e < 256; e++)
        if (lens[e] == b) {
          if (!cnt[b]) first[b] = code[e];
          cnt[b]++;
          order[m++] = e;
        }
    }
    uint64_t sum = 0;
    for (uint32_t s = 0; s < HUF_STREAMS; s++) sum += sbytes[s];
    if (sum != n_sb) return ORC_V_RECORD;
    uint64_t at = 0;
    for (uint32_t s = 0; s < HUF_STREAMS; s++) {
      const uint8_t *st = streams + at;
      uint64_t nbits = 8ull * sbytes[s], bit = 0;
      for (uint32_t i = 0; i < 64; i++) {
        uint32_t wi = stream_word(s, i);
        if (wi >= n) continue;
        uint32_t c = 0, b = 0;
        for (;;) {
          if (bit >= nbits) return ORC_V_RECORD; /* ran past the stream */
          c = (c << 1) | ((st[bit / 8] >> (bit % 8)) & 1u);
          bit++;
          b++;
          if (b > k) return ORC_V_RECORD; /* cannot happen for a complete code */
          if (cnt[b] && c - first[b] < cnt[b]) break;
        }
        e_of[wi] = (uint8_t)order[start[b] + (c - first[b])];
      }
      /* the stream is exactly its bits, rounded up to a byte of zeros */
      if ((bit + 7) / 8 != sbytes[s]) return ORC_V_RECORD;
      if (bit % 8 && (st[bit / 8] >> (bit % 8))) return ORC_V_RECORD;
      at += sbytes[s];
    }
    if (!all_zero(streams + at, pad16(at) - at)) return ORC_V_RECORD;
    sm = streams + pad16(at);
  }
  if (!all_zero(sm + n, pad16(n) - n)) return ORC_V_RECORD;
  for (uint32_t i = 0; i < n; i++)
    put_u16(out + 2 * (uint64_t)i, from_planes(codec, e_of[i], sm[i]));
  return orc_crc(kind, out, len) == src_crc ? 0u : ORC_V_DATA;
}

typedef struct {
  int kind, codec;
  const uint8_t *state;
  uint64_t nbytes;
  uint32_t chunk;
  const uint32_t *idx; /* NULL: record r is chunk r */
  uint32_t *mode, *k, *base, *esc;
  uint64_t *size, *offset;
  uint64_t table; /* byte offset of the table */
  uint8_t *payload;
} en_ctx;

static uint64_t en_chunk(const en_ctx *x, uint64_t r) {
  return x->idx ? x->idx[r] : r;
}

static void en_plan_range(void *vp, uint64_t lo, uint64_t hi) {
  en_ctx *x = (en_ctx *)vp;
  for (uint64_t r = lo; r < hi; r++) {
    uint64_t c = en_chunk(x, r);
    const uint8_t *src = x->state + c * (uint64_t)x->chunk;
    uint32_t len = chunk_len(x->nbytes, x->chunk, c);
    if (x->codec >= 2)
      orc_plan_chunk_huf(x->codec, src, len, &x->mode[r], &x->k[r], &x->base[r],
                         &x->esc[r], &x->size[r]);
    else
      orc_plan_chunk(src, len, &x->mode[r], &x->k[r], &x->base[r], &x->esc[r],
                     &x->size[r]);
  }
}

static void en_write_range(void *vp, uint64_t lo, uint64_t hi) {
  en_ctx *x = (en_ctx *)vp;
  for (uint64_t r = lo; r < hi; r++) {
    uint64_t c = en_chunk(x, r);
    const uint8_t *src = x->state + c * (uint64_t)x->chunk;
    uint32_t len = chunk_len(x->nbytes, x->chunk, c);
    uint8_t *entry = x->payload + x->table + 16 * r;
    put_u32(entry, (uint32_t)c);
    put_u32(entry + 4, orc_crc(x->kind, src, len));
    put_u64(entry + 8, x->offset[r]);
    if (x->codec >= 2)
      write_record_v2(x->kind, x->codec, src, len, x->mode[r], x->k[r], x->base[r],
                      x->esc[r], x->payload + x->offset[r]);
    else
      write_record(x->kind, src, len, x->mode[r], x->k[r], x->base[r],
                   x->esc[r], x->payload + x->offset[r]);
  }
}

uint64_t orc_payload_bound(uint64_t nbytes, uint32_t chunk_bytes,
                           uint32_t n_ship) {
  (void)nbytes; /* every record is bounded by a full RAW unit */
  if (!chunk_ok(chunk_bytes)) return 0;
  uint32_t u = unit_of(chunk_bytes);
  uint64_t units = (uint64_t)n_ship * (chunk_bytes / u);
  return 64 + units * (16 + raw_size(u / 2));
}

int64_t orc_encode(int kind, const uint8_t *state, uint64_t nbytes,
                   uint32_t chunk_bytes, const uint32_t *idx, uint32_t n_idx,
                   uint8_t *payload, uint64_t cap, int threads) {
  return orc_encode_codec(kind, 1, state, nbytes, chunk_bytes, idx, n_idx,
                          payload, cap, threads);
}

int64_t orc_encode_codec(int kind, int codec, const uint8_t *state,
                         uint64_t nbytes, uint32_t chunk_bytes,
                         const uint32_t *idx, uint32_t n_idx, uint8_t *payload,
                         uint64_t cap, int threads) {
  if (!chunk_ok(chunk_bytes) || (kind != 0 && kind != 1) || (nbytes & 1))
    return -1;
  if (codec != 1 && !((codec == 2 || codec == 3) && chunk_bytes >= ORC_TILE)) return -1;
  uint64_t n_chunks = n_chunks_of(nbytes, chunk_bytes);
  uint64_t n_ship = idx ? n_idx : n_chunks;
  if (n_ship > n_chunks) return -1;
  for (uint64_t r = 0; idx && r < n_ship; r++)
    if (idx[r] >= n_chunks || (r && idx[r] <= idx[r - 1])) return -1;
  if (cap < orc_payload_bound(nbytes, chunk_bytes, (uint32_t)n_ship)) return -2;

  /* the units shipped: every unit of each listed chunk, in order */
  uint32_t u = unit_of(chunk_bytes);
  uint64_t per = chunk_bytes / u, n_units = n_chunks_of(nbytes, u);
  uint64_t n_rec = idx ? 0 : n_units;
  uint32_t *units = NULL;
  if (idx) {
    units = (uint32_t *)malloc((n_ship * per > 0 ? n_ship * per : 1) * 4);
    for (uint64_t r = 0; r < n_ship; r++)
      for (uint64_t j = 0; j < per; j++)
        if (idx[r] * per + j < n_units) units[n_rec++] = (uint32_t)(idx[r] * per + j);
  }

  uint64_t m = n_rec ? n_rec : 1;
  en_ctx x;
  x.kind = kind;
  x.codec = codec;
  x.state = state;
  x.nbytes = nbytes;
  x.chunk = u;
  x.idx = units;
  x.mode = (uint32_t *)calloc(m, 4);
  x.k = (uint32_t *)calloc(m, 4);
  x.base = (uint32_t *)calloc(m, 4);
  x.esc = (uint32_t *)calloc(m, 4);
  x.size = (uint64_t *)calloc(m, 8);
  x.offset = (uint64_t *)calloc(m, 8);
  x.payload = payload;

  /* 1. plan every record; 2. record offsets are the exclusive prefix sum of
   * record sizes, starting right after the header; the table follows the
   * last record; 3. write records and table entries. */
  parallel_for(n_rec, threads, en_plan_range, &x);
  uint64_t at = 64;
  for (uint64_t r = 0; r < n_rec; r++) {
    x.offset[r] = at;
    at += x.size[r];
  }
  x.table = at;
  uint64_t total = at + 16 * n_rec;
  memset(payload, 0, total);
  parallel_for(n_rec, threads, en_write_range, &x);

  uint8_t *h = payload;
  h[0] = 'W';
  h[1] = 'M';
  h[2] = 'V';
  h[3] = (uint8_t)('0' + codec);
  put_u16(h + 4, (uint16_t)codec);
  h[6] = (uint8_t)kind;
  h[7] = (uint8_t)codec;
  put_u32(h + 8, chunk_bytes);
  put_u32(h + 12, (uint32_t)n_chunks);
  put_u64(h + 16, nbytes);
  put_u32(h + 24, (uint32_t)n_rec);
  put_u32(h + 28, idx ? 0u : 1u);
  put_u64(h + 32, total);
  put_u32(h + 40, orc_crc(kind, state, nbytes));
  put_u32(h + 44, orc_crc(kind, payload + x.table, 16 * n_rec));
  put_u32(h + 60, orc_crc(kind, h, 60));

  free(units);
  free(x.mode);
  free(x.k);
  free(x.base);
  free(x.esc);
  free(x.size);
  free(x.offset);
  return (int64_t)total;
}

/* --------------------------------------------------------------- decode -- */



/* Structure checks and decode of one record occupying rec[0..L).  Returns 0,
 * ORC_V_RECORD or ORC_V_DATA; on 0 the chunk's len bytes are in out. */
static uint32_t decode_record(int kind, const uint8_t *rec, uint64_t L,
                              uint32_t len, uint32_t src_crc, uint8_t *out) {
  uint32_t n = len / 2;
  if (L < 16) return ORC_V_RECORD;
  if (orc_crc(kind, rec, 12) != get_u32(rec + 12)) return ORC_V_RECORD;
  uint32_t mode = rec[0], k = rec[1], base = rec[2];
  uint32_t n_words = get_u32(rec + 4), n_esc = get_u32(rec + 8);
  if (rec[3] != 0 || n_words != n || mode > 1) return ORC_V_RECORD;
  const uint8_t *body = rec + 16;

  if (mode == 0) {
    if (k != 0 || base != 0 || n_esc != 0) return ORC_V_RECORD;
    if (L != raw_size(n)) return ORC_V_RECORD;
    const uint8_t *ex = body, *sm = body + pad16(n);
    if (!all_zero(ex + n, pad16(n) - n) || !all_zero(sm + n, pad16(n) - n))
      return ORC_V_RECORD;
    for (uint32_t i = 0; i < n; i++)
      put_u16(out + 2 * (uint64_t)i,
              (uint16_t)(((uint32_t)(sm[i] >> 7) << 15) | ((uint32_t)ex[i] << 7) |
                         (sm[i] & 127u)));
  } else {
    if (k > 7 || n_esc > n || (k == 0 && n_esc != 0)) return ORC_V_RECORD;
    if (L != pack_size(n, k, n_esc)) return ORC_V_RECORD;
    uint64_t code_bytes = ((uint64_t)n * k + 7) / 8;
    uint64_t ib = index_bytes(n, k);
    const uint8_t *codes = body;
    const uint8_t *index = codes + pad16(code_bytes);
    const uint8_t *escapes = index + pad16(ib);
    const uint8_t *sm = escapes + pad16(n_esc);
    /* padding: whole bytes after each section, and stream bits past n*k */
    if (!all_zero(codes + code_bytes, pad16(code_bytes) - code_bytes) ||
        !all_zero(index + ib, pad16(ib) - ib) ||
        !all_zero(escapes + n_esc, pad16(n_esc) - n_esc) ||
        !all_zero(sm + n, pad16(n) - n))
      return ORC_V_RECORD;
    uint64_t used_bits = (uint64_t)n * k;
    if (used_bits % 8 && (codes[used_bits / 8] >> (used_bits % 8)))
      return ORC_V_RECORD;
    uint32_t esc_code = (1u << k) - 1u;
    uint32_t esc_read = 0;
    for (uint32_t i = 0; i < n; i++) {
      uint32_t e;
      /* each index entry must equal the escapes decoded before its block */
      if (k && i % 512 == 0 &&
          (uint32_t)(index[2 * (i / 512)] | (index[2 * (i / 512) + 1] << 8)) !=
              esc_read)
        return ORC_V_RECORD;
      if (k == 0) {
        e = base;
      } else {
        uint32_t code = 0;
        for (uint32_t b = 0; b < k; b++) {
          uint64_t j = (uint64_t)i * k + b;
          code |= (uint32_t)((codes[j / 8] >> (j % 8)) & 1u) << b;
        }
        if (code == esc_code) {
          if (esc_read >= n_esc) return ORC_V_RECORD;
          e = escapes[esc_read++];
        } else {
          if (base + code > 255u) return ORC_V_RECORD;
          e = base + code;
        }
      }
      uint16_t w = (uint16_t)(((uint32_t)(sm[i] >> 7) << 15) | (e << 7) |
                              (sm[i] & 127u));
      put_u16(out + 2 * (uint64_t)i, w);
    }
    if (esc_read != n_esc) return ORC_V_RECORD;
  }
  return orc_crc(kind, out, len) == src_crc ? 0u : ORC_V_DATA;
}

typedef struct {
  int kind, codec;
  const uint8_t *payload;
  uint64_t table, nbytes;
  uint32_t chunk, n_rec;
  uint8_t *staging;
  uint32_t *status;
} de_ctx;

static void de_range(void *vp, uint64_t lo, uint64_t hi) {
  de_ctx *x = (de_ctx *)vp;
  for (uint64_t r = lo; r < hi; r++) {
    const uint8_t *e = x->payload + x->table + 16 * r;
    uint32_t c = get_u32(e);
    uint64_t off = get_u64(e + 8);
    uint64_t end = r + 1 < x->n_rec ? get_u64(e + 16 + 8) : x->table;
    uint32_t len = chunk_len(x->nbytes, x->chunk, c);
    uint8_t *out = x->staging + r * (uint64_t)x->chunk;
    x->status[r] = x->codec >= 2
                       ? decode_record_v2(x->kind, x->codec, x->payload + off, end - off,
                                          len, get_u32(e + 4), out)
                       : decode_record(x->kind, x->payload + off, end - off,
                                       len, get_u32(e + 4), out);
  }
}

uint32_t orc_decode_verify(int kind, const uint8_t *payload, uint64_t cap,
                           uint64_t nbytes, uint32_t chunk_bytes,
                           uint8_t *staging, uint64_t staging_cap,
                           uint32_t *rec_status, uint32_t n_status,
                           int threads) {
  return orc_decode_verify_codec(kind, 1, payload, cap, nbytes, chunk_bytes,
                                 staging, staging_cap, rec_status, n_status,
                                 threads);
}

uint32_t orc_decode_verify_codec(int kind, int codec, const uint8_t *payload,
                                 uint64_t cap, uint64_t nbytes,
                                 uint32_t chunk_bytes, uint8_t *staging,
                                 uint64_t staging_cap, uint32_t *rec_status,
                                 uint32_t n_status, int threads) {
  if (!chunk_ok(chunk_bytes) || (kind != 0 && kind != 1)) return ORC_V_HEADER;
  if (codec != 1 && !((codec == 2 || codec == 3) && chunk_bytes >= ORC_TILE))
    return ORC_V_HEADER;
  uint64_t n_chunks = n_chunks_of(nbytes, chunk_bytes);
  uint32_t u = unit_of(chunk_bytes);
  uint64_t per = chunk_bytes / u, n_units = n_chunks_of(nbytes, u);

  /* header */
  if (cap < 64) return ORC_V_HEADER;
  const uint8_t *h = payload;
  if (orc_crc(kind, h, 60) != get_u32(h + 60)) return ORC_V_HEADER;
  if (h[0] != 'W' || h[1] != 'M' || h[2] != 'V' ||
      h[3] != (uint8_t)('0' + codec))
    return ORC_V_HEADER;
  if ((h[4] | (h[5] << 8)) != codec || h[6] != (uint8_t)kind ||
      h[7] != (uint8_t)codec)
    return ORC_V_HEADER;
  if (get_u32(h + 8) != chunk_bytes || get_u32(h + 12) != n_chunks ||
      get_u64(h + 16) != nbytes)
    return ORC_V_HEADER;
  uint32_t n_rec = get_u32(h + 24), flags = get_u32(h + 28);
  uint64_t payload_bytes = get_u64(h + 32);
  if ((flags & ~1u) || !all_zero(h + 48, 12)) return ORC_V_HEADER;
  if (n_rec > n_units) return ORC_V_HEADER;
  if (64 + 16 * (uint64_t)n_rec > payload_bytes || payload_bytes > cap ||
      payload_bytes % 16)
    return ORC_V_HEADER;
  if ((flags & 1u) && n_rec != n_units) return ORC_V_HEADER;
  if ((uint64_t)n_rec * u > staging_cap) return ORC_V_STAGING;

  /* table: the last 16*n_records bytes of the payload */
  uint64_t table = payload_bytes - 16 * (uint64_t)n_rec;
  const uint8_t *t = payload + table;
  if (orc_crc(kind, t, 16 * (uint64_t)n_rec) != get_u32(h + 44))
    return ORC_V_TABLE;
  if (n_rec == 0 && payload_bytes != 64) return ORC_V_TABLE;
  for (uint32_t r = 0; r < n_rec; r++) {
    uint32_t c = get_u32(t + 16 * (uint64_t)r);
    uint64_t off = get_u64(t + 16 * (uint64_t)r + 8);
    uint64_t end =
        r + 1 < n_rec ? get_u64(t + 16 * (uint64_t)(r + 1) + 8) : table;
    if (c >= n_units) return ORC_V_TABLE;
    if (r && c <= get_u32(t + 16 * (uint64_t)(r - 1))) return ORC_V_TABLE;
    if (r == 0 && off != 64) return ORC_V_TABLE;
    if (off % 16 || off >= end) return ORC_V_TABLE;
    /* whole chunks: a tile other than its chunk's first comes right after
     * the tile before it, and one other than its chunk's last (and not the
     * state's last) right before the tile after it */
    if (c % per && (r == 0 || get_u32(t + 16 * (uint64_t)(r - 1)) != c - 1))
      return ORC_V_TABLE;
    if ((c + 1) % per && c + 1 < n_units &&
        (r + 1 == n_rec || get_u32(t + 16 * (uint64_t)(r + 1)) != c + 1))
      return ORC_V_TABLE;
  }

  /* records */
  uint32_t *status = (uint32_t *)calloc(n_rec ? n_rec : 1, 4);
  de_ctx x = {kind, codec, payload, table, nbytes, u, n_rec, staging, status};
  parallel_for(n_rec, threads, de_range, &x);
  uint32_t verdict = 0;
  for (uint32_t r = 0; r < n_rec; r++) {
    verdict |= status[r];
    if (rec_status && r < n_status) rec_status[r] = status[r];
  }
  free(status);
  return verdict;
}

int orc_commit(uint8_t *live, uint64_t nbytes, uint32_t chunk_bytes,
               const uint8_t *staging, const uint8_t *payload,
               uint32_t verdict) {
  if (verdict != 0) return 1;
  uint32_t u = unit_of(chunk_bytes);
  uint32_t n_rec = get_u32(payload + 24);
  uint64_t table = get_u64(payload + 32) - 16 * (uint64_t)n_rec;
  for (uint32_t r = 0; r < n_rec; r++) {
    uint32_t c = get_u32(payload + table + 16 * (uint64_t)r);
    memcpy(live + (uint64_t)c * u, staging + (uint64_t)r * u, chunk_len(nbytes, u, c));
  }
  return 0;
}

/* Re-verifying install (Table 1: commit re-verifies, then swaps).  With a
 * zero verdict, the staged records are checked again against their
 * receipts, and the state the install would produce (live with every
 * staged record in place) is checksummed whole and compared with the
 * header's global CRC, the CRC of the source state.  Only if both hold is
 * the install done.  Returns the verdict: the one given if nonzero, else 0
 * or ORC_V_REVERIFY; live is untouched unless 0 is returned. */
uint32_t orc_commit_reverify(int kind, uint8_t *live, uint64_t nbytes,
                             uint32_t chunk_bytes, const uint8_t *staging,
                             const uint8_t *payload, uint32_t verdict) {
  if (verdict != 0) return verdict;
  uint32_t u = unit_of(chunk_bytes);
  uint32_t n_rec = get_u32(payload + 24);
  uint64_t table = get_u64(payload + 32) - 16 * (uint64_t)n_rec;
  int bad = 0;
  uint8_t *result = malloc(nbytes ? nbytes : 1);
  if (!result) return ORC_V_REVERIFY;
  memcpy(result, live, nbytes);
  for (uint32_t r = 0; r < n_rec; r++) {
    uint32_t c = get_u32(payload + table + 16 * (uint64_t)r);
    uint32_t receipt = get_u32(payload + table + 16 * (uint64_t)r + 4);
    uint32_t len = chunk_len(nbytes, u, c);
    const uint8_t *src = staging + (uint64_t)r * u;
    if (orc_crc(kind, src, len) != receipt) bad = 1;
    memcpy(result + (uint64_t)c * u, src, len);
  }
  if (orc_crc(kind, result, nbytes) != get_u32(payload + 40)) bad = 1;
  if (!bad) memcpy(live, result, nbytes);
  free(result);
  return bad ? ORC_V_REVERIFY : 0u;
}

/* ---- manifest flatten / rehydrate (§4 "Sufficiency", §5 "Implementation") */

uint64_t orc_flat_layout(const uint64_t *bytes, uint32_t n, uint64_t *off) {
  uint64_t pos = 0;
  for (uint32_t i = 0; i < n; i++) {
    off[i] = pos;
    pos += bytes[i];
    while (pos % 16 != 0) pos++;
  }
  return pos;
}

void orc_flatten(const uint8_t *const *leaves, const uint64_t *bytes,
                 uint32_t n, uint8_t *flat) {
  uint64_t pos = 0;
  for (uint32_t i = 0; i < n; i++) {
    if (bytes[i]) memcpy(flat + pos, leaves[i], bytes[i]);
    pos += bytes[i];
    while (pos % 16 != 0) flat[pos++] = 0;
  }
}

void orc_rehydrate(const uint8_t *flat, uint8_t *const *leaves,
                   const uint64_t *bytes, uint32_t n) {
  uint64_t pos = 0;
  for (uint32_t i = 0; i < n; i++) {
    if (bytes[i]) memcpy(leaves[i], flat + pos, bytes[i]);
    pos += bytes[i];
    while (pos % 16 != 0) pos++;
  }
}
