/*
 * BLAKE3-256, unkeyed hash mode: a plain scalar implementation written from the
 * published BLAKE3 specification (J. O'Connor, J.-P. Aumasson, S. Neves,
 * Z. Wilcox-O'Hearn, "BLAKE3: one function, fast everywhere", 2020).
 *
 * TEST INFRASTRUCTURE ONLY: the hash function of the CPU oracle. It shares no
 * code with the HIP path and nothing in the product path links it.
 *
 * The steps, as the specification defines them:
 *   - compression: a 16-word state (chaining value, four IV words, 64-bit
 *     counter, block length, flags) mixed by 7 rounds of the G function over
 *     columns then diagonals, the message words permuted between rounds; the
 *     new chaining value is the first half of the state xor the second half;
 *   - chunk: up to 1024 bytes cut into 64-byte blocks (the last zero-padded, its
 *     true length passed as the block length), compressed in sequence from the
 *     IV with the chunk index as counter, CHUNK_START on the first block and
 *     CHUNK_END on the last;
 *   - tree: more than one chunk splits into a left subtree holding the largest
 *     power of two of chunks that leaves at least one for the right subtree;
 *     a parent compresses the two child chaining values as one 64-byte block
 *     with counter 0 and the PARENT flag;
 *   - the root (the single chunk's last block, or the top parent) also carries
 *     ROOT, and its first 32 output bytes are the digest.
 */
#include <stddef.h>
#include <stdint.h>
#include <string.h>

static const uint32_t IV[8] = {0x6A09E667u, 0xBB67AE85u, 0x3C6EF372u, 0xA54FF53Au,
                               0x510E527Fu, 0x9B05688Cu, 0x1F83D9ABu, 0x5BE0CD19u};
static const int MSG_PERMUTATION[16] = {2, 6, 3, 10, 7, 0, 4, 13, 1, 11, 12, 5, 9, 14, 15, 8};

enum { CHUNK_START = 1, CHUNK_END = 2, PARENT = 4, ROOT = 8 };
enum { BLOCK_LEN = 64, CHUNK_LEN = 1024 };

static uint32_t rotr32(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

static void g(uint32_t v[16], int a, int b, int c, int d, uint32_t mx, uint32_t my) {
  v[a] = v[a] + v[b] + mx;
  v[d] = rotr32(v[d] ^ v[a], 16);
  v[c] = v[c] + v[d];
  v[b] = rotr32(v[b] ^ v[c], 12);
  v[a] = v[a] + v[b] + my;
  v[d] = rotr32(v[d] ^ v[a], 8);
  v[c] = v[c] + v[d];
  v[b] = rotr32(v[b] ^ v[c], 7);
}

static void round_fn(uint32_t v[16], const uint32_t m[16]) {
  g(v, 0, 4, 8, 12, m[0], m[1]);     /* columns */
  g(v, 1, 5, 9, 13, m[2], m[3]);
  g(v, 2, 6, 10, 14, m[4], m[5]);
  g(v, 3, 7, 11, 15, m[6], m[7]);
  g(v, 0, 5, 10, 15, m[8], m[9]);    /* diagonals */
  g(v, 1, 6, 11, 12, m[10], m[11]);
  g(v, 2, 7, 8, 13, m[12], m[13]);
  g(v, 3, 4, 9, 14, m[14], m[15]);
}

/* New chaining value of one compression (the first 8 output words). */
static void compress(const uint32_t cv[8], const uint32_t block[16], uint64_t counter,
                     uint32_t block_len, uint32_t flags, uint32_t out[8]) {
  uint32_t v[16], m[16], t[16];
  for (int i = 0; i < 8; ++i) v[i] = cv[i];
  for (int i = 0; i < 4; ++i) v[8 + i] = IV[i];
  v[12] = (uint32_t)counter;
  v[13] = (uint32_t)(counter >> 32);
  v[14] = block_len;
  v[15] = flags;
  memcpy(m, block, sizeof m);
  for (int r = 0; r < 7; ++r) {
    round_fn(v, m);
    for (int i = 0; i < 16; ++i) t[i] = m[MSG_PERMUTATION[i]];
    memcpy(m, t, sizeof m);
  }
  for (int i = 0; i < 8; ++i) out[i] = v[i] ^ v[i + 8];
}

/* Little-endian words of a block of len <= 64 bytes, zero-padded. */
static void block_words(const uint8_t* p, size_t len, uint32_t w[16]) {
  uint8_t buf[BLOCK_LEN];
  memset(buf, 0, sizeof buf);
  if (len) memcpy(buf, p, len);
  for (int i = 0; i < 16; ++i)
    w[i] = (uint32_t)buf[4 * i] | (uint32_t)buf[4 * i + 1] << 8 | (uint32_t)buf[4 * i + 2] << 16 |
           (uint32_t)buf[4 * i + 3] << 24;
}

/* Chaining value of one chunk of len <= 1024 bytes (0 only for empty input). */
static void chunk_cv(const uint8_t* p, size_t len, uint64_t chunk_index, int is_root,
                     uint32_t out[8]) {
  const size_t nblocks = len == 0 ? 1 : (len + BLOCK_LEN - 1) / BLOCK_LEN;
  uint32_t cv[8], w[16];
  memcpy(cv, IV, sizeof cv);
  for (size_t b = 0; b < nblocks; ++b) {
    const size_t here = len - b * BLOCK_LEN < BLOCK_LEN ? len - b * BLOCK_LEN : BLOCK_LEN;
    uint32_t flags = 0;
    if (b == 0) flags |= CHUNK_START;
    if (b == nblocks - 1) flags |= CHUNK_END | (is_root ? ROOT : 0);
    block_words(p + b * BLOCK_LEN, here, w);
    compress(cv, w, chunk_index, (uint32_t)here, flags, cv);
  }
  memcpy(out, cv, sizeof cv);
}

/* Chaining value of the subtree over len bytes starting at chunk first_chunk. */
static void subtree_cv(const uint8_t* p, size_t len, uint64_t first_chunk, int is_root,
                       uint32_t out[8]) {
  if (len <= CHUNK_LEN) {
    chunk_cv(p, len, first_chunk, is_root, out);
    return;
  }
  const size_t chunks = (len + CHUNK_LEN - 1) / CHUNK_LEN;
  size_t left = 1;
  while (2 * left < chunks) left *= 2;       /* largest power of two below chunks */
  uint32_t children[16];
  subtree_cv(p, left * CHUNK_LEN, first_chunk, 0, children);
  subtree_cv(p + left * CHUNK_LEN, len - left * CHUNK_LEN, first_chunk + left, 0, children + 8);
  compress(IV, children, 0, BLOCK_LEN, PARENT | (is_root ? ROOT : 0), out);
}

/* out: 32 bytes, the BLAKE3-256 digest of data[0, len). */
void oracle_blake3(const uint8_t* data, uint64_t len, uint8_t* out) {
  uint32_t h[8];
  subtree_cv(data, (size_t)len, 0, 1, h);
  for (int i = 0; i < 8; ++i) {
    out[4 * i] = (uint8_t)h[i];
    out[4 * i + 1] = (uint8_t)(h[i] >> 8);
    out[4 * i + 2] = (uint8_t)(h[i] >> 16);
    out[4 * i + 3] = (uint8_t)(h[i] >> 24);
  }
}
