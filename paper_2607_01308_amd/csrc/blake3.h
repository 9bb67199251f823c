// BLAKE3 compression (unkeyed hash mode), written for 64-wide wavefronts: one
// lane owns one chaining value, the message words live in registers, and the 7
// rounds are fully unrolled so the per-round message permutation is register
// renaming. Each G step is the three-input add / xor / funnel-shift rotate that
// gfx950 executes in 12 VALU ops: 672 VALU ops per 64-byte block, against 960
// for BLAKE2s's 10 rounds. Host-callable too, so the CPU tests can run the very
// same code against the oracle and the published test vectors.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cm {

// Chaining value (8 words).
struct B3Cv {
  uint32_t h[8];
};

// Initial chaining value of every chunk and parent in the unkeyed hash mode
// (the same words as the SHA-256 IV).
#define CM_B3_IV0 0x6A09E667u
#define CM_B3_IV1 0xBB67AE85u
#define CM_B3_IV2 0x3C6EF372u
#define CM_B3_IV3 0xA54FF53Au
#define CM_B3_IV4 0x510E527Fu
#define CM_B3_IV5 0x9B05688Cu
#define CM_B3_IV6 0x1F83D9ABu
#define CM_B3_IV7 0x5BE0CD19u

// Domain flags of a compression.
constexpr uint32_t kB3ChunkStart = 1;
constexpr uint32_t kB3ChunkEnd = 2;
constexpr uint32_t kB3Parent = 4;
constexpr uint32_t kB3Root = 8;

// Bytes per chunk (16 blocks of 64 bytes).
constexpr int64_t kB3ChunkBytes = 1024;
constexpr int kB3ChunkBlocks = 16;

__host__ __device__ __forceinline__ uint32_t b3_rotr(uint32_t x, int n) {
  return (x >> n) | (x << (32 - n));
}

__host__ __device__ __forceinline__ void b3_init(B3Cv& s) {
  s.h[0] = CM_B3_IV0;
  s.h[1] = CM_B3_IV1;
  s.h[2] = CM_B3_IV2;
  s.h[3] = CM_B3_IV3;
  s.h[4] = CM_B3_IV4;
  s.h[5] = CM_B3_IV5;
  s.h[6] = CM_B3_IV6;
  s.h[7] = CM_B3_IV7;
}

#define CM_B3_G(a, b, c, d, x, y) \
  do {                            \
    a = a + b + (x);              \
    d = b3_rotr(d ^ a, 16);       \
    c = c + d;                    \
    b = b3_rotr(b ^ c, 12);       \
    a = a + b + (y);              \
    d = b3_rotr(d ^ a, 8);        \
    c = c + d;                    \
    b = b3_rotr(b ^ c, 7);        \
  } while (0)

// One round over the message words in the order m[p0..p15]: the four column
// steps take (p0,p1) .. (p6,p7), the four diagonal steps (p8,p9) .. (p14,p15).
#define CM_B3_ROUND(m, p0, p1, p2, p3, p4, p5, p6, p7, p8, p9, p10, p11, p12, p13, p14, p15) \
  do {                                                                                      \
    CM_B3_G(v0, v4, v8, v12, m[p0], m[p1]);                                                 \
    CM_B3_G(v1, v5, v9, v13, m[p2], m[p3]);                                                 \
    CM_B3_G(v2, v6, v10, v14, m[p4], m[p5]);                                                \
    CM_B3_G(v3, v7, v11, v15, m[p6], m[p7]);                                                \
    CM_B3_G(v0, v5, v10, v15, m[p8], m[p9]);                                                \
    CM_B3_G(v1, v6, v11, v12, m[p10], m[p11]);                                              \
    CM_B3_G(v2, v7, v8, v13, m[p12], m[p13]);                                               \
    CM_B3_G(v3, v4, v9, v14, m[p14], m[p15]);                                               \
  } while (0)

// Compress one 64-byte block m[16] into the chaining value s:
// s <- first half xor second half of the 7-round state started from
// (s, IV0..IV3, counter, block_len, flags). Round r reads the message words
// through the fixed permutation applied r times; the index lists below are
// those compositions, so no word moves at run time.
__host__ __device__ __forceinline__ void b3_compress(B3Cv& s, const uint32_t (&m)[16],
                                                     uint64_t counter, uint32_t block_len,
                                                     uint32_t flags) {
  uint32_t v0 = s.h[0], v1 = s.h[1], v2 = s.h[2], v3 = s.h[3];
  uint32_t v4 = s.h[4], v5 = s.h[5], v6 = s.h[6], v7 = s.h[7];
  uint32_t v8 = CM_B3_IV0, v9 = CM_B3_IV1, v10 = CM_B3_IV2, v11 = CM_B3_IV3;
  uint32_t v12 = (uint32_t)counter, v13 = (uint32_t)(counter >> 32);
  uint32_t v14 = block_len, v15 = flags;
  CM_B3_ROUND(m, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
  CM_B3_ROUND(m, 2, 6, 3, 10, 7, 0, 4, 13, 1, 11, 12, 5, 9, 14, 15, 8);
  CM_B3_ROUND(m, 3, 4, 10, 12, 13, 2, 7, 14, 6, 5, 9, 0, 11, 15, 8, 1);
  CM_B3_ROUND(m, 10, 7, 12, 9, 14, 3, 13, 15, 4, 0, 11, 2, 5, 8, 1, 6);
  CM_B3_ROUND(m, 12, 13, 9, 11, 15, 10, 14, 8, 7, 2, 5, 3, 0, 1, 6, 4);
  CM_B3_ROUND(m, 9, 14, 11, 5, 8, 12, 15, 1, 13, 3, 0, 10, 2, 6, 4, 7);
  CM_B3_ROUND(m, 11, 15, 5, 0, 1, 9, 8, 6, 14, 10, 2, 12, 3, 4, 7, 13);
  s.h[0] = v0 ^ v8;
  s.h[1] = v1 ^ v9;
  s.h[2] = v2 ^ v10;
  s.h[3] = v3 ^ v11;
  s.h[4] = v4 ^ v12;
  s.h[5] = v5 ^ v13;
  s.h[6] = v6 ^ v14;
  s.h[7] = v7 ^ v15;
}

#undef CM_B3_ROUND
#undef CM_B3_G

// Flags of block b of a chunk of nb blocks (root: the chunk is the whole message).
__host__ __device__ __forceinline__ uint32_t b3_chunk_flags(int64_t b, int64_t nb, bool root) {
  return (b == 0 ? kB3ChunkStart : 0u) | (b + 1 == nb ? (kB3ChunkEnd | (root ? kB3Root : 0u)) : 0u);
}

// Chaining value of a parent node whose children are l and r (root: the top node).
__host__ __device__ __forceinline__ void b3_parent(B3Cv& out, const B3Cv& l, const B3Cv& r,
                                                   bool root) {
  uint32_t m[16];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    m[k] = l.h[k];
    m[8 + k] = r.h[k];
  }
  b3_init(out);
  b3_compress(out, m, 0, 64, kB3Parent | (root ? kB3Root : 0u));
}

// Chaining value of one chunk of nb (1..16) full 64-byte blocks; load_block(b, w)
// reads block b into w[16]. Two blocks are in flight while two are compressed,
// with alternating buffers so no registers are copied between iterations.
template <class LoadBlock>
__host__ __device__ __forceinline__ void b3_chunk(B3Cv& s, int64_t nb, uint64_t chunk_index,
                                                  bool root, LoadBlock load_block) {
  uint32_t x0[16], x1[16], y0[16], y1[16];
  b3_init(s);
  load_block(0, x0);
  if (nb > 1) load_block(1, x1);
  for (int64_t b = 0; b < nb; b += 4) {
    if (b + 2 < nb) load_block(b + 2, y0);
    if (b + 3 < nb) load_block(b + 3, y1);
    b3_compress(s, x0, chunk_index, 64, b3_chunk_flags(b, nb, root));
    if (b + 1 < nb) b3_compress(s, x1, chunk_index, 64, b3_chunk_flags(b + 1, nb, root));
    if (b + 4 < nb) load_block(b + 4, x0);
    if (b + 5 < nb) load_block(b + 5, x1);
    if (b + 2 < nb) b3_compress(s, y0, chunk_index, 64, b3_chunk_flags(b + 2, nb, root));
    if (b + 3 < nb) b3_compress(s, y1, chunk_index, 64, b3_chunk_flags(b + 3, nb, root));
  }
}

}  // namespace cm
