// BLAKE2s-256 compression (RFC 7693), written for 64-wide wavefronts: one lane
// owns one hash chain, message words live in registers, the 10 rounds are fully
// unrolled so the message schedule costs nothing, and each G step is the
// three-input add / xor / funnel-shift rotate that gfx950 executes in 12 VALU ops.
// Host-callable too, so the CPU tests can run the very same code against hashlib.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cm {

struct B2sState {
  uint32_t h[8];
};

// Initial chaining values (RFC 7693, section 2.6: the SHA-256 IV).
#define CM_B2S_IV0 0x6A09E667u
#define CM_B2S_IV1 0xBB67AE85u
#define CM_B2S_IV2 0x3C6EF372u
#define CM_B2S_IV3 0xA54FF53Au
#define CM_B2S_IV4 0x510E527Fu
#define CM_B2S_IV5 0x9B05688Cu
#define CM_B2S_IV6 0x1F83D9ABu
#define CM_B2S_IV7 0x5BE0CD19u

__host__ __device__ __forceinline__ uint32_t b2s_rotr(uint32_t x, int n) {
  return (x >> n) | (x << (32 - n));
}

// Parameter block words 0..3 (RFC 7693 section 2.5 / BLAKE2 tree parameters);
// salt and personalization are zero.
//   w0 = digest_len | key_len << 8 | fanout << 16 | depth << 24
//   w1 = leaf_length
//   w2 = node_offset[31:0]
//   w3 = node_offset[47:32] | node_depth << 16 | inner_length << 24
__host__ __device__ __forceinline__ void b2s_init(B2sState& s, uint32_t p0, uint32_t p1,
                                                  uint32_t p2, uint32_t p3) {
  s.h[0] = CM_B2S_IV0 ^ p0;
  s.h[1] = CM_B2S_IV1 ^ p1;
  s.h[2] = CM_B2S_IV2 ^ p2;
  s.h[3] = CM_B2S_IV3 ^ p3;
  s.h[4] = CM_B2S_IV4;
  s.h[5] = CM_B2S_IV5;
  s.h[6] = CM_B2S_IV6;
  s.h[7] = CM_B2S_IV7;
}

// Tree-mode node parameters used for every leaf and inner node:
// 32-byte digest, no key, fanout 2, depth 255, leaf 4096 B, inner 32 B.
__host__ __device__ __forceinline__ void b2s_init_tree(B2sState& s, uint64_t node_offset,
                                                       uint32_t node_depth) {
  b2s_init(s, 32u | (2u << 16) | (255u << 24), 4096u, (uint32_t)node_offset,
           (uint32_t)((node_offset >> 32) & 0xFFFFu) | (node_depth << 16) | (32u << 24));
}

// Sequential (non-tree) BLAKE2s-256 parameters: fanout 1, depth 1.
__host__ __device__ __forceinline__ void b2s_init_sequential(B2sState& s) {
  b2s_init(s, 32u | (1u << 16) | (1u << 24), 0u, 0u, 0u);
}

#define CM_B2S_G(a, b, c, d, x, y)  \
  do {                              \
    a = a + b + (x);                \
    d = b2s_rotr(d ^ a, 16);        \
    c = c + d;                      \
    b = b2s_rotr(b ^ c, 12);        \
    a = a + b + (y);                \
    d = b2s_rotr(d ^ a, 8);         \
    c = c + d;                      \
    b = b2s_rotr(b ^ c, 7);         \
  } while (0)

// One round with message permutation (s0..s15) of RFC 7693 section 2.7.
#define CM_B2S_ROUND(m, s0, s1, s2, s3, s4, s5, s6, s7, s8, s9, s10, s11, s12, s13, s14, s15) \
  do {                                                                                        \
    CM_B2S_G(v0, v4, v8, v12, m[s0], m[s1]);                                                  \
    CM_B2S_G(v1, v5, v9, v13, m[s2], m[s3]);                                                  \
    CM_B2S_G(v2, v6, v10, v14, m[s4], m[s5]);                                                 \
    CM_B2S_G(v3, v7, v11, v15, m[s6], m[s7]);                                                 \
    CM_B2S_G(v0, v5, v10, v15, m[s8], m[s9]);                                                 \
    CM_B2S_G(v1, v6, v11, v12, m[s10], m[s11]);                                               \
    CM_B2S_G(v2, v7, v8, v13, m[s12], m[s13]);                                                \
    CM_B2S_G(v3, v4, v9, v14, m[s14], m[s15]);                                                \
  } while (0)

// Compress one 64-byte block m[16] into s. t = bytes hashed so far including
// this block; last = final block of the message (f0); last_node = final block
// of the last node of a tree level (f1).
__host__ __device__ __forceinline__ void b2s_compress(B2sState& s, const uint32_t (&m)[16],
                                                      uint64_t t, bool last, bool last_node) {
  uint32_t v0 = s.h[0], v1 = s.h[1], v2 = s.h[2], v3 = s.h[3];
  uint32_t v4 = s.h[4], v5 = s.h[5], v6 = s.h[6], v7 = s.h[7];
  uint32_t v8 = CM_B2S_IV0, v9 = CM_B2S_IV1, v10 = CM_B2S_IV2, v11 = CM_B2S_IV3;
  uint32_t v12 = CM_B2S_IV4 ^ (uint32_t)t;
  uint32_t v13 = CM_B2S_IV5 ^ (uint32_t)(t >> 32);
  uint32_t v14 = last ? ~CM_B2S_IV6 : CM_B2S_IV6;
  uint32_t v15 = last_node ? ~CM_B2S_IV7 : CM_B2S_IV7;
  CM_B2S_ROUND(m, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
  CM_B2S_ROUND(m, 14, 10, 4, 8, 9, 15, 13, 6, 1, 12, 0, 2, 11, 7, 5, 3);
  CM_B2S_ROUND(m, 11, 8, 12, 0, 5, 2, 15, 13, 10, 14, 3, 6, 7, 1, 9, 4);
  CM_B2S_ROUND(m, 7, 9, 3, 1, 13, 12, 11, 14, 2, 6, 5, 10, 4, 0, 15, 8);
  CM_B2S_ROUND(m, 9, 0, 5, 7, 2, 4, 10, 15, 14, 1, 11, 12, 6, 8, 3, 13);
  CM_B2S_ROUND(m, 2, 12, 6, 10, 0, 11, 8, 3, 4, 13, 7, 5, 15, 14, 1, 9);
  CM_B2S_ROUND(m, 12, 5, 1, 15, 14, 13, 4, 10, 0, 7, 6, 3, 9, 2, 8, 11);
  CM_B2S_ROUND(m, 13, 11, 7, 14, 12, 1, 3, 9, 5, 0, 15, 4, 8, 6, 2, 10);
  CM_B2S_ROUND(m, 6, 15, 14, 9, 11, 3, 0, 8, 12, 2, 13, 7, 1, 4, 10, 5);
  CM_B2S_ROUND(m, 10, 2, 8, 4, 7, 6, 1, 5, 15, 11, 9, 14, 3, 12, 13, 0);
  s.h[0] ^= v0 ^ v8;
  s.h[1] ^= v1 ^ v9;
  s.h[2] ^= v2 ^ v10;
  s.h[3] ^= v3 ^ v11;
  s.h[4] ^= v4 ^ v12;
  s.h[5] ^= v5 ^ v13;
  s.h[6] ^= v6 ^ v14;
  s.h[7] ^= v7 ^ v15;
}

#undef CM_B2S_ROUND
#undef CM_B2S_G

// Hash one node made of nb >= 1 64-byte message blocks; load_block(b, w) reads
// block b into w[16]. Two blocks are in flight while two are compressed, with
// alternating buffers so no registers are copied between iterations.
template <class LoadBlock>
__host__ __device__ __forceinline__ void b2s_node(B2sState& s, uint64_t nb, bool last_node,
                                                  LoadBlock load_block) {
  uint32_t x0[16], x1[16], y0[16], y1[16];
  load_block(0, x0);
  if (nb > 1) load_block(1, x1);
  for (uint64_t b = 0; b < nb; b += 4) {
    if (b + 2 < nb) load_block(b + 2, y0);
    if (b + 3 < nb) load_block(b + 3, y1);
    b2s_compress(s, x0, (b + 1) << 6, b + 1 == nb, b + 1 == nb && last_node);
    if (b + 1 < nb) b2s_compress(s, x1, (b + 2) << 6, b + 2 == nb, b + 2 == nb && last_node);
    if (b + 4 < nb) load_block(b + 4, x0);
    if (b + 5 < nb) load_block(b + 5, x1);
    if (b + 2 < nb) b2s_compress(s, y0, (b + 3) << 6, b + 3 == nb, b + 3 == nb && last_node);
    if (b + 3 < nb) b2s_compress(s, y1, (b + 4) << 6, b + 4 == nb, b + 4 == nb && last_node);
  }
}

// A node whose len bytes (a positive multiple of 64) are contiguous, read with
// the 64-byte loader load64(p, w).
template <class Load64>
__host__ __device__ __forceinline__ void b2s_node_aligned(B2sState& s, const uint8_t* p,
                                                          uint64_t len, bool last_node,
                                                          Load64 load64) {
  b2s_node(s, len >> 6, last_node,
           [&](uint64_t b, uint32_t (&w)[16]) { load64(p + (b << 6), w); });
}

}  // namespace cm
