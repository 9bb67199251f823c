// BLAKE3 compression by the four lanes of a quad, for chains of dependent
// compressions where latency counts rather than throughput: a chunk's 16 blocks
// in the fragment Id, and the last levels of a tree fold, where a handful of
// lanes would otherwise each run a whole 672-op compression while the rest of the
// wave idles. Same function as b3_compress (blake3.h); only the lanes that
// compute it differ.
//
// Lane q of a quad (lanes 4Q .. 4Q + 3) owns column q of the 4 x 4 state,
// (v[q], v[4 + q], v[8 + q], v[12 + q]), and runs that column's G step. For the
// diagonal step rows 1, 2, 3 rotate left by 1, 2, 3 lanes within the quad
// (DPP quad_perm moves, most of which the compiler folds into the VALU op
// that reads them), so lane q holds diagonal q, and rotate back after it. Every
// lane holds the whole message block and selects its round's two words by its
// column.
// Per round and lane: 24 G ops, 6 quad moves, 12 selects (against 96 G ops for
// a whole compression in one lane). The chaining value is split the same way:
// lane q holds h[q] (lo) and h[4 + q] (hi), which is exactly what the final xor
// of the state halves leaves in it, so consecutive compressions exchange
// nothing. All four lanes of a quad must be active.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "blake3.h"

namespace cm {

template <int CTRL>
__device__ __forceinline__ uint32_t b3_qperm(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

// Word A_q of the message for the lane with quad index q = q1 + 2 q2.
template <int A0, int A1, int A2, int A3>
__device__ __forceinline__ uint32_t b3_qsel(const uint32_t (&m)[16], bool q1, bool q2) {
  const uint32_t lo = q1 ? m[A1] : m[A0];
  const uint32_t hi = q1 ? m[A3] : m[A2];
  return q2 ? hi : lo;
}

#define CM_B3Q_G(x, y)               \
  do {                               \
    a = a + b + (x);                 \
    d = b3_rotr(d ^ a, 16);          \
    c = c + d;                       \
    b = b3_rotr(b ^ c, 12);          \
    a = a + b + (y);                 \
    d = b3_rotr(d ^ a, 8);           \
    c = c + d;                       \
    b = b3_rotr(b ^ c, 7);           \
  } while (0)

// One round, message words in the order m[p0..p15] as in b3_compress: column
// q takes (p[2q], p[2q+1]), diagonal q takes (p[8+2q], p[9+2q]). quad_perm
// 0x39 = [1,2,3,0] (read the lane one up), 0x4E = [2,3,0,1], 0x93 = [3,0,1,2].
#define CM_B3Q_ROUND(p0, p1, p2, p3, p4, p5, p6, p7, p8, p9, p10, p11, p12, p13, p14, p15) \
  do {                                                                                    \
    CM_B3Q_G((b3_qsel<p0, p2, p4, p6>(m, q1, q2)), (b3_qsel<p1, p3, p5, p7>(m, q1, q2)));  \
    b = b3_qperm<0x39>(b);                                                                \
    c = b3_qperm<0x4E>(c);                                                                \
    d = b3_qperm<0x93>(d);                                                                \
    CM_B3Q_G((b3_qsel<p8, p10, p12, p14>(m, q1, q2)),                                     \
             (b3_qsel<p9, p11, p13, p15>(m, q1, q2)));                                    \
    b = b3_qperm<0x93>(b);                                                                \
    c = b3_qperm<0x4E>(c);                                                                \
    d = b3_qperm<0x39>(d);                                                                \
  } while (0)

// The initial chaining words of lane q of a quad: IV[q], IV[4 + q].
__device__ __forceinline__ void b3_init_quad(uint32_t& lo, uint32_t& hi, bool q1, bool q2) {
  lo = q2 ? (q1 ? CM_B3_IV3 : CM_B3_IV2) : (q1 ? CM_B3_IV1 : CM_B3_IV0);
  hi = q2 ? (q1 ? CM_B3_IV7 : CM_B3_IV6) : (q1 ? CM_B3_IV5 : CM_B3_IV4);
}

// b3_compress on the quad's split chaining value; q1, q2: bits 0 and 1 of the
// lane's index in its quad.
__device__ __forceinline__ void b3_compress_quad(uint32_t& lo, uint32_t& hi,
                                                 const uint32_t (&m)[16], uint64_t counter,
                                                 uint32_t block_len, uint32_t flags, bool q1,
                                                 bool q2) {
  uint32_t a = lo, b = hi;
  uint32_t c = q2 ? (q1 ? CM_B3_IV3 : CM_B3_IV2) : (q1 ? CM_B3_IV1 : CM_B3_IV0);
  uint32_t d = q2 ? (q1 ? flags : block_len)
                  : (q1 ? (uint32_t)(counter >> 32) : (uint32_t)counter);
  CM_B3Q_ROUND(0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
  CM_B3Q_ROUND(2, 6, 3, 10, 7, 0, 4, 13, 1, 11, 12, 5, 9, 14, 15, 8);
  CM_B3Q_ROUND(3, 4, 10, 12, 13, 2, 7, 14, 6, 5, 9, 0, 11, 15, 8, 1);
  CM_B3Q_ROUND(10, 7, 12, 9, 14, 3, 13, 15, 4, 0, 11, 2, 5, 8, 1, 6);
  CM_B3Q_ROUND(12, 13, 9, 11, 15, 10, 14, 8, 7, 2, 5, 3, 0, 1, 6, 4);
  CM_B3Q_ROUND(9, 14, 11, 5, 8, 12, 15, 1, 13, 3, 0, 10, 2, 6, 4, 7);
  CM_B3Q_ROUND(11, 15, 5, 0, 1, 9, 8, 6, 14, 10, 2, 12, 3, 4, 7, 13);
  lo = a ^ c;
  hi = b ^ d;
}

#undef CM_B3Q_ROUND
#undef CM_B3Q_G

// b3_chunk by the four lanes of a quad: every lane loads the whole of each
// block; lane q ends with the chaining words h[q] (lo) and h[4 + q] (hi). One
// block is loaded ahead of the one compressed.
template <class LoadBlock>
__device__ __forceinline__ void b3_chunk_quad(uint32_t& lo, uint32_t& hi, int64_t nb,
                                              uint64_t chunk_index, bool root, bool q1, bool q2,
                                              LoadBlock load_block) {
  uint32_t x0[16], x1[16];
  b3_init_quad(lo, hi, q1, q2);
  load_block(0, x0);
  for (int64_t b = 0; b < nb; b += 2) {
    if (b + 1 < nb) load_block(b + 1, x1);
    b3_compress_quad(lo, hi, x0, chunk_index, 64, b3_chunk_flags(b, nb, root), q1, q2);
    if (b + 2 < nb) load_block(b + 2, x0);
    if (b + 1 < nb)
      b3_compress_quad(lo, hi, x1, chunk_index, 64, b3_chunk_flags(b + 1, nb, root), q1, q2);
  }
}

}  // namespace cm
