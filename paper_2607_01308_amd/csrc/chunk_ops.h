// Device helpers of the hash kernels (hash.hip, render_hash.hip): 64-byte block
// loads, chaining-value stores, and the BLAKE3 chunk of one lane of a stripe.
#pragma once

#include "blake3.h"
#include "internal.h"

namespace cm {

__device__ __forceinline__ void load_block64(const uint8_t* p, uint32_t (&m)[16]) {
  const CM_GLOBAL u32x4* q = global_ptr<u32x4>(p);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const u32x4 v = q[k];
    m[4 * k + 0] = v[0];
    m[4 * k + 1] = v[1];
    m[4 * k + 2] = v[2];
    m[4 * k + 3] = v[3];
  }
}

__device__ __forceinline__ void store_cv(uint8_t* out, const B3Cv& s) {
  uint4* q = reinterpret_cast<uint4*>(out);
  q[0] = make_uint4(s.h[0], s.h[1], s.h[2], s.h[3]);
  q[1] = make_uint4(s.h[4], s.h[5], s.h[6], s.h[7]);
}

// Chunk `lane` of a stripe: `stripe` points at the stripe's first byte,
// stripe_blocks (<= 1024) 64-byte blocks follow; chunk k is blocks [16k, 16k+16)
// (the last may be shorter) and has BLAKE3 chunk index chunk0 + k. root: the
// tensor is this one chunk. Returns false (s untouched) for a lane past the
// last chunk.
__device__ __forceinline__ bool hash_lane_chunk(B3Cv& s, const uint8_t* stripe,
                                                int64_t stripe_blocks, int lane, uint64_t chunk0,
                                                bool root) {
  const int64_t first = (int64_t)lane * kB3ChunkBlocks;
  if (first >= stripe_blocks) return false;
  const int64_t nb =
      stripe_blocks - first < kB3ChunkBlocks ? stripe_blocks - first : kB3ChunkBlocks;
  const uint8_t* p = stripe + first * 64;
  b3_chunk(s, nb, chunk0 + (uint64_t)lane, root,
           [&](int64_t b, uint32_t (&w)[16]) { load_block64(p + b * 64, w); });
  return true;
}

}  // namespace cm
