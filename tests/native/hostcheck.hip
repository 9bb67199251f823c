// Host-side harness for CPU tests: runs the library's BLAKE3 compression code
// (paper_2607_01308_amd/csrc/blake3.h, the same source the GPU kernels use) on
// the CPU, so chunk counters, flags and parent nodes can be compared with the
// published BLAKE3 test vectors and the oracle without a GPU. Also exposes the
// compiler's single-step fp64 -> bf16 conversion that the render kernel uses.
// Test support only.
#include <stdint.h>
#include <string.h>

#include "blake3.h"

namespace {
void store(const cm::B3Cv& s, uint8_t* out) { memcpy(out, s.h, 32); }
}  // namespace

extern "C" {

// Chaining value of one BLAKE3 chunk: len a multiple of 64 in [64, 1024].
int hc_blake3_chunk(const uint8_t* data, uint64_t len, uint64_t chunk_index, int root,
                    uint8_t* out) {
  if (len == 0 || len > 1024 || (len & 63) != 0) return -1;
  cm::B3Cv s;
  cm::b3_chunk(s, (int64_t)(len >> 6), chunk_index, root != 0,
               [&](int64_t b, uint32_t (&w)[16]) { memcpy(w, data + b * 64, 64); });
  store(s, out);
  return 0;
}

// Chaining value of a parent node over two 32-byte children.
int hc_blake3_parent(const uint8_t* left, const uint8_t* right, int root, uint8_t* out) {
  cm::B3Cv l, r, p;
  memcpy(l.h, left, 32);
  memcpy(r.h, right, 32);
  cm::b3_parent(p, l, r, root != 0);
  store(p, out);
  return 0;
}

void hc_f64_to_bf16(const double* x, uint16_t* y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) {
    const __bf16 b = (__bf16)x[i];
    memcpy(&y[i], &b, 2);
  }
}

}  // extern "C"
