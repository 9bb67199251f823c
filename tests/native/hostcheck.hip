// Host-side harness for CPU tests: runs the library's BLAKE2s compression code
// (paper_2607_01308_amd/csrc/blake2s.h, the same source the GPU kernels use) on
// the CPU, so the tree parameters, counters and flags can be compared with
// Python's hashlib without a GPU. Also exposes the compiler's single-step
// fp64 -> bf16 conversion that the render kernel uses. Test support only.
#include <stdint.h>
#include <string.h>

#include "blake2s.h"

namespace {
void load64_host(const uint8_t* p, uint32_t (&m)[16]) { memcpy(m, p, 64); }
void store(const cm::B2sState& s, uint8_t* out) { memcpy(out, s.h, 32); }
}  // namespace

extern "C" {

// One tree node (leaf or parent): len must be a positive multiple of 64.
int hc_blake2s_tree_node(const uint8_t* data, uint64_t len, uint64_t node_offset,
                         uint32_t node_depth, int last_node, uint8_t* out) {
  if (len == 0 || (len & 63) != 0) return -1;
  cm::B2sState s;
  cm::b2s_init_tree(s, node_offset, node_depth);
  cm::b2s_node_aligned(s, data, len, last_node != 0,
                       [](const uint8_t* q, uint32_t (&w)[16]) { load64_host(q, w); });
  store(s, out);
  return 0;
}

// Sequential BLAKE2s-256 of a message whose length is a positive multiple of 64.
int hc_blake2s_sequential(const uint8_t* data, uint64_t len, uint8_t* out) {
  if (len == 0 || (len & 63) != 0) return -1;
  cm::B2sState s;
  cm::b2s_init_sequential(s);
  cm::b2s_node_aligned(s, data, len, false,
                       [](const uint8_t* q, uint32_t (&w)[16]) { load64_host(q, w); });
  store(s, out);
  return 0;
}

void hc_f64_to_bf16(const double* x, uint16_t* y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) {
    const __bf16 b = (__bf16)x[i];
    memcpy(&y[i], &b, 2);
  }
}

}  // extern "C"
