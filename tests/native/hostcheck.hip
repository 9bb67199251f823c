// Host-side harness for CPU tests: runs the library's BLAKE3 compression code
// (paper_2607_01308_amd/csrc/blake3.h, the same source the GPU kernels use) on
// the CPU, so chunk counters, flags and parent nodes can be compared with the
// published BLAKE3 test vectors and the oracle without a GPU; exposes the
// compiler's single-step fp64 -> bf16 conversion that the render kernel uses;
// and walks the address maps of the fused kernel on dense and on paged storage
// (fused_geometry.h) and of the unit render (render_geometry.h), the same
// sources the kernels use, over every task, unit, lane, row and piece of a
// launch. Test support only.
#include <stdint.h>
#include <string.h>

#include <vector>

#include "blake3.h"
#include "fused_geometry.h"
#include "render_geometry.h"

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

// Every (slot, tensor stripe, lane) of a fused launch over n_u slots of
// lengths T[s] at offsets off[s] (one tensor; every tensor of a slot has the
// same geometry): checks that each lane reads whole 64-byte blocks and whole
// rows inside its tensor, that the source rows of all lanes partition the
// tensor, that each row lands at merged row h * T_out + off + t (the row's
// head h and position t), and that the merged rows [0, H * T_out) are written
// exactly once. Returns the number of violations (0: the map is right).
int64_t hc_fused_check(int32_t n_u, const int64_t* T, const int64_t* off, int32_t H, int32_t rb,
                       int64_t T_out) {
  const int rb_shift = __builtin_ctz((unsigned)rb);
  std::vector<uint8_t> seen((size_t)H * (size_t)T_out, 0);
  int64_t bad = 0;
  for (int s = 0; s < n_u; ++s) {
    const int64_t bytes = (int64_t)H * T[s] * rb;
    const int64_t stripes = ((bytes >> 6) + 1023) / 1024;
    const int64_t gap = (T_out - T[s]) << rb_shift;
    int64_t covered = 0;
    for (int64_t sidx = 0; sidx < stripes; ++sidx) {
      for (int lane = 0; lane < 64; ++lane) {
        const cm::FusedLane f = cm::fused_lane(bytes, sidx, lane, rb_shift, T[s], T_out, off[s]);
        if (f.nb < 0 || f.nb > 16) { ++bad; continue; }
        if (f.nb == 0) {
          if (f.src < bytes) ++bad;              // a lane inside the tensor must own blocks
          continue;
        }
        if (f.src != (sidx * 64 + lane) * 1024 || f.src + f.nb * 64 > bytes) ++bad;
        if ((f.nb * 64) % rb != 0) ++bad;        // whole rows only
        if (f.left < 1 || f.left > T[s]) ++bad;
        int64_t dst = f.dst, left = f.left;
        const int64_t rows = (int64_t)f.nb * 64 / rb;
        for (int64_t k = 0; k < rows; ++k) {
          const int64_t r = (f.src >> rb_shift) + k;      // source row (all heads in order)
          const int64_t h = r / T[s], t = r % T[s];
          const int64_t want = (h * T_out + off[s] + t) << rb_shift;
          if (dst != want || dst < 0 || dst + rb > ((int64_t)H * T_out) << rb_shift) {
            ++bad;
          } else {
            uint8_t& c = seen[(size_t)(dst >> rb_shift)];
            if (c) ++bad;
            c = 1;
          }
          cm::fused_next_row(dst, left, T[s], gap, rb);
          ++covered;
        }
      }
    }
    if (covered != (int64_t)H * T[s]) ++bad;      // the source rows partition the tensor
  }
  for (uint8_t c : seen)
    if (!c) ++bad;
  return bad;
}

// Every (unit, lane, piece) of a unit-render launch over rows [row0, T_out) of
// n_u slots of lengths T[s] at offsets off[s]: each piece's slot must hold its
// row, its source byte must lie inside that slot's tensor for every head, and
// the pieces must cover rows [row0, T_out) of a row block exactly once.
// Returns the number of violations.
int64_t hc_unit_check(int32_t n_u, const int64_t* T, const int64_t* off, int32_t H, int32_t rb,
                      int64_t row0, int64_t T_out) {
  const int rb_shift = __builtin_ctz((unsigned)rb);
  const int64_t end = T_out << rb_shift;
  const int64_t units = ((T_out - row0) * rb + cm::kRenderUnitBytes - 1) / cm::kRenderUnitBytes;
  std::vector<uint8_t> seen((size_t)(end >> 4), 0);
  int64_t bad = 0;
  for (int64_t x = 0; x < units; ++x) {
    const int32_t code = cm::unit_slot_code(off, n_u, T_out, rb_shift, row0, x);
    for (int lane = 0; lane < 64; ++lane) {
      for (int k = 0; k < cm::kRenderUnitPieces; ++k) {
        const int64_t b = (row0 << rb_shift) + x * cm::kRenderUnitBytes + lane * 16 + 1024 * k;
        if (b >= end) continue;                   // past the merged rows: not loaded or stored
        const int64_t r = b >> rb_shift;
        const int s = cm::unit_piece_slot(off, n_u, code, r);
        if (s < 0 || s >= n_u || r < off[s] || r >= off[s] + T[s]) { ++bad; continue; }
        for (int64_t h = 0; h < H; ++h) {
          const int64_t o = cm::unit_src_offset(h, T[s], off[s], rb_shift, b);
          const int64_t want = ((h * T[s] + r - off[s]) << rb_shift) + (b & (rb - 1));
          if (o != want || o < 0 || o + 16 > ((int64_t)H * T[s]) << rb_shift) ++bad;
        }
        uint8_t& c = seen[(size_t)(b >> 4)];
        if (c) ++bad;
        c = 1;
      }
    }
  }
  for (int64_t p = 0; p < (int64_t)seen.size(); ++p)
    if (seen[(size_t)p] != (p >= ((row0 << rb_shift) >> 4) ? 1 : 0)) ++bad;
  return bad;
}

// Every (slot, tensor stripe, lane, chunk row) of a paged fused launch
// (paged_hash_render_kernel) over n_u slots of lengths T[s] at offsets off[s],
// slot s's fragment on pages blocks[first[s] ..], into the merged K (kv = 0) or
// V (kv = 1) block table tab of a pool of P pages of B = 2^b_shift rows: each
// row the lane reads must be row tr of head h of its chunk's rows (in dense
// order) at its fragment page; each row it writes must go to merged row off + tr
// of head h in the page tab[(off + tr) / B], a page that holds no fragment row;
// a row it skips must sit in the very page it is read from; and every merged
// row [0, T_out) of every head must be written or skipped exactly once, and no
// pool row written twice. Returns the number of violations.
int64_t hc_paged_fused_check(int32_t n_u, const int64_t* T, const int64_t* off,
                             const int64_t* first, const int32_t* blocks, int64_t n_blocks,
                             int32_t H, int32_t rb, int32_t b_shift, int64_t P,
                             const int32_t* tab, int64_t T_out) {
  const int rb_shift = __builtin_ctz((unsigned)rb);
  const int64_t B = (int64_t)1 << b_shift;
  const int64_t rpc = 1024 / rb;
  std::vector<uint8_t> frag_page((size_t)P, 0), seen((size_t)H * (size_t)T_out, 0);
  std::vector<uint8_t> written((size_t)(P * H * B), 0);
  for (int64_t k = 0; k < n_blocks; ++k) frag_page[(size_t)blocks[k]] = 1;
  int64_t bad = 0;
  for (int s = 0; s < n_u; ++s) {
    const int64_t bytes = (int64_t)H * T[s] * rb;
    const int64_t stripes = ((bytes >> 6) + 1023) / 1024;
    for (int64_t sidx = 0; sidx < stripes; ++sidx) {
      for (int lane = 0; lane < 64; ++lane) {
        const int64_t chunk = sidx * 64 + lane;
        const int64_t left = (bytes >> 6) - chunk * 16;
        const int64_t nb = left < 0 ? 0 : (left > 16 ? 16 : left);
        if (nb == 0) continue;
        const int64_t rows = nb * 64 / rb;        // the chunk's rows the kernel reads
        const int64_t q0 = chunk * rpc;
        cm::ChunkRow c = cm::fused_chunk_row(sidx, lane, rb_shift, T[s]);
        for (int64_t j = 0; j < rpc; ++j) {
          const int64_t q = q0 + j;
          if (j < rows) {
            // the kernel builds the entry only for rows inside the tensor
            if (q >= (int64_t)H * T[s]) { ++bad; break; }
            if (c.h != q / T[s] || c.tr != q % T[s]) { ++bad; break; }
            uint32_t src = 0, dst = 0;
            cm::paged_row_pair(blocks, first[s], tab, P, H, b_shift, off[s], c, &src, &dst);
            const int64_t page = blocks[first[s] + c.tr / B];
            if (src != (uint32_t)((page * H + c.h) * B + c.tr % B)) ++bad;
            const int64_t m = off[s] + c.tr;
            const int64_t out = tab[m / B];
            if (dst == cm::kPagedSkipRow) {
              if (out != page) ++bad;               // only a row already in place is skipped
            } else {
              if (out < 0 || out >= P || frag_page[(size_t)out]) ++bad;
              if (dst != (uint32_t)((out * H + c.h) * B + m % B)) {
                ++bad;
              } else {
                uint8_t& w = written[dst];
                if (w) ++bad;
                w = 1;
              }
            }
            uint8_t& z = seen[(size_t)(c.h * T_out + m)];
            if (z) ++bad;
            z = 1;
          }
          cm::fused_chunk_next(c, T[s]);
        }
      }
    }
  }
  for (uint8_t z : seen)
    if (!z) ++bad;
  return bad;
}

}  // extern "C"
