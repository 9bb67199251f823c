// Address arithmetic of the unit render (render.hip), callable on the host too
// so that a CPU test can walk every unit, lane and piece of a launch and check
// that each load stays inside its slot's tensor and each store inside the
// merged cache, every merged byte written once.
//
// Every row block (layer, K/V, head) of the merged cache is T_out rows of
// 2^rb_shift bytes; slot s holds rows [off_s, off_s + T_s). The launch covers
// rows [row0, T_out) in units of kRenderUnitBytes; lane l of unit x takes the
// 16-byte pieces at row-block byte (row0 << rb_shift) + x * kRenderUnitBytes +
// 16 l + 1024 k (k = 0 .. kRenderUnitPieces - 1), those below T_out rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cm {

#ifndef CM_RENDER_UNIT_PIECES
#define CM_RENDER_UNIT_PIECES 4
#endif
constexpr int kRenderUnitPieces = CM_RENDER_UNIT_PIECES;   // 16-byte pieces per lane
constexpr int kRenderUnitBytes = 1024 * kRenderUnitPieces;
constexpr int32_t kUnitCrosses = 1 << 16;                  // a slot boundary inside the unit

// Slot of the first row of unit x (offs: the slots' offsets, increasing), with
// kUnitCrosses set when a later row of the unit lies in another slot.
__host__ __device__ __forceinline__ int32_t unit_slot_code(const int64_t* offs, int n_u,
                                                           int64_t T_out, int rb_shift,
                                                           int64_t row0, int64_t x) {
  const int64_t b0 = (row0 << rb_shift) + x * kRenderUnitBytes;
  const int64_t r0 = b0 >> rb_shift;
  int64_t r1 = (b0 + kRenderUnitBytes - 1) >> rb_shift;
  r1 = r1 < T_out ? r1 : T_out - 1;
  int lo = 0, hi = n_u - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (offs[mid] <= r0) lo = mid; else hi = mid - 1;
  }
  const bool crosses = lo + 1 < n_u && offs[lo + 1] <= r1;
  return lo | (crosses ? kUnitCrosses : 0);
}

// Slot of row r of a unit whose code is `code` (r at or after the unit's first row).
__host__ __device__ __forceinline__ int unit_piece_slot(const int64_t* offs, int n_u,
                                                        int32_t code, int64_t r) {
  int s = code & (kUnitCrosses - 1);
  if (code & kUnitCrosses)
    while (s + 1 < n_u && offs[s + 1] <= r) ++s;
  return s;
}

// Byte offset, in a tensor of slot s, of the byte read for row-block byte b of
// head h: row (b >> rb_shift) - off_s of head h, same column.
__host__ __device__ __forceinline__ int64_t unit_src_offset(int64_t h, int64_t T_s, int64_t off_s,
                                                            int rb_shift, int64_t b) {
  return ((h * T_s - off_s) << rb_shift) + b;
}

}  // namespace cm
