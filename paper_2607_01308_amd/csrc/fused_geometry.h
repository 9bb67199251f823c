// Address arithmetic of the fused hash + render (render_hash.hip), callable on
// the host too so that a CPU test can walk every task, lane and block of a
// launch and check that each load stays inside its tensor and each store
// inside the merged cache, every output byte written once.
//
// A task is one (slot, tensor, stripe): the slot's fragment has 2L tensors of
// H * T rows of RB bytes (rows of all heads in order); a stripe is 64
// consecutive BLAKE3 chunks of 1 KiB, lane k owning chunk k of the stripe,
// i.e. RPC = 1024 / RB whole rows. The merged cache holds, per tensor, H row
// blocks of T_out rows; the slot's rows [0, T) of head h go to rows
// [off, off + T) of row block h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cm {

// Slot of task `task`: the largest s in [0, n_u) with task_base[s] <= task
// (task bases strictly increase over the slots).
__host__ __device__ __forceinline__ int fused_slot(const int64_t* __restrict__ task_base, int n_u,
                                                   int64_t task) {
  int lo = 0, hi = n_u - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (task_base[mid] <= task) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Where one lane of a task reads and writes.
struct FusedLane {
  int64_t src;    // byte offset of the lane's chunk in its tensor
  int nb;         // 64-byte blocks of the chunk (0 past the tensor's end)
  int64_t dst;    // byte offset, in the tensor's part of the merged cache, of the current row
  int64_t left;   // rows of the current head from the current row on (>= 1)
};

// Lane `lane` of stripe sidx of a tensor of `bytes` = H * T * RB bytes.
// rb_shift = log2(RB); rows per chunk = 1024 >> rb_shift.
__host__ __device__ __forceinline__ FusedLane fused_lane(int64_t bytes, int64_t sidx, int lane,
                                                         int rb_shift, int64_t T, int64_t T_out,
                                                         int64_t off) {
  FusedLane f;
  const int64_t rpc = (int64_t)1024 >> rb_shift;
  const int64_t chunk = sidx * 64 + lane;
  f.src = chunk << 10;
  const int64_t blocks = (bytes >> 6) - chunk * 16;
  f.nb = blocks < 0 ? 0 : (blocks > 16 ? 16 : (int)blocks);
  // first row: row r0 + lane * rpc of the tensor, head h, row tt of that head
  const int64_t r0 = sidx * 64 * rpc;
  const int64_t h0 = r0 / T;
  const int64_t rel = r0 - h0 * T + (int64_t)lane * rpc;
  int64_t dh;
  if (T > 64 * rpc) dh = rel >= T ? 1 : 0;           // rel < 2T
  else dh = (int64_t)((uint32_t)rel / (uint32_t)T);  // rel < 2048
  const int64_t tt = rel - dh * T;
  f.dst = ((h0 + dh) * T_out + off + tt) << rb_shift;
  f.left = T - tt;
  return f;
}

// Move a lane on to its next row: the next row of the head, or row `off` of
// the next head's row block (gap = (T_out - T) rows further on). P: a byte
// offset or a byte pointer.
template <class P>
__host__ __device__ __forceinline__ void fused_next_row(P& dst, int64_t& left, int64_t T,
                                                        int64_t gap_bytes, int rb) {
  --left;
  const bool wrap = left == 0;
  dst += rb + (wrap ? gap_bytes : 0);
  left = wrap ? T : left;
}


// Paged storage: a pool [L][2][P][H][B][RB] of pages of B rows of every head,
// fragment row tr of head h in row tr % B of page blocks[first + tr / B]. The
// paged fused kernel names a pool row by its index in the (layer, K/V) slice of
// the pool, (page * H + h) * B + row (the caller keeps P * H * B below 2^32 - 1),
// so that a row is 4 bytes of a wave's LDS table.
constexpr uint32_t kPagedSkipRow = 0xFFFFFFFFu;   // a row that is not written

struct ChunkRow {
  int64_t h;    // head
  int64_t tr;   // row of that head, in [0, T)
};

// Head and row of the first row of lane `lane`'s chunk in stripe sidx of a
// tensor of H * T rows of 2^rb_shift bytes (the chunk's row 0; it exists when
// the lane's chunk holds at least one block).
__host__ __device__ __forceinline__ ChunkRow fused_chunk_row(int64_t sidx, int lane, int rb_shift,
                                                             int64_t T) {
  const int64_t rpc = (int64_t)1024 >> rb_shift;
  const int64_t r0 = sidx * 64 * rpc;
  const int64_t h0 = r0 / T;
  const int64_t rel = r0 - h0 * T + (int64_t)lane * rpc;
  int64_t dh;
  if (T > 64 * rpc) dh = rel >= T ? 1 : 0;           // rel < 2T
  else dh = (int64_t)((uint32_t)rel / (uint32_t)T);  // rel < 2048
  ChunkRow c;
  c.h = h0 + dh;
  c.tr = rel - dh * T;
  return c;
}

__host__ __device__ __forceinline__ void fused_chunk_next(ChunkRow& c, int64_t T) {
  if (++c.tr == T) {
    c.tr = 0;
    ++c.h;
  }
}

// Pool rows of row c of a slot at merged offset `off` whose fragment's page
// list starts at blocks[first]: where it is read (*src) and where the merged
// cache holds it (*dst: row off + tr of head h, in page tab[(off + tr) / B] of
// the merged K or V block table), or kPagedSkipRow for a row whose merged page
// is the page it is read from (a reused page: its bytes are already in place)
// or not a page of the pool.
__host__ __device__ __forceinline__ void paged_row_pair(const int32_t* blocks, int64_t first,
                                                        const int32_t* tab, int64_t P, int64_t H,
                                                        int b_shift, int64_t off, ChunkRow c,
                                                        uint32_t* src, uint32_t* dst) {
  const int64_t bmask = ((int64_t)1 << b_shift) - 1;
  const int64_t page = blocks[first + (c.tr >> b_shift)];
  *src = (uint32_t)(((page * H + c.h) << b_shift) + (c.tr & bmask));
  const int64_t m = off + c.tr;
  const int64_t out = tab[m >> b_shift];
  *dst = (out == page || out < 0 || out >= P) ? kPagedSkipRow
                                              : (uint32_t)(((out * H + c.h) << b_shift) + (m & bmask));
}

}  // namespace cm
