// Steps 1 and 4-5 in one pass: the render of Eq. (1)-(2) and, for the
// fragments whose Id is still missing, the chunk level of their hash (Id of
// Alg. 2), from the same loads.
//
// Hashing is VALU-bound (672 VALU ops per 64-byte block) and the render is
// HBM-bound; done separately they read every byte twice. Here one wave takes
// one (slot, tensor, stripe) task. A row holds 2P pieces of 16 bytes (P per
// half). At step j of a full 64 KiB stripe lane k loads four pieces of the 4 KiB
// step: f = (k / P) 2P + k % P, a first-half piece of a row in the step's first
// 2 KiB, its second-half partner f + P, and the same two in the second 2 KiB
// (each load covers whole rows' halves, 1 KiB across the wave). It compresses
// them as block j of its BLAKE3 chunk (exactly the message order of the hash)
// and writes each piece to its place in the merged cache: V and offset-0 K
// unchanged, other K rotated by R(off). Both halves of each of the lane's
// rotation pairs are in its own registers, all in one column: its cos/sin pairs
// are fixed for the task and no lane exchange is needed. A step covers whole
// rows; unless it straddles two heads its rows are consecutive in the merged
// cache too, so its stores take the same wave-uniform base plus lane offsets as
// its loads. The rest of a tensor after
// its last full stripe (under 64 KiB) is rendered by the same steps plus a short
// final step whose lanes keep whole 64-byte blocks, then its chunks are hashed
// in their own byte order from a second read (of bytes the render just pulled
// into the cache). HBM traffic is the algorithmic minimum (each byte read once,
// written once); the kernel is bound by the VALU work of the hash plus the fp64
// rotation.
#include <type_traits>

#include "chunk_ops.h"
#include "rotate.h"

namespace cm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
// Persistent grid of CUs x CM_FUSED_BLOCKS_PER_CU blocks; the register budget
// is capped so that CM_FUSED_WAVES_PER_EU waves fit on each SIMD (3 waves:
// 168 VGPRs, enough for the hash state, two 4 KiB step buffers and the angles),
// i.e. three blocks per CU at a time. Many more blocks than fit keep the end of
// the launch short: a block that starts late has few tasks (measured on the
// 4B-large whole path, blocks per CU -> kernel time: 4 -> 16.3-16.7 ms,
// 16 -> 15.6-15.7, 32 -> 15.4-15.5, 64 -> 15.5, one task per wave -> 16.3).
#ifndef CM_FUSED_BLOCKS_PER_CU
#define CM_FUSED_BLOCKS_PER_CU 32
#endif
#ifndef CM_FUSED_WAVES_PER_EU
#define CM_FUSED_WAVES_PER_EU 3
#endif
#define CM_FUSED_OCCUPANCY __attribute__((amdgpu_waves_per_eu(CM_FUSED_WAVES_PER_EU)))

// Short final step: lane owns block c of its row as 4 pieces with consecutive
// columns c*4 .. c*4+3 of a row of ppr pieces; ang = the slot's (cos, sin)
// table. Half-split: a row holds HB / 2 blocks and the partner block sits HB / 4
// lanes away (HB = 2: the row is this one block, pieces 0-1 pair with 2-3).
// Reached by every lane of the wave (cross-lane exchange).
template <int ESIZE, int STYLE, int HB>
__device__ __forceinline__ void rotate_block_tail(u32x4 (&x)[4], int c, int ppr,
                                                  const double* __restrict__ ang) {
  constexpr int EP = 16 / ESIZE;
  constexpr int NA = STYLE == CM_ROPE_HALF ? EP : EP / 2;
  u32x4 y[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    double cs[NA], sn[NA];
    piece_angles<ESIZE, STYLE>(ang, c * 4 + k, ppr, cs, sn);
    if constexpr (STYLE == CM_ROPE_INTERLEAVED) {
      y[k] = rotate_piece_il<ESIZE>(x[k], cs, sn);
    } else if constexpr (HB == 2) {
      y[k] = rotate_piece_half<ESIZE>(x[k], x[k ^ 2], cs, sn);
    } else {
      y[k] = rotate_piece_half<ESIZE>(x[k], lane_xor4<HB / 4>(x[k]), cs, sn);
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) x[k] = y[k];
}

__device__ __forceinline__ void compress_pieces(B3Cv& st, const u32x4 (&x)[4], uint64_t chunk,
                                                uint32_t flags) {
  uint32_t w[16];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int q = 0; q < 4; ++q) w[4 * k + q] = x[k][q];
  b3_compress(st, w, chunk, 64, flags);
}

// Destination of byte `rel` (0 <= rel < 4096) of a step whose first row is row
// tt of head hh of the fragment: rows past the head's end continue in the next
// head of the merged cache (only reached when a step straddles heads).
__device__ __forceinline__ uint8_t* dest_wrapped(uint8_t* out_t, int64_t hh, int64_t tt, int rel,
                                                 int rb_shift, int64_t T, int64_t T_out,
                                                 int64_t off) {
  int64_t rr = tt + (rel >> rb_shift);
  while (rr >= T) {
    rr -= T;
    ++hh;
  }
  return out_t + ((hh * T_out + off + rr) << rb_shift) + (rel & ((1 << rb_shift) - 1));
}

// HB: for half-split pairs, 16-byte pieces per half row (the short final step
// of a tensor's rest finds partner blocks HB / 4 lanes away); 0 for interleaved
// pairs.
template <int ESIZE, int STYLE, int HB>
__global__ __launch_bounds__(kThreads) CM_FUSED_OCCUPANCY void render_hash_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ task_base, const double* __restrict__ angles, int32_t H,
    int32_t d,
    const uint8_t* __restrict__ select, const int64_t* __restrict__ base0,
    uint8_t* __restrict__ nodes, uint8_t* __restrict__ out) {
  constexpr int EP = 16 / ESIZE;                   // elements per 16-byte piece
  constexpr int NA = STYLE == CM_ROPE_HALF ? EP : EP / 2;  // angle pairs per lane
  // the wave index is the same on every lane: say so, so that everything derived
  // from the task (slot, lengths, offsets, step positions, branches) stays in
  // scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int rb_shift = __builtin_ctz((unsigned)(d * ESIZE));   // log2 of the row bytes
  const int64_t row_bytes = (int64_t)1 << rb_shift;
  const int ppr = (int)(row_bytes >> 4);           // 16-byte pieces per row: 4 .. 64
  const int rps = 4096 >> rb_shift;                // rows per full step
  const int hp = ppr >> 1;                         // pieces per half row: 2 .. 32
  const int cp = lane % hp;                        // first-half column of the lane's pairs
  // byte offsets in a full step of the lane's pieces: f, f + P, f + 128, f + 128 + P
  const uint32_t pf = (uint32_t)((lane / hp) * ppr + cp) * 16;
  const uint32_t po[4] = {pf, pf + (uint32_t)hp * 16, pf + 2048, pf + (uint32_t)hp * 16 + 2048};
  const int64_t waves = (int64_t)gridDim.x * kWaves;
  // the plan and the task bases are read on the device: a plan the host has not
  // seen is rendered as it stands (its length T_out fits the output by contract)
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t T_out = plan[CM_PLAN_TOUT];
  const int64_t total_tasks = task_base[n];      // 0 for a plan whose status is an error
  for (int64_t task = (int64_t)blockIdx.x * kWaves + wave; task < total_tasks; task += waves) {
    int lo = 0, hi = n_u - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (task_base[mid] <= task) lo = mid; else hi = mid - 1;
    }
    const int s = lo;
    const int64_t i = plan[CM_PLAN_HEADER + s];
    const int64_t off = plan[CM_PLAN_HEADER + n + s];
    const int64_t T = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
    const bool hashing = select[i] == 0;
    const int64_t bytes = (int64_t)H * T * row_bytes;
    const int64_t stripes = stripes_of(bytes);
    const int64_t local = task - task_base[s];
    const int64_t t = local / stripes;             // tensor: 2l + kv
    const int64_t sidx = local - t * stripes;
    const bool rotate = (t & 1) == 0 && off != 0;
    const double* ang = angles + (int64_t)s * d;
    // the lane's angles: half-split, the pairs of column cp; interleaved, the
    // pairs inside columns cp (pieces 0, 2) and cp + P (pieces 1, 3)
    double cs[EP], sn[EP];
    if (rotate) {
      piece_angles<ESIZE, STYLE>(ang, cp, ppr, cs, sn);
      if constexpr (STYLE == CM_ROPE_INTERLEAVED)
        piece_angles<ESIZE, STYLE>(ang, cp + hp, ppr, cs + NA, sn + NA);
    }
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const int bh = (int)(in_stripe < kStripeBlocks ? in_stripe : kStripeBlocks);
    const bool full_stripe = bh == kStripeBlocks;
    const bool hash_steps = hashing && full_stripe;  // the lane's chunk is fed by the steps
    const int full_steps = bh / kStripeChunks;       // 16 in a full stripe
    const int rem = bh - full_steps * kStripeChunks; // 0 in a full stripe
    const uint8_t* src = reinterpret_cast<const uint8_t*>(table[i * stride + 1 + t]) +
                         ((sidx * kStripeBlocks) << 6);
    uint8_t* out_t = out + t * (int64_t)H * T_out * row_bytes;
    const uint64_t chunk0 = (uint64_t)sidx * kStripeChunks;
    const int64_t m = chunks_of(bytes);
    B3Cv st;
    b3_init(st);
    // first row of the current step: head hh, row tt of that head (scalars)
    int64_t hh, tt;
    {
      const int64_t r0 = ((sidx * kStripeBlocks) << 6) >> rb_shift;
      hh = r0 / T;
      tt = r0 - hh * T;
    }
    const int64_t gap = (T_out - T) << rb_shift;   // end of a head's rows -> next head
    // Store one step's output y at the current step position (head hh, row tt),
    // then move the position on by one step. WRAPS: the fragment is shorter than
    // a step (T < rows per step), so a step may span several heads.
    auto store_step = [&](auto wraps, const u32x4 (&y)[4]) {
      if constexpr (!decltype(wraps)::value) {
        // the step's rows are consecutive rows of the source and, unless the
        // step crosses the end of a head (at most one step per head; the rows
        // from `left` on then move on by `gap`), of the merged cache
        uint8_t* db = out_t + ((hh * T_out + off + tt) << rb_shift);   // wave-uniform base
        const int64_t left = T - tt;
        if (__builtin_expect(left >= rps, 1)) {
#pragma unroll
          for (int k = 0; k < 4; ++k) st_stream(db + po[k], y[k]);
        } else {
          uint8_t* db2 = db + gap;                                      // wave-uniform
#pragma unroll
          for (int k = 0; k < 4; ++k)
            st_stream(((int)(po[k] >> rb_shift) >= (int)left ? db2 : db) + po[k], y[k]);
        }
        tt += rps;
        const bool next_head = tt >= T;
        tt = next_head ? tt - T : tt;
        hh += next_head ? 1 : 0;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          st_stream(dest_wrapped(out_t, hh, tt, (int)po[k], rb_shift, T, T_out, off), y[k]);
        tt += rps;
        while (tt >= T) {
          tt -= T;
          ++hh;
        }
      }
    };
    // One full step j. x holds its data, loaded one step earlier. First the
    // wave waits for that data (the only memory operations older than it were
    // issued a step earlier too); then it stores the previous step's output,
    // which sits in nx (PENDING: there is one), and prefetches step j + 1 into
    // nx; then it hashes x into the lane's chunk and rotates x in place, which
    // leaves step j's output in x. Waiting before the stores and loads are
    // issued keeps every wait clear of memory operations issued in this step.
    auto step = [&](auto wraps, auto pending, u32x4 (&x)[4], u32x4 (&nx)[4], int j) {
#pragma unroll
      for (int k = 0; k < 4; ++k) launder(x[k]);   // wait for x here, before the stores
      if constexpr (decltype(pending)::value) store_step(wraps, nx);
      // the last step loads itself again: the loads stay unconditional, which
      // keeps the count of memory operations the same on every path
      const int jn = j + 1 < full_steps ? j + 1 : j;
      const uint8_t* sb = src + ((int64_t)jn << 12);     // wave-uniform base
#pragma unroll
      for (int k = 0; k < 4; ++k) nx[k] = ld16(sb + po[k]);
      if (hash_steps) compress_pieces(st, x, chunk0 + lane, b3_chunk_flags(j, full_steps, false));
      if (rotate) {
        if constexpr (STYLE == CM_ROPE_HALF) {
          rotate_pair_half<ESIZE>(x[0], x[1], cs, sn);
          rotate_pair_half<ESIZE>(x[2], x[3], cs, sn);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            x[k] = rotate_piece_il<ESIZE>(x[k], cs + (k & 1) * NA, sn + (k & 1) * NA);
        }
      }
    };
    // Software pipeline over the full steps, two buffers; the last step's
    // output is stored after the loop.
    auto run = [&](auto wraps) {
      u32x4 bufa[4], bufb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) bufa[k] = ld16(src + po[k]);
      step(wraps, std::false_type{}, bufa, bufb, 0);
      int j = 1;
      while (j + 1 < full_steps) {
        step(wraps, std::true_type{}, bufb, bufa, j);
        step(wraps, std::true_type{}, bufa, bufb, j + 1);
        j += 2;
      }
      if (j < full_steps) {
        step(wraps, std::true_type{}, bufb, bufa, j);
        store_step(wraps, bufb);
      } else {
        store_step(wraps, bufa);
      }
    };
    if (full_steps > 0) {
      if (T >= rps) run(std::false_type{});
      else run(std::true_type{});
    }
    if (rem > 0) {
      // short final step: lane < rem owns block `lane` whole (4 consecutive pieces)
      const uint8_t* sp = src + ((int64_t)full_steps << 12) + lane * 64;
      u32x4 x[4] = {};
      if (lane < rem) {
#pragma unroll
        for (int k = 0; k < 4; ++k) x[k] = ld16(sp + 16 * k);
      }
      const int cb = (int)(((lane * 64) & (row_bytes - 1)) >> 6);   // block of the row
      if (rotate) rotate_block_tail<ESIZE, STYLE, HB>(x, cb, ppr, ang);
      if (lane < rem) {
        uint8_t* dp = dest_wrapped(out_t, hh, tt, lane * 64, rb_shift, T, T_out, off);
#pragma unroll
        for (int k = 0; k < 4; ++k) st_stream(dp + 16 * k, x[k]);
      }
    }
    if (hashing) {
      uint8_t* node = nodes + (base0[i] + t * m + (int64_t)chunk0 + lane) * 32;
      if (full_stripe) {
        store_cv(node, st);
      } else {
        // the rest of the tensor: chunk `lane` is 1 KiB of consecutive bytes
        B3Cv rs;
        if (hash_rest_chunk(rs, src, bh, lane, chunk0, m == 1)) store_cv(node, rs);
      }
    }
  }
}

}  // namespace

hipError_t launch_render_hash(const SetDesc& s, const HashLayout& hlay, const RenderLayout& rlay,
                              const int64_t* plan_dev, double base, int32_t style,
                              const uint8_t* select, uint8_t* digests, void* out, uint8_t* ws,
                              hipStream_t stream, bool tables_ready, bool prep_ready) {
  uint8_t* hws = ws;
  uint8_t* rws = ws + align_up(hlay.bytes, kWsAlign);
  hipError_t e = hipSuccess;
  if (!tables_ready && (e = launch_hash_prep(s, hlay, hws, stream)) != hipSuccess) return e;
  if (!prep_ready && (e = launch_render_prep(s, rlay, plan_dev, s.n, base, style,
                                             (int32_t)kStripeBlocks, select, rws, stream)) !=
                         hipSuccess)
    return e;
  const uint8_t* hsel = rws + rlay.off_hsel;  // 0: slot delivery whose Id is computed here
  {
    const int64_t* base_tab = reinterpret_cast<const int64_t*>(hws + hlay.off_tables);
    const int64_t* tasks = reinterpret_cast<const int64_t*>(rws + rlay.off_tiles);
    const double* angles = reinterpret_cast<const double*>(rws + rlay.off_angles);
    // the task count is known on the device only: a persistent grid of a few
    // workgroups per CU strides over it
    const dim3 grid((uint32_t)(device_cu_count() * CM_FUSED_BLOCKS_PER_CU));
    ScopedTiming tm(K_RENDER_HASH, stream);
    uint8_t* nodes = hws + hlay.off_buf0;
    uint8_t* o = reinterpret_cast<uint8_t*>(out);
    auto go = [&](auto tag) {
      constexpr int STYLE = decltype(tag)::style, HB = decltype(tag)::hb;
      if (s.esize == 2)
        hipLaunchKernelGGL((render_hash_kernel<2, STYLE, HB>), grid, dim3(kThreads), 0, stream,
                           s.table_dev, s.stride, s.n, plan_dev, tasks, angles, s.H, s.d, hsel,
                           base_tab, nodes, o);
      else
        hipLaunchKernelGGL((render_hash_kernel<4, STYLE, HB>), grid, dim3(kThreads), 0, stream,
                           s.table_dev, s.stride, s.n, plan_dev, tasks, angles, s.H, s.d, hsel,
                           base_tab, nodes, o);
    };
    dispatch_style(style, s.row_bytes, go);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, hlay, hsel, 0, digests, hws, stream);
}

}  // namespace cm
