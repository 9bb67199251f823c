// Steps 1 and 4-5 in one pass: the render of Eq. (1)-(2) and, for the
// fragments whose Id is still missing, the leaf level of their hash tree (Id
// of Alg. 2), from the same loads.
//
// Hashing is VALU-bound (960 VALU ops per 64-byte block) and the render is
// HBM-bound; done separately they read every byte twice. Here one wave takes
// one (slot, tensor, stripe) task. At full step j of the 256 KiB stripe every
// lane loads the 16-byte pieces lane, lane+64, lane+128, lane+192 of the 4 KiB
// step (four loads, each 1 KiB contiguous across the wave), compresses them as
// one 64-byte block into its leaf (exactly the leaf layout of the tree) and
// writes each piece to its place in the merged cache: V and offset-0 K
// unchanged, other K rotated by R(off). A row holds row_bytes / 16 pieces and
// 64 is a multiple of that, so all four pieces of a lane sit in the same column
// of their rows: the lane's cos/sin pairs are fixed for the task (registers),
// and the other half of its pairs is in lane ^ (pieces per row / 2) (one
// cross-lane move, chosen at compile time). A step covers whole rows; unless it
// straddles two heads its rows are consecutive in the merged cache too, so its
// stores take the same wave-uniform base plus lane offsets as its loads. The
// short final step of a stripe, if any, keeps whole 64-byte blocks per lane and
// reads its angles from memory. HBM traffic is the
// algorithmic minimum (each byte read once, written once); the kernel is bound
// by the VALU work of the hash plus the fp64 rotation.
#include <type_traits>

#include "blake2s.h"
#include "internal.h"
#include "stream_ops.h"

namespace cm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
// Persistent grid of CUs x CM_FUSED_BLOCKS_PER_CU blocks; the register budget
// is capped so that CM_FUSED_WAVES_PER_EU waves fit on each SIMD (3 waves:
// 168 VGPRs, enough for the hash state, two 4 KiB step buffers and the angles).
#ifndef CM_FUSED_BLOCKS_PER_CU
#define CM_FUSED_BLOCKS_PER_CU 4
#endif
#ifndef CM_FUSED_WAVES_PER_EU
#define CM_FUSED_WAVES_PER_EU 3
#endif
#define CM_FUSED_OCCUPANCY __attribute__((amdgpu_waves_per_eu(CM_FUSED_WAVES_PER_EU)))

template <int S, int B>
struct Tag {
  static constexpr int style = S, hb = B;
};

__device__ __forceinline__ u32x4 ld16(const uint8_t* p) {
  return __builtin_nontemporal_load(global_ptr<u32x4>(p));
}

// Element e of a 16-byte piece as fp64.
template <int ESIZE>
__device__ __forceinline__ double piece_elem(const u32x4 v, int e) {
  if constexpr (ESIZE == 2) {
    const uint32_t x = v[e >> 1];
    return (double)__uint_as_float((e & 1) ? (x & 0xFFFF0000u) : (x << 16));
  } else {
    return (double)__uint_as_float(v[e]);
  }
}

template <int ESIZE>
__device__ __forceinline__ void piece_put(u32x4& y, int e, uint32_t bits) {
  if constexpr (ESIZE == 2) {
    if (e & 1) y[e >> 1] |= bits << 16;
    else y[e >> 1] = bits;
  } else {
    y[e] = bits;
  }
}

// Round EP fp64 values into a 16-byte piece. bf16: fp32 rounding first is exact
// unless an fp32 result sits on a bf16 midpoint (see bf16_bits_rne); that rare
// case is tested once for the whole piece and settled element by element.
template <int ESIZE>
__device__ __forceinline__ u32x4 round_piece(const double (&y)[16 / ESIZE]) {
  constexpr int EP = 16 / ESIZE;
  u32x4 out;
  if constexpr (ESIZE == 2) {
    float f[EP];
    bool mid = false;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      f[e] = (float)y[e];
      mid |= (__float_as_uint(f[e]) & 0xFFFFu) == 0x8000u;
    }
    if (__builtin_expect(mid, 0)) {
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        uint32_t u = __float_as_uint(f[e]);
        if ((u & 0xFFFFu) == 0x8000u) {
          const double back = (double)f[e];
          if (y[e] != back) u = (fabs(y[e]) > fabs(back)) ? u + 1u : u - 1u;
        }
        f[e] = __uint_as_float(u);
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t lo = __builtin_bit_cast(uint16_t, (__bf16)f[2 * k]);
      const uint32_t hi = __builtin_bit_cast(uint16_t, (__bf16)f[2 * k + 1]);
      out[k] = lo | (hi << 16);
    }
  } else {
#pragma unroll
    for (int e = 0; e < EP; ++e) out[e] = __float_as_uint((float)y[e]);
  }
  return out;
}

// Rotate one 16-byte piece whose pairs are (x, partner p) with the lane's fixed
// angles: y = x c - p s', where s' = s in the first half of the row and -s in
// the second (x c - p (-s) = x c + p s, bit for bit).
template <int ESIZE>
__device__ __forceinline__ u32x4 rotate_piece_half(const u32x4 x, const u32x4 p, const double* cs,
                                                   const double* sn) {
#pragma clang fp contract(off)
  constexpr int EP = 16 / ESIZE;
  double y[EP];
#pragma unroll
  for (int e = 0; e < EP; ++e)
    y[e] = piece_elem<ESIZE>(x, e) * cs[e] - piece_elem<ESIZE>(p, e) * sn[e];
  return round_piece<ESIZE>(y);
}

// Interleaved pairs (2j, 2j+1) inside the piece.
template <int ESIZE>
__device__ __forceinline__ u32x4 rotate_piece_il(const u32x4 x, const double* cs,
                                                 const double* sn) {
#pragma clang fp contract(off)
  constexpr int EP = 16 / ESIZE;
  double y[EP];
#pragma unroll
  for (int q = 0; q < EP / 2; ++q) {
    const double x1 = piece_elem<ESIZE>(x, 2 * q), x2 = piece_elem<ESIZE>(x, 2 * q + 1);
    y[2 * q] = x1 * cs[q] - x2 * sn[q];
    y[2 * q + 1] = x2 * cs[q] + x1 * sn[q];
  }
  return round_piece<ESIZE>(y);
}

// Word of the lane HB away (lane ^ HB) in the wave, without LDS traffic where
// the hardware allows: HB = 1 and 2 are quad permutations, HB = 8 a DPP rotate by 8
// within each 16-lane row, HB = 4 and 16 a ds_swizzle xor inside 32 lanes, and
// HB = 32 a ds_bpermute.
template <int HB>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v) {
  if constexpr (HB == 1) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
  else if constexpr (HB == 2) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
  else if constexpr (HB == 8) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false);
  else if constexpr (HB == 4 || HB == 16) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (HB << 10) | 0x1F);
  else return (uint32_t)__shfl_xor((int)v, HB, 64);
}

// Short final step: lane owns block c of its row as 4 pieces with consecutive
// columns; ang = the slot's (cos, sin) table in global memory. A row holds
// HB / 2 blocks (half-split pairs: the partner block c ^ (HB / 4) sits HB / 4
// lanes away). Reached by every lane of the wave (cross-lane exchange).
template <int ESIZE, int STYLE, int HB>
__device__ __forceinline__ void rotate_block_tail(u32x4 (&x)[4], int c,
                                                  const double* __restrict__ ang) {
#pragma clang fp contract(off)
  constexpr int EP = 16 / ESIZE;
  if constexpr (STYLE == CM_ROPE_INTERLEAVED) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int j0 = (c * 4 + k) * (EP / 2);
      double cs[EP / 2], sn[EP / 2];
#pragma unroll
      for (int q = 0; q < EP / 2; ++q) {
        cs[q] = ang[2 * (j0 + q)];
        sn[q] = ang[2 * (j0 + q) + 1];
      }
      x[k] = rotate_piece_il<ESIZE>(x[k], cs, sn);
    }
  } else if constexpr (HB == 2) {
    // the whole row is this block: pieces 0-1 pair with pieces 2-3
    u32x4 y[4];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      double cs[EP], sn[EP], nsn[EP];
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        cs[e] = ang[2 * (k * EP + e)];
        sn[e] = ang[2 * (k * EP + e) + 1];
        nsn[e] = -sn[e];
      }
      y[k] = rotate_piece_half<ESIZE>(x[k], x[k + 2], cs, sn);
      y[k + 2] = rotate_piece_half<ESIZE>(x[k + 2], x[k], cs, nsn);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) x[k] = y[k];
  } else {
    constexpr int hb = HB / 4;
    const bool second = c >= hb;
    const int cb = second ? c - hb : c;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      u32x4 p;
#pragma unroll
      for (int w = 0; w < 4; ++w) p[w] = lane_xor<hb>(x[k][w]);
      const int j0 = (cb * 4 + k) * EP;
      double cs[EP], sn[EP];
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        cs[e] = ang[2 * (j0 + e)];
        sn[e] = second ? -ang[2 * (j0 + e) + 1] : ang[2 * (j0 + e) + 1];
      }
      x[k] = rotate_piece_half<ESIZE>(x[k], p, cs, sn);
    }
  }
}

__device__ __forceinline__ void compress_pieces(B2sState& st, const u32x4 (&x)[4], uint64_t count,
                                                bool last, bool last_node) {
  uint32_t w[16];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int q = 0; q < 4; ++q) w[4 * k + q] = x[k][q];
  b2s_compress(st, w, count, last, last_node);
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

// HB: for half-split pairs, the lane distance between a piece and its partner
// piece in full steps (16-byte pieces per row / 2); 0 for interleaved pairs.
template <int ESIZE, int STYLE, int HB>
__global__ __launch_bounds__(kThreads) CM_FUSED_OCCUPANCY void render_hash_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ task_base, int32_t n_u, int64_t total_tasks,
    const double* __restrict__ angles, int32_t H, int32_t d, int64_t T_out,
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
  const int cp = lane & (ppr - 1);                 // column piece of this lane (full steps)
  const bool second = STYLE == CM_ROPE_HALF && cp >= (ppr >> 1);
  const int64_t waves = (int64_t)gridDim.x * kWaves;
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
    double cs[NA], sn[NA];
    if (rotate) {
      const int j0 = STYLE == CM_ROPE_HALF ? (second ? cp - (ppr >> 1) : cp) * EP : cp * (EP / 2);
#pragma unroll
      for (int e = 0; e < NA; ++e) {
        cs[e] = ang[2 * (j0 + e)];
        sn[e] = second ? -ang[2 * (j0 + e) + 1] : ang[2 * (j0 + e) + 1];
      }
    }
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const int bh = (int)(in_stripe < kStripeBlocks ? in_stripe : kStripeBlocks);
    const int full_steps = bh / kStripeLeaves;
    const int rem = bh - full_steps * kStripeLeaves;
    const int nb = full_steps + (lane < rem ? 1 : 0);
    const uint8_t* src = reinterpret_cast<const uint8_t*>(table[i * stride + 1 + t]) +
                         ((sidx * kStripeBlocks) << 6);
    uint8_t* out_t = out + t * (int64_t)H * T_out * row_bytes;
    const int64_t leaf = sidx * kStripeLeaves + lane;
    const int64_t m = leaves_of(bytes);
    B2sState st;
    b2s_init_tree(st, (uint64_t)leaf, 0);
    // first row of the current step: head hh, row tt of that head (scalars)
    int64_t hh, tt;
    {
      const int64_t r0 = ((sidx * kStripeBlocks) << 6) >> rb_shift;
      hh = r0 / T;
      tt = r0 - hh * T;
    }
    const int64_t gap = (T_out - T) << rb_shift;   // end of a head's rows -> next head
    // One full step: prefetch the next one, hash this one into the lane's leaf,
    // rotate it if needed, store it. WRAPS: the fragment is shorter than a step
    // (T < rows per step), so a step may span several heads.
    auto step = [&](auto wraps, const u32x4 (&x)[4], u32x4 (&nx)[4], int j) {
      // the last step loads itself again: the loads stay unconditional, which
      // keeps the count of memory operations the same on every path
      const int jn = j + 1 < full_steps ? j + 1 : j;
      const uint8_t* sb = src + ((int64_t)jn << 12);     // wave-uniform base
#pragma unroll
      for (int k = 0; k < 4; ++k) nx[k] = ld16(sb + (uint32_t)(lane * 16 + k * 1024));
      if (hashing) compress_pieces(st, x, (uint64_t)(j + 1) << 6, j + 1 == nb,
                                   j + 1 == nb && leaf == m - 1);
      u32x4 y[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        y[k] = x[k];
        if (rotate) {
          if constexpr (STYLE == CM_ROPE_HALF) {
            u32x4 p;
#pragma unroll
            for (int w = 0; w < 4; ++w) p[w] = lane_xor<HB>(x[k][w]);
            y[k] = rotate_piece_half<ESIZE>(x[k], p, cs, sn);
          } else {
            y[k] = rotate_piece_il<ESIZE>(x[k], cs, sn);
          }
        }
      }
      if constexpr (!decltype(wraps)::value) {
        // the step's rows are consecutive rows of the source and, up to one head
        // change (branch-free: the rows from `left` on move on by `gap`), of the
        // merged cache
        uint8_t* db = out_t + ((hh * T_out + off + tt) << rb_shift);   // wave-uniform base
        const int64_t left = T - tt;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t rel = (uint32_t)(lane * 16 + k * 1024);
          st_stream(db + rel + ((int64_t)(rel >> rb_shift) >= left ? gap : 0), y[k]);
        }
        tt += rps;
        const bool next_head = tt >= T;
        tt = next_head ? tt - T : tt;
        hh += next_head ? 1 : 0;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          st_stream(dest_wrapped(out_t, hh, tt, lane * 16 + k * 1024, rb_shift, T, T_out, off),
                    y[k]);
        tt += rps;
        while (tt >= T) {
          tt -= T;
          ++hh;
        }
      }
    };
    // Software pipeline over the full steps, two buffers. The first step is
    // peeled so that the loop is entered with the same operations in flight as
    // on its back edge (this step's loads, the previous stores): the wait for
    // a step's data then never covers the stores just issued.
    auto run = [&](auto wraps) {
      u32x4 bufa[4], bufb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) bufa[k] = ld16(src + (uint32_t)(lane * 16 + k * 1024));
      step(wraps, bufa, bufb, 0);
      int j = 1;
      while (j + 1 < full_steps) {
        step(wraps, bufb, bufa, j);
        step(wraps, bufa, bufb, j + 1);
        j += 2;
      }
      if (j < full_steps) step(wraps, bufb, bufa, j);
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
        if (hashing) compress_pieces(st, x, (uint64_t)nb << 6, true, leaf == m - 1);
      }
      const int cb = (int)(((lane * 64) & (row_bytes - 1)) >> 6);   // block of the row
      if (rotate) rotate_block_tail<ESIZE, STYLE, HB>(x, cb, ang);
      if (lane < rem) {
        uint8_t* dp = dest_wrapped(out_t, hh, tt, lane * 64, rb_shift, T, T_out, off);
#pragma unroll
        for (int k = 0; k < 4; ++k) st_stream(dp + 16 * k, x[k]);
      }
    }
    if (hashing && nb > 0) {
      uint4* q = reinterpret_cast<uint4*>(nodes + (base0[i] + t * m + leaf) * 32);
      q[0] = make_uint4(st.h[0], st.h[1], st.h[2], st.h[3]);
      q[1] = make_uint4(st.h[4], st.h[5], st.h[6], st.h[7]);
    }
  }
}

template <int ESIZE, int STYLE, int HB>
void launch_fused(dim3 grid, hipStream_t stream, const SetDesc& s, const int64_t* plan_dev,
                  const int64_t* tasks, int32_t n_unique, int64_t total_tasks,
                  const double* angles, int64_t T_out, const uint8_t* hsel,
                  const int64_t* base_tab, uint8_t* nodes, uint8_t* o) {
  hipLaunchKernelGGL((render_hash_kernel<ESIZE, STYLE, HB>), grid, dim3(kThreads), 0, stream,
                     s.table_dev, s.stride, s.n, plan_dev, tasks, n_unique, total_tasks, angles,
                     s.H, s.d, T_out, hsel, base_tab, nodes, o);
}

template <int ESIZE>
void launch_fused_es(int32_t style, dim3 grid, hipStream_t stream, const SetDesc& s,
                     const int64_t* plan_dev, const int64_t* tasks, int32_t n_unique,
                     int64_t total_tasks, const double* angles, int64_t T_out,
                     const uint8_t* hsel, const int64_t* base_tab, uint8_t* nodes, uint8_t* o) {
  auto go = [&](auto kernel_tag) {
    constexpr int STYLE = decltype(kernel_tag)::style, HB = decltype(kernel_tag)::hb;
    launch_fused<ESIZE, STYLE, HB>(grid, stream, s, plan_dev, tasks, n_unique, total_tasks,
                                   angles, T_out, hsel, base_tab, nodes, o);
  };
  if (style == CM_ROPE_INTERLEAVED) return go(Tag<CM_ROPE_INTERLEAVED, 0>{});
  switch ((int)(s.d * s.esize / 32)) {   // pieces per row / 2
    case 2: return go(Tag<CM_ROPE_HALF, 2>{});
    case 4: return go(Tag<CM_ROPE_HALF, 4>{});
    case 8: return go(Tag<CM_ROPE_HALF, 8>{});
    case 16: return go(Tag<CM_ROPE_HALF, 16>{});
    default: return go(Tag<CM_ROPE_HALF, 32>{});
  }
}

}  // namespace

int64_t render_hash_tasks(const SetDesc& s, const int64_t* plan_host) {
  const int64_t nu = plan_host[CM_PLAN_NUNIQUE];
  int64_t tasks = 0;
  for (int64_t k = 0; k < nu; ++k) {
    const int64_t len = plan_host[CM_PLAN_HEADER + 2 * (int64_t)s.n + k];
    tasks += 2 * (int64_t)s.L * stripes_of(len * token_bytes_of(s));
  }
  return tasks;
}

hipError_t launch_render_hash(const SetDesc& s, const HashLayout& hlay, const RenderLayout& rlay,
                              const int64_t* plan_dev, int32_t n_unique, int64_t total_tasks,
                              int64_t T_out, double base, int32_t style, const uint8_t* select,
                              uint8_t* digests, void* out, uint8_t* ws, hipStream_t stream) {
  uint8_t* hws = ws;
  uint8_t* rws = ws + align_up(hlay.bytes, kWsAlign);
  hipError_t e = launch_hash_prep(s, hlay, hws, stream);
  if (e != hipSuccess) return e;
  if ((e = launch_render_prep(s, rlay, plan_dev, n_unique, base, /*stripe_tasks=*/true, select,
                              rws, stream)) != hipSuccess)
    return e;
  const uint8_t* hsel = rws + rlay.off_hsel;  // 0: slot delivery whose Id is computed here
  {
    const int64_t* base_tab = reinterpret_cast<const int64_t*>(hws + hlay.off_tables);
    const int64_t* tasks = reinterpret_cast<const int64_t*>(rws + rlay.off_tiles);
    const double* angles = reinterpret_cast<const double*>(rws + rlay.off_angles);
    const int64_t full = (total_tasks + kWaves - 1) / kWaves;
    const int64_t cap = (int64_t)device_cu_count() * CM_FUSED_BLOCKS_PER_CU;
    const dim3 grid((uint32_t)(full < cap ? full : cap));
    ScopedTiming tm(K_RENDER_HASH, stream);
    uint8_t* nodes = hws + hlay.off_buf0;
    uint8_t* o = reinterpret_cast<uint8_t*>(out);
    if (s.esize == 2)
      launch_fused_es<2>(style, grid, stream, s, plan_dev, tasks, n_unique, total_tasks, angles,
                         T_out, hsel, base_tab, nodes, o);
    else
      launch_fused_es<4>(style, grid, stream, s, plan_dev, tasks, n_unique, total_tasks, angles,
                         T_out, hsel, base_tab, nodes, o);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, hlay, hsel, 0, digests, hws, stream);
}

}  // namespace cm
