// Device helpers of the render kernels for the RoPE re-encode of Eq. (1)-(2):
// 16-byte pieces of K rows rotated by R(off) in fp64, then rounded once to the
// storage dtype (round-to-nearest-even). Each output element is
// fma(x, c, -(partner * s')): the partner's product is rounded to fp64, x * c
// enters the fused multiply-add exactly. Every kernel uses these helpers, so
// the dense, fused and paged renders agree bit for bit.
//
// A K row of d elements is cut into 16-byte pieces (EP = 16 / esize elements
// each, d / EP pieces per row). Half-split pairs (j, j+d/2) put piece p of
// the first half against piece p of the second half, P = d / (2 EP) pieces
// apart; interleaved pairs (2j, 2j+1) stay inside one piece.
//
// The per-slot (cos, sin) table of the render workspace is ordered so that the
// EP angles a lane needs for its piece sit P (half-split) or d / EP
// (interleaved) entries apart and the lanes of a wave that load angle e of
// consecutive pieces read consecutive entries: entry e * P + p holds pair
// j = p * EP + e (half-split); entry q * (d / EP) + c holds pair
// j = c * EP / 2 + q (interleaved).
#pragma once

#include "internal.h"
#include "stream_ops.h"

namespace cm {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__host__ __device__ __forceinline__ int angle_slot_half(int p, int e, int P) { return e * P + p; }
__host__ __device__ __forceinline__ int angle_slot_il(int c, int q, int ppr) { return q * ppr + c; }

__device__ __forceinline__ u32x4 ld16(const uint8_t* p) {
  return __builtin_nontemporal_load(global_ptr<u32x4>(p));
}

// Element e of a 16-byte piece as fp64 (exact).
template <int ESIZE>
__device__ __forceinline__ double piece_elem(const u32x4 v, int e) {
  if constexpr (ESIZE == 2) {
    const uint32_t x = v[e >> 1];
    return (double)__uint_as_float((e & 1) ? (x & 0xFFFF0000u) : (x << 16));
  } else {
    return (double)__uint_as_float(v[e]);
  }
}

// fp32 value f of an fp64 result y, nudged one ulp towards y when f sits on a
// bf16 midpoint and y does not: rounding f to bf16 (ties to even) then gives y
// rounded to bf16 in one step: every bf16 value and midpoint is an fp32
// value, so otherwise y and its fp32 rounding lie on the same side of every
// midpoint.
__device__ __forceinline__ bool on_bf16_midpoint(float f) {
  return (__float_as_uint(f) & 0xFFFFu) == 0x8000u;
}
__device__ __forceinline__ float settle_bf16(float f, double y) {
  uint32_t u = __float_as_uint(f);
  if (on_bf16_midpoint(f)) {
    const double back = (double)f;
    if (y != back) u = (fabs(y) > fabs(back)) ? u + 1u : u - 1u;
  }
  return __uint_as_float(u);
}

// Lanes of the wave whose fp32 value f sits on a bf16 midpoint: the rare
// settling below is one wave-uniform branch, taken when any lane needs it
// (settle_bf16 leaves every other value unchanged).
__device__ __forceinline__ uint64_t midpoint_lanes(float f) {
  return __builtin_amdgcn_ballot_w64(on_bf16_midpoint(f));
}

// Two fp32 values as the bf16 pair of one word (round to nearest even).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Round EP fp64 values into a 16-byte piece. bf16: fp32 rounding first is exact
// unless an fp32 result sits on a bf16 midpoint; that rare case is tested once
// for the whole piece and settled element by element. The fp32 -> bf16 step
// converts two elements per instruction.
template <int ESIZE>
__device__ __forceinline__ u32x4 round_piece(const double (&y)[16 / ESIZE]) {
  constexpr int EP = 16 / ESIZE;
  u32x4 out;
  if constexpr (ESIZE == 2) {
    float f[EP];
    uint64_t mid = 0;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      f[e] = (float)y[e];
      mid |= midpoint_lanes(f[e]);
    }
    if (__builtin_expect(mid != 0, 0)) {
#pragma unroll
      for (int e = 0; e < EP; ++e) f[e] = settle_bf16(f[e], y[e]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
  } else {
#pragma unroll
    for (int e = 0; e < EP; ++e) out[e] = __float_as_uint((float)y[e]);
  }
  return out;
}

// The words of v, opaque to the optimiser: a value computed from them again is
// recomputed, not kept alive from an earlier computation.
__device__ __forceinline__ void launder(u32x4& v) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t x = v[w];
    asm volatile("" : "+v"(x));
    v[w] = x;
  }
}

// Rotate one 16-byte piece whose pairs are (x, partner p) with the lane's fixed
// angles: y = fma(x, c, -(p s')), where s' = s in the first half of the row and
// -s in the second (p (-s) = -(p s) exactly, so both halves match
// rotate_pair_half bit for bit).
template <int ESIZE>
__device__ __forceinline__ u32x4 rotate_piece_half(const u32x4 x, const u32x4 p, const double* cs,
                                                   const double* sn) {
#pragma clang fp contract(off)
  constexpr int EP = 16 / ESIZE;
  double y[EP];
#pragma unroll
  for (int e = 0; e < EP; ++e)
    y[e] = __builtin_fma(piece_elem<ESIZE>(x, e), cs[e], -(piece_elem<ESIZE>(p, e) * sn[e]));
  return round_piece<ESIZE>(y);
}

// Rotate a first-half piece a and its second-half partner b (same column) in
// place with the angles of that column (s not sign-flipped):
// a' = fma(a, c, -(b s)), b' = fma(b, c, a s). Each result is rounded to fp32 as
// soon as it is computed; in the rare case of a bf16 midpoint the piece's fp64
// results are computed again from the inputs (same operations, same bits), so no
// fp64 result has to stay live across the test.
template <int ESIZE>
__device__ __forceinline__ void rotate_pair_half(u32x4& a, u32x4& b, const double* cs,
                                                 const double* sn) {
#pragma clang fp contract(off)
  constexpr int EP = 16 / ESIZE;
  if constexpr (ESIZE == 2) {
    float fa[EP], fb[EP];
    uint64_t mid = 0;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      const double x1 = piece_elem<ESIZE>(a, e), x2 = piece_elem<ESIZE>(b, e);
      fa[e] = (float)__builtin_fma(x1, cs[e], -(x2 * sn[e]));
      fb[e] = (float)__builtin_fma(x2, cs[e], x1 * sn[e]);
      mid |= midpoint_lanes(fa[e]) | midpoint_lanes(fb[e]);
    }
    if (__builtin_expect(mid != 0, 0)) {
      u32x4 la = a, lb = b;
      launder(la);
      launder(lb);
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        const double x1 = piece_elem<ESIZE>(la, e), x2 = piece_elem<ESIZE>(lb, e);
        fa[e] = settle_bf16(fa[e], __builtin_fma(x1, cs[e], -(x2 * sn[e])));
        fb[e] = settle_bf16(fb[e], __builtin_fma(x2, cs[e], x1 * sn[e]));
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      a[k] = pack_bf16x2(fa[2 * k], fa[2 * k + 1]);
      b[k] = pack_bf16x2(fb[2 * k], fb[2 * k + 1]);
    }
  } else {
    u32x4 ra, rb;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      const double x1 = piece_elem<ESIZE>(a, e), x2 = piece_elem<ESIZE>(b, e);
      ra[e] = __float_as_uint((float)__builtin_fma(x1, cs[e], -(x2 * sn[e])));
      rb[e] = __float_as_uint((float)__builtin_fma(x2, cs[e], x1 * sn[e]));
    }
    a = ra;
    b = rb;
  }
}

// Interleaved pairs (2q, 2q+1) inside the piece. bf16: each result is rounded
// to fp32 as soon as it is computed, and in the rare case of a bf16 midpoint
// the piece's fp64 results are computed again from the inputs (as in
// rotate_pair_half), so no fp64 result stays live across the test.
template <int ESIZE>
__device__ __forceinline__ u32x4 rotate_piece_il(const u32x4 x, const double* cs,
                                                 const double* sn) {
#pragma clang fp contract(off)
  constexpr int EP = 16 / ESIZE;
  if constexpr (ESIZE == 2) {
    float f[EP];
    uint64_t mid = 0;
#pragma unroll
    for (int q = 0; q < EP / 2; ++q) {
      const double x1 = piece_elem<ESIZE>(x, 2 * q), x2 = piece_elem<ESIZE>(x, 2 * q + 1);
      f[2 * q] = (float)__builtin_fma(x1, cs[q], -(x2 * sn[q]));
      f[2 * q + 1] = (float)__builtin_fma(x2, cs[q], x1 * sn[q]);
      mid |= midpoint_lanes(f[2 * q]) | midpoint_lanes(f[2 * q + 1]);
    }
    if (__builtin_expect(mid != 0, 0)) {
      u32x4 lx = x;
      launder(lx);
#pragma unroll
      for (int q = 0; q < EP / 2; ++q) {
        const double x1 = piece_elem<ESIZE>(lx, 2 * q), x2 = piece_elem<ESIZE>(lx, 2 * q + 1);
        f[2 * q] = settle_bf16(f[2 * q], __builtin_fma(x1, cs[q], -(x2 * sn[q])));
        f[2 * q + 1] = settle_bf16(f[2 * q + 1], __builtin_fma(x2, cs[q], x1 * sn[q]));
      }
    }
    u32x4 out;
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
    return out;
  } else {
    double y[EP];
#pragma unroll
    for (int q = 0; q < EP / 2; ++q) {
      const double x1 = piece_elem<ESIZE>(x, 2 * q), x2 = piece_elem<ESIZE>(x, 2 * q + 1);
      y[2 * q] = __builtin_fma(x1, cs[q], -(x2 * sn[q]));
      y[2 * q + 1] = __builtin_fma(x2, cs[q], x1 * sn[q]);
    }
    return round_piece<ESIZE>(y);
  }
}

// Word of the lane HB away (lane ^ HB) in the wave, without LDS traffic where
// the hardware allows: HB = 1 and 2 are quad permutations, HB = 8 a DPP rotate
// by 8 within each 16-lane row, HB = 4 and 16 a ds_swizzle xor inside 32 lanes,
// and HB = 32 a ds_bpermute. Every lane of the wave must execute it.
template <int HB>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v) {
  if constexpr (HB == 1) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
  else if constexpr (HB == 2) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
  else if constexpr (HB == 8) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false);
  else if constexpr (HB == 4 || HB == 16) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (HB << 10) | 0x1F);
  else return (uint32_t)__shfl_xor((int)v, HB, 64);
}

template <int HB>
__device__ __forceinline__ u32x4 lane_xor4(const u32x4 v) {
  u32x4 r;
#pragma unroll
  for (int w = 0; w < 4; ++w) r[w] = lane_xor<HB>(v[w]);
  return r;
}

// The lane's angles for its piece: column piece cp of a row of ppr pieces.
// Half-split: the sines of the second half carry their sign flipped (see
// rotate_piece_half). ang = the slot's table (cos, sin per entry).
template <int ESIZE, int STYLE>
__device__ __forceinline__ void piece_angles(const double* __restrict__ ang, int cp, int ppr,
                                             double* cs, double* sn) {
  constexpr int EP = 16 / ESIZE;
  if constexpr (STYLE == CM_ROPE_HALF) {
    const int P = ppr >> 1;
    const bool second = cp >= P;
    const int p = second ? cp - P : cp;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      const int k = angle_slot_half(p, e, P);
      cs[e] = ang[2 * k];
      sn[e] = second ? -ang[2 * k + 1] : ang[2 * k + 1];
    }
  } else {
#pragma unroll
    for (int q = 0; q < EP / 2; ++q) {
      const int k = angle_slot_il(cp, q, ppr);
      cs[q] = ang[2 * k];
      sn[q] = ang[2 * k + 1];
    }
  }
}

template <int S, int B>
struct Tag {
  static constexpr int style = S, hb = B;
};

// Calls go(Tag<style, HB>) with HB the lane distance of half-split partner
// pieces (pieces per row / 2) or 0 for interleaved pairs.
template <class Go>
__host__ inline void dispatch_style(int32_t style, int64_t row_bytes, Go&& go) {
  if (style == CM_ROPE_INTERLEAVED) return go(Tag<CM_ROPE_INTERLEAVED, 0>{});
  switch ((int)(row_bytes / 32)) {
    case 2: return go(Tag<CM_ROPE_HALF, 2>{});
    case 4: return go(Tag<CM_ROPE_HALF, 4>{});
    case 8: return go(Tag<CM_ROPE_HALF, 8>{});
    case 16: return go(Tag<CM_ROPE_HALF, 16>{});
    default: return go(Tag<CM_ROPE_HALF, 32>{});
  }
}

}  // namespace cm
