// Device helpers of the render kernels for the RoPE re-encode of Eq. (1)-(2):
// a 16-byte piece of a K row rotated by R(off), in fp64 with the two products
// and the add/subtract rounded separately, then rounded once to the storage
// dtype (round-to-nearest-even).
//
// A K row of d elements is cut into 16-byte pieces (EP = 16 / esize elements
// each, d / EP pieces per row). Half-split pairs (j, j + d/2) put piece p of
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

// Round EP fp64 values into a 16-byte piece. bf16: fp32 rounding first is exact
// unless an fp32 result sits on a bf16 midpoint (see bf16_bits_rne); that rare
// case is tested once for the whole piece and settled element by element. The
// fp32 -> bf16 step converts two elements per instruction.
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
      const f32x2 v = {f[2 * k], f[2 * k + 1]};
      out[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
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

// Interleaved pairs (2q, 2q+1) inside the piece.
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
