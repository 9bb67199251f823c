// The last levels of the score tree (Eq. (3)) inside a one-workgroup kernel
// that needs the keys next (the order, the key mask), so the path spends no
// launch on them. The levels below are the knorm kernels'; the summation order
// is the same level-wise adjacent-pair tree, so the keys are bit-identical to a
// full tree of launches.
#pragma once

#include "internal.h"

namespace cm {

// Sum of squares of one 16-byte piece of a row (8 bf16 or 4 fp32 elements) by a
// fixed pair tree; the squares are exact in fp64.
template <int ESIZE>
__device__ __forceinline__ double row_chunk_sumsq(const u32x4 v) {
  const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
  if constexpr (ESIZE == 2) {
    double e[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const double lo = (double)__uint_as_float(w[k] << 16);
      const double hi = (double)__uint_as_float(w[k] & 0xFFFF0000u);
      e[2 * k] = lo * lo;
      e[2 * k + 1] = hi * hi;
    }
    return ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
  } else {
    double e[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const double x = (double)__uint_as_float(w[k]);
      e[k] = x * x;
    }
    return (e[0] + e[1]) + (e[2] + e[3]);
  }
}

// The fold's LDS: one pair of arrays per kernel, whichever entry point fills it.
__device__ __forceinline__ double* knorm_lds_a() {
  __shared__ double fa[kKnormFoldMax];
  return fa;
}
__device__ __forceinline__ double* knorm_lds_b() {
  __shared__ double fb[kKnormFoldMax / 2];
  return fb;
}

// The levels above `w` values per fragment held in knorm_lds_a() (w a power of
// two, n * w <= kKnormFoldMax); keys[i] = the root, visible to the workgroup on
// return.
__device__ __forceinline__ void knorm_fold_levels(int32_t n, int w, double* __restrict__ keys) {
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  double* src = knorm_lds_a();
  double* dst = knorm_lds_b();
  while (w > 1) {
    const int h = w >> 1;
    for (int e = tid; e < n * h; e += nt) {
      const int i = e / h;
      const int j = e - i * h;
      dst[e] = src[i * w + 2 * j] + src[i * w + 2 * j + 1];
    }
    __syncthreads();
    double* t = src;
    src = dst;
    dst = t;
    w = h;
  }
  for (int i = tid; i < n; i += nt) keys[i] = src[i];
  __syncthreads();
}

// parts holds, per fragment i, `count` consecutive partial sums (one tree
// level; count a power of two, n * count <= kKnormFoldMax). The remaining
// levels run in LDS; keys[i] = the root. Every thread of the workgroup calls it;
// the keys are visible to the workgroup on return.
__device__ __forceinline__ void knorm_fold(const double* __restrict__ parts, int32_t n,
                                           int64_t count, double* __restrict__ keys) {
  double* fa = knorm_lds_a();
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  const int w = (int)count;
  // eight loads in flight per thread before their LDS stores (one workgroup of
  // as few as 64 threads copies up to 4096 partial sums)
  const int total = n * w;
  for (int e0 = tid; e0 < total; e0 += 8 * nt) {
    double v[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int e = e0 + r * nt;
      v[r] = e < total ? parts[e] : 0.0;
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int e = e0 + r * nt;
      if (e < total) fa[e] = v[r];
    }
  }
  __syncthreads();
  knorm_fold_levels(n, w, keys);
}

// Every fragment's key from its rows, in the workgroup: the leaves are the
// same row norms the row kernel makes (each row's 16-byte pieces summed by
// row_chunk_sumsq, the pieces combined by the same butterfly over the row's
// lanes, then sqrt; zero-padded), so the fold over them gives bit-identical
// keys. Needs n * padded <= kKnormFoldMax and a workgroup of at least 64 threads.
template <int ESIZE>
__device__ __forceinline__ void knorm_direct(const int64_t* __restrict__ table, int64_t stride,
                                             int32_t n, int32_t H, int32_t d, const KnormDirect& kd,
                                             double* __restrict__ keys) {
#pragma clang fp contract(off)
  double* fa = knorm_lds_a();
  const int tid = threadIdx.x;
  const int row_bytes = d * ESIZE;
  const int rb_shift = __builtin_ctz((unsigned)row_bytes);
  const int lpr = row_bytes >> 4;                // lanes per row: 4 .. 64, within a wave
  const int rpp = (int)blockDim.x / lpr;         // rows per pass
  const int q = tid & (lpr - 1);
  const int64_t rows = (int64_t)H * kd.tail;
  const int64_t total = (int64_t)n * kd.padded;
  for (int64_t f0 = tid / lpr; f0 < total; f0 += rpp) {   // the same trip count on a row's lanes
    const int i = (int)(f0 / kd.padded);
    const int64_t f = f0 - (int64_t)i * kd.padded;
    const bool valid = f < rows;
    double acc = 0.0;
    if (valid) {
      const int64_t h = f / kd.tail;
      const int64_t r = f - h * kd.tail;
      const int64_t T = table[(int64_t)i * stride];
      const uint8_t* p = reinterpret_cast<const uint8_t*>(table[(int64_t)i * stride + 1 + 2 * kd.layer]) +
                         ((h * T + T - kd.tail + r) << rb_shift) + q * 16;
      acc = row_chunk_sumsq<ESIZE>(*global_ptr<u32x4>(p));
    }
    for (int o = 1; o < lpr; o <<= 1) acc = acc + __shfl_xor(acc, o, 64);
    if (q == 0) fa[f0] = valid ? sqrt(acc) : 0.0;
  }
  __syncthreads();
  knorm_fold_levels(n, (int)kd.padded, keys);
}

// The scores of a one-workgroup kernel: computed here (kd.layer >= 0), folded
// from the partial sums (count > 1), or already the keys.
__device__ __forceinline__ void knorm_finish(const int64_t* __restrict__ table, int64_t stride,
                                             int32_t n, int32_t H, int32_t d, const KnormDirect& kd,
                                             const double* __restrict__ parts, int64_t count,
                                             double* __restrict__ keys) {
  if (kd.layer >= 0) {
    if (kd.esize == 2) knorm_direct<2>(table, stride, n, H, d, kd, keys);
    else knorm_direct<4>(table, stride, n, H, d, kd, keys);
  } else if (count > 1) {
    knorm_fold(parts, n, count, keys);
  }
}

}  // namespace cm
