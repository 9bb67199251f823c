// The last levels of the score tree (Eq. (3)) inside a one-workgroup kernel
// that needs the keys next (the order, the key mask), so the path spends no
// launch on them. The levels below are the knorm kernels'; the summation order
// is the same level-wise adjacent-pair tree, so the keys are bit-identical to a
// full tree of launches.
#pragma once

#include "internal.h"

namespace cm {

// parts holds, per fragment i, `count` consecutive partial sums (one tree
// level; count a power of two, n * count <= kKnormFoldMax). The remaining
// levels run in LDS; keys[i] = the root. Every thread of the workgroup calls it;
// the keys are visible to the workgroup on return.
__device__ __forceinline__ void knorm_fold(const double* __restrict__ parts, int32_t n,
                                           int64_t count, double* __restrict__ keys) {
  __shared__ double fa[kKnormFoldMax];
  __shared__ double fb[kKnormFoldMax / 2];
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  int w = (int)count;
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
  double* src = fa;
  double* dst = fb;
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

}  // namespace cm
