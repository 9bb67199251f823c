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
  for (int e = tid; e < n * w; e += nt) fa[e] = parts[e];
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
