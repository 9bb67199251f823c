// mask[i] = 1 if another delivery has a bitwise-equal key (only those digests
// decide dedupe and ties), else 0. One workgroup of at least n threads.
#pragma once

#include "internal.h"

namespace cm {

__device__ __forceinline__ void equal_key_mask_body(int32_t n, const double* __restrict__ keys,
                                                    uint8_t* __restrict__ mask) {
  __shared__ double s_key[1024];
  const int tid = threadIdx.x;
  double key = 0.0;
  if (tid < n) {
    key = keys[tid];
    s_key[tid] = key;
  }
  __syncthreads();
  if (tid < n) {
    bool shared = false;
    for (int j = 0; j < n; ++j) shared |= (j != tid && s_key[j] == key);
    mask[tid] = shared ? 1 : 0;
  }
}

}  // namespace cm
