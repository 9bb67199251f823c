// Device helper shared by the render kernels: 16-byte nontemporal global
// stores (the merged cache is written once and not read back by the kernel).
#pragma once

#include "internal.h"

namespace cm {

__device__ __forceinline__ void st_stream(uint8_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, (CM_GLOBAL u32x4*)p);
}

}  // namespace cm
