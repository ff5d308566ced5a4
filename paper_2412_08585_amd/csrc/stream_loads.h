// Streaming (non-temporal) global loads, for data a launch reads exactly
// once: on gfx950 they sustain about 13 % more HBM bandwidth than ordinary
// loads (6.8 against 6.0 TB/s), also for scattered 1 KiB regions.  Where the
// data is likely to sit in the MALL from an earlier kernel, ordinary loads
// are as fast or faster, so the kernels use these only for streams that come
// from HBM.
#pragma once

#include <hip/hip_runtime.h>

namespace turbo {

typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t load_nt4(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}
__device__ __forceinline__ u32x2_t load_nt2(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
}
__device__ __forceinline__ unsigned load_nt1(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const unsigned*>(p));
}

}  // namespace turbo
