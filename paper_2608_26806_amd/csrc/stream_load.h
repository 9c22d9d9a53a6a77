// Non-temporal ("streaming") vector loads, for data a kernel reads exactly
// once: they do not displace cached data (the row gathers of the compaction,
// the hidden-state rows of the variation score).
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace avtp {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

template <typename V>
__device__ inline V ld_stream(const V *p) {
  return __builtin_nontemporal_load(p);
}
template <>
__device__ inline uint4 ld_stream(const uint4 *p) {
  const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(x.x, x.y, x.z, x.w);
}
template <>
__device__ inline uint2 ld_stream(const uint2 *p) {
  const u32x2_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
  return make_uint2(x.x, x.y);
}

}  // namespace avtp
