// Row-copy descriptors shared by the compaction kernels (compact.hip and the
// fused select + compaction in select.hip): one tensor's source and
// destination, its strides, and the vector unit its rows are copied in.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "avtp_internal.h"

namespace avtp {

struct CTensor {
  const char *src;
  char *dst;
  long long src_stride, dst_stride, src_plane_stride, dst_plane_stride;
  int units;      // vector units per row
  int vshift;     // log2 of the vector width in bytes
  int lpr_shift;  // log2 of lanes per row (a power-of-two group of lanes covers one row)
  int planes;
  int rows_per_block;    // compact.hip only
  int blocks_per_plane;  // compact.hip only
  int block_begin;       // compact.hip only
};

inline int ilog2_ll(long long v) {
  int s = 0;
  while ((1ll << (s + 1)) <= v) ++s;
  return s;
}

// Source, destination, strides and vector unit of one tensor: the widest of
// 16, 8, 4, 2, 1 bytes that divides the row size, every stride and both base
// addresses; lanes per row = units rounded up to a power of two, at most
// `threads`.
inline void describe_tensor(const avtp_tensor &x, int threads, CTensor &T) {
  long long v = 16;
  auto misaligned = [&](long long m) {
    return (x.row_bytes % m) || (x.src_stride % m) || (x.dst_stride % m) ||
           ((uintptr_t)x.src % m) || ((uintptr_t)x.dst % m) ||
           (x.planes > 1 && ((x.src_plane_stride % m) || (x.dst_plane_stride % m)));
  };
  while (v > 1 && misaligned(v)) v >>= 1;
  T.src = (const char *)x.src;
  T.dst = (char *)x.dst;
  T.src_stride = x.src_stride;
  T.dst_stride = x.dst_stride;
  T.src_plane_stride = x.src_plane_stride;
  T.dst_plane_stride = x.dst_plane_stride;
  T.vshift = ilog2_ll(v);
  T.units = (int)(x.row_bytes / v);
  long long lpr = 1;
  while (lpr < T.units && lpr < threads) lpr <<= 1;
  T.lpr_shift = ilog2_ll(lpr);
  T.planes = x.planes;
  T.rows_per_block = T.blocks_per_plane = T.block_begin = 0;
}

// Copy source row `j` of plane `plane` to destination row `r` with the
// `lpr` lanes of one group (lane = this thread's index in its group).
template <typename V>
__device__ inline void copy_one_row(const CTensor &T, int plane, long long j, long long r, int lane) {
  const int lpr = 1 << T.lpr_shift;
  const V *s = reinterpret_cast<const V *>(T.src + plane * T.src_plane_stride + j * T.src_stride);
  V *d = reinterpret_cast<V *>(T.dst + plane * T.dst_plane_stride + r * T.dst_stride);
  int u = lane;
  for (; u + lpr < T.units; u += 2 * lpr) {  // two independent loads in flight
    const V a = s[u], b = s[u + lpr];
    d[u] = a;
    d[u + lpr] = b;
  }
  if (u < T.units) d[u] = s[u];
}

}  // namespace avtp
