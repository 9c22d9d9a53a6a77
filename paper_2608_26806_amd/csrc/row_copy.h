// Row-copy descriptors shared by the compaction kernels (compact.hip and the
// fused select + compaction in select.hip): one tensor's source and
// destination, its strides, and the vector unit its rows are copied in.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "avtp_internal.h"
#include "stream_load.h"

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

// Batched row copies: a lane group works on four rows at once (their source
// and destination rows first, then every row's vector units, then the
// stores), so that several independent loads per lane are in flight; HBM
// latency is the limit otherwise.  The rows are named variables, not arrays,
// so that they stay in registers.  entry(e, j, r) gives list entry e's source
// row j and destination row r and returns false to skip it; the group handles
// entries e0, e0 + step, ... below e1.  With STREAM the source rows are read
// with non-temporal loads (for gathers larger than the caches: see
// launch_compact); the stores stay ordinary (non-temporal stores measured
// 10 % slower).
constexpr int kRowsInFlight = 4;

template <typename V>
struct RowJob {
  const V *s;
  V *d;
  bool ok;
};

template <typename V, typename Entry>
__device__ inline RowJob<V> row_job(Entry &entry, long long e, long long e1, const char *src,
                                    long long sstr, char *dst, long long dstr) {
  long long j = 0, r = 0;
  RowJob<V> w;
  w.ok = e < e1 && entry(e, j, r);
  if (!w.ok) j = r = 0;
  w.s = reinterpret_cast<const V *>(src + j * sstr);
  w.d = reinterpret_cast<V *>(dst + r * dstr);
  return w;
}

template <typename V, bool STREAM, typename Entry>
__device__ inline void copy_rows_batched(const CTensor &T, int plane, long long e0, long long e1,
                                         long long step, int lane, Entry entry) {
  const int lpr = 1 << T.lpr_shift;
  const char *src = T.src + plane * T.src_plane_stride;
  char *dst = T.dst + plane * T.dst_plane_stride;
  const long long sstr = T.src_stride, dstr = T.dst_stride;
  const int units = T.units;
  for (long long e = e0; e < e1; e += kRowsInFlight * step) {
    const RowJob<V> w0 = row_job<V>(entry, e, e1, src, sstr, dst, dstr);
    const RowJob<V> w1 = row_job<V>(entry, e + step, e1, src, sstr, dst, dstr);
    const RowJob<V> w2 = row_job<V>(entry, e + 2 * step, e1, src, sstr, dst, dstr);
    const RowJob<V> w3 = row_job<V>(entry, e + 3 * step, e1, src, sstr, dst, dstr);
    for (int u = lane; u < units; u += 2 * lpr) {
      const bool two = u + lpr < units;
      V a0{}, a1{}, a2{}, a3{}, b0{}, b1{}, b2{}, b3{};
      auto ld = [&](const RowJob<V> &w, V &x, V &y) __attribute__((always_inline)) {
        if (w.ok) {
          x = STREAM ? ld_stream(w.s + u) : w.s[u];
          if (two) y = STREAM ? ld_stream(w.s + u + lpr) : w.s[u + lpr];
        }
      };
      auto st = [&](const RowJob<V> &w, const V &x, const V &y) __attribute__((always_inline)) {
        if (w.ok) {
          w.d[u] = x;
          if (two) w.d[u + lpr] = y;
        }
      };
      ld(w0, a0, b0);
      ld(w1, a1, b1);
      ld(w2, a2, b2);
      ld(w3, a3, b3);
      st(w0, a0, b0);
      st(w1, a1, b1);
      st(w2, a2, b2);
      st(w3, a3, b3);
    }
  }
}

}  // namespace avtp
