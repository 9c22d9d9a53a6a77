// Stable compaction out[r] = in[keep_idx[r]] of up to AVTP_MAX_TENSORS
// tensors in one launch (the shortened sequence that continues through the
// layers after pruning; position ids keep their original values).
//
// HBM-bound bit copy.  Each tensor gets its own range of blocks; a block
// copies a run of output rows of one plane.  Rows are split into the widest
// aligned vector unit (16 bytes where possible); a power-of-two group of
// lanes covers one row, so small rows (position ids, per-head K/V rows) pack
// several rows per wave and large rows (hidden states) use the whole block.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"
#include "row_copy.h"

namespace avtp {
namespace {

constexpr int kThreads = 256;
constexpr int kBlockBytes = 32768;  // target bytes per block
constexpr int kRowsInFlight = 4;    // rows a thread group copies at once (copy_rows)

struct CArgs {
  CTensor t[AVTP_MAX_TENSORS];
  int n;
  const int32_t *keep_idx;
  long long n_out;
  int N_tok;
};

// A thread group works on four rows at once: their keep_idx entries are
// loaded together, then every row's vector units, then the stores, so that
// several independent loads per lane are in flight (HBM latency is the limit
// otherwise).  The rows are named variables, not arrays, so that they stay in
// registers.
template <typename V>
struct RowJob {
  const V *s;
  V *d;
  bool ok;
};

template <typename V>
__device__ inline RowJob<V> row_job(const int32_t *__restrict__ keep_idx, long long r, long long r1,
                                    int N_tok, const char *src, long long sstr, char *dst,
                                    long long dstr) {
  const int j = r < r1 ? keep_idx[r] : -1;
  RowJob<V> w;
  w.ok = (unsigned)j < (unsigned)N_tok;  // out-of-range index: row left untouched
  w.s = reinterpret_cast<const V *>(src + (w.ok ? j : 0) * sstr);
  w.d = reinterpret_cast<V *>(dst + (w.ok ? r : 0) * dstr);
  return w;
}

template <typename V>
__device__ inline void copy_rows(const CTensor &T, const int32_t *__restrict__ keep_idx,
                                 long long r0, long long r1, int N_tok, int plane) {
  const int tid = threadIdx.x;
  const int lpr = 1 << T.lpr_shift;
  const int lane = tid & (lpr - 1);
  const long long rpp = kThreads >> T.lpr_shift;  // rows per pass of the block
  const char *src = T.src + plane * T.src_plane_stride;
  char *dst = T.dst + plane * T.dst_plane_stride;
  const long long sstr = T.src_stride, dstr = T.dst_stride;
  const int units = T.units;
  for (long long rb = r0 + (tid >> T.lpr_shift); rb < r1; rb += kRowsInFlight * rpp) {
    const RowJob<V> w0 = row_job<V>(keep_idx, rb, r1, N_tok, src, sstr, dst, dstr);
    const RowJob<V> w1 = row_job<V>(keep_idx, rb + rpp, r1, N_tok, src, sstr, dst, dstr);
    const RowJob<V> w2 = row_job<V>(keep_idx, rb + 2 * rpp, r1, N_tok, src, sstr, dst, dstr);
    const RowJob<V> w3 = row_job<V>(keep_idx, rb + 3 * rpp, r1, N_tok, src, sstr, dst, dstr);
    for (int u = lane; u < units; u += 2 * lpr) {
      const bool two = u + lpr < units;
      V a0{}, a1{}, a2{}, a3{}, b0{}, b1{}, b2{}, b3{};
      auto ld = [&](const RowJob<V> &w, V &x, V &y) __attribute__((always_inline)) {
        if (w.ok) {
          x = w.s[u];
          if (two) y = w.s[u + lpr];
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

__global__ __launch_bounds__(kThreads) void compact_kernel(CArgs a) {
  int ti = 0;
  while (ti + 1 < a.n && (int)blockIdx.x >= a.t[ti + 1].block_begin) ++ti;
  const CTensor &T = a.t[ti];
  const int local = blockIdx.x - T.block_begin;
  const int plane = local / T.blocks_per_plane;
  const int rb = local - plane * T.blocks_per_plane;
  const long long r0 = (long long)rb * T.rows_per_block;
  long long r1 = r0 + T.rows_per_block;
  if (r1 > a.n_out) r1 = a.n_out;
  switch (T.vshift) {
    case 4: copy_rows<uint4>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    case 3: copy_rows<uint2>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    case 2: copy_rows<uint32_t>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    case 1: copy_rows<uint16_t>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    default: copy_rows<uint8_t>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
  }
}

}  // namespace

hipError_t launch_compact(hipStream_t st, const DevLayout &L, const int32_t *keep_idx,
                          int64_t n_out, const avtp_tensor *tensors, int n_tensors) {
  CArgs a;
  a.n = n_tensors;
  a.keep_idx = keep_idx;
  a.n_out = n_out;
  a.N_tok = L.N_tok;
  long long blocks = 0;
  for (int i = 0; i < n_tensors; ++i) {
    const avtp_tensor &x = tensors[i];
    CTensor &T = a.t[i];
    describe_tensor(x, kThreads, T);
    const long long lpr = 1ll << T.lpr_shift;
    const long long rows_per_pass = kThreads / lpr;
    long long rpb = (kBlockBytes + x.row_bytes - 1) / x.row_bytes;
    const long long batch = rows_per_pass * kRowsInFlight;
    rpb = ((rpb + batch - 1) / batch) * batch;
    T.rows_per_block = (int)rpb;
    T.blocks_per_plane = (int)((n_out + rpb - 1) / rpb);
    T.planes = x.planes;
    T.block_begin = (int)blocks;
    blocks += (long long)T.blocks_per_plane * x.planes;
  }
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(compact_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace avtp
