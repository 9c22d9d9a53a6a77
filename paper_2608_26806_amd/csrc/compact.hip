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
constexpr int kBlockBytes = 16384;  // target bytes per block (8 and 16 KB measured alike, 32 and 64 KB slower)
constexpr long long kStreamMinBytes = 256ll << 20;  // see launch_compact

struct CArgs {
  CTensor t[AVTP_MAX_TENSORS];
  int n;
  const int32_t *keep_idx;
  long long n_out;
  int N_tok;
};

template <typename V, bool STREAM>
__device__ inline void copy_rows(const CTensor &T, const int32_t *__restrict__ keep_idx,
                                 long long r0, long long r1, int N_tok, int plane) {
  const int lane = threadIdx.x & ((1 << T.lpr_shift) - 1);
  const long long rpp = kThreads >> T.lpr_shift;  // rows per pass of the block
  copy_rows_batched<V, STREAM>(T, plane, r0 + (threadIdx.x >> T.lpr_shift), r1, rpp, lane,
                       [&](long long r, long long &j, long long &dr) __attribute__((always_inline)) {
                         const int k = keep_idx[r];
                         j = k;
                         dr = r;
                         return (unsigned)k < (unsigned)N_tok;  // out-of-range index: row left untouched
                       });
}

template <bool STREAM>
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
    case 4: copy_rows<uint4, STREAM>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    case 3: copy_rows<uint2, STREAM>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    case 2: copy_rows<uint32_t, STREAM>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    case 1: copy_rows<uint16_t, STREAM>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
    default: copy_rows<uint8_t, STREAM>(T, a.keep_idx, r0, r1, a.N_tok, plane); break;
  }
}

}  // namespace

hipError_t launch_compact(hipStream_t st, const DevLayout &L, const int32_t *keep_idx,
                          int64_t n_out, const avtp_tensor *tensors, int n_tensors) {
  clear_pending_error();
  CArgs a;
  a.n = n_tensors;
  a.keep_idx = keep_idx;
  a.n_out = n_out;
  a.N_tok = L.N_tok;
  long long blocks = 0, read_bytes = 0;
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
    read_bytes += n_out * x.row_bytes * x.planes;
  }
  if (blocks == 0) return hipSuccess;
  // A gather larger than the last-level cache (256 MiB of Infinity Cache)
  // reads its source rows with non-temporal loads, which do not displace
  // cached data: at 420 MB read (8 sequences of 16 images) 0.71 -> 0.80 of
  // the HBM peak.  Smaller ones keep ordinary loads, which find part of their
  // sources in the cache: at 120 MB read non-temporal loads measured 10 %
  // slower, at 187 MB the same.
  if (read_bytes > kStreamMinBytes)
    hipLaunchKernelGGL(compact_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(compact_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace avtp
