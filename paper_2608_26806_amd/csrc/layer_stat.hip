// Architecture-aware pruning-layer selection (Sec. 3.3.2): the attention a
// layer pays to all visual tokens of each sample, and the layers' average
// rank over the samples.
//
// Both steps are latency-bound (at most a few thousand samples by a few
// hundred layers); every result is either an exactly ordered float sum or an
// integer, so reruns are bit-identical.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "avtp_internal.h"

namespace avtp {
namespace {

// A[b] = sum of the image sums of sequence b, accumulated in float64 in
// image order and rounded once.
__global__ void layer_attn_kernel(const float *__restrict__ img_sum, const int32_t *__restrict__ cu_img,
                                  int B, float *__restrict__ A) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  double s = 0.0;
#pragma unroll 8
  for (int i = cu_img[b]; i < cu_img[b + 1]; ++i) s += (double)img_sum[i];
  A[b] = (float)s;
}

// NaN ranks as the smallest value
__device__ inline float rank_key(float x) { return x != x ? -INFINITY : x; }

constexpr int kRankThreads = 256;

// Block l: rank_sum[l] = sum over samples i of the rank of A[l][i] among
// A[0..L)[i] (rank 1 = largest; an equal value ranks the lower layer first).
// Consecutive threads take consecutive samples, so every read of a layer row
// is coalesced.
__global__ __launch_bounds__(kRankThreads) void layer_rank_kernel(const float *__restrict__ A, int L,
                                                                  int N, int32_t *__restrict__ rank_sum) {
  __shared__ long long red[kRankThreads / 64];
  const int l = blockIdx.x;
  long long acc = 0;
  for (int i = threadIdx.x; i < N; i += kRankThreads) {
    const float a = rank_key(A[(size_t)l * N + i]);
    int r = 1;
    // eight layers' loads in flight at a time (the loop is latency-bound)
#pragma unroll 8
    for (int m = 0; m < L; ++m) {
      const float v = rank_key(A[(size_t)m * N + i]);
      r += (v > a) || (v == a && m < l);
    }
    acc += r;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long t = 0;
    for (int w = 0; w < kRankThreads / 64; ++w) t += red[w];
    rank_sum[l] = (int32_t)t;
  }
}

constexpr int kSelThreads = 1024;  // one thread per layer (L <= AVTP_MAX_LAYERS)
static_assert(AVTP_MAX_LAYERS <= kSelThreads, "one thread per layer");

// The k layers with the smallest rank sums (equal sums: lower layer first),
// written in ascending layer order.
__global__ __launch_bounds__(kSelThreads) void layer_select_kernel(const int32_t *__restrict__ rank_sum,
                                                                   int L, int k,
                                                                   int32_t *__restrict__ selected) {
  __shared__ int32_t rs[kSelThreads];
  __shared__ int32_t chosen[kSelThreads];
  const int l = threadIdx.x;
  if (l < L) rs[l] = rank_sum[l];
  __syncthreads();
  int pos = 0;
  if (l < L) {
    const int32_t me = rs[l];
    for (int m = 0; m < L; ++m) pos += (rs[m] < me) || (rs[m] == me && m < l);
    chosen[l] = pos < k;
  }
  __syncthreads();
  if (l < L && chosen[l]) {
    int before = 0;
    for (int m = 0; m < l; ++m) before += chosen[m];
    selected[before] = l;
  }
}

}  // namespace

hipError_t launch_layer_attention(hipStream_t st, const DevLayout &L, const float *img_sum, float *A) {
  clear_pending_error();
  if (L.B == 0) return hipSuccess;
  hipLaunchKernelGGL(layer_attn_kernel, dim3((L.B + 255) / 256), dim3(256), 0, st, img_sum, L.cu_img,
                     L.B, A);
  return hipGetLastError();
}

hipError_t launch_layer_select(hipStream_t st, const float *A, int L, int N, int k, int32_t *rank_sum,
                               int32_t *selected) {
  clear_pending_error();
  hipLaunchKernelGGL(layer_rank_kernel, dim3(L), dim3(kRankThreads), 0, st, A, L, N, rank_sum);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_select_kernel, dim3(1), dim3(kSelThreads), 0, st, rank_sum, L, k, selected);
  return hipGetLastError();
}

}  // namespace avtp
