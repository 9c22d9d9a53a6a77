// Layout of the kept tokens for the next pruning layer of a progressive
// schedule (Sec. 3.3.2 progressive pruning; the kept tokens of a sequence are
// a subsequence of it, Method, "Visual Token Pruning").
//
// keep_idx lists each sequence's kept token indices in ascending order at
// [cu_out[b], cu_out[b+1]); kept token r becomes token r of the next layer.
// The new index of an old position p of sequence b is therefore cu_out[b]
// plus the number of kept tokens of b below p, found by binary search.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"

namespace avtp {
namespace {

// number of entries of the ascending list lo[0 .. n) below p
__device__ inline int count_below(const int32_t *lo, int n, int32_t p) {
  int a = 0, b = n;
  while (a < b) {
    const int m = (a + b) >> 1;
    if (lo[m] < p) a = m + 1;
    else b = m;
  }
  return a;
}

constexpr int kThreads = 256;
constexpr int kLdsKept = 16384;  // kept lists up to this long are searched in LDS

// One block per sequence: its images and text rows, and its offsets.  The
// sequence's kept list is first copied to LDS (one coalesced pass), so that
// the binary searches' dependent reads are LDS reads; a longer list is
// searched in place.
__global__ __launch_bounds__(kThreads) void pruned_layout_kernel(
    const int32_t *__restrict__ img_start, const int32_t *__restrict__ img_len,
    const int32_t *__restrict__ cu_img, const int32_t *__restrict__ text_pos,
    const int32_t *__restrict__ cu_text, const int32_t *__restrict__ keep_idx,
    const int32_t *__restrict__ cu_out, int B, int32_t *__restrict__ cu_seqlens_out,
    int32_t *__restrict__ img_start_out, int32_t *__restrict__ img_len_out,
    int32_t *__restrict__ cu_img_out, int32_t *__restrict__ text_pos_out,
    int32_t *__restrict__ cu_text_out) {
  __shared__ int32_t kept_sh[kLdsKept];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int o0 = cu_out[b], n = cu_out[b + 1] - o0;
  const int32_t *kept = keep_idx + o0;
  auto positions = [&](const int32_t *list) __attribute__((always_inline)) {
    for (int i = cu_img[b] + tid; i < cu_img[b + 1]; i += kThreads) {
      const int s = count_below(list, n, img_start[i]);
      const int e = count_below(list, n, img_start[i] + img_len[i]);
      img_start_out[i] = o0 + s;
      img_len_out[i] = e - s;
    }
    for (int t = cu_text[b] + tid; t < cu_text[b + 1]; t += kThreads)
      text_pos_out[t] = o0 + count_below(list, n, text_pos[t]);
  };
  if (n <= kLdsKept) {  // (block-uniform)
    for (int j = tid; j < n; j += kThreads) kept_sh[j] = kept[j];
    __syncthreads();
    positions(kept_sh);
  } else {
    positions(kept);
  }
  if (tid == 0) {
    cu_seqlens_out[b + 1] = cu_out[b + 1];
    cu_img_out[b + 1] = cu_img[b + 1];
    cu_text_out[b + 1] = cu_text[b + 1];
    if (b == 0) {
      cu_seqlens_out[0] = cu_out[0];
      cu_img_out[0] = cu_img[0];
      cu_text_out[0] = cu_text[0];
    }
  }
}

}  // namespace

hipError_t launch_pruned_layout(hipStream_t st, const DevLayout &L, const int32_t *keep_idx,
                                const int32_t *cu_out, int32_t *cu_seqlens_out,
                                int32_t *img_start_out, int32_t *img_len_out, int32_t *cu_img_out,
                                int32_t *text_pos_out, int32_t *cu_text_out) {
  clear_pending_error();
  if (L.B == 0) return hipSuccess;
  hipLaunchKernelGGL(pruned_layout_kernel, dim3(L.B), dim3(kThreads), 0, st, L.img_start, L.img_len,
                     L.cu_img, L.text_pos, L.cu_text, keep_idx, cu_out, L.B, cu_seqlens_out,
                     img_start_out, img_len_out, cu_img_out, text_pos_out, cu_text_out);
  return hipGetLastError();
}

}  // namespace avtp
