// The per-image epilogue of both score modes (Sec. 3.3.2 statistic per
// visual token, and the per-image sums that Sec. 3.3.3's budgets start from).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"
#include "wave_ops.h"

namespace avtp {
namespace {

// Per-image epilogue shared by both score modes: s_j from the column sums
// (attention mode) or as stored (variation mode), NaN / empty-row flags, and
// the per-image sum in a fixed reduction order.  Extra blocks write +inf at
// the text positions.  One block of 256 threads per image.
__global__ __launch_bounds__(256) void finalize_kernel(
    const float *__restrict__ colsum, int Hq, int planes, int N_tok, int n_img, int T_tot,
    const int32_t *__restrict__ img_start, const int32_t *__restrict__ img_len,
    const int32_t *__restrict__ cu_img, const int32_t *__restrict__ cu_text,
    const int32_t *__restrict__ text_pos, int B, float *__restrict__ scores,
    float *__restrict__ img_sum, int32_t *__restrict__ status) {
  __shared__ float red[4];
  __shared__ int sh_b, sh_cnt[4];
  const int tid = threadIdx.x;
  if ((int)blockIdx.x >= n_img) {
    const int t = (blockIdx.x - n_img) * 256 + tid;
    if (t < T_tot) scores[text_pos[t]] = INFINITY;
    return;
  }
  const int i = blockIdx.x;
  for (int c = tid; c < B; c += 256)  // the sequence holding image i
    if (cu_img[c] <= i && i < cu_img[c + 1]) sh_b = c;
  __syncthreads();
  const int b = sh_b;
  const int s0 = img_start[i], n = img_len[i];
  // Tokens j = tid + 256 q (q < 4) of the first 1024 are summed over the
  // planes before the text-row count, so that all their loads are in flight
  // together; every token's plane sum runs in plane order either way.
  float v0 = 0.f, v1 = 0.f, v2 = 0.f, v3 = 0.f;
  if (colsum) {
    const float *c0 = colsum + s0 + tid;
    // a token past the image re-reads token tid (in bounds); its sum is not used
    const int o1 = tid + 256 < n ? 256 : 0, o2 = tid + 512 < n ? 512 : 0,
              o3 = tid + 768 < n ? 768 : 0;
    if (tid < n) {
#pragma unroll 4
      for (int g = 0; g < planes; ++g) {
        const float *cg = c0 + (size_t)g * N_tok;
        const float x0 = cg[0], x1 = cg[o1], x2 = cg[o2], x3 = cg[o3];
        v0 += x0;
        v1 += x1;
        v2 += x2;
        v3 += x3;
      }
    }
  }
  int nT = 0;
  if (colsum) {  // text rows after the image (their positions exceed s0)
    int c = 0;
    for (int t = cu_text[b] + tid; t < cu_text[b + 1]; t += 256) c += text_pos[t] > s0;
    c = wave::sum(c);
    if ((tid & 63) == 0) sh_cnt[tid >> 6] = c;
    __syncthreads();
    nT = sh_cnt[0] + sh_cnt[1] + sh_cnt[2] + sh_cnt[3];
  }
  float acc = 0.f;
  bool nan = false;
  for (int j = tid; j < n; j += 256) {
    float s;
    if (colsum) {
      float v;
      if (j < 1024) {
        const int q = (j - tid) >> 8;
        v = q == 0 ? v0 : (q == 1 ? v1 : (q == 2 ? v2 : v3));
      } else {
        v = 0.f;
        for (int g = 0; g < planes; ++g) v += colsum[(size_t)g * N_tok + s0 + j];
      }
      s = nT > 0 ? v / (float)((long long)Hq * nT) : 0.f;
      scores[s0 + j] = s;
    } else {
      s = scores[s0 + j];
    }
    nan |= (s != s);
    acc += s;
  }
  // the image sum in a fixed order: each thread's tokens in order, the
  // wave's lanes in the DPP pattern, then the four waves in order
  acc = wave::sum(acc);
  if ((tid & 63) == 0) red[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0) img_sum[i] = (red[0] + red[1]) + (red[2] + red[3]);
  if (status) {
    if (nan) atomicOr(status + b, AVTP_FLAG_NAN_SCORE);
    if (tid == 0 && colsum && nT == 0 && n > 0) atomicOr(status + b, AVTP_FLAG_NO_TEXT_AFTER);
  }
}

}  // namespace

hipError_t launch_finalize(hipStream_t st, const DevLayout &L, const float *colsum, int Hq,
                           int planes, float *scores, float *img_sum, int32_t *status) {
  clear_pending_error();
  const int text_blocks = (L.T_tot + 255) / 256;
  const int grid = L.n_img + text_blocks;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(finalize_kernel, dim3(grid), dim3(256), 0, st, colsum, Hq, planes, L.N_tok,
                     L.n_img, L.T_tot, L.img_start, L.img_len, L.cu_img, L.cu_text, L.text_pos,
                     L.B, scores, img_sum, status);
  return hipGetLastError();
}

}  // namespace avtp
