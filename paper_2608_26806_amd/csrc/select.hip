// Segmented top-k: inside every image keep the budget[i] highest-scoring
// tokens (the paper keeps the most important tokens of each image at its
// adaptive ratio, Sec. 3.3.3), plus every text token, and emit the kept
// global token indices of each sequence in ascending order.
//
// One 256-thread block per image finds the exact k-th largest order key by
// four 8-bit radix passes (LDS histograms, a wave suffix scan picks the
// digit), then one ordered pass keeps every key above the threshold and the
// lowest-index keys equal to it, using ballot-based block scans to place
// them.  Output offsets need no global scan: an image's kept tokens start at
//   cu_text[b] + (text rows of b before the image) + sum of earlier budgets,
// and a text row t at  t + (budgets of the images before it).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"

namespace avtp {
namespace {

constexpr int kThreads = 256;

// Monotone map float -> uint32 (larger score -> larger key); -0.0 == +0.0,
// NaN -> 0, below every other value.
__device__ inline uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline int eff_budget(const int32_t *budget, const int32_t *img_len, int i) {
  const int k = budget[i], n = img_len[i];
  return k < 0 ? 0 : (k > n ? n : k);
}

// exclusive block scan of a 0/1 flag (256 threads, 4 waves); returns the
// exclusive count and writes the block total to *total
__device__ inline int block_scan_flag(bool f, int *wsum, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long m = __ballot(f);
  const int below = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wave] = __popcll(m);
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wave; ++w) off += wsum[w];
  *total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  return off + below;
}

__global__ __launch_bounds__(kThreads) void select_kernel(
    const float *__restrict__ scores, const int32_t *__restrict__ budget,
    const int32_t *__restrict__ img_start, const int32_t *__restrict__ img_len,
    const int32_t *__restrict__ cu_img, const int32_t *__restrict__ cu_text,
    const int32_t *__restrict__ text_pos, int B, int n_img, int T_tot,
    int32_t *__restrict__ keep_idx, long long cap, int32_t *__restrict__ cu_out,
    int32_t *__restrict__ status) {
  __shared__ uint32_t hist[256];
  __shared__ int wsum[4];
  __shared__ long long red[kThreads];
  __shared__ uint32_t sh_digit;
  __shared__ int sh_krem;
  const int tid = threadIdx.x;

  if ((int)blockIdx.x >= n_img) {
    // ---- text rows and cu_out
    const int tb = blockIdx.x - n_img;
    const int t = tb * kThreads + tid;
    if (t < T_tot) {
      const int p = text_pos[t];
      int lo = 0, hi = n_img;  // images starting before p
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (img_start[mid] < p) lo = mid + 1; else hi = mid;
      }
      long long out = t;
      for (int i = 0; i < lo; ++i) out += eff_budget(budget, img_len, i);
      if (out < cap) keep_idx[out] = p;
    }
    if (tb == 0) {
      for (int b = tid; b <= B; b += kThreads) {
        long long o = cu_text[b];
        for (int i = 0; i < cu_img[b]; ++i) o += eff_budget(budget, img_len, i);
        cu_out[b] = (int32_t)o;
      }
    }
    return;
  }

  // ---- one image
  const int i = blockIdx.x;
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_img[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int st = img_start[i], n = img_len[i];
  const int k = eff_budget(budget, img_len, i);
  if (k == 0) return;
  long long part = 0;
  for (int j = tid; j < i; j += kThreads) part += eff_budget(budget, img_len, j);
  red[tid] = part;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  int a0 = cu_text[b], a1 = cu_text[b + 1];
  while (a0 < a1) {  // first text row of b at or after the image
    const int mid = (a0 + a1) >> 1;
    if (text_pos[mid] < st) a0 = mid + 1; else a1 = mid;
  }
  const long long base = (long long)a0 + red[0];
  const float *s = scores + st;

  if (k == n) {
    for (int j = tid; j < n; j += kThreads) {
      const long long o = base + j;
      if (o < cap) keep_idx[o] = st + j;
      else if (status) atomicOr(status + b, AVTP_FLAG_OUT_CAPACITY);
    }
    return;
  }

  // ---- radix select of the k-th largest key
  uint32_t prefix = 0, mask = 0;
  int krem = k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    hist[tid] = 0;
    __syncthreads();
    for (int j = tid; j < n; j += kThreads) {
      const uint32_t key = order_key(s[j]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane owns bins 4*lane .. 4*lane+3; suffix sums over lanes (high bins first)
      const int lane = tid;
      const int c = hist[4 * lane] + hist[4 * lane + 1] + hist[4 * lane + 2] + hist[4 * lane + 3];
      int suf = c;
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_down(suf, off);
        if (lane + off < 64) suf += v;
      }
      const int above = suf - c;  // keys in bins of higher lanes
      if (suf >= krem && above < krem) {
        int acc = above;
        for (int x = 4 * lane + 3; x >= 4 * lane; --x) {
          if (acc + (int)hist[x] >= krem) {
            sh_digit = (uint32_t)x;
            sh_krem = krem - acc;
            break;
          }
          acc += hist[x];
        }
      }
    }
    __syncthreads();
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    krem = sh_krem;
    __syncthreads();
  }
  const uint32_t theta = prefix;  // exactly krem keys equal to theta are kept

  // ---- ordered pass: keep > theta, and the first krem keys == theta
  int eq_carry = 0, keep_carry = 0;
  for (int c0 = 0; c0 < n; c0 += kThreads) {
    const int j = c0 + tid;
    uint32_t key = 0;
    if (j < n) key = order_key(s[j]);
    const bool gt = j < n && key > theta;
    const bool eq = j < n && key == theta;
    int tot;
    const int eq_rank = block_scan_flag(eq, wsum, &tot) + eq_carry;
    eq_carry += tot;
    const bool keep = gt || (eq && eq_rank < krem);
    const int pos = block_scan_flag(keep, wsum, &tot) + keep_carry;
    keep_carry += tot;
    if (keep) {
      const long long o = base + pos;
      if (o < cap) keep_idx[o] = st + j;
      else if (status) atomicOr(status + b, AVTP_FLAG_OUT_CAPACITY);
    }
  }
}

}  // namespace

hipError_t launch_select(hipStream_t st, const DevLayout &L, const float *scores,
                         const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                         int32_t *cu_out, int32_t *status) {
  int text_blocks = (L.T_tot + kThreads - 1) / kThreads;
  if (text_blocks < 1) text_blocks = 1;  // the first text block also writes cu_out
  hipLaunchKernelGGL(select_kernel, dim3(L.n_img + text_blocks), dim3(kThreads), 0, st, scores,
                     budget, L.img_start, L.img_len, L.cu_img, L.cu_text, L.text_pos, L.B,
                     L.n_img, L.T_tot, keep_idx, (long long)keep_capacity, cu_out, status);
  return hipGetLastError();
}

}  // namespace avtp
