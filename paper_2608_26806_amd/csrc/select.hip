// Segmented top-k: inside every image keep the budget[i] highest-scoring
// tokens (the paper keeps the most important tokens of each image at its
// adaptive ratio, Sec. 3.3.3), plus every text token, and emit the kept
// global token indices of each sequence in ascending order.
//
// One 256-thread block per image finds the exact k-th largest order key by
// four 8-bit radix passes (LDS histograms, a wave suffix scan picks the
// digit), then one ordered pass keeps every key above the threshold and the
// lowest-index keys equal to it, placed by block scans.  Output offsets need
// no global scan: an image's kept tokens start at
//   cu_text[b] + (text rows of b before the image) + sum of earlier budgets,
// and a text row t at  t + (budgets of the images before it); the image
// blocks write the text rows around them too.
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

// exclusive block scan of an integer (256 threads); block total in *total
__device__ inline int block_scan_int(int v, int *wsum, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(inc, off);
    if (lane >= off) inc += u;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wave; ++w) off += wsum[w];
  *total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  return off + inc - v;
}

// block-wide sum of a 64-bit value
__device__ inline long long block_sum_ll(long long v, long long *sh) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  const long long r = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return r;
}

constexpr int kLdsKeys = 4096;  // images up to this length keep their keys in LDS

// Digit of the krem-th largest key among those matching (prefix, mask), from
// a 256-bin histogram of byte `shift`; updates krem to the rank inside the bin.
__device__ inline void pick_digit(const uint32_t *hist, int krem, uint32_t *sh_digit, int *sh_krem) {
  if (threadIdx.x < 64) {
    // lane owns bins 4*lane .. 4*lane+3; suffix sums over lanes (high bins first)
    const int lane = threadIdx.x;
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
          *sh_digit = (uint32_t)x;
          *sh_krem = krem - acc;
          break;
        }
        acc += hist[x];
      }
    }
  }
}

// One block per image.  Besides the image's kept tokens, the block writes
// the text rows of its sequence that lie between the previous image and
// this one (all rows before it for a sequence's first image, and the rows
// after it for the last), the text rows of sequences without images whose
// output follows the same budget prefix, and the matching cu_out entries.
// A text row t goes to  t + (budgets of the images before it);  an image's
// kept tokens start at  (first text row after it) + (budgets before it).
__global__ __launch_bounds__(kThreads) void select_kernel(
    const float *__restrict__ scores, const int32_t *__restrict__ budget,
    const int32_t *__restrict__ img_start, const int32_t *__restrict__ img_len,
    const int32_t *__restrict__ cu_img, const int32_t *__restrict__ cu_text,
    const int32_t *__restrict__ text_pos, int B, int n_img, int T_tot,
    int32_t *__restrict__ keep_idx, long long cap, int32_t *__restrict__ cu_out,
    int32_t *__restrict__ status) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t keys[kLdsKeys];
  __shared__ int wsum[4];
  __shared__ long long red[4];
  __shared__ uint32_t sh_digit;
  __shared__ int sh_krem, sh_b;
  const int tid = threadIdx.x;

  auto put = [&](long long o, int32_t v, int seq) __attribute__((always_inline)) {
    if (o < cap) keep_idx[o] = v;
    else if (status) atomicOr(status + seq, AVTP_FLAG_OUT_CAPACITY);
  };

  if (n_img == 0) {  // no images at all: every text row is kept in place
    for (int t = tid; t < T_tot; t += kThreads) put(t, text_pos[t], 0);
    for (int c = tid; c <= B; c += kThreads) cu_out[c] = cu_text[c];
    return;
  }

  const int i = blockIdx.x;
  for (int c = tid; c < B; c += kThreads)  // the sequence holding image i
    if (cu_img[c] <= i && i < cu_img[c + 1]) sh_b = c;
  const int st = img_start[i], n = img_len[i];
  const int k = eff_budget(budget, img_len, i);
  long long part = 0;  // budgets of the images before i
  for (int j = tid; j < i; j += kThreads) part += eff_budget(budget, img_len, j);
  const long long pre = block_sum_ll(part, red);  // (also publishes sh_b)
  const int b = sh_b;
  const int a_lo = cu_text[b], a_hi = cu_text[b + 1];
  const bool first = i == cu_img[b], last = i + 1 == cu_img[b + 1];
  // end of the previous image of b (an empty image may share its position
  // with a text row, which then comes after it)
  const int pend = first ? 0 : img_start[i - 1] + img_len[i - 1];
  int before = 0, between = 0;  // text rows of b before the image; of those, after the previous one
  for (int t = a_lo + tid; t < a_hi; t += kThreads) {
    const int p = text_pos[t];
    before += p < st;
    between += p < st && p >= pend;
  }
  const long long cnt = block_sum_ll(((long long)before << 32) | (long long)between, red);
  const int a0 = a_lo + (int)(cnt >> 32);        // first text row after the image start
  const int am = a0 - (int)(cnt & 0xffffffffll);  // first text row after the previous image

  // text rows between the previous image and this one, and after the last
  for (int t = am + tid; t < a0; t += kThreads) put(t + pre, text_pos[t], b);
  if (last)
    for (int t = a0 + tid; t < a_hi; t += kThreads) put(t + pre + k, text_pos[t], b);
  // cu_out of b (first image) and of the sequences without images that
  // share this budget prefix; the last image also closes the array
  for (int c = tid; c <= B; c += kThreads) {
    const int ci = cu_img[c];
    const bool empty_before = c < B && ci == i && cu_img[c + 1] == i;  // image-less, before i
    const bool empty_after = last && i == n_img - 1 && ci == n_img;    // trailing ones and B
    if ((first && c == b) || empty_before) cu_out[c] = (int32_t)(cu_text[c] + pre);
    if (empty_after) cu_out[c] = (int32_t)(cu_text[c] + pre + k);
    if (empty_before || (empty_after && c < B)) {
      const long long add = empty_before ? pre : pre + k;
      for (int t = cu_text[c]; t < cu_text[c + 1]; ++t) put(t + add, text_pos[t], c);
    }
  }

  if (k == 0) return;
  const long long base = (long long)a0 + pre;
  const float *s = scores + st;
  if (k == n) {
    for (int j = tid; j < n; j += kThreads) put(base + j, st + j, b);
    return;
  }

  // ---- radix select of the k-th largest key
  const bool in_lds = n <= kLdsKeys;
  if (in_lds)
    for (int j = tid; j < n; j += kThreads) keys[j] = order_key(s[j]);
  uint32_t prefix = 0, mask = 0;
  int krem = k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    hist[tid] = 0;
    __syncthreads();
    for (int j = tid; j < n; j += kThreads) {
      const uint32_t key = in_lds ? keys[j] : order_key(s[j]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    pick_digit(hist, krem, &sh_digit, &sh_krem);
    __syncthreads();
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    krem = sh_krem;
    __syncthreads();
  }
  const uint32_t theta = prefix;  // exactly krem keys equal to theta are kept

  // ---- ordered pass: keep > theta, and the first krem keys == theta
  if (in_lds) {
    // each thread takes a contiguous run of keys; two block scans place them
    const int per = (n + kThreads - 1) / kThreads;
    const int j0 = min(n, tid * per), j1 = min(n, j0 + per);
    int ne = 0;
    for (int j = j0; j < j1; ++j) ne += keys[j] == theta;
    int tot;
    int eq_rank = block_scan_int(ne, wsum, &tot);
    int nk = 0;
    for (int j = j0, r = eq_rank; j < j1; ++j) {
      const uint32_t key = keys[j];
      if (key > theta) ++nk;
      else if (key == theta) nk += (r++ < krem);
    }
    int pos = block_scan_int(nk, wsum, &tot);
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = keys[j];
      bool keep = key > theta;
      if (key == theta) keep = eq_rank++ < krem;
      if (keep) put(base + pos++, st + j, b);
    }
    return;
  }
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
    if (keep) put(base + pos, st + j, b);
  }
}

}  // namespace

hipError_t launch_select(hipStream_t st, const DevLayout &L, const float *scores,
                         const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                         int32_t *cu_out, int32_t *status) {
  const int grid = L.n_img > 0 ? L.n_img : 1;
  hipLaunchKernelGGL(select_kernel, dim3(grid), dim3(kThreads), 0, st, scores, budget, L.img_start,
                     L.img_len, L.cu_img, L.cu_text, L.text_pos, L.B, L.n_img, L.T_tot, keep_idx,
                     (long long)keep_capacity, cu_out, status);
  return hipGetLastError();
}

}  // namespace avtp
