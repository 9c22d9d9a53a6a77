// Per-image keep budgets (Sec. 3.3.3 adaptive keep ratio, with the 5 % / 95 %
// clamp of the appendix on alpha).  One 64-thread block per sequence.
//
// The only floating-point step is the integer weight of every image,
//   W_i = max(1, rint(min(w_i, 64) * 2^28)),
// evaluated in IEEE float64 with no contraction, in a fixed operation order
// (documented in include/avtp.h).  Everything after it is exact integer
// arithmetic:
//   * the real quota q_i = clamp(lam W_i, lo_i, hi_i) with sum q_i = K lies on
//     the segment between two consecutive breakpoints lo_i/W_i, hi_i/W_i of
//     f(lam) = sum_i clamp(lam W_i, lo_i, hi_i); every thread evaluates f at
//     its breakpoints by cross-multiplication (u64), the block picks the last
//     breakpoint with f < K and the first with f >= K;
//   * on that segment lam = P/Q with P = K - (pinned bounds) and Q = (free
//     weights), so q_i = P W_i / Q for free images;
//   * largest remainder: floor(q_i), then +1 for the K - sum floor images with
//     the largest remainders (P W_i mod Q), lowest image index first.
// Limits (checked on the host): n_i <= 2^20, <= 256 images per sequence,
// alpha <= 32, so every product fits in 63 bits.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"

namespace avtp {
namespace {

constexpr int kMaxImg = AVTP_MAX_IMAGES_PER_SEQ;
constexpr int kWeightBits = 28;
constexpr double kWeightCap = 64.0;

// a/b < c/d for positive denominators (all values < 2^31 * 2^35 in range)
__device__ inline bool frac_lt(uint64_t a, uint64_t b, uint64_t c, uint64_t d) {
  return a * d < c * b;
}

__device__ double image_weight(int n, long long M, float s32, double S, bool good, int mode,
                               double alpha, int K) {
#pragma clang fp contract(off)
  if (n == 0) return 0.0;
  const double u = (double)n / (double)M;
  const double s = (double)s32;
  double w;
  if (!good || !isfinite(s)) {
    w = u;
  } else if (mode == AVTP_BUDGET_PROPORTIONAL) {
    const double t1 = (1.0 - alpha) * u;
    const double t2 = alpha * (s / S);
    w = t1 + t2;
  } else if (K > 0) {
    const double t = u * S;
    const double d = (s - t) / (double)K;
    w = u + alpha * d;
  } else {
    w = u;
  }
  if (!(w > 0.0)) w = 0.0;
  if (w > kWeightCap) w = kWeightCap;
  return w;
}

__global__ __launch_bounds__(64) void budget_kernel(const float *__restrict__ img_sum,
                                                    const int32_t *__restrict__ img_len,
                                                    const int32_t *__restrict__ cu_img,
                                                    const int32_t *__restrict__ keep_total,
                                                    int mode, float alpha, int lo_pm, int hi_pm,
                                                    int floor_abs, int32_t *__restrict__ budget,
                                                    int32_t *__restrict__ status) {
  __shared__ uint64_t W[kMaxImg];
  __shared__ int32_t lo[kMaxImg], hi[kMaxImg], kk[kMaxImg];
  __shared__ uint64_t rem[kMaxImg];
  __shared__ uint64_t nx_num[64], nx_den[64], pv_num[64], pv_den[64];
  __shared__ int nx_ok[64], pv_ok[64];
  __shared__ double sh_S;
  __shared__ long long sh_M;
  __shared__ uint64_t sh_P, sh_Q;
  __shared__ int sh_bad;

  const int b = blockIdx.x, tid = threadIdx.x;
  const int i0 = cu_img[b], m = cu_img[b + 1] - i0;
  const long long K = keep_total[b];
  if (m <= 0) return;

  for (int i = tid; i < m; i += 64) {
    const long long n = img_len[i0 + i];
    long long l = (lo_pm * n + 999) / 1000;
    if (l < floor_abs) l = floor_abs;
    if (l > n) l = n;
    long long h = (hi_pm * n) / 1000;
    if (h < l) h = l;
    lo[i] = (int32_t)l;
    hi[i] = (int32_t)h;
  }
  if (tid == 0) {
    double S = 0.0;
    long long M = 0;
    for (int i = 0; i < m; ++i) {
      S = S + (double)img_sum[i0 + i];
      M += img_len[i0 + i];
    }
    sh_S = S;
    sh_M = M;
  }
  __syncthreads();
  const double S = sh_S;
  const bool good = isfinite(S) && S > 0.0;
  for (int i = tid; i < m; i += 64) {
    const int n = img_len[i0 + i];
    const double w = image_weight(n, sh_M, img_sum[i0 + i], S, good, mode, (double)alpha, (int)K);
    uint64_t q = 0;
    if (n > 0) {
      q = (uint64_t)rint(w * (double)(1ll << kWeightBits));
      if (q < 1) q = 1;
    }
    W[i] = q;
  }
  if (tid == 0) {
    long long slo = 0, shi = 0;
    for (int i = 0; i < m; ++i) {
      slo += lo[i];
      shi += hi[i];
    }
    sh_bad = (K < slo || K > shi) ? 1 : 0;
  }
  __syncthreads();
  if (sh_bad) {  // the host checks this too; keep outputs defined anyway
    for (int i = tid; i < m; i += 64) budget[i0 + i] = lo[i];
    if (tid == 0 && status) atomicOr(status + b, AVTP_FLAG_INFEASIBLE);
    return;
  }

  // breakpoints k < m: lo_k / W_k ; k >= m: hi_(k-m) / W_(k-m); zero-length images have none
  bool has_nx = false, has_pv = false;
  uint64_t bn = 0, bd = 1, pn = 0, pd = 1;
  for (int k = tid; k < 2 * m; k += 64) {
    const int i = k < m ? k : k - m;
    if (W[i] == 0) continue;
    const uint64_t num = (uint64_t)(k < m ? lo[i] : hi[i]), den = W[i];
    uint64_t f = 0;  // f(num/den) * den
    for (int j = 0; j < m; ++j) {
      if (W[j] == 0) continue;
      uint64_t v = num * W[j];
      const uint64_t l = (uint64_t)lo[j] * den, h = (uint64_t)hi[j] * den;
      v = v < l ? l : (v > h ? h : v);
      f += v;
    }
    if (f >= (uint64_t)K * den) {
      if (!has_nx || frac_lt(num, den, bn, bd)) {
        bn = num;
        bd = den;
        has_nx = true;
      }
    } else {
      if (!has_pv || frac_lt(pn, pd, num, den)) {
        pn = num;
        pd = den;
        has_pv = true;
      }
    }
  }
  nx_num[tid] = bn;
  nx_den[tid] = bd;
  nx_ok[tid] = has_nx;
  pv_num[tid] = pn;
  pv_den[tid] = pd;
  pv_ok[tid] = has_pv;
  __syncthreads();
  if (tid == 0) {
    bool hn = false, hp = false;
    for (int t = 0; t < 64; ++t) {
      if (nx_ok[t] && (!hn || frac_lt(nx_num[t], nx_den[t], bn, bd))) {
        bn = nx_num[t];
        bd = nx_den[t];
        hn = true;
      }
      if (pv_ok[t] && (!hp || frac_lt(pn, pd, pv_num[t], pv_den[t]))) {
        pn = pv_num[t];
        pd = pv_den[t];
        hp = true;
      }
    }
    // classify images on the open segment (prev, next]
    uint64_t pinned = 0, Q = 0;
    for (int i = 0; i < m; ++i) {
      if (W[i] == 0) {
        kk[i] = 0;
        rem[i] = 0;
        continue;
      }
      const bool low = hn && !frac_lt((uint64_t)lo[i], W[i], bn, bd);       // lo/W >= next
      const bool high = hp && !frac_lt(pn, pd, (uint64_t)hi[i], W[i]);      // hi/W <= prev
      if (low || (!hn)) {
        kk[i] = lo[i];
        rem[i] = 0;
        pinned += lo[i];
      } else if (high) {
        kk[i] = hi[i];
        rem[i] = 0;
        pinned += hi[i];
      } else {
        kk[i] = -1;  // free
        Q += W[i];
      }
    }
    sh_P = (uint64_t)K - pinned;
    sh_Q = Q;
  }
  __syncthreads();
  const uint64_t P = sh_P, Q = sh_Q;
  for (int i = tid; i < m; i += 64) {
    if (kk[i] == -1) {
      const uint64_t num = P * W[i];
      kk[i] = (int32_t)(num / Q);
      rem[i] = num % Q;
    }
  }
  __syncthreads();
  __shared__ long long sh_D;
  if (tid == 0) {
    long long s = 0;
    for (int i = 0; i < m; ++i) s += kk[i];
    sh_D = K - s;
  }
  __syncthreads();
  const long long D = sh_D;
  for (int i = tid; i < m; i += 64) {
    long long rank = 0;
    for (int j = 0; j < m; ++j) rank += (rem[j] > rem[i]) || (rem[j] == rem[i] && j < i);
    budget[i0 + i] = kk[i] + (rank < D ? 1 : 0);
  }
}

}  // namespace

hipError_t launch_budget(hipStream_t st, const DevLayout &L, const float *img_sum, int mode,
                         float alpha, int lo_permille, int hi_permille, int floor_abs,
                         int32_t *budget, int32_t *status) {
  hipLaunchKernelGGL(budget_kernel, dim3(L.B), dim3(64), 0, st, img_sum, L.img_len, L.cu_img,
                     L.keep_total, mode, alpha, lo_permille, hi_permille, floor_abs, budget,
                     status);
  return hipGetLastError();
}

}  // namespace avtp
