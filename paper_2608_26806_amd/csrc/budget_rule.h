// The per-sequence budget rule (Sec. 3.3.3 adaptive keep ratio, with the
// 5 % / 95 % clamp of the appendix on alpha) as a block-level device
// function, shared by the budget kernel and the selection kernels that
// compute their sequence's budgets themselves.  One thread per image.
//
// The only floating-point step is the integer weight of every image,
//   W_i = max(1, rint((w_i / w_max) * 2^28))
// (w_max the largest weight of the sequence: only the ratios of the weights
// enter the water-filling), evaluated in IEEE float64 with no contraction,
// in a fixed operation order (documented in include/avtp.h).  Everything
// after it is exact integer arithmetic:
//   * the real quota q_i = clamp(lam W_i, lo_i, hi_i) with sum q_i = K lies on
//     the segment between two consecutive breakpoints lo_i/W_i, hi_i/W_i of
//     f(lam) = sum_i clamp(lam W_i, lo_i, hi_i); every thread evaluates f at
//     its breakpoints by cross-multiplication (32 x 32 -> 64-bit products),
//     and one block reduction picks the last breakpoint with f < K and the
//     first with f >= K;
//   * on that segment lam = P/Q with P = K - (pinned bounds) and Q = (free
//     weights), so q_i = P W_i / Q for free images;
//   * largest remainder: floor(q_i), then +1 for the K - sum floor images with
//     the largest remainders (P W_i mod Q), lowest image index first.
// Limits (checked on the host): n_i <= 2^20 and <= 256 images per sequence,
// so token counts, bounds and K (at most their sum, 2^28) fit 32 bits; with
// W_i <= 2^28 every product is below 2^48 and every sum below 2^56.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"
#include "wave_ops.h"

namespace avtp {
namespace budget_rule {

constexpr int kMaxImg = AVTP_MAX_IMAGES_PER_SEQ;
constexpr int kWeightBits = 28;

// a/b < c/d for positive denominators.  Numerators are token counts (at
// most 2^20) and denominators integer weights (at most 2^28), so both
// products are exact 32 x 32 -> 64-bit multiplies.
__device__ inline bool frac_lt(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return (uint64_t)a * d < (uint64_t)c * b;
}

__device__ inline double image_weight(int n, long long M, float s32, double S, bool good, int mode,
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
  return w;
}

// One thread per image: blocks of 256 threads, or a single wave of 64 when
// no sequence has more than 16 images (then every block-wide reduction is a
// wave butterfly, with no LDS round trip or barrier).
constexpr int kThreads = 256;
static_assert(kMaxImg <= kThreads, "one thread per image");

// The rule's barrier: the block's (NTH = 256), or, with NTH = 64, ordering
// among the lanes of the one wave that runs the rule (the whole block of the
// budget kernel, or wave 0 of a selection block while the others wait): a
// wave's LDS accesses take effect in program order, so no hardware barrier
// is needed, only that the compiler keeps that order.
template <int NTH>
__device__ inline void bsync() {
  if (NTH == 64) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}

// Block-wide reduction of a value of wave::allreduce (an integer sum, or a
// choice by exact comparison, so the combining order does not matter): the
// wave's, then the four wave results in LDS.
template <int NTH, typename V, typename F>
__device__ inline V block_reduce(V v, F combine, V *sh) {
  v = wave::allreduce(v, combine);
  if (NTH == 64) return v;
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  bsync<NTH>();
  V r = sh[0];
  for (int t = 1; t < 4; ++t) r = combine(r, sh[t]);
  bsync<NTH>();  // sh may be reused right away
  return r;
}

// One 32-bit integer sum.
using U32 = wave::One<uint32_t>;
__device__ inline U32 u32_add(const U32 &a, const U32 &b) { return U32{a.x + b.x}; }

// Three 32-bit integer sums in one reduction (the token count, the lower
// and the upper bounds of a sequence: each at most 256 * 2^20 = 2^28).
struct Sum3 {
  uint32_t x, y, z;
  template <int CTRL>
  __device__ static Sum3 shift(const Sum3 &a) {
    return Sum3{wave::dpp<CTRL>(a.x), wave::dpp<CTRL>(a.y), wave::dpp<CTRL>(a.z)};
  }
  __device__ static Sum3 at(const Sum3 &a, int lane) {
    return Sum3{wave::lane_value(a.x, lane), wave::lane_value(a.y, lane),
                wave::lane_value(a.z, lane)};
  }
};
__device__ inline Sum3 sum3_add(const Sum3 &a, const Sum3 &b) {
  return Sum3{a.x + b.x, a.y + b.y, a.z + b.z};
}

// The pinned units (at most 2^28 in all) and the free weights (each at most
// 2^28, so their sum needs 64 bits) of a segment, summed together.
struct PinFree {
  uint32_t pinned;
  uint64_t free_w;
  template <int CTRL>
  __device__ static PinFree shift(const PinFree &a) {
    return PinFree{wave::dpp<CTRL>(a.pinned), wave::dpp<CTRL>(a.free_w)};
  }
  __device__ static PinFree at(const PinFree &a, int lane) {
    return PinFree{wave::lane_value(a.pinned, lane), wave::lane_value(a.free_w, lane)};
  }
};
__device__ inline PinFree pin_free_add(const PinFree &a, const PinFree &b) {
  return PinFree{a.pinned + b.pinned, a.free_w + b.free_w};
}

// A fraction n/d with d > 0, or none (d == 0; no weight is 0 where a
// fraction is formed), as a value of wave::allreduce.
struct Frac {
  uint32_t n, d;
  template <int CTRL>
  __device__ static Frac shift(const Frac &a) {
    return Frac{wave::dpp<CTRL>(a.n), wave::dpp<CTRL>(a.d)};
  }
  __device__ static Frac at(const Frac &a, int lane) {
    return Frac{wave::lane_value(a.n, lane), wave::lane_value(a.d, lane)};
  }
};

// Block-wide extremes of two sets of fractions: the smallest of the first
// (lo) and the largest of the second (hi), in one pass.  The choice is by
// exact comparison, so equal fractions in any form give the same value
// whichever is kept.
struct Frac2 {
  Frac lo, hi;
  template <int CTRL>
  __device__ static Frac2 shift(const Frac2 &a) {
    return Frac2{Frac::shift<CTRL>(a.lo), Frac::shift<CTRL>(a.hi)};
  }
  __device__ static Frac2 at(const Frac2 &a, int lane) {
    return Frac2{Frac::at(a.lo, lane), Frac::at(a.hi, lane)};
  }
};
__device__ inline Frac2 frac_ext_combine(const Frac2 &a, const Frac2 &b) {
  Frac2 r = a;
  if (b.lo.d && (!a.lo.d || frac_lt(b.lo.n, b.lo.d, a.lo.n, a.lo.d))) r.lo = b.lo;
  if (b.hi.d && (!a.hi.d || frac_lt(a.hi.n, a.hi.d, b.hi.n, b.hi.d))) r.hi = b.hi;
  return r;
}

// The budgets of sequence b's images, by a block of NTH threads (every
// thread of the block calls it; b is block-uniform).  The thread of image
// i0 + t calls out(t, budget) once, t < the sequence's image count; a
// sequence without images calls nothing.  Sets AVTP_FLAG_INFEASIBLE in
// status[b] (if status is given) when keep_total[b] is outside the bounds.
template <int NTH, typename Out>
__device__ __attribute__((always_inline)) inline void seq_budget(
    int b, const float *__restrict__ img_sum, const int32_t *__restrict__ img_len,
    const int32_t *__restrict__ cu_img, const int32_t *__restrict__ keep_total, int mode,
    float alpha, int lo_pm, int hi_pm, int floor_abs, int32_t *__restrict__ status, Out out) {
  __shared__ uint32_t W[kMaxImg], lo[kMaxImg], hi[kMaxImg];
  __shared__ uint64_t rem[kMaxImg];
  __shared__ uint64_t fpart[NTH];  // partial f of a breakpoint, one per thread
  __shared__ __attribute__((aligned(16))) float sv[kMaxImg];
  __shared__ Sum3 red3[4];
  __shared__ PinFree red_pf[4];
  __shared__ Frac2 ext[4];
  __shared__ U32 red_k[4];
  __shared__ double sh_S, red_d[4];

  const int tid = threadIdx.x;
  const int i0 = cu_img[b], m = cu_img[b + 1] - i0;
  const long long K = keep_total[b];
  if (m <= 0) return;
  const bool mine = tid < m;  // this thread's image is tid

  // token count and bounds (at most 2^20 each; the host checks the lengths)
  uint32_t n = 0, l = 0, h = 0;
  float s32 = 0.f;
  if (mine) {
    const long long nn = img_len[i0 + tid];
    s32 = img_sum[i0 + tid];
    long long ll = (lo_pm * nn + 999) / 1000;
    if (ll < floor_abs) ll = floor_abs;
    if (ll > nn) ll = nn;
    long long hh = (hi_pm * nn) / 1000;
    if (hh < ll) hh = ll;
    n = (uint32_t)nn;
    l = (uint32_t)ll;
    h = (uint32_t)hh;
    lo[tid] = l;
    hi[tid] = h;
    sv[tid] = s32;
  }
  const Sum3 tot = block_reduce<NTH>(Sum3{n, l, h}, sum3_add, red3);
  const long long M = tot.x, slo = tot.y, shi = tot.z;
  if (NTH == 64) bsync<NTH>();  // sv is read by thread 0 below
  if (tid == 0) {  // the image sum, in image order (it fixes the weights)
    double S = 0.0;
    int i = 0;
    for (; i + 4 <= m; i += 4) {  // four values per LDS read, added one at a time
      const float4 v = *reinterpret_cast<const float4 *>(&sv[i]);
      S = S + (double)v.x;
      S = S + (double)v.y;
      S = S + (double)v.z;
      S = S + (double)v.w;
    }
    for (; i < m; ++i) S = S + (double)sv[i];
    sh_S = S;
  }
  bsync<NTH>();
  const double S = sh_S;
  const bool good = isfinite(S) && S > 0.0;
  double w = 0.0;
  if (mine) w = image_weight((int)n, M, s32, S, good, mode, (double)alpha, (int)K);
  // the largest weight (weights are >= 0; images without tokens have none)
  double wmax = wave::max(w);
  if (NTH > 64) {
    if ((tid & 63) == 0) red_d[tid >> 6] = wmax;
    bsync<NTH>();
    wmax = fmax(fmax(red_d[0], red_d[1]), fmax(red_d[2], red_d[3]));
  }
  uint32_t Wi = 0;
  if (mine) {
    if (n > 0) {
      if (wmax > 0.0) {
#pragma clang fp contract(off)
        const double r = w / wmax;
        Wi = (uint32_t)rint(r * (double)(1ll << kWeightBits));
      }
      if (Wi < 1) Wi = 1;
    }
    W[tid] = Wi;
  }
  if (K < slo || K > shi) {  // the host checks this too; keep outputs defined anyway
    if (mine) out(tid, (int32_t)l);
    if (tid == 0 && status) atomicOr(status + b, AVTP_FLAG_INFEASIBLE);
    return;
  }
  const uint32_t K32 = (uint32_t)K;  // slo <= K <= shi <= 2^28
  bsync<NTH>();

  // Breakpoints k < m: lo_k / W_k, k >= m: hi_(k-m) / W_(k-m) (zero-length
  // images have none).  f is evaluated at every breakpoint; each thread keeps
  // the smallest breakpoint with f >= K (next) and the largest with f < K
  // (prev).  With few breakpoints, np threads share one breakpoint's sum
  // over the images (np parts, combined in LDS; integer sums, so exact).
  Frac next{0, 0}, prev{0, 0};  // none yet
  auto partial_f = [&](uint32_t num, uint32_t den, int j0, int j1) __attribute__((always_inline)) {
    uint64_t f = 0;  // f(num/den) * den over images j0 .. j1-1 (below 2^56)
#pragma unroll 4
    for (int j = j0; j < j1; ++j) {
      const uint32_t wj = W[j];
      if (wj == 0) continue;
      uint64_t v = (uint64_t)num * wj;
      const uint64_t lj = (uint64_t)lo[j] * den, hj = (uint64_t)hi[j] * den;
      v = v < lj ? lj : (v > hj ? hj : v);
      f += v;
    }
    return f;
  };
  auto keep_ext = [&](uint64_t f, uint32_t num, uint32_t den) __attribute__((always_inline)) {
    // value selects (not stores through a chosen reference), so that the
    // four values stay in registers
    const bool ge = f >= (uint64_t)K32 * den;
    const bool tn = ge && (!next.d || frac_lt(num, den, next.n, next.d));
    const bool tp = !ge && (!prev.d || frac_lt(prev.n, prev.d, num, den));
    next.n = tn ? num : next.n;
    next.d = tn ? den : next.d;
    prev.n = tp ? num : prev.n;
    prev.d = tp ? den : prev.d;
  };
  const int nbp = 2 * m;
  const int np = nbp <= NTH / 4 ? 4 : (nbp <= NTH / 2 ? 2 : 1);  // parts; block-uniform
  if (np > 1) {
    const int KB = NTH / np;  // >= nbp
    const int k = tid % KB, part = tid / KB;
    const int per = (m + np - 1) / np, j0 = min(m, part * per), j1 = min(m, j0 + per);
    bool ok = false;
    uint32_t num = 0, den = 1;
    uint64_t f = 0;
    if (k < nbp) {
      const int i = k < m ? k : k - m;
      if (W[i] != 0) {
        ok = true;
        num = k < m ? lo[i] : hi[i];
        den = W[i];
        f = partial_f(num, den, j0, j1);
      }
    }
    fpart[tid] = f;
    bsync<NTH>();
    if (part == 0 && ok) {
      for (int q = 1; q < np; ++q) f += fpart[q * KB + k];
      keep_ext(f, num, den);
    }
  } else {
    for (int k = tid; k < nbp; k += NTH) {
      const int i = k < m ? k : k - m;
      if (W[i] == 0) continue;
      const uint32_t num = k < m ? lo[i] : hi[i], den = W[i];
      keep_ext(partial_f(num, den, 0, m), num, den);
    }
  }
  const Frac2 ext2 = block_reduce<NTH>(Frac2{next, prev}, frac_ext_combine, ext);
  next = ext2.lo;
  prev = ext2.hi;

  // classify the images on the segment (prev, next]: pinned at lo, at hi, or free
  uint32_t kk = 0;
  PinFree pf{0, 0};
  bool fr = false;
  if (mine && Wi != 0) {
    const bool low = next.d && !frac_lt(l, Wi, next.n, next.d);   // lo/W >= next
    const bool high = prev.d && !frac_lt(prev.n, prev.d, h, Wi);  // hi/W <= prev
    if (low || !next.d) {
      kk = l;
      pf.pinned = l;
    } else if (high) {
      kk = h;
      pf.pinned = h;
    } else {
      fr = true;
      pf.free_w = Wi;
    }
  }
  const PinFree seg = block_reduce<NTH>(pf, pin_free_add, red_pf);
  const uint32_t P = K32 - seg.pinned;  // units the free images share (P <= K)
  const uint64_t Q = seg.free_w;
  uint64_t ri = 0;
  if (fr) {
    const uint64_t num = (uint64_t)P * Wi;
    kk = (uint32_t)(num / Q);
    ri = num % Q;
  }
  if (mine) rem[tid] = ri;
  if (NTH == 64) bsync<NTH>();  // rem is read by every lane below
  // the units left to hand out (block_reduce's barriers also publish rem)
  const long long D = K - (long long)block_reduce<NTH>(U32{kk}, u32_add, red_k).x;
  // largest remainders first, lowest image index among equal ones
  if (mine) {
    long long rank = 0;
    for (int j = 0; j < m; ++j) rank += (rem[j] > ri) || (rem[j] == ri && j < tid);
    out(tid, (int32_t)(kk + (rank < D ? 1 : 0)));
  }
}

}  // namespace budget_rule
}  // namespace avtp
