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
//     its breakpoints by cross-multiplication (u64), block reductions pick the
//     last breakpoint with f < K and the first with f >= K;
//   * on that segment lam = P/Q with P = K - (pinned bounds) and Q = (free
//     weights), so q_i = P W_i / Q for free images;
//   * largest remainder: floor(q_i), then +1 for the K - sum floor images with
//     the largest remainders (P W_i mod Q), lowest image index first.
// Limits (checked on the host): n_i <= 2^20 and <= 256 images per sequence;
// with W_i <= 2^28 every product is below 2^48 and every sum below 2^56.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"
#include "wave_ops.h"

namespace avtp {
namespace budget_rule {

constexpr int kMaxImg = AVTP_MAX_IMAGES_PER_SEQ;
constexpr int kWeightBits = 28;

// a/b < c/d for positive denominators (numerators <= 2^20, denominators <= 2^28)
__device__ inline bool frac_lt(uint64_t a, uint64_t b, uint64_t c, uint64_t d) {
  return a * d < c * b;
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

// Block-wide sums: wave all-reductions (integer sums, exact in any order),
// then the four wave partials in LDS.
template <int NTH, typename T>
__device__ inline T block_sum(T v, T *sh) {
  v = wave::sum(v);
  if (NTH == 64) return v;
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  bsync<NTH>();
  const T r = sh[0] + sh[1] + sh[2] + sh[3];
  bsync<NTH>();  // sh may be reused right away
  return r;
}

// A fraction num/den and whether it is set, as a value of wave::allreduce.
struct Frac {
  uint64_t n, d;
  uint32_t ok;
  template <int CTRL>
  __device__ static Frac shift(const Frac &a) {
    return Frac{wave::dpp<CTRL>(a.n), wave::dpp<CTRL>(a.d), wave::dpp<CTRL>(a.ok)};
  }
  __device__ static Frac at(const Frac &a, int lane) {
    return Frac{wave::lane_value(a.n, lane), wave::lane_value(a.d, lane),
                wave::lane_value(a.ok, lane)};
  }
};

// Block-wide extremes of two sets of fractions num/den (den > 0), each among
// the threads with its ok set: the smallest of the first set (bn/bd, hn) and
// the largest of the second (pn/pd, hp), in one pass.  ok = false if none.
// The choice is by exact comparison, so equal fractions in any form give the
// same value whichever is kept.
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
  if (b.lo.ok && (!a.lo.ok || frac_lt(b.lo.n, b.lo.d, a.lo.n, a.lo.d))) r.lo = b.lo;
  if (b.hi.ok && (!a.hi.ok || frac_lt(a.hi.n, a.hi.d, b.hi.n, b.hi.d))) r.hi = b.hi;
  return r;
}
template <int NTH>
__device__ inline void block_frac_ext2(uint64_t &bn, uint64_t &bd, bool &hn, uint64_t &pn,
                                       uint64_t &pd, bool &hp, Frac2 *sh) {
  Frac2 f = wave::allreduce(Frac2{Frac{bn, bd, hn ? 1u : 0u}, Frac{pn, pd, hp ? 1u : 0u}},
                            frac_ext_combine);
  if (NTH > 64) {
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = f;
    bsync<NTH>();
    f = sh[0];
    for (int t = 1; t < 4; ++t) f = frac_ext_combine(f, sh[t]);
    bsync<NTH>();
  }
  bn = f.lo.n;
  bd = f.lo.d;
  hn = f.lo.ok != 0;
  pn = f.hi.n;
  pd = f.hi.d;
  hp = f.hi.ok != 0;
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
  __shared__ uint64_t W[kMaxImg], rem[kMaxImg];
  __shared__ uint64_t fpart[NTH];  // partial f of a breakpoint, one per thread
  __shared__ int32_t lo[kMaxImg], hi[kMaxImg];
  __shared__ float sv[kMaxImg];
  __shared__ long long red_i[4];
  __shared__ uint64_t red_u[4];
  __shared__ Frac2 ext[4];
  __shared__ double sh_S, red_d[4];

  const int tid = threadIdx.x;
  const int i0 = cu_img[b], m = cu_img[b + 1] - i0;
  const long long K = keep_total[b];
  if (m <= 0) return;
  const bool mine = tid < m;  // this thread's image is tid

  long long n = 0, l = 0, h = 0;
  float s32 = 0.f;
  if (mine) {
    n = img_len[i0 + tid];
    s32 = img_sum[i0 + tid];
    l = (lo_pm * n + 999) / 1000;
    if (l < floor_abs) l = floor_abs;
    if (l > n) l = n;
    h = (hi_pm * n) / 1000;
    if (h < l) h = l;
    lo[tid] = (int32_t)l;
    hi[tid] = (int32_t)h;
    sv[tid] = s32;
  }
  const long long M = block_sum<NTH>(n, red_i);
  const long long slo = block_sum<NTH>(l, red_i);
  const long long shi = block_sum<NTH>(h, red_i);
  if (NTH == 64) bsync<NTH>();  // sv is read by thread 0 below
  if (tid == 0) {  // the image sum, in image order (it fixes the weights)
    double S = 0.0;
    for (int i = 0; i < m; ++i) S = S + (double)sv[i];
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
  uint64_t Wi = 0;
  if (mine) {
    if (n > 0) {
      if (wmax > 0.0) {
#pragma clang fp contract(off)
        const double r = w / wmax;
        Wi = (uint64_t)rint(r * (double)(1ll << kWeightBits));
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
  bsync<NTH>();

  // Breakpoints k < m: lo_k / W_k, k >= m: hi_(k-m) / W_(k-m) (zero-length
  // images have none).  f is evaluated at every breakpoint; each thread keeps
  // the smallest breakpoint with f >= K (next) and the largest with f < K
  // (prev).  With few breakpoints, np threads share one breakpoint's sum
  // over the images (np parts, combined in LDS; integer sums, so exact).
  bool hn = false, hp = false;
  uint64_t bn = 0, bd = 1, pn = 0, pd = 1;
  auto partial_f = [&](uint64_t num, uint64_t den, int j0, int j1) __attribute__((always_inline)) {
    uint64_t f = 0;  // f(num/den) * den over images j0 .. j1-1
#pragma unroll 4
    for (int j = j0; j < j1; ++j) {
      const uint64_t wj = W[j];
      if (wj == 0) continue;
      uint64_t v = num * wj;
      const uint64_t lj = (uint64_t)lo[j] * den, hj = (uint64_t)hi[j] * den;
      v = v < lj ? lj : (v > hj ? hj : v);
      f += v;
    }
    return f;
  };
  auto keep_ext = [&](uint64_t f, uint64_t num, uint64_t den) __attribute__((always_inline)) {
    // value selects (not stores through a chosen reference), so that the six
    // values stay in registers
    const bool ge = f >= (uint64_t)K * den;
    const bool tn = ge && (!hn || frac_lt(num, den, bn, bd));
    const bool tp = !ge && (!hp || frac_lt(pn, pd, num, den));
    bn = tn ? num : bn;
    bd = tn ? den : bd;
    hn = hn || tn;
    pn = tp ? num : pn;
    pd = tp ? den : pd;
    hp = hp || tp;
  };
  const int nbp = 2 * m;
  const int np = nbp <= NTH / 4 ? 4 : (nbp <= NTH / 2 ? 2 : 1);  // parts; block-uniform
  if (np > 1) {
    const int KB = NTH / np;  // >= nbp
    const int k = tid % KB, part = tid / KB;
    const int per = (m + np - 1) / np, j0 = min(m, part * per), j1 = min(m, j0 + per);
    bool ok = false;
    uint64_t num = 0, den = 1, f = 0;
    if (k < nbp) {
      const int i = k < m ? k : k - m;
      if (W[i] != 0) {
        ok = true;
        num = (uint64_t)(k < m ? lo[i] : hi[i]);
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
      const uint64_t num = (uint64_t)(k < m ? lo[i] : hi[i]), den = W[i];
      keep_ext(partial_f(num, den, 0, m), num, den);
    }
  }
  block_frac_ext2<NTH>(bn, bd, hn, pn, pd, hp, ext);

  // classify the images on the segment (prev, next]: pinned at lo, at hi, or free
  int32_t kk = 0;
  uint64_t pinned = 0, freeW = 0;
  bool fr = false;
  if (mine && Wi != 0) {
    const bool low = hn && !frac_lt((uint64_t)l, Wi, bn, bd);   // lo/W >= next
    const bool high = hp && !frac_lt(pn, pd, (uint64_t)h, Wi);  // hi/W <= prev
    if (low || !hn) {
      kk = (int32_t)l;
      pinned = (uint64_t)l;
    } else if (high) {
      kk = (int32_t)h;
      pinned = (uint64_t)h;
    } else {
      fr = true;
      freeW = Wi;
    }
  }
  const uint64_t P = (uint64_t)K - block_sum<NTH>(pinned, red_u);
  const uint64_t Q = block_sum<NTH>(freeW, red_u);
  uint64_t ri = 0;
  if (fr) {
    const uint64_t num = P * Wi;
    kk = (int32_t)(num / Q);
    ri = num % Q;
  }
  if (mine) rem[tid] = ri;
  if (NTH == 64) bsync<NTH>();  // rem is read by every lane below
  const long long D = K - block_sum<NTH>((long long)kk, red_i);  // the units left to hand out
  // largest remainders first, lowest image index among equal ones
  if (mine) {
    long long rank = 0;
    for (int j = 0; j < m; ++j) rank += (rem[j] > ri) || (rem[j] == ri && j < tid);
    out(tid, (int32_t)(kk + (rank < D ? 1 : 0)));
  }
}

}  // namespace budget_rule
}  // namespace avtp
