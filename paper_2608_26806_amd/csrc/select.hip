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
#include "budget_rule.h"
#include "row_copy.h"
#include "wave_ops.h"

namespace avtp {
namespace {

constexpr int kThreads = 256;
// most images per sequence for which wave 0 alone runs the in-block budget
// rule (as the budget kernel does: with more, the four waves' share of the
// breakpoint sums pays more)
constexpr int kWaveBudgetMaxImages = 16;

// Monotone map float -> uint32 (larger score -> larger key); -0.0 == +0.0,
// NaN -> 0, below every other value.
__device__ inline uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline int clamp_budget(int k, int n) { return k < 0 ? 0 : (k > n ? n : k); }
__device__ inline int eff_budget(const int32_t *budget, const int32_t *img_len, int i) {
  return clamp_budget(budget[i], img_len[i]);
}

// Where a selection block takes the budgets from.  part(i): this thread's
// share of the budgets of every image before i (the block sums the shares);
// k(i): image i's budget, clamped to [0, len].
struct BudGlobal {  // written by the budget kernel
  const int32_t *budget, *img_len;
  __device__ long long part(int i) const {
    long long p = 0;
    for (int j = threadIdx.x; j < i; j += kThreads) p += eff_budget(budget, img_len, j);
    return p;
  }
  __device__ int k(int i) const { return eff_budget(budget, img_len, i); }
};
struct BudInBlock {  // computed by the block for its own sequence b (in LDS)
  const int32_t *bud;  // budgets of b's images, index j - i0
  const int32_t *img_len, *keep_total;
  int b, i0;
  // every earlier sequence keeps exactly its keep_total (the host rejects
  // totals its bounds cannot meet, and the rule hands out exactly K)
  __device__ long long part(int i) const {
    long long p = 0;
    for (int c = threadIdx.x; c < b; c += kThreads) p += keep_total[c];
    for (int j = i0 + threadIdx.x; j < i; j += kThreads) p += clamp_budget(bud[j - i0], img_len[j]);
    return p;
  }
  __device__ int k(int i) const { return clamp_budget(bud[i - i0], img_len[i]); }
};

// The budget rule's inputs, for the kernels that run it in-block.
struct RuleArgs {
  const float *img_sum;
  const int32_t *keep_total;
  int mode;
  float alpha;
  int lo_pm, hi_pm, floor_abs;
  int32_t *budget;  // every image's budget is also written here (by one block)
};

// How a selection block gets its budgets.
enum BudMode {
  kBudGlobal = 0,  // from the budget kernel's output
  kBudBlock = 1,   // the rule run by the whole block
  kBudWave = 2,    // the rule run by wave 0 while the other waves load the image
};

// exclusive block scans of two 0/1 flags at once (256 threads, 4 waves):
// returns the exclusive count of f, writes that of g to *g_before and the
// block totals to *f_total and *g_total
__device__ inline int block_scan_flags(bool f, bool g, int *wsum, int *f_total, int *g_before,
                                       int *g_total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long mf = __ballot(f), mg = __ballot(g);
  const unsigned long long below = (1ull << lane) - 1ull;
  // per wave: the two counts packed in one int (each at most 64)
  if (lane == 0) wsum[wave] = (__popcll(mg) << 16) | __popcll(mf);
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wave; ++w) off += wsum[w];
  const int tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  *f_total = tot & 0xffff;
  *g_total = tot >> 16;
  *g_before = (off >> 16) + __popcll(mg & below);
  return (off & 0xffff) + __popcll(mf & below);
}

// exclusive block scan of an integer (256 threads); block total in *total
__device__ inline int block_scan_int(int v, int *wsum, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int inc = (int)wave::prefix_sum((uint32_t)v);  // (v >= 0)
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
  v = wave::sum(v);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  const long long r = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return r;
}

constexpr int kLdsKeys = 4096;  // images up to this length keep their keys in LDS

// Digit of the krem-th largest key among those matching (prefix, mask), from
// a 256-bin histogram of one byte (16-byte aligned); krem becomes the rank
// inside that bin.  Every wave calls it and gets the same, wave-uniform
// result, so no wave waits for another to publish it.
__device__ inline void pick_digit(const uint32_t *hist, int &krem, uint32_t &digit) {
  // lane l owns bins 4*o .. 4*o+3 with o = 63 - l, so that a prefix sum over
  // the lanes is the sum over the bins from the highest down to its own
  const int o = 63 - (int)(threadIdx.x & 63);
  const uint4 b = *reinterpret_cast<const uint4 *>(hist + 4 * o);
  const int c = (int)(b.x + b.y + b.z + b.w);
  const int suf = (int)wave::prefix_sum((uint32_t)c);
  const int above = suf - c;  // keys in higher bins
  // exactly one lane holds the krem-th key (1 <= krem <= the keys counted)
  const bool mine = suf >= krem && above < krem;
  const int src = __builtin_ctzll(__ballot(mine));
  // that lane: its bins from the highest down
  int d = 4 * o, r = krem - above;
  if (r > (int)b.w) {
    r -= (int)b.w;
    if (r > (int)b.z) {
      r -= (int)b.z;
      if (r > (int)b.y) r -= (int)b.y;
      else d += 1;
    } else {
      d += 2;
    }
  } else {
    d += 3;
  }
  digit = (uint32_t)__builtin_amdgcn_readlane(d, src);
  krem = __builtin_amdgcn_readlane(r, src);
}

// One block per image.  Besides the image's kept tokens, the block writes
// the text rows of its sequence that lie between the previous image and
// this one (all rows before it for a sequence's first image, and the rows
// after it for the last), the text rows of sequences without images whose
// output follows the same budget prefix, and the matching cu_out entries.
// A text row t goes to  t + (budgets of the images before it);  an image's
// kept tokens start at  (first text row after it) + (budgets before it).
struct SelArgs {
  const float *scores;
  const int32_t *budget, *img_start, *img_len, *cu_img, *cu_text, *text_pos;
  int B, n_img, T_tot;
  int32_t *cu_out;  // null: not written (all but one slice of the fused kernel)
};

// The kept tokens of image i (and the text rows around it), reported as
// put(output index, token index, sequence) in no particular order.
template <int MODE, typename Put>
__device__ __attribute__((always_inline)) inline void select_image(const SelArgs &A,
                                                                   const RuleArgs &R, int i,
                                                                   bool write, int32_t *status,
                                                                   Put put) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[3][256];  // one per pass, used in turn
  __shared__ uint32_t keys[kLdsKeys];
  __shared__ int wsum[4];
  __shared__ long long red[4];
  __shared__ int sh_b, cnt[2];
  __shared__ int32_t bud_sh[AVTP_MAX_IMAGES_PER_SEQ];  // the in-block budgets of b's images
  const int tid = threadIdx.x;
  const float *__restrict__ scores = A.scores;
  const int32_t *__restrict__ img_start = A.img_start;
  const int32_t *__restrict__ img_len = A.img_len;
  const int32_t *__restrict__ cu_img = A.cu_img;
  const int32_t *__restrict__ cu_text = A.cu_text;
  const int32_t *__restrict__ text_pos = A.text_pos;
  const int B = A.B, n_img = A.n_img, T_tot = A.T_tot;
  int32_t *__restrict__ cu_out = A.cu_out;

  if (n_img == 0) {  // no images at all: every text row is kept in place
    for (int t = tid; t < T_tot; t += kThreads) put(t, text_pos[t], 0);
    if (cu_out)
      for (int c = tid; c <= B; c += kThreads) cu_out[c] = cu_text[c];
    return;
  }

  for (int c = tid; c < B; c += kThreads)  // the sequence holding image i
    if (cu_img[c] <= i && i < cu_img[c + 1]) sh_b = c;
  if (tid == 0) cnt[0] = cnt[1] = 0;
  __syncthreads();
  const int b = sh_b;
  const int st = img_start[i], n = img_len[i];
  const bool in_lds = n <= kLdsKeys;
  const int a_lo = cu_text[b], a_hi = cu_text[b + 1];
  const bool first = i == cu_img[b], last = i + 1 == cu_img[b + 1];

  // The part that needs no budget, by threads t0 .. t0 + nt - 1 and without
  // a block barrier: the image's order keys into LDS, the first radix
  // pass's histogram cleared, and the text rows of b before the image (and
  // of those, after the previous image; an empty image may share its
  // position with a text row, which then comes after it) counted in LDS.
  auto load_image = [&](int t0, int nt) __attribute__((always_inline)) {
    const int u = tid - t0;
    if (in_lds)
#pragma unroll 4
      for (int j = u; j < n; j += nt) keys[j] = order_key(scores[st + j]);
    for (int x = u; x < 256; x += nt) hist[0][x] = hist[1][x] = 0;
    const int pend = first ? 0 : img_start[i - 1] + img_len[i - 1];
    int before = 0, between = 0;
    for (int t = a_lo + u; t < a_hi; t += nt) {
      const int p = text_pos[t];
      before += p < st;
      between += p < st && p >= pend;
    }
    if (before) atomicAdd(&cnt[0], before);
    if (between) atomicAdd(&cnt[1], between);
  };
  // The budgets: read, or the rule run for b (while the image loads, when
  // wave 0 runs it).  The block with write set stores budget[i], and the one
  // of b's first image the infeasibility flag.
  const int i0 = cu_img[b];
  auto rule_out = [&](int t, int32_t v) __attribute__((always_inline)) { bud_sh[t] = v; };
  int32_t *rst = write && i == i0 ? status : nullptr;
  if constexpr (MODE == kBudWave) {
    if (tid < 64)
      budget_rule::seq_budget<64>(b, R.img_sum, img_len, cu_img, R.keep_total, R.mode, R.alpha,
                                  R.lo_pm, R.hi_pm, R.floor_abs, rst, rule_out);
    else
      load_image(64, kThreads - 64);
  } else if constexpr (MODE == kBudBlock) {
    load_image(0, kThreads);  // (its loads are in flight during the rule)
    budget_rule::seq_budget<kThreads>(b, R.img_sum, img_len, cu_img, R.keep_total, R.mode,
                                      R.alpha, R.lo_pm, R.hi_pm, R.floor_abs, rst, rule_out);
  } else {
    load_image(0, kThreads);
  }
  __syncthreads();  // keys, histogram, counts and budgets are in LDS
  long long part = 0;  // (this thread's share of) the budgets of the images before i
  int k;
  if constexpr (MODE == kBudGlobal) {
    const BudGlobal bud{A.budget, img_len};
    part = bud.part(i);
    k = bud.k(i);
  } else {
    const BudInBlock bud{bud_sh, img_len, R.keep_total, b, i0};
    part = bud.part(i);
    k = bud.k(i);
    if (write && tid == 0) R.budget[i] = bud_sh[i - i0];
  }
  const long long pre = block_sum_ll(part, red);
  const int a0 = a_lo + cnt[0];  // first text row after the image start
  const int am = a0 - cnt[1];    // first text row after the previous image

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
    if (cu_out && ((first && c == b) || empty_before)) cu_out[c] = (int32_t)(cu_text[c] + pre);
    if (cu_out && empty_after) cu_out[c] = (int32_t)(cu_text[c] + pre + k);
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
  uint32_t prefix = 0, mask = 0;
  int krem = k;
  // One barrier per pass: pass p counts into hist[p % 3], which was cleared
  // above (p < 2) or after the barrier of pass p - 2; after its own barrier
  // every wave reads the complete histogram and picks the digit itself, and
  // the block clears hist[(p + 2) % 3], which pass p - 1's picks read before
  // every wave reached this barrier.
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    uint32_t *h = hist[pass % 3];
    for (int j = tid; j < n; j += kThreads) {
      const uint32_t key = in_lds ? keys[j] : order_key(s[j]);
      if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
    }
    __syncthreads();  // the histogram is complete
    if (pass + 2 < 4) hist[(pass + 2) % 3][tid] = 0;
    uint32_t digit;
    pick_digit(h, krem, digit);
    prefix |= digit << shift;
    mask |= 255u << shift;
  }
  const uint32_t theta = prefix;  // exactly krem keys equal to theta are kept

  // ---- ordered pass: keep > theta, and the first krem keys == theta.  The
  // kept keys before a key are the keys > theta before it plus the first
  // krem of the keys == theta before it, so one scan of both counts places
  // every kept key.
  if (in_lds) {
    // each thread takes a contiguous run of keys; the two counts share one
    // 32-bit block scan (each is at most kLdsKeys < 2^16)
    const int per = (n + kThreads - 1) / kThreads;
    const int j0 = min(n, tid * per), j1 = min(n, j0 + per);
    int ne = 0, ng = 0;
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = keys[j];
      ne += key == theta;
      ng += key > theta;
    }
    int tot;
    const int before = block_scan_int((ng << 16) | ne, wsum, &tot);
    int eq_rank = before & 0xffff;
    int pos = (before >> 16) + min(krem, eq_rank);
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = keys[j];
      bool keep = key > theta;
      if (key == theta) keep = eq_rank++ < krem;
      if (keep) put(base + pos++, st + j, b);
    }
    return;
  }
  int eq_carry = 0, gt_carry = 0;
  for (int c0 = 0; c0 < n; c0 += kThreads) {
    const int j = c0 + tid;
    uint32_t key = 0;
    if (j < n) key = order_key(s[j]);
    const bool gt = j < n && key > theta;
    const bool eq = j < n && key == theta;
    int eq_tot, gt_tot;
    int gt_before;
    const int eq_rank = block_scan_flags(eq, gt, wsum, &eq_tot, &gt_before, &gt_tot) + eq_carry;
    const bool keep = gt || (eq && eq_rank < krem);
    const int pos = gt_carry + gt_before + min(krem, eq_rank);
    eq_carry += eq_tot;
    gt_carry += gt_tot;
    if (keep) put(base + pos, st + j, b);
  }
}

// MODE (BudMode): kBudGlobal reads the budget kernel's output; otherwise the
// block first runs the budget rule for its image's sequence (RuleArgs).
template <int MODE>
__global__ __launch_bounds__(kThreads) void select_kernel(SelArgs A, RuleArgs R,
                                                         int32_t *__restrict__ keep_idx,
                                                         long long cap, int32_t *__restrict__ status) {
  const int i = A.n_img > 0 ? (int)blockIdx.x : 0;
  auto put = [&](long long o, int32_t v, int seq) __attribute__((always_inline)) {
    if (o < cap) keep_idx[o] = v;
    else if (status) atomicOr(status + seq, AVTP_FLAG_OUT_CAPACITY);
  };
  select_image<MODE>(A, R, i, true, status, put);
}

// Fused selection and compaction: S blocks per image (slices).  Every slice
// runs the image's selection (its keys are few and sit in LDS), owns the
// output rows o with o mod S == slice, writes their keep_idx entries, lists
// them in LDS, and then copies those rows of every tensor with groups of
// lanes.  No block waits for another.
constexpr int kListCap = 4096;  // output rows one slice may own (the host sizes S for it)

struct SCArgs {
  SelArgs sel;
  int32_t *keep_idx;
  long long cap;    // keep_idx entries
  long long n_out;  // rows of every destination tensor (rows at or past it are not copied)
  int32_t *status;
  int S;
  int n_t;
  CTensor t[AVTP_MAX_TENSORS];
};

// The listed rows of one tensor, a power-of-two group of lanes per row (as in
// the compaction kernel), four rows per group at once.
template <typename V>
__device__ inline void copy_listed(const CTensor &T, const int *lo, const int *lj, int n) {
  const int lpr_shift = T.lpr_shift;
  const int lane = threadIdx.x & ((1 << lpr_shift) - 1);
  const int per_pass = kThreads >> lpr_shift;
  for (int p = 0; p < T.planes; ++p)
    copy_rows_batched<V, false>(T, p, (long long)(threadIdx.x >> lpr_shift), n, per_pass, lane,
                         [&](long long e, long long &j, long long &r) __attribute__((always_inline)) {
                           j = lj[e];
                           r = lo[e];
                           return true;
                         });
}

template <int MODE>
__global__ __launch_bounds__(kThreads) void select_compact_kernel(SCArgs a, RuleArgs R) {
  __shared__ int list_o[kListCap], list_j[kListCap];
  __shared__ int list_n;
  const int S = a.S;
  const int img = (int)blockIdx.x / S, sl = (int)blockIdx.x - img * S;
  if (threadIdx.x == 0) list_n = 0;
  __syncthreads();
  SelArgs A = a.sel;
  if (sl != 0) A.cu_out = nullptr;
  auto put = [&](long long o, int32_t v, int seq) __attribute__((always_inline)) {
    if ((int)(o % S) != sl) return;
    if (o >= a.cap) {
      if (a.status) atomicOr(a.status + seq, AVTP_FLAG_OUT_CAPACITY);
      return;
    }
    a.keep_idx[o] = v;
    if (o >= a.n_out) return;
    const int e = atomicAdd(&list_n, 1);
    if (e < kListCap) {
      list_o[e] = (int)o;
      list_j[e] = v;
    } else if (a.status) {  // (the host sizes S so that this does not happen)
      atomicOr(a.status + seq, AVTP_FLAG_OUT_CAPACITY);
    }
  };
  select_image<MODE>(A, R, img, sl == 0, a.status, put);
  __syncthreads();
  const int n = min(list_n, kListCap);
  for (int ti = 0; ti < a.n_t; ++ti) {
    const CTensor &T = a.t[ti];
    switch (T.vshift) {
      case 4: copy_listed<uint4>(T, list_o, list_j, n); break;
      case 3: copy_listed<uint2>(T, list_o, list_j, n); break;
      case 2: copy_listed<uint32_t>(T, list_o, list_j, n); break;
      case 1: copy_listed<uint16_t>(T, list_o, list_j, n); break;
      default: copy_listed<uint8_t>(T, list_o, list_j, n); break;
    }
  }
}

// Blocks per image of the one-launch selection + compaction: about 1024
// blocks in all, and few enough rows per slice for its list (an image block
// writes at most the image's tokens plus every text row; each contiguous run
// adds at most one to a share).
static int compact_slices(const DevLayout &L) {
  const long long bound = (long long)L.max_img_len + L.T_tot + 64;
  const int images = L.n_img > 0 ? L.n_img : 1;
  long long S = (1024 + images - 1) / images;
  if (S > 64) S = 64;
  const long long need = (bound + (kListCap - 64) - 1) / (kListCap - 64);
  if (S < need) S = need;
  if (S < 1) S = 1;
  return (int)S;
}

static SCArgs sc_args(const DevLayout &L, const float *scores, const int32_t *budget,
                      int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out, int32_t *status,
                      int64_t n_out, const avtp_tensor *tensors, int n_tensors) {
  SCArgs a;
  a.sel = SelArgs{scores, budget, L.img_start, L.img_len, L.cu_img, L.cu_text, L.text_pos,
                  L.B, L.n_img, L.T_tot, cu_out};
  a.keep_idx = keep_idx;
  a.cap = (long long)keep_capacity;
  a.n_out = n_out;
  a.status = status;
  a.n_t = n_tensors;
  for (int i = 0; i < n_tensors; ++i) describe_tensor(tensors[i], kThreads, a.t[i]);
  a.S = compact_slices(L);
  return a;
}

static RuleArgs rule_args(const DevLayout &L, const float *img_sum, int mode, float alpha,
                          int lo_permille, int hi_permille, int floor_abs, int32_t *budget) {
  return RuleArgs{img_sum, L.keep_total, mode, alpha, lo_permille, hi_permille, floor_abs, budget};
}

}  // namespace

hipError_t launch_select_compact(hipStream_t st, const DevLayout &L, const float *scores,
                                 const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                                 int32_t *cu_out, int32_t *status, int64_t n_out,
                                 const avtp_tensor *tensors, int n_tensors) {
  clear_pending_error();
  const SCArgs a = sc_args(L, scores, budget, keep_idx, keep_capacity, cu_out, status, n_out,
                           tensors, n_tensors);
  const int images = L.n_img > 0 ? L.n_img : 1;
  hipLaunchKernelGGL(select_compact_kernel<kBudGlobal>, dim3((unsigned)(images * a.S)), dim3(kThreads),
                     0, st, a, RuleArgs{});
  return hipGetLastError();
}

hipError_t launch_select(hipStream_t st, const DevLayout &L, const float *scores,
                         const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                         int32_t *cu_out, int32_t *status) {
  clear_pending_error();
  const int grid = L.n_img > 0 ? L.n_img : 1;
  const SelArgs A{scores, budget, L.img_start, L.img_len, L.cu_img, L.cu_text, L.text_pos,
                  L.B, L.n_img, L.T_tot, cu_out};
  hipLaunchKernelGGL(select_kernel<kBudGlobal>, dim3(grid), dim3(kThreads), 0, st, A, RuleArgs{},
                     keep_idx, (long long)keep_capacity, status);
  return hipGetLastError();
}

hipError_t launch_budget_select(hipStream_t st, const DevLayout &L, const float *img_sum, int mode,
                                float alpha, int lo_permille, int hi_permille, int floor_abs,
                                const float *scores, int32_t *budget, int32_t *keep_idx,
                                int64_t keep_capacity, int32_t *cu_out, int32_t *status) {
  clear_pending_error();
  const int grid = L.n_img > 0 ? L.n_img : 1;
  const SelArgs A{scores, budget, L.img_start, L.img_len, L.cu_img, L.cu_text, L.text_pos,
                  L.B, L.n_img, L.T_tot, cu_out};
  const RuleArgs R =
      rule_args(L, img_sum, mode, alpha, lo_permille, hi_permille, floor_abs, budget);
  if (L.max_img_per_seq <= kWaveBudgetMaxImages)
    hipLaunchKernelGGL(select_kernel<kBudWave>, dim3(grid), dim3(kThreads), 0, st, A, R, keep_idx,
                       (long long)keep_capacity, status);
  else
    hipLaunchKernelGGL(select_kernel<kBudBlock>, dim3(grid), dim3(kThreads), 0, st, A, R,
                       keep_idx, (long long)keep_capacity, status);
  return hipGetLastError();
}

hipError_t launch_budget_select_compact(hipStream_t st, const DevLayout &L, const float *img_sum,
                                        int mode, float alpha, int lo_permille, int hi_permille,
                                        int floor_abs, const float *scores, int32_t *budget,
                                        int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out,
                                        int32_t *status, int64_t n_out, const avtp_tensor *tensors,
                                        int n_tensors) {
  clear_pending_error();
  const SCArgs a = sc_args(L, scores, budget, keep_idx, keep_capacity, cu_out, status, n_out,
                           tensors, n_tensors);
  const int images = L.n_img > 0 ? L.n_img : 1;
  const RuleArgs R =
      rule_args(L, img_sum, mode, alpha, lo_permille, hi_permille, floor_abs, budget);
  const dim3 grid((unsigned)(images * a.S));
  if (L.max_img_per_seq <= kWaveBudgetMaxImages)
    hipLaunchKernelGGL(select_compact_kernel<kBudWave>, grid, dim3(kThreads), 0, st, a, R);
  else
    hipLaunchKernelGGL(select_compact_kernel<kBudBlock>, grid, dim3(kThreads), 0, st, a, R);
  return hipGetLastError();
}

}  // namespace avtp
