// Attention-to-visual-token score on gfx950 (MFMA, wave64).
//
// The score of visual token j is the attention the text rows pay to it,
// averaged over the query heads and over the rows that can see it (the
// per-token form of the statistic summed in Sec. 3.3.2 of the paper):
//   P[h,t,j] = exp(c q_{t,h}.k_{j,g(h)} - lse[h,t]),  lse = causal row LSE
//   s_j      = 1/Hq sum_h 1/|T_j| sum_{t in T_j} P[h,t,j]
// The row normaliser has to exist before any column can be summed, so the
// work is split into two tiled passes over the keys, neither of which stores
// the T x L attention matrix:
//   pass 1 (row statistics): queries stay in VGPRs as MFMA B operands, key
//     tiles stream through LDS; the 32x32 MFMA output puts one query column
//     in each lane, so the running max / sum of a row never leaves its lane.
//     The key range is split in chunks; a small kernel merges the chunk
//     partials into the natural-log LSE.
//   pass 2 (column sums): keys stay in VGPRs, query tiles (and their LSE)
//     stream through LDS; the output transposes, so each lane owns one key
//     column and accumulates its column sum locally.
// Both passes use v_mfma_f32_32x32x16_bf16 (bf16 inputs) or
// v_mfma_f32_32x32x2_f32 (fp32 inputs), accumulate in fp32, and use exp2
// with c*log2(e) folded into one FMA per logit.  Every reduction has a fixed
// order, so results are bit-reproducible and identical key rows give
// identical scores.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"

namespace avtp {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kThreads = 256;  // 4 waves per block in both passes
constexpr int kStage = 64;     // rows (keys or queries) per LDS stage

template <typename T>
struct Mma;
template <>
struct Mma<__bf16> {
  static constexpr int E = 8;  // elements each lane feeds per k-step
  typedef __bf16 frag __attribute__((ext_vector_type(8)));
  __device__ static inline f32x16 run(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mma<float> {
  static constexpr int E = 1;
  typedef float frag;
  __device__ static inline f32x16 run(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Register budget (two waves per SIMD = 256 VGPRs per wave): the stationary
// operand of a wave, NT tiles of 32 rows, takes at most 128 VGPRs in pass 1
// (queries; accumulators 16 per tile) and at most 96 in pass 2 (keys; the
// per-row LSE values of the streamed tile need registers too).
__host__ __device__ constexpr int tiles_cap(int budget, int row_bytes) {
  return (budget / (row_bytes / 8)) > 4 ? 4 : (budget / (row_bytes / 8));
}
__host__ __device__ constexpr int tiles_pass1(int row_bytes) { return tiles_cap(128, row_bytes); }
__host__ __device__ constexpr int tiles_pass2(int row_bytes) { return tiles_cap(96, row_bytes); }

template <typename T, int D>
struct Geo {
  static constexpr int E = Mma<T>::E;
  static constexpr int NS = D / (2 * E);          // k-steps per 32x32 tile
  static constexpr int ROWB = D * (int)sizeof(T);  // bytes of one head row
  static constexpr int LS = ROWB + 16;             // padded LDS row stride (conflict-free b128 reads)
  static constexpr int NT1 = tiles_pass1(ROWB);   // stationary 32-row tiles per wave, pass 1
  static constexpr int NT2 = tiles_pass2(ROWB);   // same for pass 2
  static constexpr int V16 = kStage * ROWB / 16 / kThreads;  // 16-byte loads per thread per stage
  static constexpr int V16_ROW = ROWB / 16;
  static constexpr int NCH = ROWB / 16;                // 16-byte chunks per row
  static constexpr int SWZ = (NCH < 16 ? NCH : 16) - 1;  // XOR swizzle of the chunk index
  static constexpr int DMA = kStage * NCH / 64 / 4;    // direct-to-LDS loads per wave per stage
  static_assert(DMA >= 1 && kStage * NCH % 256 == 0, "stage must split into whole wave loads");
};

// Byte offset in a swizzled LDS stage of element offset `eo` of row `row`:
// row-major rows without padding, the 16-byte chunk index XOR-ed with the
// row so that the 32 rows read by one MFMA operand load hit distinct banks.
template <typename T, int D>
__device__ inline int swz_off(int row, int eo) {
  using G_ = Geo<T, D>;
  const int bo = eo * (int)sizeof(T);
  return row * G_::ROWB + (((bo >> 4) ^ (row & G_::SWZ)) << 4) + (bo & 15);
}

// Enqueue one stage (kStage rows of ROWB bytes) with global_load_lds: wave w
// fills LDS bytes [1 KB * (w*DMA + i), +1 KB) for i < DMA, lane l writing
// the 16 bytes at +16*l, i.e. physical chunk p = 64*(w*DMA+i) + l.
// row_src(row) returns the global address of a row (always a valid row).
template <typename T, int D, typename F>
__device__ inline void dma_stage(char *lds, int wave, int lane, F row_src) {
  using G_ = Geo<T, D>;
#pragma unroll
  for (int i = 0; i < G_::DMA; ++i) {
    const int gi = wave * G_::DMA + i;
    const int p = gi * 64 + lane;
    const int row = p / G_::NCH, pc = p % G_::NCH;
    const int c = pc ^ (row & G_::SWZ);
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void *)(row_src(row) + c * 16),
        (__attribute__((address_space(3))) void *)(lds + gi * 1024), 16, 0, 0);
  }
}

// wait for this wave's outstanding global loads (including direct-to-LDS ones)
__device__ inline void wait_vmem() { __builtin_amdgcn_s_waitcnt(0xF70); }

template <typename F>
__device__ inline F load_frag(const char *p) {
  return *reinterpret_cast<const F *>(p);
}

// Positions spanned by query rows [r0, r1) of one (sequence, key head);
// row r is text row t = r % Tb of head r / Tb, positions ascend with t.
__device__ inline void rows_pos_range(const int32_t *tp, int Tb, int r0, int r1, int &pmin,
                                      int &pmax) {
  if (r0 / Tb == (r1 - 1) / Tb) {
    pmin = tp[r0 % Tb];
    pmax = tp[(r1 - 1) % Tb];
  } else {
    pmin = tp[0];
    pmax = tp[Tb - 1];
  }
}

struct P1Args {
  const char *q, *k;
  const int32_t *cu_seqlens, *cu_text, *text_pos;
  int B, Hq, Hkv, G, T_tot;
  int nqb, nkc, kchunk;
  float cl2e;
  float *part_m, *part_l;  // [nkc][Hq * T_tot]
};

// Pass 1: per (sequence b, key head g, query block, key chunk), partial
// row statistics (max in log2 units, sum of 2^(z - max)) of every query row.
//
// Per 32-key tile a wave runs NT chains of 8 MFMAs (one per stationary
// query tile).  The exp/sum of chain i-1 is issued in the same basic block
// as the MFMAs of chain i, so the transcendental work runs while the matrix
// core is busy.  The running maximum is only raised when a tile's sum of
// 2^(z - m) exceeds 2^64 (first visible tile, or a big jump): the common
// case costs one FMA, one exp and one add per logit.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void rowstats_kernel(P1Args a) {
  using G_ = Geo<T, D>;
  using MM = Mma<T>;
  using frag = typename MM::frag;
  constexpr int NT = G_::NT1, NS = G_::NS, ROWB = G_::ROWB, LS = G_::LS, E = G_::E;
  constexpr int QB = 4 * NT * 32;  // query rows per block
  __shared__ __attribute__((aligned(16))) char smem[2][kStage * LS];

  // Blocks that share one key chunk (the nqb query blocks of a unit) get
  // ids that are equal mod 8, i.e. land on one XCD and share its L2.
  const int nunits = a.B * a.Hkv * a.nkc;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int qb = local % a.nqb;
  const int unit = (local / a.nqb) * 8 + xcd;
  if (unit >= nunits) return;
  const int kc = unit % a.nkc, bg = unit / a.nkc, g = bg % a.Hkv, b = bg / a.Hkv;

  const int s0 = a.cu_seqlens[b], L = a.cu_seqlens[b + 1] - s0;
  const int t0 = a.cu_text[b], Tb = a.cu_text[b + 1] - t0;
  const int R = a.G * Tb;
  const int row0 = qb * QB;
  const int kbeg = kc * a.kchunk;
  if (row0 >= R || kbeg >= L) return;
  const int kend = min(L, kbeg + a.kchunk);
  const int32_t *tp = a.text_pos + t0;
  int bmin, bmax;
  rows_pos_range(tp, Tb, row0, min(R, row0 + QB), bmin, bmax);
  if (s0 + kbeg > bmax) return;                  // chunk starts after every row of the block
  const int kstop = min(kend, bmax - s0 + 1);    // keys after the last row are never visible

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hi = lane >> 5, col = lane & 31;
  const int wr0 = row0 + wave * NT * 32;
  const bool active = wr0 < R;
  int wmin = 0, wmax = -1;
  if (active) rows_pos_range(tp, Tb, wr0, min(R, wr0 + NT * 32), wmin, wmax);

  // stationary operand: this wave's query rows
  frag qf[NT][NS];
  int qrel[NT];  // query position relative to the sequence start (-1: padding row)
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    const int r = wr0 + i * 32 + col;
    qrel[i] = -1;
    if (r < R) {
      const int hh = r / Tb, t = r - hh * Tb, h = g * a.G + hh;
      qrel[i] = tp[t] - s0;
      const char *src = a.q + ((size_t)(t0 + t) * a.Hq + h) * ROWB + hi * E * sizeof(T);
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[i][s] = load_frag<frag>(src + s * 2 * E * sizeof(T));
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[i][s] = frag{};
    }
  }

  float m2[NT], l[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    m2[i] = -INFINITY;
    l[i] = 0.f;
  }
  const float cl2e = a.cl2e;

  // keys of one stage, rows clamped into the chunk (rows past kend are masked)
  auto issue_stage = [&](int ks, int bufi) {
    dma_stage<T, D>(smem[bufi], wave, lane, [&](int row) {
      const int key = min(ks + row, kend - 1);
      return a.k + ((size_t)(s0 + key) * a.Hkv + g) * ROWB;
    });
  };

  // Accumulator element e of this lane holds key kb + hi*4 + eoff(e) of its
  // query column; it is visible iff eoff(e) <= vlim, with the per-lane limit
  // vlim = min(q - kb, kend - 1 - kb) - hi*4 (causal row and chunk end).
  auto eoff = [](int e) { return 8 * (e >> 2) + (e & 3); };
  auto vlimit = [&](int qi, int kb) { return min(qrel[qi] - kb, kend - 1 - kb) - hi * 4; };

  // Exact update of row qi with tile kb (any visibility pattern; raises the max).
  auto exact_update = [&](const f32x16 &acc, int qi, int kb) {
    const int vl = vlimit(qi, kb);
    float tm = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (eoff(e) <= vl) tm = fmaxf(tm, acc[e] * cl2e);
    if (tm == -INFINITY) return;
    const float nm = fmaxf(m2[qi], tm);
    float ns = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float x = __builtin_amdgcn_exp2f(acc[e] * cl2e - nm);
      ns += eoff(e) <= vl ? x : 0.f;
    }
    l[qi] = l[qi] * __builtin_amdgcn_exp2f(m2[qi] - nm) + ns;
    m2[qi] = nm;
  };

  f32x16 pacc = f32x16{};  // accumulators waiting for their exp/sum
  int pend_kb = 0;
  bool pend = false;

  const int nstage = (kstop - kbeg + kStage - 1) / kStage;
  issue_stage(kbeg, 0);
  for (int st = 0; st < nstage; ++st) {
    const int ks = kbeg + st * kStage;
    wait_vmem();
    __syncthreads();  // stage st is in LDS; every wave is done with the other buffer
    if (st + 1 < nstage) issue_stage(ks + kStage, (st + 1) & 1);
    const char *buf = smem[st & 1];
    if (active) {
#pragma unroll
      for (int kt = 0; kt < kStage / 32; ++kt) {
        const int kb = ks + kt * 32;  // first key (relative) of this 32-key tile
        if (kb < kstop && s0 + kb <= wmax) {
          frag av[NS];
#pragma unroll
          for (int s = 0; s < NS; ++s)
            av[s] = load_frag<frag>(buf + swz_off<T, D>(kt * 32 + col, s * 2 * E + hi * E));
#pragma unroll
          for (int qi = 0; qi < NT; ++qi) {
            const int pqi = qi == 0 ? NT - 1 : qi - 1;
            const int pkb = qi == 0 ? pend_kb : kb;
            const bool has = qi > 0 || pend;
            // visibility of the pending tile for this lane: all, none, or partial
            const int vl = vlimit(pqi, pkb);
            const bool none = qrel[pqi] - pkb < 0;
            const bool all = qrel[pqi] - pkb >= 31 && pkb + 32 <= kend;
            const bool fast = __ballot(!(none || all)) == 0ull;
            f32x16 acc = f32x16{};
            float ts = 0.f;
            if (has && fast) {
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                acc = MM::run(av[s], qf[qi][s], acc);
#pragma unroll
                for (int e = (s * 16) / NS; e < ((s + 1) * 16) / NS; ++e)
                  ts += __builtin_amdgcn_exp2f(pacc[e] * cl2e - m2[pqi]);
              }
              if (none) ts = 0.f;
            } else if (has) {
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                acc = MM::run(av[s], qf[qi][s], acc);
#pragma unroll
                for (int e = (s * 16) / NS; e < ((s + 1) * 16) / NS; ++e) {
                  const float x = __builtin_amdgcn_exp2f(pacc[e] * cl2e - m2[pqi]);
                  ts += eoff(e) <= vl ? x : 0.f;
                }
              }
            } else {
#pragma unroll
              for (int s = 0; s < NS; ++s) acc = MM::run(av[s], qf[qi][s], acc);
            }
            if (has) {
              if (ts <= 0x1p64f) l[pqi] += ts;
              else exact_update(pacc, pqi, pkb);  // first visible tile, a jump, or NaN
            }
            pacc = acc;
          }
          pend = true;
          pend_kb = kb;
        }
      }
    }
  }
  if (!active) return;
  if (pend) {
    const int vl = vlimit(NT - 1, pend_kb);
    float ts = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float x = __builtin_amdgcn_exp2f(pacc[e] * cl2e - m2[NT - 1]);
      ts += eoff(e) <= vl ? x : 0.f;
    }
    if (ts <= 0x1p64f) l[NT - 1] += ts;
    else exact_update(pacc, NT - 1, pend_kb);
  }
  // merge the two half-waves (same query column, disjoint keys) and store
  const size_t HqT = (size_t)a.Hq * a.T_tot;
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    const float om = __shfl_xor(m2[i], 32), ol = __shfl_xor(l[i], 32);
    const float nm = fmaxf(m2[i], om);
    float tot = 0.f;
    if (nm != -INFINITY)
      tot = l[i] * __builtin_amdgcn_exp2f(m2[i] - nm) + ol * __builtin_amdgcn_exp2f(om - nm);
    const int r = wr0 + i * 32 + col;
    if (hi == 0 && r < R) {
      const int hh = r / Tb, qidx = (g * a.G + hh) * a.T_tot + t0 + (r - hh * Tb);
      a.part_m[kc * HqT + qidx] = nm;
      a.part_l[kc * HqT + qidx] = tot;
    }
  }
}

// Merge the chunk partials of every text row into lse = ln(sum exp(z)).
// Only the chunks that start at or before the row's position hold keys it
// can see, and exactly those were written by pass 1.
__global__ void lse_combine_kernel(const float *__restrict__ part_m, const float *__restrict__ part_l,
                                   const int32_t *__restrict__ cu_seqlens,
                                   const int32_t *__restrict__ cu_text,
                                   const int32_t *__restrict__ text_pos, int B, int Hq, int T_tot,
                                   int kchunk, float *__restrict__ lse) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= Hq * T_tot) return;
  const int t = idx % T_tot;
  int lo = 0, hi = B - 1;  // sequence of text row t
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_text[mid] <= t) lo = mid; else hi = mid - 1;
  }
  const int last = (text_pos[t] - cu_seqlens[lo]) / kchunk;
  const size_t HqT = (size_t)Hq * T_tot;
  float M = -INFINITY;
  for (int c = 0; c <= last; ++c) M = fmaxf(M, part_m[c * HqT + idx]);
  float S = 0.f;
  for (int c = 0; c <= last; ++c) {
    const float m = part_m[c * HqT + idx];
    if (m != -INFINITY) S += part_l[c * HqT + idx] * __builtin_amdgcn_exp2f(m - M);
  }
  lse[idx] = (M + __builtin_amdgcn_logf(S)) * kLn2;
}

struct P2Args {
  const char *q, *k;
  const float *lse;
  const int32_t *cu_seqlens, *cu_text, *text_pos;
  int B, Hq, Hkv, G, T_tot, N_tok, nkb;
  float cl2e;
  float *colsum;  // [Hkv][N_tok]
};

// Pass 2: per (sequence b, key head g, key block), the column sums
// sum_{h in group g} sum_t exp(c q_{t,h}.k_j - lse[h,t]) over visible rows.
//
// Query tiles (and their LSE, positions and position range) stream through
// double-buffered LDS; keys are the stationary MFMA operand.  For a 32-row
// tile that sees every key of the wave, the exp/sum of key tile j-1 is
// issued between the MFMAs of key tile j; tiles that see only part of the
// wave's keys take a masked path, tiles that see none are skipped.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void colsum_kernel(P2Args a) {
  using G_ = Geo<T, D>;
  using MM = Mma<T>;
  using frag = typename MM::frag;
  constexpr int NKT = G_::NT2, NS = G_::NS, ROWB = G_::ROWB, E = G_::E;
  constexpr int KB = 4 * NKT * 32;  // keys per block
  __shared__ __attribute__((aligned(16))) char smem[2][kStage * ROWB];
  __shared__ __attribute__((aligned(16))) float s_lse2[2][kStage];
  __shared__ __attribute__((aligned(16))) int s_pos[2][kStage];
  __shared__ int s_meta[2][4];  // per 32-row half: min and max position

  // the nkb key blocks of one (sequence, key head) read the same queries:
  // keep them on one XCD
  const int nunits = a.B * a.Hkv;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int kb = local % a.nkb;
  const int unit = (local / a.nkb) * 8 + xcd;
  if (unit >= nunits) return;
  const int g = unit % a.Hkv, b = unit / a.Hkv;
  const int s0 = a.cu_seqlens[b], L = a.cu_seqlens[b + 1] - s0;
  const int t0 = a.cu_text[b], Tb = a.cu_text[b + 1] - t0;
  const int R = a.G * Tb;
  const int kb0 = kb * KB;
  if (kb0 >= L) return;
  const int32_t *tp = a.text_pos + t0;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hi = lane >> 5, col = lane & 31;
  const int kw0 = kb0 + wave * NKT * 32;
  const bool active = kw0 < L;
  const int kmin = s0 + kw0, kmax = s0 + min(L, kw0 + NKT * 32) - 1;

  frag kf[NKT][NS];
  int kpos[NKT];
#pragma unroll
  for (int j = 0; j < NKT; ++j) {
    const int key = kw0 + j * 32 + col;
    if (key < L) {
      kpos[j] = s0 + key;
      const char *src = a.k + ((size_t)(s0 + key) * a.Hkv + g) * ROWB + hi * E * sizeof(T);
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[j][s] = load_frag<frag>(src + s * 2 * E * sizeof(T));
    } else {
      kpos[j] = 0x7fffffff;
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[j][s] = frag{};
    }
  }
  float cs[NKT];
#pragma unroll
  for (int j = 0; j < NKT; ++j) cs[j] = 0.f;
  const float cl2e = a.cl2e;

  auto issue_stage = [&](int rs, int bufi) {
    dma_stage<T, D>(smem[bufi], wave, lane, [&](int row) {
      const int r = min(rs + row, R - 1);  // padding rows re-read row R-1; their lse is +inf
      const int hh = r / Tb, t = r - hh * Tb;
      return a.q + ((size_t)(t0 + t) * a.Hq + g * a.G + hh) * ROWB;
    });
  };
  float pre_lse = INFINITY;
  int pre_pos = -1;
  auto load_meta = [&](int rs) {  // wave 0: LSE (log2 units) and position of each row
    if (wave == 0) {
      const int r = rs + lane;
      pre_lse = INFINITY;
      pre_pos = -1;
      if (r < R) {
        const int hh = r / Tb, t = r - hh * Tb;
        pre_lse = a.lse[(size_t)(g * a.G + hh) * a.T_tot + t0 + t] * kLog2e;
        pre_pos = tp[t];
      }
    }
  };
  auto store_meta = [&](int bufi) {
    if (wave == 0) {
      s_lse2[bufi][lane] = pre_lse;
      s_pos[bufi][lane] = pre_pos;
      int vmin = pre_pos >= 0 ? pre_pos : 0x7fffffff, vmax = pre_pos;
#pragma unroll
      for (int off = 16; off > 0; off >>= 1) {  // reduce within each 32-lane half
        vmin = min(vmin, __shfl_xor(vmin, off));
        vmax = max(vmax, __shfl_xor(vmax, off));
      }
      if (col == 0) {
        s_meta[bufi][2 * hi] = vmin;
        s_meta[bufi][2 * hi + 1] = vmax;
      }
    }
  };

  auto exp_sum = [&](const f32x16 &acc, const float *lv) {
    float t = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) t += __builtin_amdgcn_exp2f(acc[e] * cl2e - lv[e]);
    return t;
  };

  f32x16 pacc = f32x16{};
  float plv[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) plv[e] = INFINITY;
  bool pend = false;  // pacc holds key tile NKT-1 of an earlier row tile

  const int nstage = (R + kStage - 1) / kStage;
  if (nstage > 0) {
    issue_stage(0, 0);
    load_meta(0);
    store_meta(0);
  }
  for (int st = 0; st < nstage; ++st) {
    const int rs = st * kStage;
    const int bi = st & 1;
    wait_vmem();
    __syncthreads();  // stage st is in LDS; every wave is done with the other buffer
    if (st + 1 < nstage) {
      issue_stage(rs + kStage, bi ^ 1);
      load_meta(rs + kStage);
    }
    if (active) {
#pragma unroll
      for (int sub = 0; sub < kStage / 32; ++sub) {
        if (rs + sub * 32 >= R) break;
        const int qmin = s_meta[bi][2 * sub], qmax = s_meta[bi][2 * sub + 1];
        if (qmax < kmin) continue;  // no row of this tile sees any key of the wave
        frag av[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s)
          av[s] = load_frag<frag>(smem[bi] + swz_off<T, D>(sub * 32 + col, s * 2 * E + hi * E));
        // lane's rows: sub*32 + hi*4 + 8*(e/4) + e%4
        float lv[16];
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const float4 v = *reinterpret_cast<const float4 *>(&s_lse2[bi][sub * 32 + hi * 4 + 8 * e4]);
          lv[4 * e4 + 0] = v.x;
          lv[4 * e4 + 1] = v.y;
          lv[4 * e4 + 2] = v.z;
          lv[4 * e4 + 3] = v.w;
        }
        if (qmin >= kmax) {
          // every row sees every key of the wave: pipelined MFMA + exp/sum
#pragma unroll
          for (int j = 0; j < NKT; ++j) {
            f32x16 acc = f32x16{};
            float ts = 0.f;
            if (j > 0 || pend) {
              const float *pl = j > 0 ? lv : plv;
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                acc = MM::run(av[s], kf[j][s], acc);
#pragma unroll
                for (int e = (s * 16) / NS; e < ((s + 1) * 16) / NS; ++e)
                  ts += __builtin_amdgcn_exp2f(pacc[e] * cl2e - pl[e]);
              }
              cs[j > 0 ? j - 1 : NKT - 1] += ts;
            } else {
#pragma unroll
              for (int s = 0; s < NS; ++s) acc = MM::run(av[s], kf[j][s], acc);
            }
            pacc = acc;
          }
#pragma unroll
          for (int e = 0; e < 16; ++e) plv[e] = lv[e];
          pend = true;
        } else {
          // some rows see only part of the wave's keys: masked, not pipelined
          if (pend) {
            cs[NKT - 1] += exp_sum(pacc, plv);
            pend = false;
          }
          int qp[16];
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4) {
            const int4 v = *reinterpret_cast<const int4 *>(&s_pos[bi][sub * 32 + hi * 4 + 8 * e4]);
            qp[4 * e4 + 0] = v.x;
            qp[4 * e4 + 1] = v.y;
            qp[4 * e4 + 2] = v.z;
            qp[4 * e4 + 3] = v.w;
          }
#pragma unroll
          for (int j = 0; j < NKT; ++j) {
            f32x16 acc = f32x16{};
#pragma unroll
            for (int s = 0; s < NS; ++s) acc = MM::run(av[s], kf[j][s], acc);
            float ts = 0.f;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const float x = __builtin_amdgcn_exp2f(acc[e] * cl2e - lv[e]);
              ts += kpos[j] <= qp[e] ? x : 0.f;
            }
            cs[j] += ts;
          }
        }
      }
    }
    if (st + 1 < nstage) store_meta(bi ^ 1);
  }
  if (!active) return;
  if (pend) cs[NKT - 1] += exp_sum(pacc, plv);
#pragma unroll
  for (int j = 0; j < NKT; ++j) {
    const float v = cs[j] + __shfl_xor(cs[j], 32);
    const int key = kw0 + j * 32 + col;
    if (hi == 0 && key < L) a.colsum[(size_t)g * a.N_tok + s0 + key] = v;
  }
}

// Per-image epilogue shared by both score modes: s_j from the column sums
// (attention mode) or as stored (variation mode), NaN / empty-row flags, and
// the per-image sum in a fixed reduction order.  Extra blocks write +inf at
// the text positions.
__global__ __launch_bounds__(256) void finalize_kernel(
    const float *__restrict__ colsum, int Hq, int Hkv, int N_tok, int n_img, int T_tot,
    const int32_t *__restrict__ img_start, const int32_t *__restrict__ img_len,
    const int32_t *__restrict__ cu_img, const int32_t *__restrict__ cu_text,
    const int32_t *__restrict__ text_pos, int B, float *__restrict__ scores,
    float *__restrict__ img_sum, int32_t *__restrict__ status) {
  __shared__ float red[256];
  const int tid = threadIdx.x;
  if ((int)blockIdx.x >= n_img) {
    const int t = (blockIdx.x - n_img) * 256 + tid;
    if (t < T_tot) scores[text_pos[t]] = INFINITY;
    return;
  }
  const int i = blockIdx.x;
  int lo = 0, hi = B - 1;  // sequence of image i
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_img[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int s0 = img_start[i], n = img_len[i];
  int nT = 0;
  if (colsum) {  // text rows after the image: those past the first one beyond s0
    int a0 = cu_text[b], a1 = cu_text[b + 1];
    while (a0 < a1) {
      const int mid = (a0 + a1) >> 1;
      if (text_pos[mid] < s0) a0 = mid + 1; else a1 = mid;
    }
    nT = cu_text[b + 1] - a0;
  }
  float acc = 0.f;
  bool nan = false;
  for (int j = tid; j < n; j += 256) {
    float s;
    if (colsum) {
      float v = 0.f;
      for (int g = 0; g < Hkv; ++g) v += colsum[(size_t)g * N_tok + s0 + j];
      s = nT > 0 ? v / (float)((long long)Hq * nT) : 0.f;
      scores[s0 + j] = s;
    } else {
      s = scores[s0 + j];
    }
    nan |= (s != s);
    acc += s;
  }
  red[tid] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) img_sum[i] = red[0];
  if (status) {
    if (nan) atomicOr(status + b, AVTP_FLAG_NAN_SCORE);
    if (tid == 0 && colsum && nT == 0 && n > 0) atomicOr(status + b, AVTP_FLAG_NO_TEXT_AFTER);
  }
}

template <typename T, int D>
hipError_t run_row_lse(hipStream_t st, const DevLayout &L, const AttnPlan &P, const void *q,
                       const void *k, int Hq, int Hkv, float scale, float *row_lse, char *ws) {
  P1Args a;
  a.q = (const char *)q;
  a.k = (const char *)k;
  a.cu_seqlens = L.cu_seqlens;
  a.cu_text = L.cu_text;
  a.text_pos = L.text_pos;
  a.B = L.B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = P.G;
  a.T_tot = L.T_tot;
  a.nqb = P.nqb;
  a.nkc = P.nkc;
  a.kchunk = P.kchunk;
  a.cl2e = scale * kLog2e;
  a.part_m = (float *)(ws + P.off_part_m);
  a.part_l = (float *)(ws + P.off_part_l);
  const int nunits = L.B * Hkv * P.nkc;
  const int grid = ((nunits + 7) / 8) * 8 * P.nqb;
  hipLaunchKernelGGL((rowstats_kernel<T, D>), dim3(grid), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rows = Hq * L.T_tot;
  hipLaunchKernelGGL(lse_combine_kernel, dim3((rows + 255) / 256), dim3(256), 0, st, a.part_m,
                     a.part_l, L.cu_seqlens, L.cu_text, L.text_pos, L.B, Hq, L.T_tot, P.kchunk,
                     row_lse);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t run_colsum(hipStream_t st, const DevLayout &L, const AttnPlan &P, const void *q,
                      const void *k, int Hq, int Hkv, float scale, const float *lse, char *ws) {
  P2Args a;
  a.q = (const char *)q;
  a.k = (const char *)k;
  a.lse = lse;
  a.cu_seqlens = L.cu_seqlens;
  a.cu_text = L.cu_text;
  a.text_pos = L.text_pos;
  a.B = L.B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = P.G;
  a.T_tot = L.T_tot;
  a.N_tok = L.N_tok;
  a.nkb = P.nkb;
  a.cl2e = scale * kLog2e;
  a.colsum = (float *)(ws + P.off_colsum);
  const int nunits = L.B * Hkv;
  const int grid = ((nunits + 7) / 8) * 8 * P.nkb;
  hipLaunchKernelGGL((colsum_kernel<T, D>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

AttnPlan attn_plan(const DevLayout &L, int Hq, int Hkv, int d, int dtype) {
  AttnPlan P;
  P.G = Hq / Hkv;
  const int row_bytes = d * (dtype == AVTP_FP32 ? 4 : 2);
  const int rows_per_block = 4 * tiles_pass1(row_bytes) * 32;  // pass 1 query rows per block
  const int keys_per_block = 4 * tiles_pass2(row_bytes) * 32;  // pass 2 keys per block
  P.rows_max = P.G * L.max_text;
  P.nqb = (P.rows_max + rows_per_block - 1) / rows_per_block;
  if (P.nqb < 1) P.nqb = 1;
  // split keys so that pass 1 launches about 2048 blocks (8 per CU)
  const long long base = (long long)L.B * Hkv * P.nqb;
  long long want = (2048 + base - 1) / base;
  if (want < 1) want = 1;
  long long kc = (L.max_seqlen + want - 1) / want;
  kc = ((kc + kStage - 1) / kStage) * kStage;
  if (kc < 256) kc = 256;
  P.kchunk = (int)kc;
  P.nkc = (L.max_seqlen + P.kchunk - 1) / P.kchunk;
  if (P.nkc < 1) P.nkc = 1;
  P.nkb = (L.max_seqlen + keys_per_block - 1) / keys_per_block;
  if (P.nkb < 1) P.nkb = 1;
  const size_t rows = (size_t)Hq * L.T_tot;
  size_t off = 0;
  P.off_part_m = off;
  off = align256(off + sizeof(float) * rows * P.nkc);
  P.off_part_l = off;
  off = align256(off + sizeof(float) * rows * P.nkc);
  P.off_lse = off;
  off = align256(off + sizeof(float) * rows);
  P.off_colsum = off;
  off = align256(off + sizeof(float) * (size_t)Hkv * L.N_tok);
  P.bytes = off;
  return P;
}

hipError_t launch_row_lse(hipStream_t st, const DevLayout &L, const AttnPlan &P, int dtype,
                          const void *q, const void *k, int Hq, int Hkv, int d, float scale,
                          float *row_lse, char *ws) {
  if (dtype == AVTP_BF16)
    return d == 128 ? run_row_lse<__bf16, 128>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws)
                    : run_row_lse<__bf16, 64>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws);
  return d == 128 ? run_row_lse<float, 128>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws)
                  : run_row_lse<float, 64>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws);
}

hipError_t launch_colsum(hipStream_t st, const DevLayout &L, const AttnPlan &P, int dtype,
                         const void *q, const void *k, int Hq, int Hkv, int d, float scale,
                         const float *row_lse, char *ws) {
  if (dtype == AVTP_BF16)
    return d == 128 ? run_colsum<__bf16, 128>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws)
                    : run_colsum<__bf16, 64>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws);
  return d == 128 ? run_colsum<float, 128>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws)
                  : run_colsum<float, 64>(st, L, P, q, k, Hq, Hkv, scale, row_lse, ws);
}

hipError_t launch_finalize(hipStream_t st, const DevLayout &L, const float *colsum, int Hq,
                           int Hkv, float *scores, float *img_sum, int32_t *status) {
  const int text_blocks = (L.T_tot + 255) / 256;
  const int grid = L.n_img + text_blocks;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(finalize_kernel, dim3(grid), dim3(256), 0, st, colsum, Hq, Hkv, L.N_tok,
                     L.n_img, L.T_tot, L.img_start, L.img_len, L.cu_img, L.cu_text, L.text_pos,
                     L.B, scores, img_sum, status);
  return hipGetLastError();
}

}  // namespace avtp
