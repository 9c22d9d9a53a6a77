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

#include <type_traits>

#include "avtp_internal.h"

namespace avtp {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kThreads = 256;  // 4 waves per block in both passes
constexpr int kStage = 128;    // query rows per LDS stage in pass 2
constexpr int kStage1 = 128;   // key rows per LDS stage in pass 1
// A chain of 16 exp2 terms above this means the lazily kept reference of a
// row is too far below the row's logits: that chain is redone exactly.
constexpr float kLazyLimit = 18446744073709551616.f;  // 2^64

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

// Register budget, two waves per SIMD (256 VGPRs per wave).  Pass 1 keeps
// at most two 32-row query tiles per wave and two accumulator sets per tile;
// pass 2 keeps up to 96 registers of stationary key tiles, one accumulator
// set each (fewer tiles on small grids, see attn_plan).  fp32
// operands at d = 128 do not fit that budget and run one wave per SIMD.
constexpr int kTiles1 = 2;
template <typename T, int D>
struct Occ {
  static constexpr int value = (sizeof(T) == 4 && D == 128) ? 1 : 2;
};
// pass 2: stationary key fragments take at most 96 registers
__host__ __device__ constexpr int tiles_pass2(int row_bytes) {
  return 96 / (row_bytes / 8) < 1 ? 1 : (96 / (row_bytes / 8) > 4 ? 4 : 96 / (row_bytes / 8));
}

template <typename T, int D>
struct Geo {
  static constexpr int E = Mma<T>::E;
  static constexpr int NS = D / (2 * E);          // k-steps per 32x32 tile
  static constexpr int ROWB = D * (int)sizeof(T);  // bytes of one head row
  static constexpr int LS = ROWB + 16;             // padded LDS row stride (conflict-free b128 reads)
  static constexpr int NT2 = tiles_pass2(ROWB);   // same for pass 2
  static constexpr int V16 = kStage * ROWB / 16 / kThreads;  // 16-byte loads per thread per stage
  static constexpr int V16_ROW = ROWB / 16;
  static constexpr int NCH = ROWB / 16;                // 16-byte chunks per row
  static constexpr int SWZ = (NCH < 16 ? NCH : 16) - 1;  // XOR swizzle of the chunk index
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

// Enqueue one stage (ROWS rows of ROWB bytes) with global_load_lds: wave w
// fills LDS bytes [1 KB * (w*DMA + i), +1 KB) for i < DMA, lane l writing
// the 16 bytes at +16*l, i.e. physical chunk p = 64*(w*DMA+i) + l.
// row_off(row) is the byte offset of a (valid) source row from the
// wave-uniform `base`.  The lane id is made opaque so that the few integer
// ops per load are redone per stage instead of pinning registers.
template <typename T, int D, int ROWS, typename F>
__device__ inline void dma_stage(char *lds, const char *base, int wave, int lane, F row_off) {
  using G_ = Geo<T, D>;
  constexpr int DMA = ROWS * G_::NCH / 64 / 4;  // 1 KB loads per wave
  static_assert(DMA >= 1 && ROWS * G_::NCH % 256 == 0, "stage must split into whole wave loads");
  int ln = lane;
  asm volatile("" : "+v"(ln));
#pragma unroll
  for (int i = 0; i < DMA; ++i) {
    const int gi = wave * DMA + i;
    const unsigned p = (unsigned)(gi * 64 + ln);
    const int row = (int)(p / G_::NCH), pc = (int)(p % G_::NCH);
    const int c = pc ^ (row & G_::SWZ);
    const uint32_t off = row_off(row) + (uint32_t)(c * 16);
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)(base + off),
                                     (__attribute__((address_space(3))) void *)(lds + gi * 1024),
                                     16, 0, 0);
  }
}

// Lane part of the source offsets of a dma_stage whose rows are consecutive
// with a uniform stride: load i of a wave reads row wave*ROWS/4 + i*RPL +
// lane/NCH, chunk (lane%NCH) ^ (row & SWZ); the row bits that reach the
// swizzle repeat with period PER in i, so PER lane offsets cover every load.
template <typename T, int D, int ROWS>
struct DmaPlan {
  using G_ = Geo<T, D>;
  static constexpr int NCH = G_::NCH;
  static constexpr int RPL = 64 / NCH;                     // rows per wave load
  static constexpr int DMA = ROWS * NCH / 64 / 4;          // loads per wave
  static constexpr int SPAN = G_::SWZ + 1;
  static constexpr int PER0 = RPL >= SPAN ? 1 : SPAN / RPL;
  static constexpr int PER = PER0 < DMA ? PER0 : DMA;
  static_assert(NCH <= 64 && (ROWS / 4) % SPAN == 0, "wave row blocks must align to the swizzle");
  __device__ static inline void lane_offsets(uint32_t (&lo)[PER], int lane, uint32_t stride) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int r = j * RPL + lane / NCH;
      lo[j] = (uint32_t)(lane / NCH) * stride + (uint32_t)(((lane % NCH) ^ (r & G_::SWZ)) * 16);
    }
  }
  // rows [0, ROWS) from `base` (row 0) with stride `stride` bytes.  The
  // wave index and lane offsets are made opaque so that the per-load
  // constants are rebuilt here (a few scalar ops) instead of being kept live
  // across the whole loop.
  __device__ static inline void issue(char *lds, const char *base, int wave, const uint32_t (&lo)[PER],
                                      uint32_t stride) {
    int w = wave;
    asm volatile("" : "+s"(w));
    uint32_t l[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      l[j] = lo[j];
      asm volatile("" : "+v"(l[j]));
    }
#pragma unroll
    for (int i = 0; i < DMA; ++i) {
      const int gi = w * DMA + i;
      const char *row = base + (uint32_t)(w * (ROWS / 4) + i * RPL) * stride;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)(row + l[i % PER]),
                                       (__attribute__((address_space(3))) void *)(lds + gi * 1024), 16, 0, 0);
    }
  }
  // Token-major rows: row r of the source is token r >> lg, head r & (G-1)
  // (G = 2^lg), at byte offset (r >> lg) * tok + (r & (G-1)) * ROWB.  The
  // rows of one wave load start at a multiple of RPL, so the offset of row
  // r0 + lane/NCH splits into a part of r0 and a lane part (no carries for
  // any power-of-two G).
  __device__ static inline void lane_offsets_tm(uint32_t (&lo)[PER], int lane, int lg, uint32_t tok) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int lr = lane / NCH, r = j * RPL + lr;
      lo[j] = (uint32_t)(lr >> lg) * tok + (uint32_t)(lr & ((1 << lg) - 1)) * G_::ROWB +
              (uint32_t)(((lane % NCH) ^ (r & G_::SWZ)) * 16);
    }
  }
  // rows [r0, r0 + ROWS) of a token-major source (r0 a multiple of ROWS)
  __device__ static inline void issue_tm(char *lds, const char *base, int r0, int wave,
                                         const uint32_t (&lo)[PER], int lg, uint32_t tok) {
    int w = wave;
    asm volatile("" : "+s"(w));
    uint32_t l[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      l[j] = lo[j];
      asm volatile("" : "+v"(l[j]));
    }
#pragma unroll
    for (int i = 0; i < DMA; ++i) {
      const int gi = w * DMA + i;
      const int rr = r0 + w * (ROWS / 4) + i * RPL;
      const char *row = base + (uint32_t)(rr >> lg) * tok + (uint32_t)(rr & ((1 << lg) - 1)) * G_::ROWB;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)(row + l[i % PER]),
                                       (__attribute__((address_space(3))) void *)(lds + gi * 1024), 16, 0, 0);
    }
  }
};

// Scheduling hint for one MFMA chain of NS steps sharing a basic block with
// independent VALU work: issue one MFMA, then up to V VALU ops, repeat.  The
// chain's first MFMA goes out before any VALU, so work that depends on the
// previous chain's result cannot hold back the matrix core.
template <int NS, int V>
__device__ inline void interleave_mfma_valu() {
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, V, 0);  // VALU
  }
}

// Scheduling hint for one pass-1 key tile: the LDS reads of the first LEAD
// k-steps (none if they were read before the tile), then per k-step the NT
// MFMAs of the step, each followed by up to V VALU ops working on the
// previous tile, then the LDS read of the fragment PF steps ahead.
template <int NS, int NT, int V, int LEAD, bool NX = false>
__device__ inline void interleave_tile() {
  constexpr int PF = NS < 3 ? NS : 3;
  if (LEAD > 0) __builtin_amdgcn_sched_group_barrier(0x100, LEAD, 0);  // DS read
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, V, 0);  // VALU
    }
    // the fragment PF steps ahead: of this tile, or (NX) of the next one
    if (s + PF < NS || NX) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
  }
}

// wait for this wave's outstanding global loads (including direct-to-LDS ones)
__device__ inline void wait_vmem() { __builtin_amdgcn_s_waitcnt(0xF70); }

template <typename F>
__device__ inline F load_frag(const char *p) {
  return *reinterpret_cast<const F *>(p);
}

// Positions spanned by pass-1 query rows [r0, r1) of one (sequence, key
// head).  Rows are token-major: row r is text token r / G under query head
// r % G of the group, so positions ascend with r.
__device__ inline void rows_pos_range(const int32_t *tp, int G, int r0, int r1, int &pmin,
                                      int &pmax) {
  pmin = tp[r0 / G];
  pmax = tp[(r1 - 1) / G];
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
// row statistics of every query row: a reference m (log2 units) and the sum
// l of 2^(z c log2e - m) over the row's visible keys of the chunk.
//
// Each wave holds NT 32-row query tiles (two; one on grids that fit in one
// round, see attn_plan).  Per 32-key tile the MFMAs of the NT tiles advance
// k-step by k-step, while the VALU turns the two accumulators
// of the previous key tile into exp2 sums (one FMA, one exp2 and one add per
// logit), so no instruction waits on a result of the running MFMAs.  The
// reference of a row is kept lazily: it is raised (and the row's sum
// rescaled) only when a 16-term chain exceeds 2^64, which the exact
// recomputation of that chain then resolves.  A tile that some lane sees
// only in part takes a per-element masked variant.  Query rows are
// token-major (the G heads of one text token adjacent), so a block's rows
// span few positions and a block of early text rows stops at its last row.
template <typename T, int D, int NT>
__global__ __launch_bounds__(kThreads, (Occ<T, D>::value)) void rowstats_kernel(P1Args a) {
  using G_ = Geo<T, D>;
  using MM = Mma<T>;
  using frag = typename MM::frag;
  constexpr int NS = G_::NS, ROWB = G_::ROWB, E = G_::E;
  constexpr int QB = 4 * NT * 32;  // query rows per block
  constexpr int KS = kStage1;      // keys per LDS stage
  constexpr int TPS = KS / 32;     // key tiles per stage
  static_assert(TPS % 2 == 0, "accumulator sets alternate between consecutive key tiles");
  // two stage buffers as distinct objects, so the compiler can tell the
  // buffer being read from the one the in-flight DMA writes
  __shared__ __attribute__((aligned(16))) char smA[KS * ROWB];
  __shared__ __attribute__((aligned(16))) char smB[KS * ROWB];

  // Blocks that share one key chunk (the nqb query blocks of a unit) get
  // ids that are equal mod 8, i.e. land on one XCD and share its L2.  Units
  // are numbered (sequence, key head) fastest, so each XCD gets every chunk
  // of its heads (chunks differ in work: the last is short, early text rows
  // see only the first ones) and the short last chunks are dispatched last.
  const int nbg = a.B * a.Hkv, nunits = nbg * a.nkc;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int qb = local % a.nqb;
  const int unit = (local / a.nqb) * 8 + xcd;
  if (unit >= nunits) return;
  const int kc = unit / nbg, bg = unit - kc * nbg, g = bg % a.Hkv, b = bg / a.Hkv;

  const int s0 = a.cu_seqlens[b], L = a.cu_seqlens[b + 1] - s0;
  const int t0 = a.cu_text[b], Tb = a.cu_text[b + 1] - t0;
  const int R = a.G * Tb;
  const int row0 = qb * QB;
  const int kbeg = kc * a.kchunk;
  if (row0 >= R) return;
  const size_t HqT = (size_t)a.Hq * a.T_tot;
  const int32_t *tp = a.text_pos + t0;
  int bmin = 0, bmax = -1;
  if (kbeg < L) rows_pos_range(tp, a.G, row0, min(R, row0 + QB), bmin, bmax);
  if (kbeg >= L || s0 + kbeg > bmax) {
    // no row of the block sees a key of the chunk: empty partials, so that
    // the combine can read every chunk of every row
    for (int r = row0 + (int)threadIdx.x; r < min(R, row0 + QB); r += kThreads) {
      const int t = r / a.G, qidx = (g * a.G + (r - t * a.G)) * a.T_tot + t0 + t;
      a.part_m[kc * HqT + qidx] = -INFINITY;
      a.part_l[kc * HqT + qidx] = 0.f;
    }
    return;
  }
  const int kend = min(L, kbeg + a.kchunk);
  const int kstop = min(kend, bmax - s0 + 1);    // keys after the last row are never visible

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (SGPR)
  const int hi = lane >> 5, col = lane & 31;
  const int wr0 = row0 + wave * NT * 32;
  const bool active = wr0 < R;
  int wmin = 0, wmax = -1;
  if (active) rows_pos_range(tp, a.G, wr0, min(R, wr0 + NT * 32), wmin, wmax);

  // stationary operand: this wave's query rows
  frag qf[NT][NS];
  int qrel[NT];  // query position relative to the sequence start (-1: padding row)
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    const int r = wr0 + i * 32 + col;
    qrel[i] = -1;
    if (r < R) {
      const int t = r / a.G, h = g * a.G + (r - t * a.G);
      qrel[i] = tp[t] - s0;
      const char *src = a.q + ((size_t)(t0 + t) * a.Hq + h) * ROWB + hi * E * sizeof(T);
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[i][s] = load_frag<frag>(src + s * 2 * E * sizeof(T));
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[i][s] = frag{};
    }
  }

  float ref[NT], l[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    ref[i] = -INFINITY;
    l[i] = 0.f;
  }
  const float cl2e = a.cl2e;

  // keys of one stage, rows clamped into the chunk (rows past kend are masked)
  const char *kbase = a.k + ((size_t)s0 * a.Hkv + g) * ROWB;  // key 0 of this sequence, head g
  const uint32_t kstride = (uint32_t)a.Hkv * ROWB;
  using DP = DmaPlan<T, D, KS>;
  uint32_t dlo[DP::PER];
  DP::lane_offsets(dlo, lane, kstride);
  auto issue_stage = [&](int ks, char *dst) __attribute__((always_inline)) {
    if (ks + KS <= kend) {
      DP::issue(dst, kbase + (size_t)ks * kstride, wave, dlo, kstride);
    } else {  // last stage of the chunk: rows past its end re-read row kend-1
      dma_stage<T, D, KS>(dst, kbase, wave, lane, [&](int row) __attribute__((always_inline)) {
        return (uint32_t)min(ks + row, kend - 1) * kstride;
      });
    }
  };

  // Accumulator element e of this lane holds key kb + hi*4 + eoff(e) of its
  // query column; it is visible iff eoff(e) <= vl, with the per-lane limit
  // vl = min(q - kb, kend - 1 - kb) - hi*4 (causal row and chunk end).
  auto eoff = [](int e) __attribute__((always_inline)) { return 8 * (e >> 2) + (e & 3); };
  auto vlimit = [&](int qi, int kb) __attribute__((always_inline)) {
    return min(qrel[qi] - kb, kend - 1 - kb) - hi * 4;
  };

  // Accumulator sets: the key tile of parity p is computed into acc[p*NT ..]
  // while the other parity's sets hold the pending tile at key pend_kb.
  f32x16 acc[2 * NT];
#pragma unroll
  for (int i = 0; i < 2 * NT; ++i) acc[i] = f32x16{};
  constexpr int kNone = 1 << 30;  // pend_kb of an empty pending tile: no lane sees it
  int pend_kb = kNone;
  constexpr int kAll = 0, kAllOrNone = 1, kPerElem = 2;
  using All = std::integral_constant<int, kAll>;
  using AllOrNone = std::integral_constant<int, kAllOrNone>;
  using PerElem = std::integral_constant<int, kPerElem>;

  // One key tile: MFMAs of the tile at buf row `lrow` into the sets of
  // parity P (if MF), and the exp2 sums of the pending tile (sets of parity
  // P^1).  Mode M: kAll (every lane sees the whole pending tile), kAllOrNone
  // (every lane sees all or none of it) or kPerElem (per-element mask).
  // With NX the tile's last PF k-steps read the first PF fragments of the
  // next tile (at lrow + 32) into pf, for that tile's PRE.
  constexpr int PF = NS < 3 ? NS : 3;  // key fragments are read PF k-steps ahead of their MFMAs
  frag pf[PF];                          // a tile's first PF fragments, if read before it (PRE)
  using NoNext = std::false_type;
  auto tile = [&](const char *buf, int lrow, auto par_tag, auto mode_tag, auto mf_tag, auto pre_tag,
                  auto nx_tag) __attribute__((always_inline)) {
    constexpr int P = decltype(par_tag)::value;
    constexpr int M = decltype(mode_tag)::value;
    constexpr bool MF = decltype(mf_tag)::value;
    constexpr bool PRE = decltype(pre_tag)::value;
    constexpr bool NX = decltype(nx_tag)::value;
    constexpr int CS = P * NT, PS = (P ^ 1) * NT;
    // per-element limit (kPerElem); in kAllOrNone a lane sees the whole
    // pending tile unless its row precedes it, and only lanes that see it
    // all can take the exact redo below
    int vl[NT];
    bool none[NT];
    float r[NT], ts[NT][2];
#pragma unroll
    for (int qi = 0; qi < NT; ++qi) {
      vl[qi] = M == kPerElem ? vlimit(qi, pend_kb) : 31;
      none[qi] = qrel[qi] < pend_kb;
      r[qi] = ref[qi];
    }
    if (MF) {
#pragma unroll
      for (int qi = 0; qi < NT; ++qi) acc[CS + qi] = f32x16{};
    }
    frag av[NS];
    if (MF) {
#pragma unroll
      for (int s = 0; s < PF; ++s)
        av[s] = PRE ? pf[s] : load_frag<frag>(buf + swz_off<T, D>(lrow + col, s * 2 * E + hi * E));
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (MF) {
        if (s + PF < NS)
          av[s + PF] = load_frag<frag>(buf + swz_off<T, D>(lrow + col, (s + PF) * 2 * E + hi * E));
        else if (NX)
          pf[s + PF - NS] =
              load_frag<frag>(buf + swz_off<T, D>(lrow + 32 + col, (s + PF - NS) * 2 * E + hi * E));
#pragma unroll
        for (int qi = 0; qi < NT; ++qi) acc[CS + qi] = MM::run(av[s], qf[qi][s], acc[CS + qi]);
      }
#pragma unroll
      for (int qi = 0; qi < NT; ++qi) {
#pragma unroll
        for (int e = (s * 16) / NS; e < ((s + 1) * 16) / NS; ++e) {
          float x = acc[PS + qi][e];
          if (M == kPerElem) x = eoff(e) <= vl[qi] ? x : -INFINITY;
          const float v = __builtin_amdgcn_exp2f(x * cl2e - r[qi]);
          if (e < 2) ts[qi][e] = v;  // each of the two chains starts at its first term
          else ts[qi][e & 1] += v;
        }
      }
    }
    if (MF)
      interleave_tile<NS, NT, ((M == kPerElem ? 64 : 40) / NS > 0 ? (M == kPerElem ? 64 : 40) / NS : 1),
                      PRE ? 0 : PF, NX>();
    float t[NT];
    bool bad = false;
#pragma unroll
    for (int qi = 0; qi < NT; ++qi) {
      t[qi] = ts[qi][0] + ts[qi][1];
      if (M == kAllOrNone && none[qi]) t[qi] = 0.f;  // lane sees none of the pending tile
      bad = bad || !(t[qi] <= kLazyLimit);
    }
    if (__ballot(bad) != 0ull) {
      // exact redo of the chains whose sum left the range: raise the
      // reference to the chain's maximum and rescale the row sum
#pragma unroll
      for (int qi = 0; qi < NT; ++qi) {
        if (!(t[qi] <= kLazyLimit)) {
          float mx = -INFINITY;
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (eoff(e) <= vl[qi]) mx = fmaxf(mx, acc[PS + qi][e]);
          const float nm = fmaxf(ref[qi], mx * cl2e);
          float u = 0.f;
          if (nm != -INFINITY) {
            l[qi] = ref[qi] == -INFINITY ? 0.f : l[qi] * __builtin_amdgcn_exp2f(ref[qi] - nm);
            ref[qi] = nm;
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (eoff(e) <= vl[qi]) u += __builtin_amdgcn_exp2f(acc[PS + qi][e] * cl2e - nm);
          }
          t[qi] = u;
        }
      }
    }
#pragma unroll
    for (int qi = 0; qi < NT; ++qi) l[qi] += t[qi];
  };
  using P0 = std::integral_constant<int, 0>;

  const int nstage = (kstop - kbeg + KS - 1) / KS;
  // key tiles this wave processes: those below kstop that start at or
  // before its last row (a prefix of the chunk's tiles)
  const int kw_end = active ? min(kstop, wmax - s0 + 1) : kbeg;
  const int ntw = kw_end > kbeg ? (kw_end - kbeg + 31) / 32 : 0;
  issue_stage(kbeg, smA);
  auto step = [&](const char *buf, char *nxt, int st) __attribute__((always_inline)) {
    const int ks = kbeg + st * KS;
    wait_vmem();
    __syncthreads();  // stage st is in LDS; every wave is done with the other buffer
    if (st + 1 < nstage) issue_stage(ks + KS, nxt);
    // every lane sees every pending tile of the stage (the previous stage's
    // last tile and this stage's first TPS-1): no per-tile checks, and each
    // tile reads the next one's first fragments
    bool allvis = false;
    if ((st + 1) * TPS <= ntw && pend_kb != kNone) {
#pragma unroll
      for (int s = 0; s < PF; ++s) pf[s] = load_frag<frag>(buf + swz_off<T, D>(col, s * 2 * E + hi * E));
      bool part = false;
#pragma unroll
      for (int qi = 0; qi < NT; ++qi) part = part || qrel[qi] < ks + (TPS - 1) * 32 - 1;
      allvis = __ballot(part) == 0ull;
    }
    if (allvis) {
      using P0_ = std::integral_constant<int, 0>;
      using P1_ = std::integral_constant<int, 1>;
      using Yes = std::true_type;
      tile(buf, 0, P0_{}, All{}, Yes{}, Yes{}, Yes{});
      tile(buf, 32, P1_{}, All{}, Yes{}, Yes{}, Yes{});
      if constexpr (TPS == 4) {
        tile(buf, 64, P0_{}, All{}, Yes{}, Yes{}, Yes{});
        tile(buf, 96, P1_{}, All{}, Yes{}, Yes{}, NoNext{});
      }
      pend_kb = ks + (TPS - 1) * 32;
    } else if ((st + 1) * TPS <= ntw) {
      // every tile of the stage is this wave's: no per-tile bounds
      auto one = [&](auto kt_tag) __attribute__((always_inline)) {
        constexpr int KT = decltype(kt_tag)::value;
        using par_tag = std::integral_constant<int, KT & 1>;
        // a lane that sees only part of the pending tile needs the masked
        // variant; the tile's first fragments are read before this check,
        // whose VALU work then covers their latency
#pragma unroll
        for (int s = 0; s < PF; ++s)
          pf[s] = load_frag<frag>(buf + swz_off<T, D>(KT * 32 + col, s * 2 * E + hi * E));
        bool part = false;
#pragma unroll
        for (int qi = 0; qi < NT; ++qi) part = part || (unsigned)(qrel[qi] - pend_kb) < 31u;
        if (__ballot(part) == 0ull)
          tile(buf, KT * 32, par_tag{}, AllOrNone{}, std::true_type{}, std::true_type{}, NoNext{});
        else
          tile(buf, KT * 32, par_tag{}, PerElem{}, std::true_type{}, std::true_type{}, NoNext{});
        pend_kb = ks + KT * 32;
      };
      static_assert(TPS == 2 || TPS == 4, "one stage is two or four key tiles");
      one(std::integral_constant<int, 0>{});
      one(std::integral_constant<int, 1>{});
      if constexpr (TPS == 4) {
        one(std::integral_constant<int, 2>{});
        one(std::integral_constant<int, 3>{});
      }
    } else if (st * TPS < ntw) {
      // the wave's last tiles, then settle the pending one (masked variant)
      auto one = [&](auto kt_tag) __attribute__((always_inline)) {
        constexpr int KT = decltype(kt_tag)::value;
        using par_tag = std::integral_constant<int, KT & 1>;
        if (st * TPS + KT < ntw) {
          tile(buf, KT * 32, par_tag{}, PerElem{}, std::true_type{}, std::false_type{}, NoNext{});
          pend_kb = ks + KT * 32;
        } else if (st * TPS + KT == ntw) {
          tile(buf, 0, par_tag{}, PerElem{}, std::false_type{}, std::false_type{}, NoNext{});
          pend_kb = kNone;
        }
      };
      one(std::integral_constant<int, 0>{});
      one(std::integral_constant<int, 1>{});
      if constexpr (TPS == 4) {
        one(std::integral_constant<int, 2>{});
        one(std::integral_constant<int, 3>{});
      }
    }
  };
  for (int st = 0; st < nstage; st += 2) {
    step(smA, smB, st);
    if (st + 1 < nstage) step(smB, smA, st + 1);
  }
  if (!active) return;
  // with a whole number of stages the pending tile is the last (odd) one
  if (ntw > 0 && ntw % TPS == 0) tile(smA, 0, P0{}, PerElem{}, std::false_type{}, std::false_type{}, NoNext{});

  // merge the two half-waves (same query column, disjoint keys) and store
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    const float om = __shfl_xor(ref[i], 32), ol = __shfl_xor(l[i], 32);
    const float nm = fmaxf(ref[i], om);
    float tot = 0.f;
    if (nm != -INFINITY)
      tot = (ref[i] == -INFINITY ? 0.f : l[i] * __builtin_amdgcn_exp2f(ref[i] - nm)) +
            (om == -INFINITY ? 0.f : ol * __builtin_amdgcn_exp2f(om - nm));
    const int r = wr0 + i * 32 + col;
    if (hi == 0 && r < R) {
      const int t = r / a.G, qidx = (g * a.G + (r - t * a.G)) * a.T_tot + t0 + t;
      a.part_m[kc * HqT + qidx] = nm;
      a.part_l[kc * HqT + qidx] = tot;
    }
  }
}

// Merge the chunk partials of every text row into lse = ln(sum exp(z)), and
// (if lse2 is given) the same in log2 units for pass 2.  Pass 1 writes a
// partial for every (chunk, row), empty (-inf, 0) where the row sees no key
// of the chunk.  Max and sum run over the chunks in ascending order.
//
// The loads of G chunks are issued together (a chunk index past nkc re-reads
// the last chunk and is then ignored).  With at most G chunks, every partial
// of the row is held in registers and read once: the kernel waits on one
// round of loads; with more, the groups are read twice (max, then sum).
template <int G>
__global__ void lse_combine_kernel(const float *__restrict__ part_m, const float *__restrict__ part_l,
                                   int rows, int nkc, float *__restrict__ lse,
                                   float *__restrict__ lse2) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows) return;
  auto at = [&](int c) __attribute__((always_inline)) {
    return (size_t)min(c, nkc - 1) * rows + idx;
  };
  float M = -INFINITY, S = 0.f;
  if (nkc <= G) {
    float m[G], l[G];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      m[u] = part_m[at(u)];
      l[u] = part_l[at(u)];
    }
#pragma unroll
    for (int u = 0; u < G; ++u)
      if (u < nkc) M = fmaxf(M, m[u]);
#pragma unroll
    for (int u = 0; u < G; ++u)
      if (u < nkc && m[u] != -INFINITY) S += l[u] * __builtin_amdgcn_exp2f(m[u] - M);
  } else {
    for (int c0 = 0; c0 < nkc; c0 += G) {
      float m[G];
#pragma unroll
      for (int u = 0; u < G; ++u) m[u] = part_m[at(c0 + u)];
#pragma unroll
      for (int u = 0; u < G; ++u)
        if (c0 + u < nkc) M = fmaxf(M, m[u]);
    }
    for (int c0 = 0; c0 < nkc; c0 += G) {
      float m[G], l[G];
#pragma unroll
      for (int u = 0; u < G; ++u) {
        m[u] = part_m[at(c0 + u)];
        l[u] = part_l[at(c0 + u)];
      }
#pragma unroll
      for (int u = 0; u < G; ++u)
        if (c0 + u < nkc && m[u] != -INFINITY) S += l[u] * __builtin_amdgcn_exp2f(m[u] - M);
    }
  }
  const float v = (M + __builtin_amdgcn_logf(S)) * kLn2;
  lse[idx] = v;
  // log2 units from the rounded natural value, exactly as for a supplied LSE
  if (lse2) lse2[idx] = v * kLog2e;
}

// Row LSE in natural log -> log2 units (for an LSE the caller supplies).
__global__ void lse_to_log2_kernel(const float *__restrict__ lse, int rows, float *__restrict__ lse2) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < rows) lse2[idx] = lse[idx] * kLog2e;
}

// Pass-2 LDS stage: kStage query rows (swizzled) with their row LSE and
// positions, double-buffered.  Rows past the end of the split get LSE +inf
// and position -1, copied from these two constants, so they add nothing and
// are never visible.
__device__ const float kRowNone = INFINITY;
__device__ const int kPosNone = -1;
template <int ROWB>
struct __attribute__((aligned(16))) QTile2 {
  char q[kStage * ROWB];
  float lse[kStage];  // log2 units
  int pos[kStage];
};

struct P2Args {
  const char *q, *k;
  const float *lse2;  // row LSE in log2 units, [Hq][T_tot]
  const int32_t *cu_seqlens, *cu_text, *text_pos;
  int B, Hq, Hkv, G, T_tot, N_tok, nkb, nqs;
  int nsl, ppx, kps;  // key-block slices per unit, (unit, slice) pairs per XCD, blocks per pair
  float cl2e;
  float *colsum;  // [nqs][Hkv][N_tok]
};

// Pass 2: per (sequence b, key head g, key block, query split), the column
// sums sum_{h in group g} sum_t exp(c q_{t,h}.k_j - lse[h,t]) over the split's
// rows t that see key j.
//
// Keys are the stationary MFMA operand: each wave holds NKT 32-key tiles.
// Query sub-tiles of 32 rows stream through double-buffered LDS together
// with their row LSE and positions, all brought in by direct-to-LDS loads.
// Per sub-tile the wave runs one chain of MFMAs per key tile, chain j into
// accumulator set j; the VALU work interleaved with chain j turns the
// accumulators of the chain DIST chains earlier (of this sub-tile or the
// previous one processed) into exp2 terms, one FMA, one exp2 and one add
// per logit, so it never waits on a running MFMA.  A sub-tile some rows of
// which see only part of the wave's keys is done unpipelined with a
// per-element mask; sub-tiles that see none are skipped.
template <typename T, int D, int NKT>
__global__ __launch_bounds__(kThreads, (Occ<T, D>::value)) void colsum_kernel(P2Args a) {
  using G_ = Geo<T, D>;
  using MM = Mma<T>;
  using frag = typename MM::frag;
  constexpr int NS = G_::NS, ROWB = G_::ROWB, E = G_::E;
  constexpr int DIST = NKT >= 3 ? 2 : NKT - 1;  // pipeline distance in chains
  constexpr int KB = 4 * NKT * 32;  // keys per block
  constexpr int QR = kStage;        // query rows per stage
  constexpr int SUBS = QR / 32;     // sub-tiles per stage
  static_assert(SUBS == 4, "one stage is four query sub-tiles");
  // two query buffers as distinct objects (see pass 1)
  __shared__ QTile2<ROWB> qtA, qtB;

  // The key blocks of one (sequence, key head) read the same queries, so
  // they stay on few XCDs: a unit's key blocks are dealt to nsl slices
  // (kb mod nsl, enough (unit, slice) pairs for the 8 XCDs), and the blocks
  // of one pair land on XCD pair mod 8, one pair after the other, so that
  // an XCD's L2 holds the queries of few units at a time.
  const int npairs = a.B * a.Hkv * a.nsl;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int per = a.kps * a.nqs;
  const int kk = local % per, pj = local / per;
  const int pair = pj * 8 + xcd;
  if (pair >= npairs) return;
  const int unit = pair / a.nsl, sl = pair - unit * a.nsl;
  const int kbl = kk % a.kps, qsp = kk / a.kps;
  const int kb = kbl * a.nsl + sl;
  if (kb >= a.nkb || qsp >= a.nqs) return;
  const int g = unit % a.Hkv, b = unit / a.Hkv;
  const int s0 = a.cu_seqlens[b], L = a.cu_seqlens[b + 1] - s0;
  const int t0 = a.cu_text[b], Tb = a.cu_text[b + 1] - t0;
  const int R = a.G * Tb;
  const int kb0 = kb * KB;
  if (kb0 >= L) return;
  // rows of this split: [r_lo, r_hi), split boundaries on whole stages
  const int rps = ((R + a.nqs - 1) / a.nqs + QR - 1) / QR * QR;
  const int r_lo = min(R, qsp * rps), r_hi = min(R, r_lo + rps);
  const int32_t *tp = a.text_pos + t0;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (SGPR)
  const int hi = lane >> 5, col = lane & 31;
  const int kw0 = kb0 + wave * NKT * 32;
  const bool active = kw0 < L;
  const int kmin = s0 + kw0, kmax = s0 + min(L, kw0 + NKT * 32) - 1;

  frag kf[NKT][NS];
#pragma unroll
  for (int j = 0; j < NKT; ++j) {
    const int key = kw0 + j * 32 + col;
    if (key < L) {
      const char *src = a.k + ((size_t)(s0 + key) * a.Hkv + g) * ROWB + hi * E * sizeof(T);
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[j][s] = load_frag<frag>(src + s * 2 * E * sizeof(T));
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[j][s] = frag{};
    }
  }
  // position of this lane's key in key tile j (padding keys: never visible)
  auto kpos = [&](int j) __attribute__((always_inline)) {
    const int key = kw0 + j * 32 + col;
    return key < L ? s0 + key : 0x7fffffff;
  };
  float cs[NKT];
#pragma unroll
  for (int j = 0; j < NKT; ++j) cs[j] = 0.f;
  const float cl2e = a.cl2e;

  const char *qbase = a.q + ((size_t)t0 * a.Hq + g * a.G) * ROWB;  // text row 0, head g*G
  const uint32_t qstride = (uint32_t)a.Hq * ROWB;
  const float *lbase = a.lse2 + (size_t)g * a.G * a.T_tot + t0;    // head g*G, text row 0
  using DP = DmaPlan<T, D, QR>;
  // Rows are token-major: row r is text token r / G under query head
  // g*G + r % G, so positions ascend with r.  With G a power of two every
  // stage load has per-lane offsets fixed across stages.
  const int lg = __builtin_ctz((unsigned)a.G);
  const bool g_pow2 = (a.G & (a.G - 1)) == 0;
  // One stage: query rows [rs, rs + QR), their LSE and positions.  Wave 0
  // loads the LSE, wave 1 the positions, 64 rows per instruction.
  auto issue_stage = [&](int rs, QTile2<ROWB> &dst) __attribute__((always_inline)) {
    if (g_pow2 && rs + QR <= R) {
      int ln = lane;
      asm volatile("" : "+v"(ln));
      uint32_t dlo[DP::PER];
      DP::lane_offsets_tm(dlo, ln, lg, qstride);
      DP::issue_tm(dst.q, qbase, rs, wave, dlo, lg, qstride);
    } else {
      dma_stage<T, D, QR>(dst.q, qbase, wave, lane, [&](int row) __attribute__((always_inline)) {
        const int r = min(rs + row, R - 1);  // rows past R re-read row R-1; their lse is +inf
        const int t = r / a.G;
        return (uint32_t)(t * a.Hq + (r - t * a.G)) * ROWB;
      });
    }
    if (wave < 2) {
#pragma unroll
      for (int i = 0; i < QR / 64; ++i) {
        const int r = rs + i * 64 + lane;
        const void *src;
        if (r < r_hi) {
          const int t = r / a.G;
          src = wave == 0 ? (const void *)(lbase + (size_t)(r - t * a.G) * a.T_tot + t) : (const void *)(tp + t);
        } else {
          src = wave == 0 ? (const void *)&kRowNone : (const void *)&kPosNone;
        }
        void *dstp = wave == 0 ? (void *)(dst.lse + i * 64) : (void *)(dst.pos + i * 64);
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src,
                                         (__attribute__((address_space(3))) void *)dstp, 4, 0, 0);
      }
    }
  };

  // acc[j]: chain j of the latest sub-tile processed.  The chains
  // NKT-DIST .. NKT-1 of the previous sub-tile processed are still pending,
  // with that sub-tile's LSE (log2 units) in plv (+inf: nothing pending).
  f32x16 acc[NKT];
#pragma unroll
  for (int j = 0; j < NKT; ++j) acc[j] = f32x16{};
  float plv[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) plv[e] = INFINITY;

  // exp2 terms of chain c (its accumulators in set c) for elements [e0, e1);
  // the two partial sums start at elements 0 and 1 (the same bits as 0 +
  // term, since no term is negative)
  auto terms = [&](int c, int e0, int e1, const float *lv, float (&ts)[2])
      __attribute__((always_inline)) {
#pragma unroll
    for (int e = e0; e < e1; ++e) {
      const float v = __builtin_amdgcn_exp2f(acc[c][e] * cl2e - lv[e]);
      if (e < 2) ts[e] = v;
      else ts[e & 1] += v;
    }
  };
  // the sub-tile's LSE of this lane's rows (log2 units)
  auto load_lv = [&](const QTile2<ROWB> &cur, int U, float (&lv)[16]) __attribute__((always_inline)) {
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const float4 x = *reinterpret_cast<const float4 *>(&cur.lse[U * 32 + hi * 4 + 8 * e4]);
      lv[4 * e4 + 0] = x.x;
      lv[4 * e4 + 1] = x.y;
      lv[4 * e4 + 2] = x.z;
      lv[4 * e4 + 3] = x.w;
    }
  };
  // a sub-tile in stage slot U that every row of which sees every key of the
  // wave: chain j of MFMAs with the terms of chain j-DIST in between
  auto sub_tile = [&](const QTile2<ROWB> &cur, auto u_tag, const frag (&av)[NS]) __attribute__((always_inline)) {
    constexpr int U = decltype(u_tag)::value;
    // this sub-tile's LSE, read once the pending chains no longer need plv
    float clv[16];
#pragma unroll
    for (int j = 0; j < NKT; ++j) {
      if (j == DIST) load_lv(cur, U, clv);
      const int pj = j - DIST;       // chain processed by the VALU alongside chain j
      const bool prev = pj < 0;      // (of the previous sub-tile)
      const int pc = prev ? pj + NKT : pj;
      float ts[2] = {0.f, 0.f};
      acc[j] = f32x16{};
      if (DIST > 0) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          acc[j] = MM::run(av[s], kf[j][s], acc[j]);
          terms(pc, (s * 16) / NS, ((s + 1) * 16) / NS, prev ? plv : clv, ts);
        }
        interleave_mfma_valu<NS, (24 / NS > 0 ? 24 / NS : 1)>();
      } else {
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[j] = MM::run(av[s], kf[j][s], acc[j]);
        terms(pc, 0, 16, clv, ts);
      }
      cs[pc] += ts[0] + ts[1];
    }
    // the last DIST chains of this sub-tile are now the pending ones
#pragma unroll
    for (int e = 0; e < 16; ++e) plv[e] = clv[e];
  };
  // settle the pending chains
  auto settle = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = NKT - DIST; c < NKT; ++c) {
      float ts[2] = {0.f, 0.f};
      terms(c, 0, 16, plv, ts);
      cs[c] += ts[0] + ts[1];
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) plv[e] = INFINITY;
  };
  // a sub-tile in slot U some rows of which see only part of the wave's
  // keys: settle what is pending, then MFMAs and masked terms, unpipelined.
  // The terms are summed in the order of the unmasked path (two alternating
  // partial sums per chain, elements ascending) and a masked term is an
  // exact 0, so a key that sees every row of the sub-tile gets the same bits
  // on either path.
  auto sub_masked = [&](const QTile2<ROWB> &cur, auto u_tag, const frag (&av)[NS]) __attribute__((always_inline)) {
    constexpr int U = decltype(u_tag)::value;
    settle();
#pragma unroll
    for (int j = 0; j < NKT; ++j) {
      acc[j] = f32x16{};
#pragma unroll
      for (int s = 0; s < NS; ++s) acc[j] = MM::run(av[s], kf[j][s], acc[j]);
    }
    float ts[NKT][2];
#pragma unroll
    for (int j = 0; j < NKT; ++j) ts[j][0] = ts[j][1] = 0.f;
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const int ro = U * 32 + hi * 4 + 8 * e4;
      const float4 lv4 = *reinterpret_cast<const float4 *>(&cur.lse[ro]);
      const int4 qp4 = *reinterpret_cast<const int4 *>(&cur.pos[ro]);
      const float lv[4] = {lv4.x, lv4.y, lv4.z, lv4.w};
      const int qp[4] = {qp4.x, qp4.y, qp4.z, qp4.w};
#pragma unroll
      for (int j = 0; j < NKT; ++j) {
        const int kp = kpos(j);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * e4 + i;
          ts[j][e & 1] += kp <= qp[i] ? __builtin_amdgcn_exp2f(acc[j][e] * cl2e - lv[i]) : 0.f;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NKT; ++j) cs[j] += ts[j][0] + ts[j][1];
  };

  const int nstage = (r_hi - r_lo + QR - 1) / QR;
  if (nstage > 0) issue_stage(r_lo, qtA);
  auto step = [&](QTile2<ROWB> &cur, QTile2<ROWB> &nxt, int st) __attribute__((always_inline)) {
    const int rs = r_lo + st * QR;
    wait_vmem();
    __syncthreads();  // stage st is in LDS; every wave is done with the other buffer
    if (st + 1 < nstage) issue_stage(rs + QR, nxt);
    if (active) {
      auto one = [&](auto u_tag) __attribute__((always_inline)) {
        constexpr int U = decltype(u_tag)::value;
        const int nv = min(32, r_hi - (rs + U * 32));  // valid rows of the sub-tile
        if (nv > 0) {
          // the query fragments are read together with the positions that
          // classify the sub-tile: one LDS round trip before the first MFMA
          frag av[NS];
#pragma unroll
          for (int s = 0; s < NS; ++s)
            av[s] = load_frag<frag>(cur.q + swz_off<T, D>(U * 32 + col, s * 2 * E + hi * E));
          const int qmin = cur.pos[U * 32], qmax = cur.pos[U * 32 + nv - 1];
          if (qmax >= kmin) {  // else no row of the sub-tile sees a key of the wave
            if (qmin >= kmax) sub_tile(cur, u_tag, av);
            else sub_masked(cur, u_tag, av);
          }
        }
      };
      one(std::integral_constant<int, 0>{});
      one(std::integral_constant<int, 1>{});
      one(std::integral_constant<int, 2>{});
      one(std::integral_constant<int, 3>{});
    }
  };
  for (int st = 0; st < nstage; st += 2) {
    step(qtA, qtB, st);
    if (st + 1 < nstage) step(qtB, qtA, st + 1);
  }
  if (!active) return;
  settle();  // the chains still pending
#pragma unroll
  for (int j = 0; j < NKT; ++j) {
    const float v = cs[j] + __shfl_xor(cs[j], 32);
    const int key = kw0 + j * 32 + col;
    if (hi == 0 && key < L) a.colsum[((size_t)qsp * a.Hkv + g) * a.N_tok + s0 + key] = v;
  }
}

template <typename T, int D>
hipError_t run_row_lse(hipStream_t st, const DevLayout &L, const AttnPlan &P, const void *q,
                       const void *k, int Hq, int Hkv, float scale, float *row_lse, float *lse2,
                       char *ws) {
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
  if (P.nt1 == 1)  // one query tile per wave on small grids (attn_plan)
    hipLaunchKernelGGL((rowstats_kernel<T, D, 1>), dim3(grid), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((rowstats_kernel<T, D, kTiles1>), dim3(grid), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rows = Hq * L.T_tot;
  const dim3 cg((rows + 255) / 256), cb(256);
  if (P.nkc <= 8)
    hipLaunchKernelGGL(lse_combine_kernel<8>, cg, cb, 0, st, a.part_m, a.part_l, rows, P.nkc,
                       row_lse, lse2);
  else if (P.nkc <= 16)
    hipLaunchKernelGGL(lse_combine_kernel<16>, cg, cb, 0, st, a.part_m, a.part_l, rows, P.nkc,
                       row_lse, lse2);
  else
    hipLaunchKernelGGL(lse_combine_kernel<32>, cg, cb, 0, st, a.part_m, a.part_l, rows, P.nkc,
                       row_lse, lse2);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t run_colsum(hipStream_t st, const DevLayout &L, const AttnPlan &P, const void *q,
                      const void *k, int Hq, int Hkv, float scale, const float *lse2, char *ws) {
  P2Args a;
  a.q = (const char *)q;
  a.k = (const char *)k;
  a.lse2 = lse2;
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
  a.nqs = P.nqs;
  a.cl2e = scale * kLog2e;
  a.colsum = (float *)(ws + P.off_colsum);
  a.nsl = P.nsl;
  a.ppx = (L.B * Hkv * P.nsl + 7) / 8;
  a.kps = (P.nkb + P.nsl - 1) / P.nsl;
  const int grid = 8 * a.ppx * a.kps * P.nqs;
  if constexpr (Geo<T, D>::NT2 == 3) {  // narrower blocks for small grids (attn_plan)
    if (P.nkt2 == 2) {
      hipLaunchKernelGGL((colsum_kernel<T, D, 2>), dim3(grid), dim3(kThreads), 0, st, a);
      return hipGetLastError();
    }
    if (P.nkt2 == 1) {
      hipLaunchKernelGGL((colsum_kernel<T, D, 1>), dim3(grid), dim3(kThreads), 0, st, a);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((colsum_kernel<T, D, Geo<T, D>::NT2>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

AttnPlan attn_plan(const DevLayout &L, int Hq, int Hkv, int d, int dtype) {
  AttnPlan P;
  P.G = Hq / Hkv;
  const int row_bytes = d * (dtype == AVTP_FP32 ? 4 : 2);
  int nkt2 = tiles_pass2(row_bytes);                            // pass 2 key tiles per wave
  P.rows_max = P.G * L.max_text;
  // Pass 1 geometry for nt query tiles per wave: query blocks per unit and
  // the key chunk.
  auto pass1 = [&](int nt, int &nqb, long long &kc) {
    const int rows_per_block = 4 * nt * 32;
    nqb = (P.rows_max + rows_per_block - 1) / rows_per_block;
    if (nqb < 1) nqb = 1;
    // split keys so that pass 1 launches about 1536 blocks (6 per CU, three
    // rounds of two); chunks of at least two stages, or one on a grid of less
    // than one block per CU, where a block's latency is what counts.  Against
    // 2048 blocks: 8 sequences of 16 images 135 -> 129 us, 4 x 32 images of
    // 1,024 tokens 488 -> 482 us sustained; 2560-4096 blocks were 3-4 %
    // slower there
    const long long base = (long long)L.B * Hkv * nqb;
    long long want = (1536 + base - 1) / base;
    if (want < 1) want = 1;
    kc = (L.max_seqlen + want - 1) / want;
    kc = ((kc + kStage1 - 1) / kStage1) * kStage1;
    if (kc < 2 * kStage1) {
      const long long two = (L.max_seqlen + 2 * kStage1 - 1) / (2 * kStage1);  // chunks of two stages
      kc = base * two < 256 ? (kc < kStage1 ? kStage1 : kc) : 2 * kStage1;
    }
    // Where that gives blocks of at most two stages but more than 512 of them
    // (more than one round at two blocks per CU), a block's fixed latency
    // (layout reads, query loads, the first stage's wait, the flush) outweighs
    // its work: take chunks long enough for at most 512 blocks, one round.
    // Two sequences of 8 images with 96 text rows: 1,024 blocks of two stages
    // -> 512 of four, pass 1 33.3 -> 28.8 us (384 or 256 blocks: 34.7, 29.7).
    if (kc <= 2 * kStage1 && base <= 512 && base * ((L.max_seqlen + kc - 1) / kc) > 512) {
      const long long per = 512 / base;  // chunks per unit
      long long k2 = (L.max_seqlen + per - 1) / per;
      k2 = ((k2 + kStage1 - 1) / kStage1) * kStage1;
      if (k2 > kc) kc = k2;
    }
    return base * ((L.max_seqlen + kc - 1) / kc);  // blocks
  };
  // Two query tiles per wave (a key fragment read from LDS serves two
  // MFMAs).  A grid that fits in one round (at most 512 blocks) is bound by
  // latency instead: there blocks of one tile per wave
  // (128 rows, more blocks and rows of closer positions) measured faster:
  // one sequence of 4 x 729 tokens 13.4 -> 12.9 us, two sequences of 8
  // images 28.4 -> 26.2 us; on the larger grids they were slower (8 x 16
  // images 127-131 -> 134-137 us, 4 x 32 images 536-540 -> 602-606 us).
  int nqb = 1;
  long long kc = 0;
  P.nt1 = kTiles1;
  if (pass1(kTiles1, nqb, kc) <= 512) {
    P.nt1 = 1;
    pass1(1, nqb, kc);
  }
  P.nqb = nqb;
  P.kchunk = (int)kc;
  P.nkc = (L.max_seqlen + P.kchunk - 1) / P.kchunk;
  if (P.nkc < 1) P.nkc = 1;
  // Pass 2: three key tiles per wave (384 keys per block) where that gives
  // at least 512 blocks; on smaller grids two, and one where two give fewer
  // than 256 blocks, so that more blocks share the chip (the rows a block
  // streams are the same whatever its width).  Two sequences of 8 images with
  // 96 text rows (336 -> 512 blocks): pass 2 34.5 -> 29.2 us; one sequence of
  // 4 x 729 tokens: 15.3 -> 12.8 (two tiles) -> 12.3 us (one).  At 2,432
  // blocks three tiles stay faster (8 x 16 images: 108-113 against 119-124).
  auto key_blocks = [&](int nt) { return (L.max_seqlen + 4 * nt * 32 - 1) / (4 * nt * 32); };
  P.nkb = key_blocks(nkt2);
  if (nkt2 == 3 && (long long)L.B * Hkv * P.nkb < 512) {
    nkt2 = 2;
    P.nkb = key_blocks(nkt2);
    if ((long long)L.B * Hkv * P.nkb < 256) {
      nkt2 = 1;
      P.nkb = key_blocks(nkt2);
    }
  }
  if (P.nkb < 1) P.nkb = 1;
  P.nkt2 = nkt2;
  {  // slices per unit: the fewest that make the (unit, slice) pairs a multiple of 8
    int a8 = L.B * Hkv, b8 = 8;
    while (b8 != 0) {
      const int t = a8 % b8;
      a8 = b8;
      b8 = t;
    }
    P.nsl = 8 / a8;
    if (P.nsl > P.nkb) P.nsl = P.nkb;
  }
  // Split the query rows of pass 2 only when its grid would not fill the
  // chip twice over (512 blocks): a block pays for loading its keys and for
  // filling its pipeline, so fewer, longer blocks are faster; keep at least
  // 512 rows (four stages) per split.  A grid of less than one block per CU
  // is latency-bound instead: there a split may go down to one stage.
  {
    const long long base2 = (long long)L.B * Hkv * P.nkb;
    long long nq = base2 >= 512 ? 1 : (512 + base2 - 1) / base2;
    const long long min_rows = base2 < 256 ? kStage : 512;
    const long long cap = (P.rows_max + min_rows - 1) / min_rows;
    if (nq > cap) nq = cap;
    P.nqs = nq < 1 ? 1 : (int)nq;
  }
  const size_t rows = (size_t)Hq * L.T_tot;
  size_t off = 0;
  P.off_part_m = off;
  off = align256(off + sizeof(float) * rows * P.nkc);
  P.off_part_l = off;
  off = align256(off + sizeof(float) * rows * P.nkc);
  P.off_lse = off;
  off = align256(off + sizeof(float) * rows);
  P.off_lse2 = off;
  off = align256(off + sizeof(float) * rows);
  P.off_colsum = off;
  off = align256(off + sizeof(float) * (size_t)P.nqs * Hkv * L.N_tok);
  P.bytes = off;
  return P;
}

hipError_t launch_row_lse(hipStream_t st, const DevLayout &L, const AttnPlan &P, int dtype,
                          const void *q, const void *k, int Hq, int Hkv, int d, float scale,
                          float *row_lse, float *lse2, char *ws) {
  clear_pending_error();
  if (dtype == AVTP_BF16)
    return d == 128 ? run_row_lse<__bf16, 128>(st, L, P, q, k, Hq, Hkv, scale, row_lse, lse2, ws)
                    : run_row_lse<__bf16, 64>(st, L, P, q, k, Hq, Hkv, scale, row_lse, lse2, ws);
  return d == 128 ? run_row_lse<float, 128>(st, L, P, q, k, Hq, Hkv, scale, row_lse, lse2, ws)
                  : run_row_lse<float, 64>(st, L, P, q, k, Hq, Hkv, scale, row_lse, lse2, ws);
}

hipError_t launch_lse_to_log2(hipStream_t st, int rows, const float *lse, float *lse2) {
  clear_pending_error();
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(lse_to_log2_kernel, dim3((rows + 255) / 256), dim3(256), 0, st, lse, rows, lse2);
  return hipGetLastError();
}

hipError_t launch_colsum(hipStream_t st, const DevLayout &L, const AttnPlan &P, int dtype,
                         const void *q, const void *k, int Hq, int Hkv, int d, float scale,
                         const float *lse2, char *ws) {
  clear_pending_error();
  if (dtype == AVTP_BF16)
    return d == 128 ? run_colsum<__bf16, 128>(st, L, P, q, k, Hq, Hkv, scale, lse2, ws)
                    : run_colsum<__bf16, 64>(st, L, P, q, k, Hq, Hkv, scale, lse2, ws);
  return d == 128 ? run_colsum<float, 128>(st, L, P, q, k, Hq, Hkv, scale, lse2, ws)
                  : run_colsum<float, 64>(st, L, P, q, k, Hq, Hkv, scale, lse2, ws);
}

}  // namespace avtp
