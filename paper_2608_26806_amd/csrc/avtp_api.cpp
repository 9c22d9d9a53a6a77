// Host layer of libavtp.so: argument validation (pure host code, runs before
// any HIP call and therefore also without a GPU), workspace sizing and the
// C entry points declared in include/avtp.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "avtp_internal.h"

namespace avtp {
namespace {

inline int hip_status(hipError_t e) { return e == hipSuccess ? AVTP_OK : AVTP_ERR_HIP; }

// Validate the packed layout from its host mirrors and derive launch maxima.
// Checks: array presence; monotone offsets; images ascending, non-overlapping,
// inside their sequence; text ascending and inside the sequence; every token
// is text or visual (the lengths partition each sequence); size limits.
int check_layout(const avtp_layout *lay, DevLayout *out) {
  if (!lay) return AVTP_ERR_INVALID_ARG;
  const int B = lay->B, n_img = lay->n_img, N = lay->N_tok, T = lay->T_tot;
  if (B < 1 || n_img < 0 || N < 1 || T < 0) return AVTP_ERR_INVALID_ARG;
  // the image arrays may be NULL without images, text_pos without text rows
  // (an empty array may have no address)
  if (!lay->cu_seqlens || !lay->cu_img || !lay->cu_text || !lay->keep_total ||
      (n_img > 0 && (!lay->img_start || !lay->img_len)) || (T > 0 && !lay->text_pos))
    return AVTP_ERR_INVALID_ARG;
  if (!lay->h_cu_seqlens || !lay->h_cu_img || !lay->h_cu_text || !lay->h_keep_total ||
      (n_img > 0 && (!lay->h_img_start || !lay->h_img_len)) || (T > 0 && !lay->h_text_pos))
    return AVTP_ERR_INVALID_ARG;
  if (n_img > AVTP_MAX_IMAGES) return AVTP_ERR_UNSUPPORTED;
  const int32_t *cs = lay->h_cu_seqlens, *ci = lay->h_cu_img, *ct = lay->h_cu_text;
  if (cs[0] != 0 || ci[0] != 0 || ct[0] != 0) return AVTP_ERR_INVALID_ARG;
  if (cs[B] != N || ci[B] != n_img || ct[B] != T) return AVTP_ERR_INVALID_ARG;
  int max_seq = 0, max_text = 0, max_img = 0, max_ips = 0;
  for (int b = 0; b < B; ++b) {
    const int s0 = cs[b], s1 = cs[b + 1];
    if (s1 < s0 || ci[b + 1] < ci[b] || ct[b + 1] < ct[b]) return AVTP_ERR_INVALID_ARG;
    if (ci[b + 1] - ci[b] > AVTP_MAX_IMAGES_PER_SEQ) return AVTP_ERR_UNSUPPORTED;
    max_ips = std::max(max_ips, ci[b + 1] - ci[b]);
    int64_t covered = ct[b + 1] - ct[b];
    int prev_end = s0;
    for (int i = ci[b]; i < ci[b + 1]; ++i) {
      const int st = lay->h_img_start[i], n = lay->h_img_len[i];
      if (n < 0 || st < prev_end || (int64_t)st + n > s1) return AVTP_ERR_INVALID_ARG;
      if (n > AVTP_MAX_IMAGE_LEN) return AVTP_ERR_UNSUPPORTED;
      prev_end = st + n;
      covered += n;
      max_img = std::max(max_img, n);
    }
    if (covered != s1 - s0) return AVTP_ERR_INVALID_ARG;
    // text rows: ascending, inside the sequence, outside every image (merge walk)
    int img = ci[b], prev = s0 - 1;
    for (int t = ct[b]; t < ct[b + 1]; ++t) {
      const int p = lay->h_text_pos[t];
      if (p <= prev || p >= s1) return AVTP_ERR_INVALID_ARG;
      while (img < ci[b + 1] && lay->h_img_start[img] + lay->h_img_len[img] <= p) ++img;
      if (img < ci[b + 1] && lay->h_img_start[img] <= p) return AVTP_ERR_INVALID_ARG;
      prev = p;
    }
    if (lay->h_keep_total[b] < 0) return AVTP_ERR_INVALID_ARG;
    max_seq = std::max(max_seq, s1 - s0);
    max_text = std::max(max_text, ct[b + 1] - ct[b]);
  }
  if (out) {
    *out = DevLayout{B,        n_img,        N,           T,           max_seq,        max_text,
                     max_img,  max_ips,      lay->cu_seqlens, lay->img_start, lay->img_len,
                     lay->cu_img, lay->text_pos, lay->cu_text, lay->keep_total};
  }
  return AVTP_OK;
}

int check_attn_args(int dtype, int Hq, int Hkv, int d) {
  if (dtype != AVTP_BF16 && dtype != AVTP_FP32) return AVTP_ERR_UNSUPPORTED;
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return AVTP_ERR_INVALID_ARG;
  if (d != 64 && d != 128) return AVTP_ERR_UNSUPPORTED;
  if (Hq > 256) return AVTP_ERR_UNSUPPORTED;
  return AVTP_OK;
}

// The score kernels address a sequence's keys (from its first token) and its
// text-row queries (from its first text row) with 32-bit byte offsets.
int check_attn_extent(const DevLayout &L, int dtype, int Hq, int Hkv, int d) {
  const long long row = (long long)d * (dtype == AVTP_FP32 ? 4 : 2);
  if ((long long)L.max_seqlen * Hkv * row >= AVTP_MAX_SEQ_BYTES ||
      (long long)L.max_text * Hq * row >= AVTP_MAX_SEQ_BYTES)
    return AVTP_ERR_UNSUPPORTED;
  return AVTP_OK;
}

// avtp_select_compact, avtp_budget_select_compact: bytes moved above which
// they run the selection and compaction kernels back to back
constexpr int64_t kFusedMaxBytes = 4ll << 20;
// avtp_budget_select_compact: most images per sequence for which the
// selection blocks run the budget rule themselves
constexpr int kInBlockBudgetMaxImages = 64;

int64_t n_out_of(const avtp_layout *lay) {
  int64_t n = lay->T_tot;
  for (int b = 0; b < lay->B; ++b) n += lay->h_keep_total[b];
  return n;
}

}  // namespace
}  // namespace avtp

using namespace avtp;

extern "C" {

int avtp_version(void) { return (1 << 16) | 0; }

const char *avtp_status_string(int s) {
  switch (s) {
    case AVTP_OK: return "AVTP_OK";
    case AVTP_ERR_INVALID_ARG: return "AVTP_ERR_INVALID_ARG: invalid argument or layout";
    case AVTP_ERR_UNSUPPORTED: return "AVTP_ERR_UNSUPPORTED: unsupported dtype, head_dim or size";
    case AVTP_ERR_INFEASIBLE: return "AVTP_ERR_INFEASIBLE: keep_total outside the per-image bounds";
    case AVTP_ERR_WORKSPACE: return "AVTP_ERR_WORKSPACE: workspace missing or too small";
    case AVTP_ERR_HIP: return "AVTP_ERR_HIP: a HIP launch failed";
    default: return "unknown avtp status";
  }
}

size_t avtp_score_workspace_size(const avtp_layout *layout, int mode, int dtype, int Hq, int Hkv,
                                 int d) {
  DevLayout L;
  if (check_layout(layout, &L) != AVTP_OK) return 0;
  if (mode == AVTP_SCORE_VARIATION) return variation_workspace_bytes(L);
  if (mode != AVTP_SCORE_ATTN || check_attn_args(dtype, Hq, Hkv, d) != AVTP_OK ||
      check_attn_extent(L, dtype, Hq, Hkv, d) != AVTP_OK)
    return 0;
  return attn_plan(L, Hq, Hkv, d, dtype).bytes;
}

int avtp_row_lse(avtp_stream_t stream, const avtp_layout *layout, int dtype, const void *q_text,
                 const void *k, int Hq, int Hkv, int d, float softmax_scale, float *row_lse_out,
                 void *ws, size_t ws_bytes) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  if ((rc = check_attn_args(dtype, Hq, Hkv, d)) != AVTP_OK) return rc;
  if ((rc = check_attn_extent(L, dtype, Hq, Hkv, d)) != AVTP_OK) return rc;
  // without text rows there is nothing to read or write through q_text and
  // row_lse_out (an empty buffer may have no address)
  if ((L.T_tot > 0 && (!q_text || !row_lse_out)) || !k || !(std::isfinite(softmax_scale)) ||
      softmax_scale <= 0.f)
    return AVTP_ERR_INVALID_ARG;
  if ((uintptr_t)q_text % 16 || (uintptr_t)k % 16) return AVTP_ERR_INVALID_ARG;
  AttnPlan P = attn_plan(L, Hq, Hkv, d, dtype);
  if (!ws || ws_bytes < P.bytes || (uintptr_t)ws % 256) return AVTP_ERR_WORKSPACE;
  if (L.T_tot == 0) return AVTP_OK;
  return hip_status(launch_row_lse((hipStream_t)stream, L, P, dtype, q_text, k, Hq, Hkv, d,
                                   softmax_scale, row_lse_out, nullptr, (char *)ws));
}

}  // extern "C"

namespace avtp {

int score_impl(avtp_stream_t stream, const avtp_layout *layout, int mode, int dtype,
               const void *q_text, const void *k, int Hq, int Hkv, int d, float softmax_scale,
               const float *row_lse, const void *h_cur, const void *h_prior, int hidden,
               float *scores, float *img_sum, int32_t *status, void *ws, size_t ws_bytes,
               size_t *ws_need) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  if (!scores || (L.n_img > 0 && !img_sum)) return AVTP_ERR_INVALID_ARG;
  hipStream_t st = (hipStream_t)stream;
  if (mode == AVTP_SCORE_VARIATION) {
    if (dtype != AVTP_BF16 && dtype != AVTP_FP32) return AVTP_ERR_UNSUPPORTED;
    if (!h_cur || !h_prior || hidden < 1) return AVTP_ERR_INVALID_ARG;
    if (hidden % 8 != 0) return AVTP_ERR_UNSUPPORTED;
    if ((uintptr_t)h_cur % 16 || (uintptr_t)h_prior % 16) return AVTP_ERR_INVALID_ARG;
    if (ws_need) {
      *ws_need = variation_workspace_bytes(L);
      return AVTP_OK;
    }
    if (ws_bytes < variation_workspace_bytes(L)) return AVTP_ERR_WORKSPACE;
    hipError_t e = launch_variation(st, L, dtype, h_cur, h_prior, hidden, scores);
    if (e == hipSuccess) e = launch_finalize(st, L, nullptr, 0, 0, scores, img_sum, status);
    return hip_status(e);
  }
  if (mode != AVTP_SCORE_ATTN) return AVTP_ERR_INVALID_ARG;
  if ((rc = check_attn_args(dtype, Hq, Hkv, d)) != AVTP_OK) return rc;
  if ((rc = check_attn_extent(L, dtype, Hq, Hkv, d)) != AVTP_OK) return rc;
  // without text rows no query is read (an empty buffer may have no address)
  if ((L.T_tot > 0 && !q_text) || !k || !(std::isfinite(softmax_scale)) || softmax_scale <= 0.f)
    return AVTP_ERR_INVALID_ARG;
  if ((uintptr_t)q_text % 16 || (uintptr_t)k % 16 || (row_lse && (uintptr_t)row_lse % 4))
    return AVTP_ERR_INVALID_ARG;
  AttnPlan P = attn_plan(L, Hq, Hkv, d, dtype);
  if (ws_need) {
    *ws_need = P.bytes;
    return AVTP_OK;
  }
  if (!ws || ws_bytes < P.bytes || (uintptr_t)ws % 256) return AVTP_ERR_WORKSPACE;
  char *w = (char *)ws;
  hipError_t e = hipSuccess;
  float *lse2 = (float *)(w + P.off_lse2);  // row LSE in log2 units, for pass 2
  if (L.T_tot > 0) {
    if (row_lse)
      e = launch_lse_to_log2(st, Hq * L.T_tot, row_lse, lse2);
    else
      e = launch_row_lse(st, L, P, dtype, q_text, k, Hq, Hkv, d, softmax_scale,
                         (float *)(w + P.off_lse), lse2, w);
  }
  if (e == hipSuccess && L.T_tot > 0)
    e = launch_colsum(st, L, P, dtype, q_text, k, Hq, Hkv, d, softmax_scale, lse2, w);
  if (e == hipSuccess)
    e = launch_finalize(st, L, (const float *)(w + P.off_colsum), Hq, Hkv * P.nqs, scores, img_sum,
                        status);
  return hip_status(e);
}

}  // namespace avtp

extern "C" {

int avtp_score(avtp_stream_t stream, const avtp_layout *layout, int mode, int dtype,
               const void *q_text, const void *k, int Hq, int Hkv, int d, float softmax_scale,
               const float *row_lse, const void *h_cur, const void *h_prior, int hidden,
               float *scores, float *img_sum, int32_t *status, void *ws, size_t ws_bytes) {
  return score_impl(stream, layout, mode, dtype, q_text, k, Hq, Hkv, d, softmax_scale, row_lse,
                    h_cur, h_prior, hidden, scores, img_sum, status, ws, ws_bytes, nullptr);
}

// The budget rule's arguments, and that every sequence's keep total lies
// between the sums of its images' bounds.
static int check_budget(const avtp_layout *layout, const DevLayout &L, const float *img_sum,
                        int mode, float alpha, int lo_permille, int hi_permille, int floor_abs,
                        const int32_t *budget) {
  if (mode != AVTP_BUDGET_PROPORTIONAL && mode != AVTP_BUDGET_RAW) return AVTP_ERR_INVALID_ARG;
  if (!(alpha >= 0.f && alpha <= 32.f)) return AVTP_ERR_INVALID_ARG;
  if (lo_permille < 0 || hi_permille > 1000 || lo_permille > hi_permille || floor_abs < 0)
    return AVTP_ERR_INVALID_ARG;
  if (L.n_img > 0 && (!img_sum || !budget)) return AVTP_ERR_INVALID_ARG;
  // feasibility: sum lo <= keep_total <= sum hi for every sequence
  for (int b = 0; b < L.B; ++b) {
    int64_t slo = 0, shi = 0;
    for (int i = layout->h_cu_img[b]; i < layout->h_cu_img[b + 1]; ++i) {
      const int64_t n = layout->h_img_len[i];
      const int64_t lo = std::min<int64_t>(n, std::max<int64_t>((lo_permille * n + 999) / 1000, floor_abs));
      const int64_t hi = std::max<int64_t>(lo, (hi_permille * n) / 1000);
      slo += lo;
      shi += hi;
    }
    const int64_t K = layout->h_keep_total[b];
    if (K < slo || K > shi) return AVTP_ERR_INFEASIBLE;
  }
  return AVTP_OK;
}

int avtp_budget(avtp_stream_t stream, const avtp_layout *layout, const float *img_sum, int mode,
                float alpha, int lo_permille, int hi_permille, int floor_abs, int32_t *budget,
                int32_t *status) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  rc = check_budget(layout, L, img_sum, mode, alpha, lo_permille, hi_permille, floor_abs, budget);
  if (rc != AVTP_OK) return rc;
  if (L.n_img == 0) return AVTP_OK;
  return hip_status(launch_budget((hipStream_t)stream, L, img_sum, mode, alpha, lo_permille,
                                  hi_permille, floor_abs, budget, status));
}

int avtp_select(avtp_stream_t stream, const avtp_layout *layout, const float *scores,
                const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out,
                int32_t *status) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  if (!scores || !cu_out || (L.n_img > 0 && !budget)) return AVTP_ERR_INVALID_ARG;
  const int64_t need = n_out_of(layout);
  if (keep_capacity < need || (need > 0 && !keep_idx)) return AVTP_ERR_INVALID_ARG;
  return hip_status(launch_select((hipStream_t)stream, L, scores, budget, keep_idx,
                                  keep_capacity, cu_out, status));
}

int avtp_pruned_layout(avtp_stream_t stream, const avtp_layout *layout, const int32_t *keep_idx,
                       const int32_t *cu_out, int32_t *cu_seqlens_out, int32_t *img_start_out,
                       int32_t *img_len_out, int32_t *cu_img_out, int32_t *text_pos_out,
                       int32_t *cu_text_out) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  if (!cu_out || !cu_seqlens_out || !cu_img_out || !cu_text_out) return AVTP_ERR_INVALID_ARG;
  if (L.n_img > 0 && (!img_start_out || !img_len_out)) return AVTP_ERR_INVALID_ARG;
  if (L.T_tot > 0 && !text_pos_out) return AVTP_ERR_INVALID_ARG;
  if (n_out_of(layout) > 0 && !keep_idx) return AVTP_ERR_INVALID_ARG;
  return hip_status(launch_pruned_layout((hipStream_t)stream, L, keep_idx, cu_out, cu_seqlens_out,
                                         img_start_out, img_len_out, cu_img_out, text_pos_out,
                                         cu_text_out));
}

int avtp_layer_attention(avtp_stream_t stream, const avtp_layout *layout, const float *img_sum,
                         float *A_out) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  if ((L.B > 0 && !A_out) || (L.n_img > 0 && !img_sum)) return AVTP_ERR_INVALID_ARG;
  return hip_status(launch_layer_attention((hipStream_t)stream, L, img_sum, A_out));
}

int avtp_layer_select(avtp_stream_t stream, const float *A, int L, int N, int k, int32_t *rank_sum,
                      int32_t *selected) {
  if (!A || !rank_sum || !selected) return AVTP_ERR_INVALID_ARG;
  if (L < 1 || L > AVTP_MAX_LAYERS || N < 1 || N > AVTP_MAX_SAMPLES || k < 1 || k > L)
    return AVTP_ERR_INVALID_ARG;
  return hip_status(launch_layer_select((hipStream_t)stream, A, L, N, k, rank_sum, selected));
}

// tensor descriptors of a compaction to n_out rows
static int check_tensors(const DevLayout &L, int64_t n_out, const avtp_tensor *tensors,
                         int n_tensors) {
  if (n_tensors < 0 || n_out < 0) return AVTP_ERR_INVALID_ARG;
  if (n_tensors > AVTP_MAX_TENSORS) return AVTP_ERR_UNSUPPORTED;
  if (n_tensors > 0 && !tensors) return AVTP_ERR_INVALID_ARG;
  for (int i = 0; i < n_tensors; ++i) {
    const avtp_tensor &t = tensors[i];
    // (nothing is written when no row is kept: dst may then be NULL)
    if (!t.src || (n_out > 0 && !t.dst) || t.row_bytes < 1 || t.planes < 1)
      return AVTP_ERR_INVALID_ARG;
    if (t.src_stride < t.row_bytes || t.dst_stride < t.row_bytes) return AVTP_ERR_INVALID_ARG;
    if (t.planes > 1 && (t.src_plane_stride < (int64_t)L.N_tok * t.src_stride ||
                         t.dst_plane_stride < n_out * t.dst_stride))
      return AVTP_ERR_INVALID_ARG;
  }
  return AVTP_OK;
}

int avtp_compact(avtp_stream_t stream, const avtp_layout *layout, const int32_t *keep_idx,
                 int64_t n_out, const avtp_tensor *tensors, int n_tensors) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  rc = check_tensors(L, n_out, tensors, n_tensors);
  if (rc != AVTP_OK) return rc;
  if (n_out > 0 && !keep_idx) return AVTP_ERR_INVALID_ARG;
  if (n_out > n_out_of(layout)) return AVTP_ERR_INVALID_ARG;
  if (n_out == 0 || n_tensors == 0) return AVTP_OK;
  return hip_status(launch_compact((hipStream_t)stream, L, keep_idx, n_out, tensors, n_tensors));
}

// bytes a compaction of n_out rows of these tensors reads and writes
static int64_t bytes_moved(int64_t n_out, const avtp_tensor *tensors, int n_tensors) {
  int64_t moved = 0;
  for (int i = 0; i < n_tensors; ++i) moved += 2 * n_out * tensors[i].row_bytes * tensors[i].planes;
  return moved;
}

int avtp_select_compact(avtp_stream_t stream, const avtp_layout *layout, const float *scores,
                        const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                        int32_t *cu_out, int32_t *status, const avtp_tensor *tensors,
                        int n_tensors) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  if (!scores || !cu_out || (L.n_img > 0 && !budget)) return AVTP_ERR_INVALID_ARG;
  const int64_t need = n_out_of(layout);
  if (keep_capacity < need || (need > 0 && !keep_idx)) return AVTP_ERR_INVALID_ARG;
  rc = check_tensors(L, need, tensors, n_tensors);
  if (rc != AVTP_OK) return rc;
  // One launch pays where launches and the selection's latency dominate (few
  // bytes to move).  Every block of the fused kernel runs its image's
  // selection before it copies, so the copies cannot start before the
  // selections end; with more bytes to move the two kernels back to back are
  // as fast or faster (measured with events around the calls: 0.4 MB moved
  // (128 visual tokens): one launch 12.2 us, two 12.8; 15 MB (4 images of
  // 729 tokens): 17.0 and 16.2; 240 MB (2 sequences of 8 images): 39 and
  // 34), and are used instead.
  const int64_t moved = bytes_moved(need, tensors, n_tensors);
  hipStream_t st = (hipStream_t)stream;
  if (moved > kFusedMaxBytes) {
    hipError_t e = launch_select(st, L, scores, budget, keep_idx, keep_capacity, cu_out, status);
    if (e == hipSuccess && need > 0 && n_tensors > 0)
      e = launch_compact(st, L, keep_idx, need, tensors, n_tensors);
    return hip_status(e);
  }
  return hip_status(launch_select_compact(st, L, scores, budget, keep_idx, keep_capacity, cu_out,
                                          status, need, tensors, n_tensors));
}

int avtp_budget_select_compact(avtp_stream_t stream, const avtp_layout *layout,
                               const float *img_sum, int mode, float alpha, int lo_permille,
                               int hi_permille, int floor_abs, const float *scores, int32_t *budget,
                               int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out,
                               int32_t *status, const avtp_tensor *tensors, int n_tensors) {
  DevLayout L;
  int rc = check_layout(layout, &L);
  if (rc != AVTP_OK) return rc;
  rc = check_budget(layout, L, img_sum, mode, alpha, lo_permille, hi_permille, floor_abs, budget);
  if (rc != AVTP_OK) return rc;
  if (!scores || !cu_out) return AVTP_ERR_INVALID_ARG;
  const int64_t need = n_out_of(layout);
  if (keep_capacity < need || (need > 0 && !keep_idx)) return AVTP_ERR_INVALID_ARG;
  rc = check_tensors(L, need, tensors, n_tensors);
  if (rc != AVTP_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  // Every selection block runs the budget rule for its own sequence, which
  // costs less than a launch while sequences have few images; with many, the
  // budget kernel runs once per sequence first.
  if (L.max_img_per_seq > kInBlockBudgetMaxImages) {
    hipError_t e = hipSuccess;
    if (L.n_img > 0)
      e = launch_budget(st, L, img_sum, mode, alpha, lo_permille, hi_permille, floor_abs, budget,
                        status);
    if (e != hipSuccess) return hip_status(e);
    return avtp_select_compact(stream, layout, scores, budget, keep_idx, keep_capacity, cu_out,
                               status, tensors, n_tensors);
  }
  if (bytes_moved(need, tensors, n_tensors) > kFusedMaxBytes) {
    hipError_t e = launch_budget_select(st, L, img_sum, mode, alpha, lo_permille, hi_permille,
                                        floor_abs, scores, budget, keep_idx, keep_capacity, cu_out,
                                        status);
    if (e == hipSuccess && need > 0 && n_tensors > 0)
      e = launch_compact(st, L, keep_idx, need, tensors, n_tensors);
    return hip_status(e);
  }
  return hip_status(launch_budget_select_compact(st, L, img_sum, mode, alpha, lo_permille,
                                                 hi_permille, floor_abs, scores, budget, keep_idx,
                                                 keep_capacity, cu_out, status, need, tensors,
                                                 n_tensors));
}

}  // extern "C"
