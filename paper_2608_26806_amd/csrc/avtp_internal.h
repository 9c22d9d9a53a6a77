// Internal interface between the host layer (avtp_api.cpp) and the HIP
// kernels.  Every launcher enqueues on `stream` and returns the hipError_t of
// its launches; all arguments were validated by the host layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/avtp.h"

namespace avtp {

// hipGetLastError() reports the last failed HIP call of the calling thread,
// including calls the library's caller made before entering it.  Every
// launch function reads it (which clears it) before its first launch, so
// that the read after a launch reports that launch alone; an error of the
// device itself (a broken context) still fails the launch and is reported.
inline void clear_pending_error() { (void)hipGetLastError(); }

// Device view of a validated layout (device pointers plus host-derived maxima).
struct DevLayout {
  int B, n_img, N_tok, T_tot;
  int max_seqlen, max_text, max_img_len;
  int max_img_per_seq;
  const int32_t *cu_seqlens, *img_start, *img_len, *cu_img, *text_pos, *cu_text, *keep_total;
};

// Launch geometry of the two attention passes, derived from the layout only
// (so the workspace size and the launches always agree).
struct AttnPlan {
  int G;          // query heads per key head
  int rows_max;   // max over sequences of G * T_b
  int nqb;        // query blocks per (sequence, key head) in pass 1
  int nt1;        // 32-row query tiles per wave in pass 1
  int kchunk;     // keys per pass-1 chunk (multiple of 64)
  int nkc;        // chunks per sequence (max)
  int nkb;        // key blocks per (sequence, key head) in pass 2
  int nkt2;       // 32-key tiles per wave in pass 2
  int nqs;        // query splits of pass 2 (column-sum planes per key head)
  int nsl;        // pass 2: each (sequence, key head)'s key blocks are dealt to nsl
                  // slices (kb mod nsl), so that there are units for all 8 XCDs
  size_t off_part_m, off_part_l, off_lse, off_lse2, off_colsum, bytes;
};

AttnPlan attn_plan(const DevLayout &L, int Hq, int Hkv, int d, int dtype);

// avtp_score with its workspace argument.  With ws_need set, only validates
// the arguments (returning their error, if any) and stores the workspace the
// call needs; nothing is launched and ws is not read.
int score_impl(avtp_stream_t stream, const avtp_layout *layout, int mode, int dtype,
               const void *q_text, const void *k, int Hq, int Hkv, int d, float softmax_scale,
               const float *row_lse, const void *h_cur, const void *h_prior, int hidden,
               float *scores, float *img_sum, int32_t *status, void *ws, size_t ws_bytes,
               size_t *ws_need);
size_t variation_workspace_bytes(const DevLayout &L);

// Pass 1 and the combine: the row LSE (natural log) into row_lse and, if
// lse2 is not null, in log2 units into lse2.
hipError_t launch_row_lse(hipStream_t stream, const DevLayout &L, const AttnPlan &P, int dtype,
                          const void *q, const void *k, int Hq, int Hkv, int d, float scale,
                          float *row_lse, float *lse2, char *ws);
// lse2 = lse * log2(e) for `rows` rows (an LSE the caller supplies)
hipError_t launch_lse_to_log2(hipStream_t stream, int rows, const float *lse, float *lse2);
// Pass 2: column sums from the row LSE in log2 units.
hipError_t launch_colsum(hipStream_t stream, const DevLayout &L, const AttnPlan &P, int dtype,
                         const void *q, const void *k, int Hq, int Hkv, int d, float scale,
                         const float *lse2, char *ws);
// Per-image finalisation shared by both score modes.  colsum == nullptr:
// scores already hold the per-token values (variation mode); otherwise the
// score of token j is the sum of `planes` column-sum planes at j over
// (Hq * rows after j).
hipError_t launch_finalize(hipStream_t stream, const DevLayout &L, const float *colsum, int Hq,
                           int planes, float *scores, float *img_sum, int32_t *status);
hipError_t launch_variation(hipStream_t stream, const DevLayout &L, int dtype, const void *h_cur,
                            const void *h_prior, int hidden, float *scores);
hipError_t launch_budget(hipStream_t stream, const DevLayout &L, const float *img_sum, int mode,
                         float alpha, int lo_permille, int hi_permille, int floor_abs,
                         int32_t *budget, int32_t *status);
hipError_t launch_select(hipStream_t stream, const DevLayout &L, const float *scores,
                         const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                         int32_t *cu_out, int32_t *status);
hipError_t launch_compact(hipStream_t stream, const DevLayout &L, const int32_t *keep_idx,
                          int64_t n_out, const avtp_tensor *tensors, int n_tensors);
// avtp_select and avtp_compact (to the n_out of the layout) in one launch.
hipError_t launch_select_compact(hipStream_t stream, const DevLayout &L, const float *scores,
                                 const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                                 int32_t *cu_out, int32_t *status, int64_t n_out,
                                 const avtp_tensor *tensors, int n_tensors);
// The budget rule run inside the selection blocks (each block for its
// image's sequence), then the selection (and the compaction); budget[] is
// written too.  Needs keep totals the per-image bounds can meet.
hipError_t launch_budget_select(hipStream_t stream, const DevLayout &L, const float *img_sum,
                                int mode, float alpha, int lo_permille, int hi_permille,
                                int floor_abs, const float *scores, int32_t *budget,
                                int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out,
                                int32_t *status);
hipError_t launch_budget_select_compact(hipStream_t stream, const DevLayout &L,
                                        const float *img_sum, int mode, float alpha,
                                        int lo_permille, int hi_permille, int floor_abs,
                                        const float *scores, int32_t *budget, int32_t *keep_idx,
                                        int64_t keep_capacity, int32_t *cu_out, int32_t *status,
                                        int64_t n_out, const avtp_tensor *tensors, int n_tensors);

// Layout of the kept tokens for the next pruning layer.
hipError_t launch_pruned_layout(hipStream_t stream, const DevLayout &L, const int32_t *keep_idx,
                                const int32_t *cu_out, int32_t *cu_seqlens_out,
                                int32_t *img_start_out, int32_t *img_len_out, int32_t *cu_img_out,
                                int32_t *text_pos_out, int32_t *cu_text_out);

// Pruning-layer selection (Sec. 3.3.2): per-sample attention of one layer,
// and the per-sample ranks, their sums and the top-k layers.
hipError_t launch_layer_attention(hipStream_t stream, const DevLayout &L, const float *img_sum,
                                  float *A);
hipError_t launch_layer_select(hipStream_t stream, const float *A, int L, int N, int k,
                               int32_t *rank_sum, int32_t *selected);

}  // namespace avtp
