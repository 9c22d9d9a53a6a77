/*
 * avtp.h -- C ABI of libavtp.so, the MI355X (gfx950) pruning-layer operator of
 * "Multi-Image Visual Token Pruning in Large Visual Language Models" (AVTP).
 *
 * A pruning layer turns the n visual tokens of each sequence into a shorter
 * subsequence (Method, "Visual Token Pruning": E_pruned = p(E_v)).  The four
 * calls below are the four steps of that map:
 *
 *   avtp_score   importance of every visual token and its per-image sum
 *   avtp_budget  per-image keep counts from the image importances
 *   avtp_select  per-image top-k -> ascending list of kept token indices
 *   avtp_compact gather of hidden states, position ids and the layer's K/V
 *
 * Conventions shared by every call
 *   - Every data pointer is caller-owned DEVICE memory unless its name starts
 *     with h_ or the comment says "host".  The library allocates nothing.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = null stream).
 *     Argument errors are detected on the host, before anything is enqueued,
 *     and returned synchronously; nothing is launched in that case.
 *   - Return value: AVTP_OK or a negative avtp_status.  HIP launch errors map
 *     to AVTP_ERR_HIP.
 *   - Data-dependent conditions found on the device are OR-ed into the
 *     optional per-sequence status word (int32 [B], caller zero-fills it).
 *   - Outputs must not alias inputs.  No global mutable state (except the
 *     per-GPU scratch of avtp_score_noalloc, below): calls on different
 *     streams with different buffers may run concurrently.
 */
#ifndef AVTP_H
#define AVTP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *avtp_stream_t; /* a hipStream_t */

typedef enum {
  AVTP_OK = 0,
  AVTP_ERR_INVALID_ARG = -1, /* null pointer, inconsistent layout, bad size */
  AVTP_ERR_UNSUPPORTED = -2, /* head_dim, dtype, or a size beyond the limits below */
  AVTP_ERR_INFEASIBLE = -3,  /* keep_total outside [sum of lower, sum of upper bounds] */
  AVTP_ERR_WORKSPACE = -4,   /* workspace missing or smaller than *_workspace_size */
  AVTP_ERR_HIP = -5          /* a HIP launch failed */
} avtp_status;

typedef enum { AVTP_BF16 = 0, AVTP_FP32 = 1 } avtp_dtype;

typedef enum {
  AVTP_SCORE_ATTN = 0,      /* attention paid by the text rows to each visual token */
  AVTP_SCORE_VARIATION = 1  /* 1 - cos(h^l, h^prior), the hidden-state variation  */
} avtp_score_mode;

typedef enum {
  AVTP_BUDGET_PROPORTIONAL = 0, /* keep ratio scaled by importance / mean importance */
  AVTP_BUDGET_RAW = 1           /* keep ratio shifted by alpha (importance - mean)   */
} avtp_budget_mode;

/* per-sequence device status bits */
#define AVTP_FLAG_NAN_SCORE 1       /* a visual score was NaN (ranked last)           */
#define AVTP_FLAG_NO_TEXT_AFTER 2   /* an image has no text row after it (scores = 0) */
#define AVTP_FLAG_INFEASIBLE 4      /* budget bounds cannot meet keep_total           */
#define AVTP_FLAG_OUT_CAPACITY 8    /* kept list longer than keep_capacity (truncated) */

/* Limits checked on the host (AVTP_ERR_UNSUPPORTED beyond them). */
#define AVTP_MAX_IMAGES_PER_SEQ 256
#define AVTP_MAX_IMAGES 8192
#define AVTP_MAX_IMAGE_LEN (1 << 20)
#define AVTP_MAX_TENSORS 8
#define AVTP_MAX_LAYERS 1024       /* avtp_layer_select: layers               */
#define AVTP_MAX_SAMPLES (1 << 20) /* avtp_layer_select: samples              */
/* The attention score (avtp_score in attention mode, avtp_row_lse) addresses
 * one sequence's keys and text-row queries with 32-bit byte offsets: every
 * sequence must have (its tokens) * Hkv * d * elem and (its text rows) *
 * Hq * d * elem below AVTP_MAX_SEQ_BYTES (elem: 2 for bf16, 4 for fp32). */
#define AVTP_MAX_SEQ_BYTES (1ll << 32)

/*
 * Packed ("THD") description of one batch of B sequences, N_tok tokens.
 * Sequence b owns tokens [cu_seqlens[b], cu_seqlens[b+1]).  Every token is
 * either a text token or belongs to exactly one image:
 *   image i: tokens [img_start[i], img_start[i] + img_len[i]) (global
 *            indices); the images of sequence b are cu_img[b] .. cu_img[b+1]-1,
 *            in ascending position order;
 *   text t:  token text_pos[t]; the text rows of sequence b are
 *            cu_text[b] .. cu_text[b+1]-1, in ascending position order.
 * keep_total[b] is the number of visual tokens sequence b keeps.
 * Each int32 array is given twice: as device memory (read by the kernels)
 * and as a host mirror with identical contents (read by the host-side
 * validation and launch sizing; never dereferenced on the device).  Arrays
 * of length 0 may be NULL (img_start, img_len when n_img = 0; text_pos when
 * T_tot = 0).
 */
typedef struct {
  int32_t B, n_img, N_tok, T_tot;
  const int32_t *cu_seqlens, *img_start, *img_len, *cu_img, *text_pos, *cu_text, *keep_total;
  const int32_t *h_cu_seqlens, *h_img_start, *h_img_len, *h_cu_img, *h_text_pos, *h_cu_text,
      *h_keep_total;
} avtp_layout;

/*
 * One tensor to compact.  For every plane p < planes and output row r:
 *   dst + p*dst_plane_stride + r*dst_stride  <-  row_bytes bytes from
 *   src + p*src_plane_stride + keep_idx[r]*src_stride
 * (token-major [N_tok, ...] tensors use planes = 1; position ids [P, N_tok]
 * use planes = P; head-major K/V [Hkv, N_tok, d] use planes = Hkv).
 * All strides and offsets in bytes.  dst may be NULL when no row is kept.
 */
typedef struct {
  const void *src;
  void *dst;
  int64_t row_bytes, src_stride, dst_stride;
  int32_t planes;
  int64_t src_plane_stride, dst_plane_stride;
} avtp_tensor;

/* ------------------------------------------------------------------------
 * avtp_score -- importance of every visual token.
 *
 * AVTP_SCORE_ATTN (the attention a layer pays to visual tokens, the quantity
 * summed in Sec. 3.3.2, here kept per token).  With c = softmax_scale, query
 * head h using key head g = h / (Hq/Hkv) (grouped-query attention), text row t
 * at position p_t and the causal row normaliser
 *   lse[h,t] = log sum_{j <= p_t, j in seq} exp(c q_{t,h}.k_{j,g}),
 * the score of visual token j is
 *   s_j = 1/Hq sum_h 1/|T_j| sum_{t in T_j} exp(c q_{t,h}.k_{j,g} - lse[h,t])
 * where T_j are the text rows after j.  Computed in two tiled passes over
 * the keys (row statistics, then column sums) with bf16 MFMA and fp32
 * accumulation; the attention matrix is never stored.  If row_lse is given
 * (e.g. the softmax LSE of the layer's own fused attention, natural log,
 * [Hq, T_tot] fp32) the first pass is skipped.
 *   q_text [T_tot, Hq, d]  queries of the text rows (dtype; may be NULL when
 *                          T_tot = 0: every image then has no text row after it)
 *   k      [N_tok, Hkv, d] the layer's keys (dtype)
 *   d in {64, 128}, Hq % Hkv == 0.
 *
 * AVTP_SCORE_VARIATION (Sec. 3.3.1, importance = 1 - Sim(h^l, h^prior),
 * Sim = cosine similarity with a 1e-8 norm guard):
 *   h_cur, h_prior [N_tok, hidden] (dtype); q_text, k, row_lse unused.
 *
 * Outputs: scores [N_tok] fp32 (+inf at text positions), img_sum [n_img]
 * fp32 = sum of the image's scores (Sec. 3.3.3 mean importance times |V_i|).
 * An image with no text row after it scores 0 and flags
 * AVTP_FLAG_NO_TEXT_AFTER.  Deterministic: bit-identical key rows in one
 * image give bit-identical scores, and reruns are bit-identical.
 * ws: device scratch of at least avtp_score_workspace_size() bytes (0 for an
 * invalid layout or arguments); its contents need no initialisation.
 * ---------------------------------------------------------------------- */
size_t avtp_score_workspace_size(const avtp_layout *layout, int mode, int dtype, int Hq, int Hkv,
                                 int d);
int avtp_score(avtp_stream_t stream, const avtp_layout *layout, int mode, int dtype,
               const void *q_text, const void *k, int Hq, int Hkv, int d, float softmax_scale,
               const float *row_lse, const void *h_cur, const void *h_prior, int hidden,
               float *scores, float *img_sum, int32_t *status, void *ws, size_t ws_bytes);

/* The first pass of AVTP_SCORE_ATTN alone: row_lse_out [Hq, T_tot] fp32,
 * natural-log LSE of each text row's causal attention logits (definition
 * above).  Same arguments and workspace as avtp_score; q_text and
 * row_lse_out may be NULL when T_tot = 0 (nothing is launched). */
int avtp_row_lse(avtp_stream_t stream, const avtp_layout *layout, int dtype, const void *q_text,
                 const void *k, int Hq, int Hkv, int d, float softmax_scale, float *row_lse_out,
                 void *ws, size_t ws_bytes);

/* ------------------------------------------------------------------------
 * avtp_budget -- per-image keep counts (Sec. 3.3.3 ratio rule, clamp of the
 * appendix on alpha).  For sequence b with images of n_i tokens and sums S_i,
 * M = sum n_i, S = sum S_i, K = keep_total[b]:
 *   PROPORTIONAL: quota share w_i = (1-alpha) n_i/M + alpha S_i/S
 *   RAW:          w_i = n_i/M + alpha (S_i - n_i S/M) / K
 * (each the ratio r_i = r_base + alpha (Ibar_i - Ibar_avg) of the paper with
 * r_base = K/M; PROPORTIONAL measures importance in units of its mean).
 * w_i < 0 -> 0; only the ratios of the shares matter, so with w_max the
 * largest share of the sequence W_i = max(1, rint((w_i / w_max) * 2^28))
 * (float64, one operation at a time, no FMA contraction); if S is not
 * positive and finite, w_i = n_i/M.  Bounds
 *   lo_i = min(n_i, max(ceil(lo_permille n_i / 1000), floor_abs)),
 *   hi_i = max(lo_i, floor(hi_permille n_i / 1000))
 * (paper: 5 % and 95 %, i.e. 50 and 950).  Exact integer water-filling finds
 * q_i = clamp(lam W_i, lo_i, hi_i) with sum q_i = K; largest-remainder
 * rounding (ties to the lowest image index) gives budget[i], sum = K.
 * alpha in [0, 32].  AVTP_ERR_INFEASIBLE (host check) if K is outside
 * [sum lo_i, sum hi_i].  budget: [n_img] int32 output.
 * ---------------------------------------------------------------------- */
int avtp_budget(avtp_stream_t stream, const avtp_layout *layout, const float *img_sum, int mode,
                float alpha, int lo_permille, int hi_permille, int floor_abs, int32_t *budget,
                int32_t *status);

/* ------------------------------------------------------------------------
 * avtp_select -- the pruned subsequence (Method, "Visual Token Pruning": the
 * pruning map keeps a subset of the visual tokens and every text token),
 * with the per-image keep counts of Sec. 3.3.3 (an image keeps budget[i]
 * tokens, so more important images keep more).  Inside every image the
 * budget[i] highest-scoring tokens are kept (score descending; an exact tie
 * keeps the lowest token index; -0.0 equals +0.0; NaN ranks last), plus
 * every text token.  Writes the kept global token indices of each sequence
 * in ascending order to keep_idx[cu_out[b] .. cu_out[b+1]), and cu_out [B+1].
 *   scores [N_tok] fp32 (device; text positions are not read), budget
 *   [n_img] int32 (device), keep_idx [keep_capacity] int32 and cu_out [B+1]
 *   int32 (device outputs).
 * keep_capacity: entries available in keep_idx; must be at least
 * T_tot + sum(keep_total) (checked on the host); writes past it are dropped
 * and flag AVTP_FLAG_OUT_CAPACITY (budgets not summing to keep_total).
 * No workspace: the selection of an image runs inside one block, from its
 * keys cached in LDS (or re-read from scores for images above 4096 tokens),
 * and each block knows its output offset from the budgets; so there is no
 * avtp_select_workspace_size.
 * ---------------------------------------------------------------------- */
int avtp_select(avtp_stream_t stream, const avtp_layout *layout, const float *scores,
                const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out,
                int32_t *status);

/* ------------------------------------------------------------------------
 * avtp_compact -- the pruned sequence that the following layers run on
 * (Method, "Visual Token Pruning": E_pruned replaces E_v; Sec. 3.3.3: the
 * kept tokens of each image): stable gather out[r] = in[keep_idx[r]] for up
 * to AVTP_MAX_TENSORS tensors in one launch (hidden states, position ids with
 * their original values, K and V of the layer).  n_out = number of entries
 * of keep_idx to apply (normally T_tot + sum(keep_total)); every keep_idx
 * entry should lie in [0, N_tok): an entry outside it reads nothing and
 * leaves its output row as it was.  tensors: HOST array of n_tensors
 * descriptors.  Copies are bit-exact.
 * ---------------------------------------------------------------------- */
int avtp_compact(avtp_stream_t stream, const avtp_layout *layout, const int32_t *keep_idx,
                 int64_t n_out, const avtp_tensor *tensors, int n_tensors);

/* ------------------------------------------------------------------------
 * avtp_pruned_layout -- the layout of the kept tokens, for the next pruning
 * layer of a progressive schedule (Sec. 3.3.2: pruning at several selected
 * layers; Sec. 3.3.1: the next layer's h^prior is the hidden state after this
 * pruning, i.e. this layer's compacted hidden rows).  Pruning keeps a
 * subsequence of every sequence (Method, "Visual Token Pruning"): kept token
 * r of the batch (keep_idx[r], from avtp_select, ascending per sequence)
 * becomes token r of the next layer.  Writes, as device int32 arrays of the
 * next layer's avtp_layout:
 *   cu_seqlens_out [B+1] = cu_out;
 *   img_start_out, img_len_out [n_img]: image i's first new index and its
 *     number of kept tokens (an image that keeps none has length 0 and sits
 *     where its tokens were);
 *   text_pos_out [T_tot]: the new index of every text token (all are kept);
 *   cu_img_out, cu_text_out [B+1]: unchanged copies.
 * The next layer's keep totals (the schedule) are the caller's.  Host
 * mirrors of the next layout are the caller's copies of these arrays.
 * ---------------------------------------------------------------------- */
int avtp_pruned_layout(avtp_stream_t stream, const avtp_layout *layout, const int32_t *keep_idx,
                       const int32_t *cu_out, int32_t *cu_seqlens_out, int32_t *img_start_out,
                       int32_t *img_len_out, int32_t *cu_img_out, int32_t *text_pos_out,
                       int32_t *cu_text_out);

/* ------------------------------------------------------------------------
 * Architecture-aware pruning-layer selection (Sec. 3.3.2), computed from
 * calibration prefills.  For sample i and layer l the paper sums the
 * attention the layer pays to every visual token,
 *   A_l^(i) = sum_j Attention(l, v_j^(i)),
 * ranks the layers within each sample, averages the ranks over the N samples,
 *   R_l = 1/N sum_i Rank(A_l^(i)),
 * and prunes at the k layers of highest average attention.
 *
 * avtp_layer_attention -- A of one layer for every sequence of a batch (each
 * sequence is one sample): A_out[b] = sum of img_sum over the images of
 * sequence b (img_sum from avtp_score in AVTP_SCORE_ATTN mode, whose
 * per-token score stands for Attention(l, v_j)), accumulated in float64 in
 * image order and rounded once to fp32; 0 for a sequence without images.
 *   img_sum [n_img] fp32 (device), A_out [B] fp32 (device; typically row l
 *   of the caller's [L][N] table, at the batch's sample offset).
 *
 * avtp_layer_select -- ranks and selection from the whole table.
 *   A [L][N] fp32 (device, row-major: layer l, sample i at A[l*N + i]);
 *   1 <= L <= AVTP_MAX_LAYERS, 1 <= N <= AVTP_MAX_SAMPLES, 1 <= k <= L.
 *   Within each sample, rank 1 is the largest A; equal values rank the lower
 *   layer index first (each sample's ranks are a permutation of 1..L); NaN
 *   ranks as the smallest value; -0.0 equals +0.0.
 *   rank_sum [L] int32 (device, output): sum_i Rank(A_l^(i)) = N * R_l exactly.
 *   selected [k] int32 (device, output): the k layers with the smallest rank
 *   sums (equal sums: lower layer index first), in ascending layer order.
 * Both calls: AVTP_ERR_INVALID_ARG for null pointers or sizes out of range.
 * ---------------------------------------------------------------------- */
int avtp_layer_attention(avtp_stream_t stream, const avtp_layout *layout, const float *img_sum,
                         float *A_out);
int avtp_layer_select(avtp_stream_t stream, const float *A, int L, int N, int k,
                      int32_t *rank_sum, int32_t *selected);

/* ------------------------------------------------------------------------
 * avtp_select_compact -- avtp_select followed by avtp_compact of the same
 * tensors to n_out = T_tot + sum(keep_total) rows (the pruned subsequence of
 * Method, "Visual Token Pruning", gathered in one call).  Same arguments and
 * outputs as the two calls; the kept rows and keep_idx are bit-identical to
 * theirs.  When the compaction moves at most 4 MiB (reads plus writes) it is
 * one launch, for the small configurations where launches and the
 * selection's latency dominate: every image is handled by several blocks
 * that each redo its selection and copy an interleaved share of its output
 * rows, so no block waits for another.  Above that the two kernels run back
 * to back (one block's copies cannot start before its selection ends, so the
 * one-launch form is slower there).
 * ---------------------------------------------------------------------- */
int avtp_select_compact(avtp_stream_t stream, const avtp_layout *layout, const float *scores,
                        const int32_t *budget, int32_t *keep_idx, int64_t keep_capacity,
                        int32_t *cu_out, int32_t *status, const avtp_tensor *tensors,
                        int n_tensors);

/* ------------------------------------------------------------------------
 * avtp_budget_select_compact -- avtp_budget, then avtp_select_compact: the
 * per-image budgets of Sec. 3.3.3 (adaptive keep ratio, appendix clamp on
 * alpha), the top-budget selection of every image and the gather of the
 * pruned subsequence (Method, "Visual Token Pruning"), in one call.
 * Arguments: those of avtp_budget (img_sum, mode, alpha, lo/hi permille,
 * floor_abs; budget[n_img] is written) followed by those of
 * avtp_select_compact.  Every output (budget, keep_idx, cu_out, the compacted
 * tensors, status flags) is bit-identical to the separate calls'.  Errors: as
 * the separate calls, all checked on the host before any launch, including
 * AVTP_ERR_INFEASIBLE.  While no sequence has more than 64 images, the
 * selection blocks each run the budget rule for their own sequence (the
 * same integer arithmetic as the budget kernel), so no budget launch is
 * needed: one launch in all when the compaction moves at most 4 MiB, else
 * the selection and the compaction kernels.  With more images per sequence
 * the budget kernel runs first.
 * ---------------------------------------------------------------------- */
int avtp_budget_select_compact(avtp_stream_t stream, const avtp_layout *layout,
                               const float *img_sum, int mode, float alpha, int lo_permille,
                               int hi_permille, int floor_abs, const float *scores, int32_t *budget,
                               int32_t *keep_idx, int64_t keep_capacity, int32_t *cu_out,
                               int32_t *status, const avtp_tensor *tensors, int n_tensors);

/* ------------------------------------------------------------------------
 * avtp_score_noalloc -- avtp_score for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, outputs and results as avtp_score
 * (bit-identical: the same kernels run), but no workspace argument: the
 * scratch space lives in a device array of AVTP_NOALLOC_MAX_WORKSPACE bytes
 * inside the library, one per GPU, held until the process ends.  Its address
 * on a device is looked up on the first call with that device current (a
 * hipGetSymbolAddress, which allocates nothing); the stream must belong to the
 * calling thread's current device.  Nothing is allocated, on any call.
 * Returns AVTP_ERR_WORKSPACE when the layout needs more scratch than that
 * (avtp_score_workspace_size tells how much); every other argument error as
 * avtp_score, before any HIP call.  All calls on one GPU share its array:
 * calls that overlap on one GPU (other streams or threads) race; calls in
 * stream order do not.  No scratch contents need clearing between calls.
 * ---------------------------------------------------------------------- */
#define AVTP_NOALLOC_MAX_WORKSPACE (16 << 20) /* bytes of the library's scratch per GPU */
int avtp_score_noalloc(avtp_stream_t stream, const avtp_layout *layout, int mode, int dtype,
                       const void *q_text, const void *k, int Hq, int Hkv, int d,
                       float softmax_scale, const float *row_lse, const void *h_cur,
                       const void *h_prior, int hidden, float *scores, float *img_sum,
                       int32_t *status);

/* Human-readable name of an avtp_status value (static string). */
const char *avtp_status_string(int status);

/* ABI version: (major << 16) | minor. */
int avtp_version(void);

#ifdef __cplusplus
}
#endif
#endif /* AVTP_H */
