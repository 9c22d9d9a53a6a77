// avtp_score_noalloc: avtp_score for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc).  The score passes' scratch (pass-1 partials, the row LSE
// in both units, the pass-2 column-sum planes) lives in one file-scope device
// array of AVTP_NOALLOC_MAX_WORKSPACE bytes instead of a caller workspace.
//
// Each GPU holds its own copy of the array at its own address.  The address
// is looked up once per device, on the first call with that device current,
// with hipGetSymbolAddress; host code never passes the array's name itself to
// a kernel (on the host that name is only a stand-in, not a device address).
// Nothing here allocates: no hipMalloc, hipFree or allocating library call.
// The passes write every scratch entry they read before reading it, so the
// contents left by an earlier call need no clearing.  Calls that overlap on
// one GPU (other streams, other threads) share the array and race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "avtp_internal.h"

namespace {

static __device__ __align__(256) char scratch[AVTP_NOALLOC_MAX_WORKSPACE];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of `scratch` on each device (null: not yet looked up)

// The scratch array's address on the current device (looked up on the first
// call there).  Returns AVTP_OK and sets *out, or AVTP_ERR_HIP.
int scratch_ptr(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return AVTP_ERR_HIP;
  if (dev >= kMaxDevices) return AVTP_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return AVTP_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return AVTP_OK;
}

}  // namespace

extern "C" int avtp_score_noalloc(avtp_stream_t stream, const avtp_layout *layout, int mode,
                                  int dtype, const void *q_text, const void *k, int Hq, int Hkv,
                                  int d, float softmax_scale, const float *row_lse,
                                  const void *h_cur, const void *h_prior, int hidden,
                                  float *scores, float *img_sum, int32_t *status) {
  // every argument error first, on the host, before any HIP call
  size_t need = 0;
  int rc = avtp::score_impl(stream, layout, mode, dtype, q_text, k, Hq, Hkv, d, softmax_scale,
                            row_lse, h_cur, h_prior, hidden, scores, img_sum, status, nullptr, 0,
                            &need);
  if (rc != AVTP_OK) return rc;
  if (need > (size_t)AVTP_NOALLOC_MAX_WORKSPACE) return AVTP_ERR_WORKSPACE;
  void *ws = nullptr;
  if ((rc = scratch_ptr(&ws)) != AVTP_OK) return rc;
  return avtp::score_impl(stream, layout, mode, dtype, q_text, k, Hq, Hkv, d, softmax_scale,
                          row_lse, h_cur, h_prior, hidden, scores, img_sum, status, ws,
                          (size_t)AVTP_NOALLOC_MAX_WORKSPACE, nullptr);
}
