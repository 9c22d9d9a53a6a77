// Per-image keep budgets (Sec. 3.3.3 adaptive keep ratio, with the 5 % / 95 %
// clamp of the appendix on alpha).  One block per sequence, one thread per
// image.
//
// The rule itself is in budget_rule.h (shared with the selection kernels
// that compute their sequence's budgets in-block).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"
#include "budget_rule.h"

namespace avtp {
namespace {

template <int NTH>
__global__ __launch_bounds__(NTH) void budget_kernel(const float *__restrict__ img_sum,
                                                     const int32_t *__restrict__ img_len,
                                                     const int32_t *__restrict__ cu_img,
                                                     const int32_t *__restrict__ keep_total,
                                                     int mode, float alpha, int lo_pm, int hi_pm,
                                                     int floor_abs, int32_t *__restrict__ budget,
                                                     int32_t *__restrict__ status) {
  const int b = blockIdx.x;
  int32_t *out = budget + cu_img[b];
  budget_rule::seq_budget<NTH>(b, img_sum, img_len, cu_img, keep_total, mode, alpha, lo_pm, hi_pm,
                               floor_abs, status,
                               [&](int t, int32_t v) __attribute__((always_inline)) { out[t] = v; });
}

}  // namespace

hipError_t launch_budget(hipStream_t st, const DevLayout &L, const float *img_sum, int mode,
                         float alpha, int lo_permille, int hi_permille, int floor_abs,
                         int32_t *budget, int32_t *status) {
  clear_pending_error();
  if (L.max_img_per_seq <= 16)
    hipLaunchKernelGGL(budget_kernel<64>, dim3(L.B), dim3(64), 0, st, img_sum, L.img_len, L.cu_img,
                       L.keep_total, mode, alpha, lo_permille, hi_permille, floor_abs, budget,
                       status);
  else
    hipLaunchKernelGGL(budget_kernel<budget_rule::kThreads>, dim3(L.B),
                       dim3(budget_rule::kThreads), 0, st, img_sum, L.img_len, L.cu_img,
                       L.keep_total, mode, alpha, lo_permille, hi_permille, floor_abs, budget,
                       status);
  return hipGetLastError();
}

}  // namespace avtp
