// Hidden-state-variation score (Sec. 3.3.1 of the paper): for visual token j
//   I_j = 1 - <h_j, h'_j> / max(|h_j| |h'_j|, 1e-8)
// with h the hidden state at the pruning layer and h' the state saved after
// the previous pruning (the input embeddings before the first one).
// HBM-bound: one wave streams the rows of two tokens at a time with 16-byte
// non-temporal loads and reduces each token's three fp32 sums over its lanes
// in a fixed order.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "avtp_internal.h"
#include "stream_load.h"
#include "wave_ops.h"

namespace avtp {
namespace {

constexpr int kTokPerWave = 4;
constexpr int kTokPerBlock = 4 * kTokPerWave;
static_assert(kTokPerWave % 2 == 0, "a wave takes its tokens two at a time");

__device__ inline void acc8(const uint4 &x, const uint4 &y, float &dot, float &nx, float &ny,
                            __bf16 *) {
  const uint32_t xs[4] = {x.x, x.y, x.z, x.w}, ys[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float x0 = __uint_as_float(xs[w] << 16), x1 = __uint_as_float(xs[w] & 0xffff0000u);
    const float y0 = __uint_as_float(ys[w] << 16), y1 = __uint_as_float(ys[w] & 0xffff0000u);
    dot += x0 * y0;
    dot += x1 * y1;
    nx += x0 * x0;
    nx += x1 * x1;
    ny += y0 * y0;
    ny += y1 * y1;
  }
}
__device__ inline void acc8(const uint4 &x, const uint4 &y, float &dot, float &nx, float &ny,
                            float *) {
  const float xs[4] = {__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z),
                       __uint_as_float(x.w)};
  const float ys[4] = {__uint_as_float(y.x), __uint_as_float(y.y), __uint_as_float(y.z),
                       __uint_as_float(y.w)};
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    dot += xs[w] * ys[w];
    nx += xs[w] * xs[w];
    ny += ys[w] * ys[w];
  }
}

// Every row is read once, and the two tensors are far larger than the
// caches: the loads are non-temporal (ld_stream) so that they do not
// displace cached data (measured 368 -> 334 us at 4 x 32,768 visual tokens of
// 4,096 bf16 values).

// three fp32 sums, as a value of wave::allreduce
struct Sums3 {
  float a, b, c;
  template <int CTRL>
  __device__ static Sums3 shift(const Sums3 &v) {
    return Sums3{__uint_as_float(wave::dpp<CTRL>(__float_as_uint(v.a))),
                 __uint_as_float(wave::dpp<CTRL>(__float_as_uint(v.b))),
                 __uint_as_float(wave::dpp<CTRL>(__float_as_uint(v.c)))};
  }
  __device__ static Sums3 at(const Sums3 &v, int lane) {
    return Sums3{__uint_as_float(wave::lane_value(__float_as_uint(v.a), lane)),
                 __uint_as_float(wave::lane_value(__float_as_uint(v.b), lane)),
                 __uint_as_float(wave::lane_value(__float_as_uint(v.c), lane))};
  }
};

template <typename T>
__global__ __launch_bounds__(256) void variation_kernel(const char *__restrict__ hc,
                                                        const char *__restrict__ hp, int hidden,
                                                        const int32_t *__restrict__ img_start,
                                                        const int32_t *__restrict__ img_len,
                                                        float *__restrict__ scores) {
  const int i = blockIdx.y;
  const int n = img_len[i];
  const int base = blockIdx.x * kTokPerBlock;
  if (base >= n) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t row_bytes = (size_t)hidden * sizeof(T);
  const int nvec = (int)(row_bytes / 16);
  // the three sums over the wave in a fixed order (DPP lane network), then
  // the score of the token at `row`
  auto finish = [&](float dot, float nx, float ny, size_t row) __attribute__((always_inline)) {
    const Sums3 r = wave::allreduce(Sums3{dot, nx, ny}, [](const Sums3 &x, const Sums3 &y) {
      return Sums3{x.a + y.a, x.b + y.b, x.c + y.c};
    });
    if (lane == 0) scores[row] = 1.f - r.a / fmaxf(sqrtf(r.b) * sqrtf(r.c), 1e-8f);
  };
  // two tokens per iteration, their loads in flight together; each token's
  // sums run over its row in the same order as for one token at a time (a
  // missing second token re-reads the first, and its sums are dropped)
  for (int tt = 0; tt < kTokPerWave; tt += 2) {
    const int tok = base + wave * kTokPerWave + tt;
    if (tok >= n) break;
    const bool two = tok + 1 < n;
    const size_t row = (size_t)img_start[i] + tok, row1 = two ? row + 1 : row;
    const uint4 *a = reinterpret_cast<const uint4 *>(hc + row * row_bytes);
    const uint4 *b = reinterpret_cast<const uint4 *>(hp + row * row_bytes);
    const uint4 *a1 = reinterpret_cast<const uint4 *>(hc + row1 * row_bytes);
    const uint4 *b1 = reinterpret_cast<const uint4 *>(hp + row1 * row_bytes);
    float dot = 0.f, nx = 0.f, ny = 0.f, dot1 = 0.f, nx1 = 0.f, ny1 = 0.f;
    for (int v = lane; v < nvec; v += 64) {
      const uint4 x0 = ld_stream(a + v), y0 = ld_stream(b + v);
      const uint4 x1 = ld_stream(a1 + v), y1 = ld_stream(b1 + v);
      acc8(x0, y0, dot, nx, ny, (T *)nullptr);
      acc8(x1, y1, dot1, nx1, ny1, (T *)nullptr);
    }
    finish(dot, nx, ny, row);
    if (two) finish(dot1, nx1, ny1, row1);
  }
}

}  // namespace

size_t variation_workspace_bytes(const DevLayout &) { return 0; }

hipError_t launch_variation(hipStream_t st, const DevLayout &L, int dtype, const void *h_cur,
                            const void *h_prior, int hidden, float *scores) {
  clear_pending_error();
  if (L.n_img == 0 || L.max_img_len == 0) return hipSuccess;
  const dim3 grid((L.max_img_len + kTokPerBlock - 1) / kTokPerBlock, L.n_img);
  if (dtype == AVTP_BF16)
    hipLaunchKernelGGL(variation_kernel<__bf16>, grid, dim3(256), 0, st, (const char *)h_cur,
                       (const char *)h_prior, hidden, L.img_start, L.img_len, scores);
  else
    hipLaunchKernelGGL(variation_kernel<float>, grid, dim3(256), 0, st, (const char *)h_cur,
                       (const char *)h_prior, hidden, L.img_start, L.img_len, scores);
  return hipGetLastError();
}

}  // namespace avtp
