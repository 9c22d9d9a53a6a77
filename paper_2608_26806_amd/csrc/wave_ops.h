// Wave-wide all-reductions on the DPP lane network (CDNA, wave64).
//
// A butterfly written with __shfl_xor goes through the LDS crossbar
// (ds_bpermute) at every step; here the lanes of a quad are combined with
// quad permutes, the four quads of each 16-lane row with two row rotates,
// and the four rows by reading one lane of each (v_readlane), so the result
// is wave-uniform.  The operation must be associative and commutative.  The
// combining pattern is fixed, so results are the same on every run; integer
// sums, max / min and choices by exact comparison are also independent of
// it, while a floating-point sum rounds in this pattern's order.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <type_traits>

namespace avtp {
namespace wave {

// DPP controls (GCN / CDNA encoding)
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1, 0, 3, 2]
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2, 3, 0, 1]
constexpr int kRowRor4 = 0x124;  // row_ror:4
constexpr int kRowRor8 = 0x128;  // row_ror:8

template <int CTRL>
__device__ inline uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ inline uint64_t dpp(uint64_t v) {
  return (uint64_t)dpp<CTRL>((uint32_t)v) | ((uint64_t)dpp<CTRL>((uint32_t)(v >> 32)) << 32);
}
__device__ inline uint32_t lane_value(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}
__device__ inline uint64_t lane_value(uint64_t v, int lane) {
  return (uint64_t)lane_value((uint32_t)v, lane) | ((uint64_t)lane_value((uint32_t)(v >> 32), lane) << 32);
}

// All-reduce of a value held as W 32-bit or 64-bit words (a struct the
// caller packs), with combine(a, b) -> the combination of a and b.
template <typename V, typename F>
__device__ inline V allreduce(V v, F combine) {
  v = combine(v, V::template shift<kQuadXor1>(v));
  v = combine(v, V::template shift<kQuadXor2>(v));
  v = combine(v, V::template shift<kRowRor4>(v));
  v = combine(v, V::template shift<kRowRor8>(v));
  V r = V::at(v, 0);
  r = combine(r, V::at(v, 16));
  r = combine(r, V::at(v, 32));
  return combine(r, V::at(v, 48));
}

// One integer or floating-point scalar.
template <typename T>
struct One {
  T x;
  template <int CTRL>
  __device__ static One shift(const One &a) {
    if constexpr (sizeof(T) == 8) {
      return One{__builtin_bit_cast(T, dpp<CTRL>(__builtin_bit_cast(uint64_t, a.x)))};
    } else {
      return One{__builtin_bit_cast(T, dpp<CTRL>(__builtin_bit_cast(uint32_t, a.x)))};
    }
  }
  __device__ static One at(const One &a, int lane) {
    if constexpr (sizeof(T) == 8) {
      return One{__builtin_bit_cast(T, lane_value(__builtin_bit_cast(uint64_t, a.x), lane))};
    } else {
      return One{__builtin_bit_cast(T, lane_value(__builtin_bit_cast(uint32_t, a.x), lane))};
    }
  }
};

// Inclusive prefix sum over the 64 lanes (lane i: lanes 0 .. i), by the
// row shifts and row broadcasts of the DPP network: a window of four lanes
// from row_shr 1-3, then the row's lower half and quarter added into the
// upper banks, then the last lane of each row broadcast into the rows above.
__device__ inline uint32_t prefix_sum(uint32_t v) {
  auto sh = [](uint32_t x, auto ctrl_tag, auto row_tag, auto bank_tag) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, decltype(ctrl_tag)::value,
                                                 decltype(row_tag)::value,
                                                 decltype(bank_tag)::value, false);
  };
  using std::integral_constant;
  using I = int;
  uint32_t r = v + sh(v, integral_constant<I, 0x111>{}, integral_constant<I, 0xF>{},
                      integral_constant<I, 0xF>{});          // + lane i-1 (row_shr:1)
  r += sh(v, integral_constant<I, 0x112>{}, integral_constant<I, 0xF>{},
          integral_constant<I, 0xF>{});                      // + lane i-2
  r += sh(v, integral_constant<I, 0x113>{}, integral_constant<I, 0xF>{},
          integral_constant<I, 0xF>{});                      // + lane i-3
  r += sh(r, integral_constant<I, 0x114>{}, integral_constant<I, 0xF>{},
          integral_constant<I, 0xE>{});                      // row_shr:4 into banks 1-3
  r += sh(r, integral_constant<I, 0x118>{}, integral_constant<I, 0xF>{},
          integral_constant<I, 0xC>{});                      // row_shr:8 into banks 2-3
  r += sh(r, integral_constant<I, 0x142>{}, integral_constant<I, 0xA>{},
          integral_constant<I, 0xF>{});                      // row_bcast:15 into rows 1, 3
  r += sh(r, integral_constant<I, 0x143>{}, integral_constant<I, 0xC>{},
          integral_constant<I, 0xF>{});                      // row_bcast:31 into rows 2, 3
  return r;
}

template <typename T>
__device__ inline T sum(T v) {
  return allreduce(One<T>{v}, [](One<T> a, One<T> b) { return One<T>{a.x + b.x}; }).x;
}
__device__ inline double max(double v) {
  return allreduce(One<double>{v}, [](One<double> a, One<double> b) {
           return One<double>{fmax(a.x, b.x)};
         }).x;
}

}  // namespace wave
}  // namespace avtp
