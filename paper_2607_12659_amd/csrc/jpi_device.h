// Device helpers shared by the libjpi kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

#include "jpi_internal.h"

namespace jpi {

// Launch with optional start/stop events tied to the dispatch itself.
#define JPI_LAUNCH(kern, grid, block, shm, strm, evs, eve, ...)                           \
  do {                                                                                    \
    if ((evs) || (eve))                                                                   \
      hipExtLaunchKernelGGL(kern, grid, block, shm, strm, evs, eve, 0, __VA_ARGS__);      \
    else                                                                                  \
      hipLaunchKernelGGL(kern, grid, block, shm, strm, __VA_ARGS__);                      \
  } while (0)

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T>
struct Mfma;

template <>
struct Mfma<bf16> {
  static constexpr int KPL = 8;    // k values per lane per instruction
  static constexpr int KSUB = 32;  // k depth of one instruction
  typedef bf16x8 frag;
  static __device__ __forceinline__ frag load(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<float> {
  static constexpr int KPL = 1;
  static constexpr int KSUB = 4;
  typedef float frag;
  static __device__ __forceinline__ frag load(const float* p) { return *p; }
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

template <typename T>
__device__ __forceinline__ T from_f32(float v) { return static_cast<T>(v); }

// Value of another lane of the same 16-lane row through a DPP operand
// modifier (one VALU move; no LDS crossbar round trip).
template <int CTRL>
__device__ __forceinline__ float dpp_row(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
constexpr int DPP_QUAD_XOR1 = 0xb1;   // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_XOR2 = 0x4e;   // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane i <-> 7 - i within each half-row
constexpr int DPP_MIRROR = 0x140;       // lane i <-> 15 - i within each row

// Sum over the 16 lanes that share lane / 16 (one row group of an MFMA tile).
// Every stage pairs lanes whose partial results are equal, so all 16 lanes
// end with the same bits.
__device__ __forceinline__ float group16_sum(float v) {
  v += dpp_row<DPP_QUAD_XOR1>(v);
  v += dpp_row<DPP_QUAD_XOR2>(v);
  v += dpp_row<DPP_HALF_MIRROR>(v);
  v += dpp_row<DPP_MIRROR>(v);
  return v;
}
__device__ __forceinline__ float group16_max(float v) {
  v = fmaxf(v, dpp_row<DPP_QUAD_XOR1>(v));
  v = fmaxf(v, dpp_row<DPP_QUAD_XOR2>(v));
  v = fmaxf(v, dpp_row<DPP_HALF_MIRROR>(v));
  v = fmaxf(v, dpp_row<DPP_MIRROR>(v));
  return v;
}

// Whole-wave sum, the same in every lane: row sums, then the four rows in order.
__device__ __forceinline__ float wave_sum(float v) {
  v = group16_sum(v);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return ((r0 + r1) + r2) + r3;
}

__device__ __forceinline__ float wave_max(float v) {
  v = group16_max(v);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}


// Block of 256 threads: fixed-order sum (wave sums, then the 4 wave totals in order).
__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// GELU, tanh form: 0.5 z (1 + tanh(u)), u = sqrt(2/pi) (z + 0.044715 z^3),
// evaluated through the identity 0.5 (1 + tanh u) = 1 / (1 + 2^(-2u log2 e)):
// one exp2 and one reciprocal instead of the library tanh (whose cost showed
// in every GeGLU epilogue); relative error about 2e-6, below the bf16 rounding
// of its uses.  Saturates correctly: the exponential overflows to inf (result
// -0) for large negative z and underflows to 0 (result z) for large positive z.
__device__ __forceinline__ float gelu_tanh(float z) {
  const float u2 = 2.f * 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return z * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * u2));
}


}  // namespace jpi
