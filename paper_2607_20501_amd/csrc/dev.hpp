// Device helpers shared by the HIP kernels: storage conversion, activations
// and the element-wise chain.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"
#include "plan_codes.hpp"

namespace mk {

using bf16 = uint16_t;

__device__ __forceinline__ float bf2f(bf16 b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest even (gfx950 converts in hardware, NaN preserved).
__device__ __forceinline__ bf16 f2bf(float f) {
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(bf16, h);
}

template <typename T> __device__ __forceinline__ float ld(const T* p, int64_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16>(const bf16* p, int64_t i) {
  return bf2f(p[i]);
}

template <typename T> __device__ __forceinline__ void st(T* p, int64_t i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16>(bf16* p, int64_t i, float v) {
  p[i] = f2bf(v);
}

// Value after a round trip through the storage type.
template <typename T> __device__ __forceinline__ float rnd(float v);
template <> __device__ __forceinline__ float rnd<float>(float v) { return v; }
template <> __device__ __forceinline__ float rnd<bf16>(float v) { return bf2f(f2bf(v)); }

__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_tanh(float x) {
  const float c = 0.79788456080286536f;  // sqrt(2 / pi)
  return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}

// Apply the chain to v.  col: column (BIAS_COL); ch: channel (BIAS_CH);
// flat: element offset shared with residual operands; (row, col) for CAUSAL.
template <typename T>
__device__ __forceinline__ float epi_apply(const EpiDev& e, float v, int64_t row, int64_t col,
                                           int64_t ch, int64_t flat) {
  for (int i = 0; i < e.n; ++i) {
    switch (e.code[i]) {
      case EPI_BIAS_COL: v += ld<T>((const T*)e.ptr[i], col); break;
      case EPI_BIAS_CH: v += ld<T>((const T*)e.ptr[i], ch); break;
      case EPI_RELU: v = fmaxf(v, 0.0f); break;
      case EPI_GELU_ERF: v = gelu_erf(v); break;
      case EPI_GELU_TANH: v = gelu_tanh(v); break;
      case EPI_SCALE: v *= e.s[i]; break;
      case EPI_ADD: v += ld<T>((const T*)e.ptr[i], flat); break;
      case EPI_CAUSAL: if (col > row) v = -INFINITY; break;
      case EPI_GELU_SIGMOID: v = v / (1.0f + __expf(-1.702f * v)); break;
      case EPI_CAUSAL_STRICT: if (col >= row) v = -INFINITY; break;
      default: break;
    }
  }
  return v;
}

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide reductions for blockDim.x a multiple of 64 (<= 1024); `red` is
// a __shared__ float[16].  Every thread receives the result.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = warp_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = warp_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, red[i]);
  return t;
}

}  // namespace mk
