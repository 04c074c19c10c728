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

// Two values rounded to bf16 and packed (lo in the low half): one packed
// conversion instruction.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
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

// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),
// t = 1 / (1 + p x) for x >= 0 (|error| <= 1.5e-7), odd extension for x < 0.
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  float poly = 1.061405429f;
  poly = fmaf(poly, t, -1.453152027f);
  poly = fmaf(poly, t, 1.421413741f);
  poly = fmaf(poly, t, -0.284496736f);
  poly = fmaf(poly, t, 0.254829592f);
  poly *= t;
  // exp(-x^2) = 2^(-x^2 log2 e)
  const float y = 1.0f - poly * __builtin_amdgcn_exp2f(-1.4426950408889634f * ax * ax);
  return copysignf(y, x);
}

__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f));
}
// GELU (erf form) for results stored as bf16: x * Phi(x) with the normal CDF
// in logistic form (as in Bowling et al., J. Ind. Eng. Manag. 2009, with an
// x^4 term added), Phi(x) ~= sigmoid(x (c0 + c1 x^2 + c2 x^4)), x^2 capped
// at 49.  The coefficients (folded with -log2 e for exp2 below) minimise the
// largest |x (Phi~ - Phi)| over [0, 7]; evaluated in fp32 the result is
// within 2.6e-5 of x Phi(x) for every x (1/150 of a bf16 half-ulp at 1).
// The exponent is odd in x, so Phi~(-x) = 1 - Phi~(x) as for Phi.
__device__ __forceinline__ float gelu_erf_bf16out(float x) {
  const float x2 = fminf(x * x, 49.0f);
  const float p = fmaf(fmaf(0.001014263f, x2, -0.10677572f), x2, -2.3011212f);
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * p));
}

// 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)) exactly, so the tanh form of GELU is
// x * sigmoid(2u) with u = sqrt(2/pi) (x + 0.044715 x^3).  exp(-2u) is taken
// as 2^(-2u log2 e); the reciprocal is the hardware one (1 ulp): for very
// negative x it sees +inf and gives 0.
// The exponent -2u log2 e = x (k0 + k1 x^2) with k0 = -2 sqrt(2/pi) log2 e,
// k1 = 0.044715 k0: one multiply, one FMA, one multiply.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = -2.3022081983f;           // -2 sqrt(2 / pi) log2(e)
  const float k1 = -0.10294324f;             // 0.044715 k0
  const float e = __builtin_amdgcn_exp2f(x * fmaf(k1, x * x, k0));
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

// Apply the chain to v.  col: column (BIAS_COL); ch: channel (BIAS_CH);
// flat: element offset shared with residual operands; (row, col) for CAUSAL.
// The loop over the (at most kMaxEpi) steps is unrolled so that the step codes
// are read once per kernel, not once per element.
template <typename T>
__device__ __forceinline__ float epi_apply(const EpiDev& e, float v, int64_t row, int64_t col,
                                           int64_t ch, int64_t flat) {
#pragma unroll
  for (int i = 0; i < kMaxEpi; ++i) {
    if (i >= e.n) break;
    switch (e.code[i]) {
      case EPI_BIAS_COL: v += ld<T>((const T*)e.ptr[i], col); break;
      case EPI_BIAS_CH: v += ld<T>((const T*)e.ptr[i], ch); break;
      case EPI_RELU: v = fmaxf(v, 0.0f); break;
      case EPI_GELU_ERF: v = sizeof(T) == 2 ? gelu_erf_bf16out(v) : gelu_erf(v); break;
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

// Load 8 consecutive values p[0..7] as floats; `vec` allows one 16-byte (bf16)
// or two 16-byte (fp32) accesses, otherwise only the first `valid` are read.
template <typename T>
__device__ __forceinline__ void ld8(const T* p, bool vec, int valid, float (&out)[8]) {
  if (vec) {
    if constexpr (sizeof(T) == 2) {
      const uint4 r = *(const uint4*)p;
      const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        out[2 * k] = __uint_as_float(w[k] << 16);
        out[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
      }
    } else {
      const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
      out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
      out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) out[k] = k < valid ? ld<T>(p, k) : 0.f;
  }
}

// Store 8 consecutive values to p[0..7] (16-byte aligned): one 16-byte store
// of bf16, two of fp32.
template <typename T>
__device__ __forceinline__ void st8(T* p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    uint4 o;
    o.x = pack2_bf16(v[0], v[1]);
    o.y = pack2_bf16(v[2], v[3]);
    o.z = pack2_bf16(v[4], v[5]);
    o.w = pack2_bf16(v[6], v[7]);
    *(uint4*)p = o;
  } else {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// The chain applied to 8 consecutive columns col0.. of one row (flat0 is the
// offset of column col0 in residual operands).  One uniform switch per step;
// `vec` says that 16-byte operand accesses are aligned and in range.
// Step `pre` (if >= 0) is a BIAS_CH whose value for this row the caller has
// already loaded (`bpre`).
template <typename T>
__device__ __forceinline__ void epi_apply8(const EpiDev& e, float (&v)[8], int64_t row,
                                           int64_t col0, int64_t ch, int valid, int64_t flat0,
                                           bool vec, int pre = -1, float bpre = 0.f) {
#pragma unroll
  for (int i = 0; i < kMaxEpi; ++i) {
    if (i >= e.n) break;
    float t[8];
    switch (e.code[i]) {
      case EPI_BIAS_COL:
        ld8<T>((const T*)e.ptr[i] + col0, vec, valid, t);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] += t[k];
        break;
      case EPI_ADD:
        ld8<T>((const T*)e.ptr[i] + flat0, vec, valid, t);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] += t[k];
        break;
      case EPI_BIAS_CH: {
        const float bch = i == pre ? bpre : ld<T>((const T*)e.ptr[i], ch);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] += bch;
        break;
      }
      case EPI_RELU:
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = fmaxf(v[k], 0.0f);
        break;
      case EPI_GELU_ERF:   // (the logistic form where the result is stored as bf16)
#pragma unroll
        for (int k = 0; k < 8; ++k)
          v[k] = sizeof(T) == 2 ? gelu_erf_bf16out(v[k]) : gelu_erf(v[k]);
        break;
      case EPI_GELU_TANH:
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = gelu_tanh(v[k]);
        break;
      case EPI_SCALE:
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] *= e.s[i];
        break;
      case EPI_CAUSAL:
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (col0 + k > row) v[k] = -INFINITY;
        break;
      case EPI_GELU_SIGMOID:
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = v[k] / (1.0f + __expf(-1.702f * v[k]));
        break;
      case EPI_CAUSAL_STRICT:
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (col0 + k >= row) v[k] = -INFINITY;
        break;
      default:
        break;
    }
  }
}

// Global pooling over positions (GAP mean, GMP max, LPPOOL sign(S)|S|^(1/p)
// of S = sum x^p): each value's contribution, the identity and combination of
// partial results, and the final value over `count` positions.
__device__ __forceinline__ float pool_in(int kind, float p, float v) {
  return kind == MK_OP_LPPOOL ? powf(v, p) : v;
}
__device__ __forceinline__ float pool_id(int kind) {
  return kind == MK_OP_GMP ? -INFINITY : 0.f;
}
__device__ __forceinline__ float pool_comb(int kind, float a, float b) {
  return kind == MK_OP_GMP ? fmaxf(a, b) : a + b;
}
__device__ __forceinline__ float pool_out(int kind, float p, float s, float count) {
  if (kind == MK_OP_GAP) return s / count;
  if (kind == MK_OP_LPPOOL) return copysignf(powf(fabsf(s), 1.0f / p), s);
  return s;
}

// Row moments (count, mean, sum of squared deviations M2): Welford's update
// for one value, Chan et al.'s pairwise combination for two partial results
// (no E[x^2] - mean^2 cancellation).
struct Moments {
  float n, mean, m2;
};
__device__ __forceinline__ void mom_add(Moments& a, float v) {
  a.n += 1.f;
  const float d = v - a.mean;
  a.mean += d / a.n;
  a.m2 += d * (v - a.mean);
}
__device__ __forceinline__ Moments mom_comb(const Moments& a, const Moments& b) {
  const float n = a.n + b.n;
  const float d = b.mean - a.mean, f = n > 0.f ? b.n / n : 0.f;   // (n = 0: both empty)
  return {n, a.mean + d * f, a.m2 + b.m2 + d * d * a.n * f};
}
__device__ __forceinline__ Moments mom_shfl_xor(const Moments& a, int o) {
  return {__shfl_xor(a.n, o, 64), __shfl_xor(a.mean, o, 64), __shfl_xor(a.m2, o, 64)};
}

// The value of lane (this lane ^ O), O = 8, 16 or 32, by VALU lane
// exchanges instead of an LDS permute: a DPP rotate by 8 within each 16-lane
// row; the gfx950 swaps of odd with even 16-lane rows and of the two 32-lane
// halves (each returns both operands after the swap; a lane takes the half
// that came from its partner).
template <int O>
__device__ __forceinline__ float lane_xor(float x) {
  const int b = __builtin_bit_cast(int, x);
  if constexpr (O == 8) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, b, 0x128, 0xF, 0xF, false));
  } else if constexpr (O == 16) {
    const auto p = __builtin_amdgcn_permlane16_swap((unsigned)b, (unsigned)b, false, false);
    return __builtin_bit_cast(float, (threadIdx.x & 16) ? p[0] : p[1]);
  } else {
    static_assert(O == 32, "lane_xor: 8, 16 or 32");
    const auto p = __builtin_amdgcn_permlane32_swap((unsigned)b, (unsigned)b, false, false);
    return __builtin_bit_cast(float, (threadIdx.x & 32) ? p[0] : p[1]);
  }
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
