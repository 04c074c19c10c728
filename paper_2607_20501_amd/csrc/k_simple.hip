// Simple implementations of every subkernel family: plain HIP with fp32
// FMA, no MFMA.  They are the swap alternatives of the tuned kernels (MKEvolve
// Sec. 3 "Swap": a subkernel can be replaced by an alternative implementation)
// and cover every shape and dtype the plan accepts.
#include "dev.hpp"

namespace mk {

// ----------------------------------------------------------------- element-wise

template <typename T>
__global__ void ew_simple_kernel(EwArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < a.numel; i += stride) {
    float v = ld<T>((const T*)a.x, i);
    v = epi_apply<T>(a.epi, v, (i / a.S) % a.S, i % a.last, (i / a.HW) % a.C, i);
    st<T>((T*)a.y, i, v);
  }
}

// Vectorised form: a thread owns groups of 8 consecutive elements (one
// 16-byte bf16 or two 16-byte fp32 accesses) and keeps 4 groups in flight;
// index arithmetic is done once per group.
template <typename T>
__device__ __forceinline__ void ew_load8(const T* x, int64_t i0, float (&v)[8]) {
  ld8<T>(x + i0, true, 8, v);
}

template <typename T>
__device__ __forceinline__ void ew_store8(T* y, int64_t i0, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    uint4 raw;
    raw.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    raw.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    raw.z = (uint32_t)f2bf(v[4]) | ((uint32_t)f2bf(v[5]) << 16);
    raw.w = (uint32_t)f2bf(v[6]) | ((uint32_t)f2bf(v[7]) << 16);
    *(uint4*)(y + i0) = raw;
  } else {
    *(float4*)(y + i0) = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(y + i0 + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

template <typename T>
__device__ __forceinline__ void ew_chain8(const EwArgs& a, int64_t i0, float (&v)[8]) {
  int64_t col = i0 % a.last, row = (i0 / a.S) % a.S, ch = (i0 / a.HW) % a.C;
  int64_t inrow = i0 % a.HW;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    v[k] = epi_apply<T>(a.epi, v[k], row, col, ch, i0 + k);
    if (++col == a.last) {
      col = 0;
      if (++row == a.S) row = 0;
    }
    if (++inrow == a.HW) {
      inrow = 0;
      if (++ch == a.C) ch = 0;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void ew_vec_kernel(EwArgs a) {
  constexpr int kIn = 4;   // groups in flight per thread
  const int64_t groups = a.numel / 8;
  const int64_t span = (int64_t)gridDim.x * blockDim.x * kIn;
  for (int64_t g0 = (int64_t)blockIdx.x * blockDim.x * kIn + threadIdx.x; g0 < groups;
       g0 += span) {
    float v[kIn][8];
#pragma unroll
    for (int j = 0; j < kIn; ++j) {
      const int64_t g = g0 + (int64_t)j * blockDim.x;
      if (g < groups) ew_load8<T>((const T*)a.x, g * 8, v[j]);
    }
#pragma unroll
    for (int j = 0; j < kIn; ++j) {
      const int64_t g = g0 + (int64_t)j * blockDim.x;
      if (g < groups) {
        if (a.epi.n) ew_chain8<T>(a, g * 8, v[j]);
        ew_store8<T>((T*)a.y, g * 8, v[j]);
      }
    }
  }
  // ragged tail
  const int64_t tail0 = groups * 8;
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t < a.numel - tail0) {
    const int64_t i = tail0 + t;
    float v = ld<T>((const T*)a.x, i);
    v = epi_apply<T>(a.epi, v, (i / a.S) % a.S, i % a.last, (i / a.HW) % a.C, i);
    st<T>((T*)a.y, i, v);
  }
}

static int grid_for(int64_t work, int per_block) {
  int64_t g = (work + per_block - 1) / per_block;
  if (g > 65536) g = 65536;
  return (int)(g < 1 ? 1 : g);
}

hipError_t launch_ew(int dtype, const EwArgs& a, hipStream_t st, int impl) {
  if (a.numel == 0) return hipSuccess;
  if (impl != MK_IMPL_SIMPLE && ew_fast_supported(a)) return launch_ew_fast(dtype, a, st);
  const bool aligned = ((uintptr_t)a.x % 16 == 0) && ((uintptr_t)a.y % 16 == 0);
  if (aligned) {
    const int g = grid_for(a.numel / 32 + 1, 256);
    if (dtype == 1)
      hipLaunchKernelGGL(ew_vec_kernel<bf16>, dim3(g), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(ew_vec_kernel<float>, dim3(g), dim3(256), 0, st, a);
  } else {
    const int g = grid_for(a.numel, 256);
    if (dtype == 1)
      hipLaunchKernelGGL(ew_simple_kernel<bf16>, dim3(g), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(ew_simple_kernel<float>, dim3(g), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------- row ops

template <typename T>
__device__ __forceinline__ float row_in(const RowArgs& a, int64_t r, int64_t j) {
  const int64_t flat = r * a.len + j;
  float v = ld<T>((const T*)a.x, flat);
  if (a.pre.epi.n)
    v = epi_apply<T>(a.pre.epi, v, (flat / a.pre.S) % a.pre.S, flat % a.pre.last,
                     (flat / a.pre.HW) % a.pre.C, flat);
  return v;
}

// One workgroup per row.  Softmax subtracts the row maximum; LayerNorm takes
// the mean, then the biased variance of the centred values (two passes).
template <typename T>
__global__ __launch_bounds__(256) void row_kernel(RowArgs a) {
  __shared__ float red[16];
  const int64_t r = blockIdx.x;
  const int64_t L = a.len;
  switch (a.op) {
    case MK_OP_ROWSUM: case MK_OP_GAP: {
      float s = 0.f;
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x) s += row_in<T>(a, r, j);
      s = block_sum(s, red);
      if (threadIdx.x == 0) st<T>((T*)a.y, r, a.op == MK_OP_GAP ? s / (float)L : s);
      break;
    }
    case MK_OP_GMP: case MK_OP_LPPOOL: {
      const int kind = a.op;
      float s = pool_id(kind);
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x)
        s = pool_comb(kind, s, pool_in(kind, a.p, row_in<T>(a, r, j)));
      s = kind == MK_OP_GMP ? block_max(s, red) : block_sum(s, red);
      if (threadIdx.x == 0) st<T>((T*)a.y, r, pool_out(kind, a.p, s, (float)L));
      break;
    }
    case MK_OP_SOFTMAX: {
      float m = -INFINITY;
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x) m = fmaxf(m, row_in<T>(a, r, j));
      m = block_max(m, red);
      if (a.variant == 1) m = 0.f;   // test-only: the max is not subtracted
      float s = 0.f;
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x) s += __expf(row_in<T>(a, r, j) - m);
      s = block_sum(s, red);
      const float inv = 1.0f / s;
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x)
        st<T>((T*)a.y, r * L + j, __expf(row_in<T>(a, r, j) - m) * inv);
      break;
    }
    case MK_OP_LAYERNORM: {
      float s = 0.f;
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x) s += row_in<T>(a, r, j);
      const float mu = block_sum(s, red) / (float)L;
      float q = 0.f;
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x) {
        const float d = row_in<T>(a, r, j) - mu;
        q += d * d;
      }
      const float rstd = rsqrtf(block_sum(q, red) / (float)L + a.eps);
      const float shift = a.variant == 3 ? 0.f : mu;   // test-only: no centring
      for (int64_t j = threadIdx.x; j < L; j += blockDim.x) {
        const float v = (row_in<T>(a, r, j) - shift) * rstd * ld<T>((const T*)a.gamma, j) +
                        ld<T>((const T*)a.beta, j);
        st<T>((T*)a.y, r * L + j, v);
      }
      break;
    }
    default:
      break;
  }
}

// Test-only: softmax over dim -2, i.e. down each column of every group of n2
// consecutive rows.  One thread per column.
template <typename T>
__global__ void softmax_col_kernel(RowArgs a) {
  const int64_t L = a.len, groups = a.rows / a.n2;
  const int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (c >= groups * L) return;
  const int64_t g = c / L, j = c % L, r0 = g * a.n2;
  float m = -INFINITY;
  for (int64_t i = 0; i < a.n2; ++i) m = fmaxf(m, row_in<T>(a, r0 + i, j));
  float s = 0.f;
  for (int64_t i = 0; i < a.n2; ++i) s += __expf(row_in<T>(a, r0 + i, j) - m);
  for (int64_t i = 0; i < a.n2; ++i)
    st<T>((T*)a.y, (r0 + i) * L + j, __expf(row_in<T>(a, r0 + i, j) - m) / s);
}

hipError_t launch_row(int dtype, const RowArgs& a, hipStream_t st, int impl) {
  if (a.rows == 0) return hipSuccess;
  if (a.variant == 2) {
    if (a.op != MK_OP_SOFTMAX || a.n2 < 1 || a.rows % a.n2) return hipErrorInvalidValue;
    const unsigned g = (unsigned)((a.rows / a.n2 * a.len + 255) / 256);
    if (dtype == 1)
      hipLaunchKernelGGL(softmax_col_kernel<bf16>, dim3(g), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(softmax_col_kernel<float>, dim3(g), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  if (a.variant == 0 && impl != MK_IMPL_SIMPLE && row_wave_supported(dtype, a))
    return launch_row_wave(dtype, a, st);
  if (dtype == 1)
    hipLaunchKernelGGL(row_kernel<bf16>, dim3((unsigned)a.rows), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(row_kernel<float>, dim3((unsigned)a.rows), dim3(256), 0, st, a);
  return hipGetLastError();
}

// Per-row (mean, rstd) for a LayerNorm applied as a GEMM prologue.
template <typename T>
__global__ __launch_bounds__(256) void ln_stats_kernel(const T* x, int64_t len, float eps,
                                                       float* stats, int unsafe) {
  __shared__ float red[16];
  const int64_t r = blockIdx.x;
  const T* xr = x + r * len;
  float s = 0.f;
  for (int64_t j = threadIdx.x; j < len; j += blockDim.x) s += ld<T>(xr, j);
  const float mu = block_sum(s, red) / (float)len;
  float q = 0.f;
  for (int64_t j = threadIdx.x; j < len; j += blockDim.x) {
    const float d = ld<T>(xr, j) - mu;
    q += d * d;
  }
  const float var = block_sum(q, red) / (float)len;
  if (threadIdx.x == 0) {
    stats[2 * r] = unsafe ? 0.f : mu;   // test-only: no centring
    stats[2 * r + 1] = rsqrtf(var + eps);
  }
}

hipError_t launch_ln_stats(int dtype, const void* x, int64_t rows, int64_t len, float eps,
                           float* stats, hipStream_t st, int unsafe) {
  if (rows == 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(ln_stats_kernel<bf16>, dim3((unsigned)rows), dim3(256), 0, st,
                       (const bf16*)x, len, eps, stats, unsafe);
  else
    hipLaunchKernelGGL(ln_stats_kernel<float>, dim3((unsigned)rows), dim3(256), 0, st,
                       (const float*)x, len, eps, stats, unsafe);
  return hipGetLastError();
}

// ----------------------------------------------------------------- GEMM

// 64x64 output tile per workgroup, 16-deep K slices through LDS, 4x4
// outputs per thread.  Handles LN prologue, alpha, the element-wise chain and
// the terminal row-sum / softmax partials.
template <typename T>
__global__ __launch_bounds__(256) void gemm_simple_kernel(GemmArgs a) {
  __shared__ float As[16][68];
  __shared__ float Bs[16][68];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const int64_t z = blockIdx.z, bb = z / a.heads, hh = z % a.heads;
  const T* A = (const T*)a.A + a.a_off + bb * a.a_sb + hh * a.a_sh;
  const T* B = (const T*)a.B + a.b_off + bb * a.b_sb + hh * a.b_sh;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int64_t k0 = 0; k0 < a.K; k0 += 16) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int idx = threadIdx.x + t * 256;
      const int mm = idx >> 4, kk = idx & 15;
      const int64_t gm = m0 + mm, gk = k0 + kk;
      float v = 0.f;
      if (gm < a.M && gk < a.K) {
        v = ld<T>(A, gm * a.lda + gk);
        if (a.ln_stats) {
          v = (v - a.ln_stats[2 * gm]) * a.ln_stats[2 * gm + 1] * ld<T>((const T*)a.ln_g, gk) +
              ld<T>((const T*)a.ln_b, gk);
          v = rnd<T>(v);
        }
      }
      As[kk][mm] = v;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int idx = threadIdx.x + t * 256;
      int kk, nn;
      if (a.layout == 1) {
        kk = idx >> 6;
        nn = idx & 63;
      } else {
        nn = idx >> 4;
        kk = idx & 15;
      }
      const int64_t gk = k0 + kk, gn = n0 + nn;
      float v = 0.f;
      if (gk < a.K && gn < a.N) v = ld<T>(B, a.layout == 1 ? gk * a.ldb + gn : gn * a.ldb + gk);
      Bs[kk][nn] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float ar[4], br[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) ar[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) br[j] = Bs[kk][tx * 4 + j];
      if (a.acc_bf16) {   // test-only: a bf16 accumulator
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = rnd<bf16>(fmaf(ar[i], br[j], acc[i][j]));
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], br[j], acc[i][j]);
      }
    }
    __syncthreads();
  }
  const int64_t cbase = a.c_off + bb * a.c_sb + hh * a.c_sh;
  T* C = (T*)a.C + cbase;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t gm = m0 + ty * 4 + i;
    float rs = 0.f, rm = -INFINITY, re = 0.f;
    Moments mo{0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t gn = n0 + tx * 4 + j;
      if (gm < a.M && gn < a.N) {
        float v = acc[i][j] * a.alpha;
        v = epi_apply<T>(a.epi, v, gm, gn, 0, cbase + gm * a.ldc + gn);
        if (a.terminal == TERM_ROWSUM) {
          rs += v;
        } else if (a.terminal == TERM_SOFTMAX) {
          v = rnd<T>(v);
          st<T>(C, gm * a.ldc + gn, v);
          const float nm = fmaxf(rm, v);
          re = re * __expf(rm - nm) + __expf(v - nm);
          rm = nm;
        } else if (a.terminal == TERM_LAYERNORM) {
          v = rnd<T>(v);
          st<T>(C, gm * a.ldc + gn, v);
          mom_add(mo, v);
        } else {
          st<T>(C, gm * a.ldc + gn, v);
        }
      }
    }
    if (a.terminal == TERM_ROWSUM) {
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) rs += __shfl_xor(rs, o, 64);
      if (tx == 0 && gm < a.M) a.partial[gm * a.n_tiles + blockIdx.x] = rs;
    } else if (a.terminal == TERM_SOFTMAX) {
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) {
        const float om = __shfl_xor(rm, o, 64), oe = __shfl_xor(re, o, 64);
        const float nm = fmaxf(rm, om);
        if (nm != -INFINITY) {
          re = re * __expf(rm - nm) + oe * __expf(om - nm);
          rm = nm;
        }
      }
      if (tx == 0 && gm < a.M) {
        a.partial[(gm * a.n_tiles + blockIdx.x) * 2] = rm;
        a.partial[(gm * a.n_tiles + blockIdx.x) * 2 + 1] = re;
      }
    } else if (a.terminal == TERM_LAYERNORM) {
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) mo = mom_comb(mo, mom_shfl_xor(mo, o));
      if (tx == 0 && gm < a.M) {
        a.partial[(gm * a.n_tiles + blockIdx.x) * 2] = mo.mean;
        a.partial[(gm * a.n_tiles + blockIdx.x) * 2 + 1] = mo.m2;
      }
    }
  }
}

hipError_t launch_gemm_simple(int dtype, const GemmArgs& a, hipStream_t st) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  dim3 grid((unsigned)((a.N + 63) / 64), (unsigned)((a.M + 63) / 64),
            (unsigned)(a.batch * a.heads));
  if (dtype == 1)
    hipLaunchKernelGGL(gemm_simple_kernel<bf16>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(gemm_simple_kernel<float>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// Row-sum finisher: adds a row's column-tile partials in tile order.
template <typename T>
__global__ void rowsum_finish_kernel(const float* partial, int64_t rows, int64_t nt, T* out) {
  const int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (r >= rows) return;
  float s = 0.f;
  for (int64_t t = 0; t < nt; ++t) s += partial[r * nt + t];
  st<T>(out, r, s);
}

hipError_t launch_rowsum_finish(int dtype, const float* partial, int64_t rows, int64_t nt,
                                void* out, hipStream_t st) {
  const unsigned g = (unsigned)((rows + 255) / 256);
  if (dtype == 1)
    hipLaunchKernelGGL(rowsum_finish_kernel<bf16>, dim3(g), dim3(256), 0, st, partial, rows, nt,
                       (bf16*)out);
  else
    hipLaunchKernelGGL(rowsum_finish_kernel<float>, dim3(g), dim3(256), 0, st, partial, rows, nt,
                       (float*)out);
  return hipGetLastError();
}

// Softmax finisher: merges the (max, sum of exp) partials of a row and
// normalises the row in place: y = exp(c - M) / S.
template <typename T>
__global__ __launch_bounds__(256) void softmax_finish_kernel(const float* partial, int64_t nt,
                                                             int64_t N, T* out) {
  const int64_t r = blockIdx.x;
  float M = -INFINITY;
  for (int64_t t = 0; t < nt; ++t) M = fmaxf(M, partial[(r * nt + t) * 2]);
  float S = 0.f;
  for (int64_t t = 0; t < nt; ++t) {
    const float m = partial[(r * nt + t) * 2];
    if (m != -INFINITY) S += partial[(r * nt + t) * 2 + 1] * __expf(m - M);
  }
  const float inv = 1.0f / S;
  T* row = out + r * N;
  for (int64_t j = threadIdx.x; j < N; j += blockDim.x)
    st<T>(row, j, __expf(ld<T>(row, j) - M) * inv);
}

hipError_t launch_softmax_finish(int dtype, const float* partial, int64_t rows, int64_t nt,
                                 int64_t N, void* out, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  if (softmax_finish_wave_supported(dtype, N, out))
    return launch_softmax_finish_wave(dtype, partial, rows, nt, N, out, st);
  if (dtype == 1)
    hipLaunchKernelGGL(softmax_finish_kernel<bf16>, dim3((unsigned)rows), dim3(256), 0, st,
                       partial, nt, N, (bf16*)out);
  else
    hipLaunchKernelGGL(softmax_finish_kernel<float>, dim3((unsigned)rows), dim3(256), 0, st,
                       partial, nt, N, (float*)out);
  return hipGetLastError();
}

// ----------------------------------------------------------------- conv

template <typename T>
__device__ __forceinline__ float conv_at(const ConvArgs& a, int64_t n, int64_t k, int64_t p,
                                         int64_t q) {
  const T* x = (const T*)a.x;
  const T* w = (const T*)a.w;
  float acc = 0.f;
  for (int64_t c = 0; c < a.C; ++c)
    for (int64_t r = 0; r < a.R; ++r) {
      const int64_t h = p * a.stride + r - a.pad;
      if (h < 0 || h >= a.H) continue;
      for (int64_t s = 0; s < a.S; ++s) {
        const int64_t ww = q * a.stride + s - a.pad;
        if (ww < 0 || ww >= a.W) continue;
        acc = fmaf(ld<T>(x, ((n * a.C + c) * a.H + h) * a.W + ww),
                   ld<T>(w, ((k * a.C + c) * a.R + r) * a.S + s), acc);
      }
    }
  return acc;
}

template <typename T>
__global__ void conv_simple_kernel(ConvArgs a) {
  const int64_t total = a.N * a.K * a.P * a.Q;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t q = i % a.Q, p = (i / a.Q) % a.P, k = (i / (a.P * a.Q)) % a.K,
                  n = i / (a.K * a.P * a.Q);
    float v = conv_at<T>(a, n, k, p, q);
    v = epi_apply<T>(a.epi, v, 0, 0, k, i);
    st<T>((T*)a.y, i, v);
  }
}

// Conv + chain + global pool: one workgroup per (image, channel).
template <typename T>
__global__ __launch_bounds__(256) void conv_gap_simple_kernel(ConvArgs a) {
  __shared__ float red[16];
  const int64_t nk = blockIdx.x, n = nk / a.K, k = nk % a.K;
  const int64_t PQ = a.P * a.Q;
  const int kind = a.pool;
  float s = pool_id(kind);
  for (int64_t pos = threadIdx.x; pos < PQ; pos += blockDim.x) {
    float v = conv_at<T>(a, n, k, pos / a.Q, pos % a.Q);
    v = epi_apply<T>(a.epi, v, 0, 0, k, nk * PQ + pos);
    s = pool_comb(kind, s, pool_in(kind, a.pool_p, v));
  }
  s = kind == MK_OP_GMP ? block_max(s, red) : block_sum(s, red);
  if (threadIdx.x == 0) st<T>((T*)a.y, nk, pool_out(kind, a.pool_p, s, (float)PQ));
}

hipError_t launch_conv_simple(int dtype, const ConvArgs& a, hipStream_t st) {
  if (a.gap) {
    const unsigned g = (unsigned)(a.N * a.K);
    if (dtype == 1)
      hipLaunchKernelGGL(conv_gap_simple_kernel<bf16>, dim3(g), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(conv_gap_simple_kernel<float>, dim3(g), dim3(256), 0, st, a);
  } else {
    const int g = grid_for(a.N * a.K * a.P * a.Q, 256);
    if (dtype == 1)
      hipLaunchKernelGGL(conv_simple_kernel<bf16>, dim3(g), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(conv_simple_kernel<float>, dim3(g), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------- attention

// One workgroup per (batch, head, query row): scores into LDS, safe softmax,
// then each thread accumulates output columns.
template <typename T>
__global__ __launch_bounds__(256) void attn_simple_kernel(AttnArgs a) {
  extern __shared__ float sc[];
  __shared__ float red[16];
  const int64_t z = blockIdx.x, i = z % a.S, bh = z / a.S, h = bh % a.H, b = bh / a.H;
  const int64_t ld3 = 3 * a.H * a.dh;
  const T* qkv = (const T*)a.qkv;
  const T* q = qkv + (b * a.S + i) * ld3 + h * a.dh;
  const int64_t jmax = a.causal == 2 ? i : (a.causal ? i + 1 : a.S);
  float m = -INFINITY;
  for (int64_t j = threadIdx.x; j < jmax; j += blockDim.x) {
    const T* k = qkv + (b * a.S + j) * ld3 + a.H * a.dh + h * a.dh;
    float s = 0.f;
    for (int64_t e = 0; e < a.kdim; ++e) s = fmaf(ld<T>(q, e), ld<T>(k, e), s);
    s *= a.scale;
    sc[j] = s;
    m = fmaxf(m, s);
  }
  m = block_max(m, red);
  float l = 0.f;
  for (int64_t j = threadIdx.x; j < jmax; j += blockDim.x) {
    const float p = __expf(sc[j] - m);
    sc[j] = p;
    l += p;
  }
  l = block_sum(l, red);   // contains __syncthreads: sc is complete
  const float inv = 1.0f / l;
  T* o = (T*)a.o + (b * a.S + i) * a.H * a.dh + h * a.dh;
  for (int64_t e = threadIdx.x; e < a.dh; e += blockDim.x) {
    float acc = 0.f;
    for (int64_t j = 0; j < jmax; ++j)
      acc = fmaf(sc[j], ld<T>(qkv, (b * a.S + j) * ld3 + 2 * a.H * a.dh + h * a.dh + e), acc);
    st<T>(o, e, acc * inv);
  }
}

hipError_t launch_attn_simple(int dtype, const AttnArgs& a, hipStream_t st) {
  const unsigned g = (unsigned)(a.B * a.H * a.S);
  const size_t lds = (size_t)a.S * sizeof(float);
  if (dtype == 1)
    hipLaunchKernelGGL(attn_simple_kernel<bf16>, dim3(g), dim3(256), lds, st, a);
  else
    hipLaunchKernelGGL(attn_simple_kernel<float>, dim3(g), dim3(256), lds, st, a);
  return hipGetLastError();
}

}  // namespace mk
