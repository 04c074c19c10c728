// Tuned row kernels (HBM-bound, no element-wise prologue): one wave per row,
// the row held in registers after one pass of 16-byte loads, reductions by
// wave shuffles.  Row-sum, global average / max / LP pool, softmax (max
// subtracted, App. D), LayerNorm (mean, then the biased variance of the
// centred values; App. H.2 / App. I.2).  Each value is read from HBM once and
// each output written once.
#include <algorithm>

#include "dev.hpp"

namespace mk {

namespace {

template <typename T>
constexpr int kEpv = 16 / sizeof(T);   // elements per 16-byte vector

template <typename T>
__device__ __forceinline__ void ld_vec(const T* p, float* out) {
  float t[8];
  ld8<T>(p, true, 8, t);
#pragma unroll
  for (int k = 0; k < kEpv<T>; ++k) out[k] = t[k];
}

template <typename T>
__device__ __forceinline__ void st_vec(T* p, const float* v) {
  if constexpr (sizeof(T) == 2) {
    uint4 o;
    o.x = pack2_bf16(v[0], v[1]);
    o.y = pack2_bf16(v[2], v[3]);
    o.z = pack2_bf16(v[4], v[5]);
    o.w = pack2_bf16(v[6], v[7]);
    *(uint4*)p = o;
  } else {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
  }
}

// NV 16-byte vectors per lane cover the row (L <= 64 * NV * kEpv, L a
// multiple of kEpv); lane l owns vectors l, l + 64, ...
template <typename T, int NV>
__global__ __launch_bounds__(64) void row_wave_kernel(RowArgs a) {
  constexpr int E = kEpv<T>;
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x;   // one wave (one row) per workgroup
  if (r >= a.rows) return;
  const int64_t L = a.len;
  const T* x = (const T*)a.x + r * L;
  float v[NV][E];
  bool ok[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int64_t c = (int64_t)(i * 64 + lane) * E;
    ok[i] = c < L;
    if (ok[i]) ld_vec<T>(x + c, v[i]);
  }
  if (a.op == MK_OP_GMP || a.op == MK_OP_LPPOOL) {
    const int kind = a.op;
    float s = pool_id(kind);
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (ok[i])
#pragma unroll
        for (int k = 0; k < E; ++k) s = pool_comb(kind, s, pool_in(kind, a.p, v[i][k]));
    s = kind == MK_OP_GMP ? warp_max(s) : warp_sum(s);
    if (lane == 0) st<T>((T*)a.y, r, pool_out(kind, a.p, s, (float)L));
    return;
  }
  if (a.op == MK_OP_ROWSUM || a.op == MK_OP_GAP) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (ok[i])
#pragma unroll
        for (int k = 0; k < E; ++k) s += v[i][k];
    s = warp_sum(s);
    if (lane == 0) st<T>((T*)a.y, r, a.op == MK_OP_GAP ? s / (float)L : s);
    return;
  }
  T* y = (T*)a.y + r * L;
  if (a.op == MK_OP_SOFTMAX) {
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (ok[i])
#pragma unroll
        for (int k = 0; k < E; ++k) m = fmaxf(m, v[i][k]);
    m = warp_max(m);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (ok[i])
#pragma unroll
        for (int k = 0; k < E; ++k) {
          v[i][k] = __expf(v[i][k] - m);
          s += v[i][k];
        }
    const float inv = 1.0f / warp_sum(s);
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (ok[i]) {
#pragma unroll
        for (int k = 0; k < E; ++k) v[i][k] *= inv;
        st_vec<T>(y + (int64_t)(i * 64 + lane) * E, v[i]);
      }
    return;
  }
  // LayerNorm
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (ok[i])
#pragma unroll
      for (int k = 0; k < E; ++k) s += v[i][k];
  const float mu = warp_sum(s) / (float)L;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (ok[i])
#pragma unroll
      for (int k = 0; k < E; ++k) {
        const float d = v[i][k] - mu;
        q += d * d;
      }
  const float rstd = rsqrtf(warp_sum(q) / (float)L + a.eps);
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (ok[i]) {
      const int64_t c = (int64_t)(i * 64 + lane) * E;
      float g[E], b[E];
      ld_vec<T>((const T*)a.gamma + c, g);
      ld_vec<T>((const T*)a.beta + c, b);
#pragma unroll
      for (int k = 0; k < E; ++k) v[i][k] = (v[i][k] - mu) * rstd * g[k] + b[k];
      st_vec<T>(y + c, v[i]);
    }
}

// LayerNorm over rows with persistent waves: gamma and beta of the lane's
// columns stay in registers across rows, and the next row is requested
// before the current one is reduced (two row buffers in alternation), so a
// wave keeps a row of loads in flight while it computes.  Rows past the end
// and columns past L read valid memory (clamped) and are not stored.
template <typename T, int NV>
__global__ __launch_bounds__(64) void ln_rows_kernel(RowArgs a) {
  constexpr int E = kEpv<T>;
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  const int lane = threadIdx.x & 63;
  const int64_t L = a.len, rows = a.rows, step = gridDim.x;
  const T* X = (const T*)a.x;
  T* Y = (T*)a.y;
  bool ok[NV];
  int64_t col[NV];
  u32x4_t g[NV], be[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    col[i] = (int64_t)(i * 64 + lane) * E;
    ok[i] = col[i] < L;
    const int64_t cc = ok[i] ? col[i] : 0;
    g[i] = *(const u32x4_t*)((const T*)a.gamma + cc);
    be[i] = *(const u32x4_t*)((const T*)a.beta + cc);
  }
  auto load_row = [&](int64_t r, u32x4_t (&dst)[NV]) {
    const int64_t rr = r < rows ? r : rows - 1;
#pragma unroll
    for (int i = 0; i < NV; ++i) dst[i] = *(const u32x4_t*)(X + rr * L + (ok[i] ? col[i] : 0));
  };
  auto unpack = [&](const u32x4_t& w, float (&out)[E]) {
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        out[2 * k] = __uint_as_float(w[k] << 16);
        out[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) out[k] = __uint_as_float(w[k]);
    }
  };
  // (The row stays packed: each pass unpacks it again, which keeps the
  // register count at two occupancy levels above float copies.)
  auto do_row = [&](int64_t r, const u32x4_t (&src)[NV]) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float v[E];
      unpack(src[i], v);
#pragma unroll
      for (int k = 0; k < E; ++k) s += ok[i] ? v[k] : 0.f;
    }
    const float mu = warp_sum(s) / (float)L;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float v[E];
      unpack(src[i], v);
#pragma unroll
      for (int k = 0; k < E; ++k) {
        const float d = v[k] - mu;
        q += ok[i] ? d * d : 0.f;
      }
    }
    const float rstd = rsqrtf(warp_sum(q) / (float)L + a.eps);
    if (r >= rows) return;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (!ok[i]) continue;
      float v[E], gg[E], bb[E];
      // gamma and beta are unpacked per row: an opaque copy keeps the
      // compiler from hoisting 2 * NV * E floats out of the row loop.
      u32x4_t gi = g[i], bi = be[i];
      asm volatile("" : "+v"(gi), "+v"(bi));
      unpack(src[i], v);
      unpack(gi, gg);
      unpack(bi, bb);
#pragma unroll
      for (int k = 0; k < E; ++k) v[k] = (v[k] - mu) * rstd * gg[k] + bb[k];
      st_vec<T>(Y + r * L + col[i], v);
    }
  };
  int64_t r = blockIdx.x;
  u32x4_t xa[NV], xb[NV];
  load_row(r, xa);
  for (; r < rows; r += 2 * step) {
    load_row(r + step, xb);
    do_row(r, xa);
    if (r + step >= rows) break;
    load_row(r + 2 * step, xa);
    do_row(r + step, xb);
  }
}

// Softmax over rows (max subtracted) on persistent waves, like the LayerNorm
// rows: the next row is requested before the current one is reduced; the
// exponentials stay in registers between the sum and the normalisation.
template <typename T, int NV>
__global__ __launch_bounds__(64) void softmax_rows_kernel(RowArgs a) {
  constexpr int E = kEpv<T>;
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  const int lane = threadIdx.x & 63;
  const int64_t L = a.len, rows = a.rows, step = gridDim.x;
  const T* X = (const T*)a.x;
  T* Y = (T*)a.y;
  bool ok[NV];
  int64_t col[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    col[i] = (int64_t)(i * 64 + lane) * E;
    ok[i] = col[i] < L;
  }
  auto load_row = [&](int64_t r, u32x4_t (&dst)[NV]) {
    const int64_t rr = r < rows ? r : rows - 1;
#pragma unroll
    for (int i = 0; i < NV; ++i) dst[i] = *(const u32x4_t*)(X + rr * L + (ok[i] ? col[i] : 0));
  };
  auto unpack = [&](const u32x4_t& w, float (&out)[E]) {
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        out[2 * k] = __uint_as_float(w[k] << 16);
        out[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) out[k] = __uint_as_float(w[k]);
    }
  };
  auto do_row = [&](int64_t r, const u32x4_t (&src)[NV]) {
    float e[NV][E];
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      unpack(src[i], e[i]);
#pragma unroll
      for (int k = 0; k < E; ++k) m = fmaxf(m, ok[i] ? e[i][k] : -INFINITY);
    }
    m = warp_max(m);
    // exp(v - m) = 2^(v log2 e - m log2 e)
    const float ml = m * 1.4426950408889634f;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int k = 0; k < E; ++k) {
        e[i][k] = __builtin_amdgcn_exp2f(fmaf(e[i][k], 1.4426950408889634f, -ml));
        s += ok[i] ? e[i][k] : 0.f;
      }
    const float inv = 1.0f / warp_sum(s);
    if (r >= rows) return;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (!ok[i]) continue;
#pragma unroll
      for (int k = 0; k < E; ++k) e[i][k] *= inv;
      st_vec<T>(Y + r * L + col[i], e[i]);
    }
  };
  int64_t r = blockIdx.x;
  u32x4_t xa[NV], xb[NV];
  load_row(r, xa);
  for (; r < rows; r += 2 * step) {
    load_row(r + step, xb);
    do_row(r, xa);
    if (r + step >= rows) break;
    load_row(r + 2 * step, xa);
    do_row(r + step, xb);
  }
}

// Persistent row waves: eight per CU (LayerNorm; softmax takes twice as many).
static int ln_waves() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
    n = 256;
  return 8 * n;
}

template <typename T>
hipError_t launch_row_wave_t(const RowArgs& a, hipStream_t st) {
  constexpr int E = kEpv<T>;
  const int64_t nv = (a.len + 64 * E - 1) / (64 * E);
  const dim3 grid((unsigned)a.rows), block(64);
  if (a.op == MK_OP_SOFTMAX) {
    // (sixteen waves per CU: fewer registers than the LayerNorm waves)
    const dim3 pg((unsigned)std::min<int64_t>(a.rows, 2 * ln_waves()));
    switch (nv) {
      case 1: hipLaunchKernelGGL((softmax_rows_kernel<T, 1>), pg, block, 0, st, a); break;
      case 2: hipLaunchKernelGGL((softmax_rows_kernel<T, 2>), pg, block, 0, st, a); break;
      case 3: case 4: hipLaunchKernelGGL((softmax_rows_kernel<T, 4>), pg, block, 0, st, a); break;
      default: hipLaunchKernelGGL((softmax_rows_kernel<T, 8>), pg, block, 0, st, a); break;
    }
    return hipGetLastError();
  }
  if (a.op == MK_OP_LAYERNORM) {
    const dim3 pg((unsigned)std::min<int64_t>(a.rows, ln_waves()));
    switch (nv) {
      case 1: hipLaunchKernelGGL((ln_rows_kernel<T, 1>), pg, block, 0, st, a); break;
      case 2: hipLaunchKernelGGL((ln_rows_kernel<T, 2>), pg, block, 0, st, a); break;
      case 3: case 4: hipLaunchKernelGGL((ln_rows_kernel<T, 4>), pg, block, 0, st, a); break;
      default: hipLaunchKernelGGL((ln_rows_kernel<T, 8>), pg, block, 0, st, a); break;
    }
    return hipGetLastError();
  }
  switch (nv) {
    case 1: hipLaunchKernelGGL((row_wave_kernel<T, 1>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((row_wave_kernel<T, 2>), grid, block, 0, st, a); break;
    case 3: case 4: hipLaunchKernelGGL((row_wave_kernel<T, 4>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((row_wave_kernel<T, 8>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

// Softmax finisher over the per-(row, column tile) partials (m_t, s_t) of a
// GEMM epilogue: M = max_t m_t, S = sum_t s_t exp(m_t - M), then the row is
// normalised in place, y = exp(c - M) / S.  One wave per row; lanes merge
// the partials in parallel, and the row moves in 16-byte chunks, four in
// flight per lane.
template <typename T>
__global__ __launch_bounds__(256) void softmax_finish_wave_kernel(const float* partial, int64_t rows,
                                                                  int64_t nt, int64_t N, T* out) {
  constexpr int E = kEpv<T>;
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;   // whole wave exits together
  const float* pr = partial + r * nt * 2;
  float m = -INFINITY;
  for (int64_t t = lane; t < nt; t += 64) m = fmaxf(m, pr[t * 2]);
  const float M = warp_max(m);
  float s = 0.f;
  for (int64_t t = lane; t < nt; t += 64) {
    const float mt = pr[t * 2];
    if (mt != -INFINITY) s += pr[t * 2 + 1] * __expf(mt - M);
  }
  const float inv = 1.0f / warp_sum(s);
  T* y = out + r * N;
  const int64_t chunks = N / E;
  for (int64_t c0 = lane; c0 < chunks; c0 += 64 * 4) {
    float v[4][E];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (c0 + u * 64 < chunks) ld_vec<T>(y + (c0 + u * 64) * E, v[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (c0 + u * 64 < chunks) {
#pragma unroll
        for (int k = 0; k < E; ++k) v[u][k] = __expf(v[u][k] - M) * inv;
        st_vec<T>(y + (c0 + u * 64) * E, v[u]);
      }
  }
}

// LayerNorm finisher over the per-(row, column tile) moments (mean_t, M2_t) of
// a GEMM epilogue (tile t holds min(tile, N - t*tile) columns): the moments
// are merged (Chan et al.), then the stored row is normalised in place,
// y = (x - mean) / sqrt(M2 / N + eps) * gamma + beta.  One wave per row.
template <typename T>
__global__ __launch_bounds__(256) void ln_finish_wave_kernel(const float* partial, int64_t rows,
                                                             int64_t nt, int64_t N, int64_t tile,
                                                             const T* gamma, const T* beta,
                                                             float eps, T* out) {
  constexpr int E = kEpv<T>;
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;   // whole wave exits together
  const float* pr = partial + r * nt * 2;
  Moments mo{0.f, 0.f, 0.f};
  for (int64_t t = lane; t < nt; t += 64) {
    const float cnt = (float)min<int64_t>(tile, N - t * tile);
    mo = mom_comb(mo, Moments{cnt, pr[t * 2], pr[t * 2 + 1]});
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mo = mom_comb(mo, mom_shfl_xor(mo, o));
  const float mean = mo.mean, rstd = rsqrtf(mo.m2 / (float)N + eps);
  T* y = out + r * N;
  const bool vec = N % E == 0 && ((uintptr_t)out | (uintptr_t)gamma | (uintptr_t)beta) % 16 == 0;
  if (vec) {
    for (int64_t c = lane; c < N / E; c += 64) {
      float v[E], g[E], b[E];
      ld_vec<T>(y + c * E, v);
      ld_vec<T>(gamma + c * E, g);
      ld_vec<T>(beta + c * E, b);
#pragma unroll
      for (int k = 0; k < E; ++k) v[k] = (v[k] - mean) * rstd * g[k] + b[k];
      st_vec<T>(y + c * E, v);
    }
  } else {
    for (int64_t j = lane; j < N; j += 64)
      st<T>(y, j, (ld<T>(y, j) - mean) * rstd * ld<T>(gamma, j) + ld<T>(beta, j));
  }
}

}  // namespace

hipError_t launch_ln_finish(int dtype, const float* partial, int64_t rows, int64_t nt, int64_t N,
                            int64_t tile, const void* gamma, const void* beta, float eps,
                            void* out, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  if (dtype == MK_BF16)
    hipLaunchKernelGGL(ln_finish_wave_kernel<bf16>, grid, block, 0, st, partial, rows, nt, N, tile,
                       (const bf16*)gamma, (const bf16*)beta, eps, (bf16*)out);
  else
    hipLaunchKernelGGL(ln_finish_wave_kernel<float>, grid, block, 0, st, partial, rows, nt, N,
                       tile, (const float*)gamma, (const float*)beta, eps, (float*)out);
  return hipGetLastError();
}

bool softmax_finish_wave_supported(int dtype, int64_t N, const void* out) {
  const int E = dtype == MK_BF16 ? 8 : 4;
  return N % E == 0 && (uintptr_t)out % 16 == 0;
}

hipError_t launch_softmax_finish_wave(int dtype, const float* partial, int64_t rows, int64_t nt,
                                      int64_t N, void* out, hipStream_t st) {
  const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  if (dtype == MK_BF16)
    hipLaunchKernelGGL(softmax_finish_wave_kernel<bf16>, grid, block, 0, st, partial, rows, nt, N,
                       (bf16*)out);
  else
    hipLaunchKernelGGL(softmax_finish_wave_kernel<float>, grid, block, 0, st, partial, rows, nt, N,
                       (float*)out);
  return hipGetLastError();
}

bool row_wave_supported(int dtype, const RowArgs& a) {
  const int E = dtype == MK_BF16 ? 8 : 4;
  // (Groups with an element-wise prologue run on the simple row kernel.)
  if (a.pre.epi.n || a.len % E || a.len > 64 * 8 * E || a.rows < 1) return false;
  if (((uintptr_t)a.x | (uintptr_t)a.y) % 16) return false;
  if (a.op == MK_OP_LAYERNORM && ((uintptr_t)a.gamma | (uintptr_t)a.beta) % 16) return false;
  return a.rows < (1ll << 31);   // one workgroup per row
}

hipError_t launch_row_wave(int dtype, const RowArgs& a, hipStream_t st) {
  return dtype == MK_BF16 ? launch_row_wave_t<bf16>(a, st) : launch_row_wave_t<float>(a, st);
}

}  // namespace mk
