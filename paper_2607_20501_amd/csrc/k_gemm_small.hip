// Small-problem GEMM on the matrix cores: 64 x 64 output tiles, four waves
// of one 32 x 32 MFMA tile each, operand fragments loaded straight into
// registers.
//
//   C[z][m, n] = chain(alpha * sum_k A[z][m, k] B[z][n, k])     (fp32 accumulate)
//
// The same contraction and fused epilogue as the 256 x 256 kernel
// (k_gemm_mfma.hip; MKEvolve App. H.2 linear kernels, App. I.1 fusion of the
// element-wise chain and a split at full-row reductions).  A problem with
// few 256 x 256 tiles would leave most of the 256 CUs idle there (a
// 128 x 256 fp32 Linear is one tile on one CU), so such problems take this
// kernel: 16x as many workgroups, no LDS staging of operands (each
// fragment is used by two waves and stays in L1/L2), and row-reduction
// partials per 64-column tile.
#include "dev.hpp"

namespace mk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr uint32_t kOob = 0x80000000u;
constexpr int kSubs = 4;   // sub-steps (two 16-byte chunks of K) per load group

template <typename T>
struct SmallFrag;
template <>
struct SmallFrag<bf16> {
  typedef bf16x8 type;
};
template <>
struct SmallFrag<float> {
  typedef f32x4 type;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t small_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// One MFMA sub-step: lane (lr, lh) holds the 16-byte chunk 2s+lh of its A row
// and B row (bf16: the 32x32x16 instruction's k = 8lh..8lh+7; fp32: four
// 32x32x2 instructions, instruction t taking the chunk's element t).
template <typename T>
__device__ __forceinline__ void small_mfma(const typename SmallFrag<T>::type& fa,
                                           const typename SmallFrag<T>::type& fb, f32x16& acc) {
  if constexpr (sizeof(T) == 2) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, acc, 0, 0, 0);
  } else {
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[t], fb[t], acc, 0, 0, 0);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void gemm_small_kernel(GemmArgs a) {
  typedef typename SmallFrag<T>::type F;
  constexpr int E = 16 / (int)sizeof(T);   // elements per 16-byte chunk
  __shared__ float red[2][64][2];          // [wave column][tile row][2] row-reduction exchange
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int lr = lane & 31, lh = lane >> 5;
  const int64_t z = blockIdx.z, bb = z / a.heads, hh = z % a.heads;
  const T* A = (const T*)a.A + a.a_off + bb * a.a_sb + hh * a.a_sh;
  const T* B = (const T*)a.B + a.b_off + bb * a.b_sb + hh * a.b_sh;
  const int64_t tm0 = (int64_t)blockIdx.y * 64, tn0 = (int64_t)blockIdx.x * 64;
  const int64_t m0 = tm0 + wm * 32, n0 = tn0 + wn * 32;   // this wave's 32 x 32 tile

  // Operand rows through buffer descriptors: rows past M / N and chunks past
  // K read zeros.
  const __amdgpu_buffer_rsrc_t ra = small_rsrc(A, a.M * a.lda * (int64_t)sizeof(T));
  const __amdgpu_buffer_rsrc_t rb = small_rsrc(B, a.N * a.ldb * (int64_t)sizeof(T));
  const int64_t arow = m0 + lr, brow = n0 + lr;
  const uint32_t va = arow < a.M ? (uint32_t)(arow * a.lda * (int64_t)sizeof(T)) : kOob;
  const uint32_t vb = brow < a.N ? (uint32_t)(brow * a.ldb * (int64_t)sizeof(T)) : kOob;
  const int nsub = (int)((a.K + 2 * E - 1) / (2 * E));
  auto load_group = [&](int g, F (&fa)[kSubs], F (&fb)[kSubs]) {
#pragma unroll
    for (int s = 0; s < kSubs; ++s) {
      const int64_t chunk = (int64_t)(g * kSubs + s) * 2 + lh;
      const bool in_k = chunk * E < a.K;
      const int off = (int)(chunk * 16);
      fa[s] = __builtin_bit_cast(F, __builtin_amdgcn_raw_buffer_load_b128(
                                        ra, (int)(in_k ? va : kOob), off, 0));
      fb[s] = __builtin_bit_cast(F, __builtin_amdgcn_raw_buffer_load_b128(
                                        rb, (int)(in_k ? vb : kOob), off, 0));
    }
  };
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  const int ngroups = (nsub + kSubs - 1) / kSubs;
  F fa0[kSubs], fb0[kSubs], fa1[kSubs], fb1[kSubs];
  load_group(0, fa0, fb0);
  // Two register groups: the loads of group g+1 are in flight during the
  // MFMAs of group g (loads past K read zeros, so every group is whole).
  for (int g = 0; g < ngroups; g += 2) {
    load_group(g + 1, fa1, fb1);
#pragma unroll
    for (int s = 0; s < kSubs; ++s) small_mfma<T>(fa0[s], fb0[s], acc);
    if (g + 1 >= ngroups) break;
    load_group(g + 2, fa0, fb0);
#pragma unroll
    for (int s = 0; s < kSubs; ++s) small_mfma<T>(fa1[s], fb1[s], acc);
  }

  // Epilogue.  acc[r] is C[row, col], row = m0 + (r/4)*8 + lh*4 + r%4,
  // col = n0 + lr.
  const int64_t cbase = a.c_off + bb * a.c_sb + hh * a.c_sh;
  T* C = (T*)a.C + cbase;
  const int64_t col = n0 + lr;
  const bool col_ok = col < a.N;
  const bool softmax = a.terminal == TERM_SOFTMAX;
  float v[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t row = m0 + (r >> 2) * 8 + lh * 4 + (r & 3);
    float x = acc[r] * a.alpha;
    if (row < a.M && col_ok) {
      if (a.epi.n) x = epi_apply<T>(a.epi, x, row, col, row, cbase + row * a.ldc + col);
      // stored values are rounded to the storage type; reductions that need
      // the whole row read them back as stored
      if (a.terminal != TERM_ROWSUM) x = rnd<T>(x);
      if (a.terminal != TERM_ROWSUM) st<T>(C, row * a.ldc + col, x);
    }
    v[r] = x;
  }
  if (a.terminal == TERM_NONE) return;
  // Per-row partials over this wave's 32 columns (lanes of one half), then
  // over the two waves of the tile's 64 columns.
  if (a.terminal == TERM_ROWSUM) {
    // All 16 rows at once by a halving butterfly over the 32 lanes lr: at
    // the step across lane bit b a lane keeps the half of its values
    // selected by that bit and adds the partner's copy of it; after bits
    // 4..1 lane lr holds row r = lr / 2, and a last exchange across bit 0
    // completes it (16 exchanges instead of 5 per row).
    float x[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = col_ok ? v[r] : 0.f;
#define MK_SMALL_STEP(O, H)                                                         \
  {                                                                                 \
    const bool up = (lr & (O)) != 0;                                                \
    _Pragma("unroll") for (int k = 0; k < (H); ++k) {                               \
      const float keep = up ? x[k + (H)] : x[k];                                    \
      const float send = up ? x[k] : x[k + (H)];                                    \
      x[k] = keep + __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(send), \
                                                               ((O) << 10) | 0x1F));  \
    }                                                                               \
  }
    MK_SMALL_STEP(16, 8)
    MK_SMALL_STEP(8, 4)
    MK_SMALL_STEP(4, 2)
    MK_SMALL_STEP(2, 1)
#undef MK_SMALL_STEP
    x[0] += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x[0]), (1 << 10) | 0x1F));
    if ((lr & 1) == 0) {
      const int r = lr >> 1;
      red[wn][wm * 32 + (r >> 2) * 8 + lh * 4 + (r & 3)][1] = x[0];
    }
  }
  const float cnt = (float)min<int64_t>(32, max<int64_t>(0, a.N - n0));
#pragma unroll
  for (int r = 0; r < 16 && a.terminal != TERM_ROWSUM; ++r) {
    const int trow = wm * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
    float p0, p1;
    if (a.terminal == TERM_LAYERNORM) {
      float s = col_ok ? v[r] : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) s += __shfl_xor(s, o, 64);
      const float mean = cnt > 0.f ? s / cnt : 0.f;
      const float d = v[r] - mean;
      float m2 = col_ok ? d * d : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) m2 += __shfl_xor(m2, o, 64);
      p0 = mean;
      p1 = m2;
    } else if (softmax) {
      float m = col_ok ? v[r] : -INFINITY;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
      float s = (col_ok && m != -INFINITY) ? __expf(v[r] - m) : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) s += __shfl_xor(s, o, 64);
      p0 = m;
      p1 = s;
    } else {
      float s = col_ok ? v[r] : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) s += __shfl_xor(s, o, 64);
      p0 = 0.f;
      p1 = s;
    }
    if (lr == 0) {
      red[wn][trow][0] = p0;
      red[wn][trow][1] = p1;
    }
  }
  __syncthreads();
  if (threadIdx.x >= 64) return;
  const int trow = threadIdx.x;
  const int64_t row = tm0 + trow;
  if (row >= a.M) return;
  const int64_t tile = blockIdx.x;
  if (a.terminal == TERM_LAYERNORM) {
    Moments mo{0.f, 0.f, 0.f};
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const float c = (float)min<int64_t>(32, max<int64_t>(0, a.N - (tn0 + g * 32)));
      mo = mom_comb(mo, Moments{c, red[g][trow][0], red[g][trow][1]});
    }
    a.partial[(row * a.n_tiles + tile) * 2] = mo.mean;
    a.partial[(row * a.n_tiles + tile) * 2 + 1] = mo.m2;
  } else if (softmax) {
    const float mm = fmaxf(red[0][trow][0], red[1][trow][0]);
    float ss = 0.f;
    if (mm != -INFINITY) {
#pragma unroll
      for (int g = 0; g < 2; ++g)
        if (red[g][trow][0] != -INFINITY) ss += red[g][trow][1] * __expf(red[g][trow][0] - mm);
    }
    a.partial[(row * a.n_tiles + tile) * 2] = mm;
    a.partial[(row * a.n_tiles + tile) * 2 + 1] = ss;
  } else {
    a.partial[row * a.n_tiles + tile] = red[0][trow][1] + red[1][trow][1];
  }
}

}  // namespace

hipError_t launch_gemm_small(int dtype, const GemmArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.N + 63) / 64), (unsigned)((a.M + 63) / 64),
                  (unsigned)(a.batch * a.heads));
  if (dtype == MK_BF16)
    hipLaunchKernelGGL(gemm_small_kernel<bf16>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(gemm_small_kernel<float>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace mk
