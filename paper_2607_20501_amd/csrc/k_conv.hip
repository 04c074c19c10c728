// Implicit-GEMM convolution support on gfx950: layout passes around the MFMA
// GEMM kernel (k_gemm_mfma.hip, conv mode) and the global-average-pool
// finisher.
//
// The conv y[n,k,p,q] = sum_{c,r,s} x[n,c,p*st+r-pad,q*st+s-pad] w[k,c,r,s]
// (cross-correlation; a KernelBench L2-style conv + bias + ReLU + pool chain,
// MKEvolve Sec. 4 "Setup") is run as the GEMM
//   C[k][m] = sum_{(r,s,c)} W'[k][(r,s,c)] X'[m][(r,s,c)],  m = (n, p, q),
// where W' is w repacked to [K][R][S][C] and X' rows are gathered from a
// zero-padded NHWC copy of x: for a fixed (r, s) the C channels of a window
// element are contiguous, so every MFMA operand chunk is a 16-byte load and
// the padding needs no bounds checks.
#include "dev.hpp"

namespace mk {

namespace {

template <typename T>
struct KrscArgs {
  const T* w;
  T* wp;
  int64_t K, R, S;
};

// w [K][C][R][S] -> wp [K][R][S][C], done by the workgroups past the last
// image of the input-packing grid (one launch packs both operands): workgroup
// b of nb takes elements b*256*8 + t, stepping by 256, for 8 steps, and the
// rest in grid-stride order.
// Eight elements per pass: all eight loads are issued before the stores.
template <typename T>
__device__ __forceinline__ void pack_krsc_part(const T* __restrict__ w, T* __restrict__ wp,
                                               int64_t K, int64_t C, int64_t R, int64_t S,
                                               int64_t b, int64_t nb) {
  const int64_t total = K * R * S * C, step = nb * 256;
  for (int64_t i0 = b * 256 + threadIdx.x; i0 < total; i0 += 8 * step) {
    T v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      // 32-bit: the weight tensor has fewer than 2^31 elements
      const int64_t i = i0 + u * step;
      const uint32_t iu = (uint32_t)i, Cu = (uint32_t)C, Su = (uint32_t)S, Ru = (uint32_t)R;
      const uint32_t q1 = iu / Cu, c = iu - q1 * Cu, q2 = q1 / Su, s = q1 - q2 * Su;
      const uint32_t k = q2 / Ru, r = q2 - k * Ru;
      v[u] = i < total ? w[((k * Cu + c) * Ru + r) * Su + s] : T(0);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (i0 + u * step < total) wp[i0 + u * step] = v[u];
  }
}

// x [N][C][H][W] -> xp [N][H+2pad][W+2pad][C], zero border.
//
// Row form (W <= 64, rows of whole 16-byte chunks): one workgroup per (padded
// row hp, 64 channels, image).  Each (c, h) input row is one contiguous run
// of W values, read in 16-byte chunks; the tile is transposed in LDS and the
// padded row written as 16-byte channel chunks, border positions as zeros.
template <typename T>
__global__ __launch_bounds__(256) void pack_nhwc_rows_kernel(const T* x, T* xp, int64_t N,
                                                             int64_t C, int64_t H, int64_t W,
                                                             int64_t pad, KrscArgs<T> kw) {
  constexpr int E = 16 / (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) T tile[64][64 + E];   // [w][channel]
  if (blockIdx.z >= N) {
    const int64_t per = (int64_t)gridDim.x * gridDim.y;
    pack_krsc_part(kw.w, kw.wp, kw.K, C, kw.R, kw.S,
                   (blockIdx.z - N) * per + (int64_t)blockIdx.y * gridDim.x + blockIdx.x,
                   (gridDim.z - N) * per);
    return;
  }
  const int64_t Hp = H + 2 * pad, Wp = W + 2 * pad;
  const int64_t hp = blockIdx.x, c0 = (int64_t)blockIdx.y * 64, n = blockIdx.z;
  const int64_t h = hp - pad;
  const bool inside = h >= 0 && h < H;
  const int t = threadIdx.x;
  const int cpr = (int)(W / E);             // chunks per input row
  if (inside) {
    for (int idx = t; idx < 64 * cpr; idx += 256) {
      const int cl = idx / cpr, j = idx % cpr;
      const int64_t c = c0 + cl;
      if (c >= C) continue;
      const uint4 v = *(const uint4*)(x + ((n * C + c) * H + h) * W + j * E);
      const T* e = (const T*)&v;
#pragma unroll
      for (int k = 0; k < E; ++k) tile[j * E + k][cl] = e[k];
    }
  }
  __syncthreads();
  constexpr int CPP = 64 / E;               // channel chunks per position
  T* dst = xp + ((n * Hp + hp) * Wp) * C + c0;
  for (int idx = t; idx < (int)Wp * CPP; idx += 256) {
    const int64_t wp = idx / CPP;
    const int cc = idx % CPP;
    if (c0 + cc * E >= C) continue;
    const int64_t w = wp - pad;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (inside && w >= 0 && w < W) v = *(const uint4*)&tile[w][cc * E];
    *(uint4*)(dst + wp * C + cc * E) = v;
  }
}

// Block form (C and W multiples of the 16-byte chunk E): no LDS.  Thread g
// takes an E x E block (E channels at E consecutive positions of one input
// row): E 16-byte loads, one per channel row, transposed in registers into E
// 16-byte stores, one per position.  Channel blocks vary fastest across
// threads, so a wave's stores cover whole positions (all C channels
// contiguous).  Threads past the blocks write the zero border (one 16-byte
// chunk each).  The weights are packed by the first workgroups, which start
// first (their element-wise gathers are latency-bound).
template <typename T>
__global__ __launch_bounds__(256) void pack_nhwc_blocks_kernel(const T* x, T* xp, int N, int C,
                                                               int H, int W, int pad,
                                                               int64_t n_blk, int64_t n_zero,
                                                               int wg_data, KrscArgs<T> kw) {
  constexpr int E = 16 / (int)sizeof(T);
  const int wg_w = (int)gridDim.x - wg_data;   // weight workgroups come first
  if ((int)blockIdx.x < wg_w) {
    pack_krsc_part(kw.w, kw.wp, kw.K, C, kw.R, kw.S, (int64_t)blockIdx.x, (int64_t)wg_w);
    return;
  }
  const int CB = C / E, PB = W / E;
  const int64_t Hp = H + 2 * pad, Wp = W + 2 * pad;
  const int64_t g = (int64_t)(blockIdx.x - wg_w) * 256 + threadIdx.x;
  if (g < n_blk) {
    // 32-bit index arithmetic: block and chunk counts stay below 2^31
    uint32_t t = (uint32_t)g;
    const int cb = (int)(t % (uint32_t)CB);
    t /= (uint32_t)CB;
    const int pb = (int)(t % (uint32_t)PB);
    t /= (uint32_t)PB;
    const int h = (int)(t % (uint32_t)H);
    const int64_t n = t / (uint32_t)H;
    const T* src = x + ((n * C + (int64_t)cb * E) * H + h) * W + (int64_t)pb * E;
    union Chunk {
      uint4 u;
      T e[E];
    } v[E], o;
#pragma unroll
    for (int k = 0; k < E; ++k) v[k].u = *(const uint4*)(src + (int64_t)k * H * W);
    T* dst = xp + ((n * Hp + h + pad) * Wp + (int64_t)pb * E + pad) * C + (int64_t)cb * E;
#pragma unroll
    for (int q = 0; q < E; ++q) {
#pragma unroll
      for (int k = 0; k < E; ++k) o.e[k] = v[k].e[q];
      *(uint4*)(dst + (int64_t)q * C) = o.u;
    }
  } else if (g < n_blk + n_zero) {
    // border chunk: the 2*pad padded rows, then the 2*pad side positions of
    // each interior row, per image
    const uint32_t CBu = (uint32_t)CB, Wpu = (uint32_t)Wp, p2 = 2u * (uint32_t)pad;
    const uint32_t rows_part = p2 * Wpu * CBu;
    const uint32_t per_img = rows_part + (uint32_t)H * p2 * CBu;
    const uint32_t z = (uint32_t)(g - n_blk), n = z / per_img;
    uint32_t r = z - n * per_img, hp, wp;
    const int cb = (int)(r % CBu);
    if (r < rows_part) {
      const uint32_t row = r / (Wpu * CBu);
      hp = row < (uint32_t)pad ? row : (uint32_t)H + row;
      wp = (r / CBu) % Wpu;
    } else {
      r -= rows_part;
      const uint32_t sd = (r / CBu) % p2;
      hp = r / (p2 * CBu) + (uint32_t)pad;
      wp = sd < (uint32_t)pad ? sd : (uint32_t)W + sd;
    }
    *(uint4*)(xp + (((int64_t)n * Hp + hp) * Wp + wp) * C + (int64_t)cb * E) = make_uint4(0, 0, 0, 0);
  }
}

// General form: one workgroup per (64 padded positions, 64 channels, image),
// one element per thread on the read side.
template <typename T>
__global__ __launch_bounds__(256) void pack_nhwc_kernel(const T* x, T* xp, int64_t N, int64_t C,
                                                        int64_t H, int64_t W, int64_t pad,
                                                        KrscArgs<T> kw) {
  constexpr int E = 16 / (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) T tile[64][64 + E];
  if (blockIdx.z >= N) {
    const int64_t per = (int64_t)gridDim.x * gridDim.y;
    pack_krsc_part(kw.w, kw.wp, kw.K, C, kw.R, kw.S,
                   (blockIdx.z - N) * per + (int64_t)blockIdx.y * gridDim.x + blockIdx.x,
                   (gridDim.z - N) * per);
    return;
  }
  const int64_t Hp = H + 2 * pad, Wp = W + 2 * pad, HWp = Hp * Wp;
  const int64_t pos0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64, n = blockIdx.z;
  const int t = threadIdx.x;
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int idx = it * 256 + t, cl = idx >> 6, pl = idx & 63;
    const int64_t pos = pos0 + pl, c = c0 + cl;
    T v = T(0);
    if (pos < HWp && c < C) {
      const int64_t h = pos / Wp - pad, w = pos % Wp - pad;
      if (h >= 0 && h < H && w >= 0 && w < W) v = x[((n * C + c) * H + h) * W + w];
    }
    tile[pl][cl] = v;
  }
  __syncthreads();
  constexpr int CPP = 64 / E;
  for (int idx = t; idx < 64 * CPP; idx += 256) {
    const int pl = idx / CPP, ch = idx % CPP;
    const int64_t pos = pos0 + pl, c = c0 + ch * E;
    if (pos < HWp && c < C)
      *(uint4*)(xp + (n * HWp + pos) * C + c) = *(const uint4*)&tile[pl][ch * E];
  }
}

// out[n][k] = the pool of image n from the partials of the position tiles
// that cover it, combined in tile order (sum, or max for GMP), then finished
// (mean over PQ, or sign(S)|S|^(1/p) for LPPOOL).  Partial (tile t, slot)
// holds the reduction of the tile's positions in image (t*tile)/PQ + slot.
template <typename T>
__global__ void gap_finish_kernel(const float* partial, int64_t N, int64_t K, int64_t PQ,
                                  int64_t tile, int kind, float p, T* out) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= N * K) return;
  const int64_t n = i / K, k = i % K;
  const int64_t t0 = (n * PQ) / tile, t1 = ((n + 1) * PQ - 1) / tile;
  float s = pool_id(kind);
  // A tile that starts before image n holds it in its second slot.  The
  // loads are independent: unrolled, several are in flight at once.
#pragma unroll 4
  for (int64_t t = t0; t <= t1; ++t) {
    const int64_t slot = t * tile < n * PQ ? 1 : 0;
    s = pool_comb(kind, s, partial[(t * 2 + slot) * K + k]);
  }
  st<T>(out, i, pool_out(kind, p, s, (float)PQ));
}

}  // namespace

static int64_t esize(int dtype) { return dtype == MK_BF16 ? 2 : 4; }

int conv_mfma_limit(int dtype, const ConvArgs& a) {
  if (dtype != MK_BF16 && dtype != MK_F32) return MK_LIMIT_DTYPE;
  // A K slice (32 bf16 / 16 fp32 channels of one (r, s)) must not cross an
  // (r, s) boundary; 8 consecutive positions stay in one image.
  const int64_t bk = dtype == MK_BF16 ? 32 : 16;
  if (a.C % bk || (a.P * a.Q) % 8) return MK_LIMIT_SHAPE;
  // a tile spans at most two images
  if (a.gap && a.P * a.Q < conv_gemm_tile_n(dtype, a.C, a.P * a.Q, a.epi, a.gap, a.pool))
    return MK_LIMIT_SHAPE;
  const int64_t xp = a.N * (a.H + 2 * a.pad) * (a.W + 2 * a.pad) * a.C * esize(dtype);
  return xp < ((int64_t)1 << 31) && a.K * a.R * a.S * a.C * esize(dtype) < ((int64_t)1 << 31)
             ? MK_LIMIT_NONE
             : MK_LIMIT_RANGE;
}

bool conv_mfma_supported(int dtype, const ConvArgs& a) {
  return conv_mfma_limit(dtype, a) == MK_LIMIT_NONE;
}

ConvScratch conv_mfma_scratch(int dtype, const ConvArgs& a) {
  ConvScratch s{};
  auto al = [](int64_t b) { return (b + 255) / 256 * 256; };
  s.xp_bytes = al(a.N * (a.H + 2 * a.pad) * (a.W + 2 * a.pad) * a.C * esize(dtype));
  s.wp_bytes = al(a.K * a.R * a.S * a.C * esize(dtype));
  const int64_t tn = conv_gemm_tile_n(dtype, a.C, a.P * a.Q, a.epi, a.gap, a.pool);
  const int64_t tiles = (a.N * a.P * a.Q + tn - 1) / tn;
  s.partial_bytes = a.gap ? al(tiles * 2 * a.K * 4) : 0;
  return s;
}

// Workgroups for the weight repack appended to the input-packing grid: whole
// z slices of the grid, about one workgroup per 2048 weights.
static unsigned krsc_slices(const ConvArgs& a, int64_t per_slice) {
  const int64_t blocks = (a.K * a.R * a.S * a.C + 2047) / 2048;
  return (unsigned)std::max<int64_t>(1, (blocks + per_slice - 1) / per_slice);
}

template <typename T>
static void launch_pack_t(const ConvArgs& a, void* xp, void* wp, hipStream_t st) {
  constexpr int E = 16 / (int)sizeof(T);
  const int64_t Hp = a.H + 2 * a.pad, HWp = Hp * (a.W + 2 * a.pad);
  const unsigned cb = (unsigned)((a.C + 63) / 64);
  const KrscArgs<T> kw{(const T*)a.w, (T*)wp, a.K, a.R, a.S};
  if (a.C % E == 0 && a.W % E == 0 && (uintptr_t)a.x % 16 == 0) {
    const int64_t n_blk = a.N * a.H * (a.W / E) * (a.C / E);
    const int64_t Wp = a.W + 2 * a.pad;
    const int64_t n_zero = a.N * (2 * a.pad * Wp + a.H * 2 * a.pad) * (a.C / E);
    const int64_t wg_data = (n_blk + n_zero + 255) / 256;
    const unsigned wg_w = krsc_slices(a, 1);
    hipLaunchKernelGGL(pack_nhwc_blocks_kernel<T>, dim3((unsigned)(wg_data + wg_w)), dim3(256), 0,
                       st, (const T*)a.x, (T*)xp, (int)a.N, (int)a.C, (int)a.H, (int)a.W,
                       (int)a.pad, n_blk, n_zero, (int)wg_data, kw);
  } else if (a.W <= 64 && a.W % E == 0 && (uintptr_t)a.x % 16 == 0) {
    const unsigned z = (unsigned)a.N + krsc_slices(a, Hp * cb);
    hipLaunchKernelGGL(pack_nhwc_rows_kernel<T>, dim3((unsigned)Hp, cb, z), dim3(256), 0, st,
                       (const T*)a.x, (T*)xp, a.N, a.C, a.H, a.W, a.pad, kw);
  } else {
    const unsigned gx = (unsigned)((HWp + 63) / 64);
    const unsigned z = (unsigned)a.N + krsc_slices(a, (int64_t)gx * cb);
    hipLaunchKernelGGL(pack_nhwc_kernel<T>, dim3(gx, cb, z), dim3(256), 0, st, (const T*)a.x,
                       (T*)xp, a.N, a.C, a.H, a.W, a.pad, kw);
  }
}

hipError_t launch_conv_pack(int dtype, const ConvArgs& a, void* xp, void* wp, hipStream_t st) {
  if (dtype == MK_BF16)
    launch_pack_t<bf16>(a, xp, wp, st);
  else
    launch_pack_t<float>(a, xp, wp, st);
  return hipGetLastError();
}

GemmArgs conv_gemm_args(const ConvArgs& a, const void* xp, const void* wp, float* partial) {
  GemmArgs g{};
  g.A = wp;
  g.B = xp;
  g.C = a.y;
  g.M = a.K;
  g.N = a.N * a.P * a.Q;
  g.K = a.R * a.S * a.C;
  g.lda = g.K;
  g.ldb = g.K;
  g.ldc = g.N;
  g.batch = g.heads = 1;
  g.layout = 0;
  g.alpha = 1.f;
  g.epi = a.epi;
  g.terminal = a.gap ? TERM_GAP : TERM_NONE;
  g.pool = a.pool;
  g.pool_p = a.pool_p;
  g.partial = partial;
  // (n_tiles is not read in conv mode: partials are indexed by tile.)
  g.n_tiles = 0;
  g.conv = 1;
  g.cv_C = a.C;
  g.cv_Hp = a.H + 2 * a.pad;
  g.cv_Wp = a.W + 2 * a.pad;
  g.cv_P = a.P;
  g.cv_Q = a.Q;
  g.cv_S = a.S;
  g.cv_stride = a.stride;
  return g;
}

hipError_t launch_gap_finish(int dtype, const ConvArgs& a, const float* partial, hipStream_t st) {
  const int64_t total = a.N * a.K;
  const int64_t tn = conv_gemm_tile_n(dtype, a.C, a.P * a.Q, a.epi, a.gap, a.pool);
  // One wave per workgroup: N*K outputs are few (16384 for 64 images of 256
  // channels), so small workgroups spread them over every CU.
  const dim3 grid((unsigned)((total + 63) / 64));
  if (dtype == MK_BF16)
    hipLaunchKernelGGL(gap_finish_kernel<bf16>, grid, dim3(64), 0, st, partial, a.N, a.K,
                       a.P * a.Q, tn, (int)a.pool, a.pool_p, (bf16*)a.y);
  else
    hipLaunchKernelGGL(gap_finish_kernel<float>, grid, dim3(64), 0, st, partial, a.N, a.K,
                       a.P * a.Q, tn, (int)a.pool, a.pool_p, (float*)a.y);
  return hipGetLastError();
}

}  // namespace mk
