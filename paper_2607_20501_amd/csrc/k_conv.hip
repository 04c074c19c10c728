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

// x [N][C][H][W] -> xp [N][H+2pad][W+2pad][C], zero border.  One workgroup per
// (64 padded positions, 64 channels, image); the tile is transposed in LDS so
// both the reads (along positions) and the 16-byte writes (along channels)
// are coalesced.
__global__ __launch_bounds__(256) void pack_nhwc_kernel(const bf16* x, bf16* xp, int64_t C,
                                                        int64_t H, int64_t W, int64_t pad) {
  __shared__ bf16 tile[64][72];
  const int64_t Hp = H + 2 * pad, Wp = W + 2 * pad, HWp = Hp * Wp;
  const int64_t pos0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64, n = blockIdx.z;
  const int t = threadIdx.x;
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int idx = it * 256 + t, cl = idx >> 6, pl = idx & 63;
    const int64_t pos = pos0 + pl, c = c0 + cl;
    bf16 v = 0;
    if (pos < HWp && c < C) {
      const int64_t h = pos / Wp - pad, w = pos % Wp - pad;
      if (h >= 0 && h < H && w >= 0 && w < W) v = x[((n * C + c) * H + h) * W + w];
    }
    tile[pl][cl] = v;
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int idx = it * 256 + t, pl = idx >> 3, ch = idx & 7;
    const int64_t pos = pos0 + pl, c = c0 + ch * 8;
    if (pos < HWp && c < C)
      *(uint4*)(xp + (n * HWp + pos) * C + c) = *(const uint4*)&tile[pl][ch * 8];
  }
}

// w [K][C][R][S] -> wp [K][R][S][C].
__global__ void pack_krsc_kernel(const bf16* w, bf16* wp, int64_t K, int64_t C, int64_t R,
                                 int64_t S) {
  const int64_t total = K * R * S * C;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = i % C, s = (i / C) % S, r = (i / (C * S)) % R, k = i / (C * S * R);
    wp[i] = w[((k * C + c) * R + r) * S + s];
  }
}

// out[n][k] = (sum of the GAP partials of the position tiles that cover image
// n, in tile order) / PQ.  Partial (tile t, slot) holds the column sums of the
// tile's positions in image (t*256)/PQ + slot.
__global__ void gap_finish_kernel(const float* partial, int64_t N, int64_t K, int64_t PQ,
                                  int64_t tile, bf16* out) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= N * K) return;
  const int64_t n = i / K, k = i % K;
  const int64_t t0 = (n * PQ) / tile, t1 = ((n + 1) * PQ - 1) / tile;
  float s = 0.f;
  for (int64_t t = t0; t <= t1; ++t) {
    const int64_t slot = n - (t * tile) / PQ;
    s += partial[(t * 2 + slot) * K + k];
  }
  out[i] = f2bf(s / (float)PQ);
}

}  // namespace

bool conv_mfma_supported(int dtype, const ConvArgs& a) {
  if (dtype != MK_BF16 || a.C % 32 || (a.P * a.Q) % 8) return false;
  if (a.gap && a.P * a.Q < kConvTileN) return false;   // a tile spans at most two images
  const int64_t xp = a.N * (a.H + 2 * a.pad) * (a.W + 2 * a.pad) * a.C * 2;
  return xp < ((int64_t)1 << 31) && a.K * a.R * a.S * a.C * 2 < ((int64_t)1 << 31);
}

ConvScratch conv_mfma_scratch(const ConvArgs& a) {
  ConvScratch s{};
  auto al = [](int64_t b) { return (b + 255) / 256 * 256; };
  s.xp_bytes = al(a.N * (a.H + 2 * a.pad) * (a.W + 2 * a.pad) * a.C * 2);
  s.wp_bytes = al(a.K * a.R * a.S * a.C * 2);
  const int64_t tiles = (a.N * a.P * a.Q + kConvTileN - 1) / kConvTileN;
  s.partial_bytes = a.gap ? al(tiles * 2 * a.K * 4) : 0;
  return s;
}

hipError_t launch_pack_nhwc(const ConvArgs& a, void* xp, hipStream_t st) {
  const int64_t HWp = (a.H + 2 * a.pad) * (a.W + 2 * a.pad);
  dim3 grid((unsigned)((HWp + 63) / 64), (unsigned)((a.C + 63) / 64), (unsigned)a.N);
  hipLaunchKernelGGL(pack_nhwc_kernel, grid, dim3(256), 0, st, (const bf16*)a.x, (bf16*)xp, a.C,
                     a.H, a.W, a.pad);
  return hipGetLastError();
}

hipError_t launch_pack_krsc(const ConvArgs& a, void* wp, hipStream_t st) {
  const int64_t total = a.K * a.R * a.S * a.C;
  const unsigned g = (unsigned)std::min<int64_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(pack_krsc_kernel, dim3(g), dim3(256), 0, st, (const bf16*)a.w, (bf16*)wp,
                     a.K, a.C, a.R, a.S);
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
  g.partial = partial;
  g.n_tiles = (g.N + kConvTileN - 1) / kConvTileN;
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

hipError_t launch_gap_finish(const ConvArgs& a, const float* partial, hipStream_t st) {
  const int64_t total = a.N * a.K;
  hipLaunchKernelGGL(gap_finish_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                     partial, a.N, a.K, a.P * a.Q, kConvTileN, (bf16*)a.y);
  return hipGetLastError();
}

}  // namespace mk
