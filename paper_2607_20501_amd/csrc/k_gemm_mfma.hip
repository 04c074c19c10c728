// bf16 / fp32 GEMM with fused epilogue on gfx950 matrix cores.
//
//   C[z][m, n] = chain(alpha * sum_k A[z][m, k] B[z](k, n))     (fp32 accumulate)
//
// The contraction is the dense GEMM of a Linear layer / conv / attention
// product (MKEvolve App. H.2 linear kernels; the fusion guidance of App. I.1:
// GEMM followed by bias, activations, scaling and the residual add in one
// kernel, never materialising the intermediate).  A terminal row reduction
// that needs a full row (softmax, row-sum, post-LN LayerNorm) is split at the
// column tile: the epilogue emits per-(row, tile) partials and a finisher
// combines them (App. I.1: "may need split at softmax due to reduction").
//
// Design for CDNA4:
//  * Plain GEMMs: a 256 x 256 output tile per workgroup, eight waves (two per
//    SIMD) in a 2 x 4 arrangement, each owning 128 x 64 = 4 x 2 tiles of
//    v_mfma_f32_32x32x16_bf16 (fp32: v_mfma_f32_32x32x2_f32), 128 fp32
//    accumulators per lane.  Conv GEMMs: 256 x 128 tiles, four waves, two
//    workgroups per CU.
//  * The four-wave form (bf16 chains without a terminal, K a multiple of 64)
//    gives each wave a 128 x 128 quarter as 8 x 8 tiles of
//    v_mfma_f32_16x16x32_bf16.  Same flops per cycle as the 32 x 32 x 16
//    instruction, but it moves a quarter of the accumulator bytes per
//    multiply-add (4 registers per 16 x 16 x 32 against 16 per 32 x 32 x 16):
//    on random operands, with every CU busy, a stream of them holds a clock
//    about 12% higher under the power limit (2.15 against 1.91 GHz).
//  * Operands move HBM -> LDS with buffer_load ... lds (no register staging).
//    An LDS row holds one K stage of one operand row: 128 bytes for plain
//    GEMMs (64 bf16 / 32 fp32; eight 16-byte chunks), so every 8 lanes of a
//    load read one whole 128-byte line and the L2 sees 128-byte requests
//    (64-byte rows issue twice the requests and the operand stream, not the
//    matrix cores, bounds the loop).  Conv GEMMs keep 64-byte rows (a slice
//    must not cross a filter tap at C = 128 bf16 ... and two workgroups fit).
//    Out-of-range lanes read zeros through the buffer descriptor's range
//    check (ragged M / N / K).
//  * Plain GEMMs double-buffer two 64 KB stages; within a stage the MFMA
//    fragments are read one 16-deep sub-step ahead of the MFMAs that use them,
//    and the one barrier per stage sits before its last sub-step, where the
//    next stage is known landed and the freed slot is refilled.
//  * LDS chunk c of row r sits at chunk c ^ swz(r), so the lanes served together
//    by a 128-bit fragment read hit distinct banks; each lane's global address
//    is chosen so that the lane-ordered LDS write lands in that layout.
//  * MFMA operands must be K-contiguous; a weight given as [K, N] is first
//    transposed to [N, K] in scratch by a tiled transpose launch.
//  * Tiles are remapped so that consecutive workgroups of one XCD (the
//    hardware deals workgroups round-robin over the 8 XCDs) take a compact
//    group of tiles and share operand slices in that XCD's L2.
//  * The epilogue stages 16-row slabs of accumulators through LDS so each
//    lane finishes 8 consecutive columns and writes them with one 16-byte
//    store.

#include <algorithm>
#include <type_traits>

#include "dev.hpp"

namespace mk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

namespace {

// MfmaType<T>: the MFMA fragment (one 16-byte chunk: 8 bf16 / 4 fp32
// consecutive k of one row / column).
template <typename T>
struct MfmaType;
template <>
struct MfmaType<bf16> {
  typedef bf16x8 frag;
};
template <>
struct MfmaType<float> {
  typedef f32x4 frag;
};

constexpr int BM = 256;
// Epilogue signatures with straight-line code (kSigGeneric interprets any
// chain step by step; the others are compiled for one chain and terminal).
constexpr int kSigGeneric = 0;
constexpr int kSigConvBiasReluGap = 1;   // conv: channel bias, ReLU, global average pool
constexpr int kSigNone = 2;              // no chain, no terminal
constexpr int kSigGeluErf = 3;           // exact GELU
constexpr int kSigAdd = 4;               // residual add (operand laid out as C)
constexpr int kSigBiasGeluTanhScaleSoftmax = 5;   // bias, tanh GELU, scale; softmax partials
constexpr int kSigBiasGeluTanhScale = 6;          // bias, tanh GELU, scale
constexpr int kSigBias = 7;                       // column bias

// The compiled chains without a terminal (stored through a buffer resource).
constexpr bool sig_plain(int sig) {
  return sig == kSigNone || sig == kSigGeluErf || sig == kSigAdd || sig == kSigBiasGeluTanhScale ||
         sig == kSigBias;
}
// Chains that start with a column bias (alpha * acc + bias as one FMA).
constexpr bool sig_bias(int sig) {
  return sig == kSigBiasGeluTanhScaleSoftmax || sig == kSigBiasGeluTanhScale || sig == kSigBias;
}

// Terminal of a signature (-1: read at run time).
constexpr int sig_terminal(int sig) {
  return sig == kSigBiasGeluTanhScaleSoftmax ? TERM_SOFTMAX : sig_plain(sig) ? TERM_NONE : -1;
}
constexpr int kGroupM = 8;                        // tile rows per locality group
constexpr int kXcds = 8;

// Chunk swizzles: 64-byte rows (4 chunks) and 128-byte rows (8 chunks); the 8
// consecutive rows read together by a 128-bit fragment read map to distinct
// physical chunks.
template <int RB>
__device__ __forceinline__ int swz(int r) {
  if constexpr (RB == 64)
    return ((r >> 1) ^ (r >> 3)) & 3;
  else
    return (r ^ (r >> 3)) & 7;
}

// Byte offset of logical chunk c of row r in an operand stage of RB-byte rows.
template <int RB>
__device__ __forceinline__ int lds_off(int r, int c) {
  return r * RB + ((c ^ swz<RB>(r)) << 4);
}

struct TileCoord {
  int tm, tn;
};

// Logical tile of this workgroup: XCD-aware remap, then grouped (column-major
// within groups of kGroupM tile rows) order.
__device__ __forceinline__ TileCoord tile_of(int bid, int tiles_m, int tiles_n) {
  const int total = tiles_m * tiles_n;
  if (total % kXcds == 0) bid = (bid % kXcds) * (total / kXcds) + bid / kXcds;
  const int per_group = kGroupM * tiles_n;
  const int g = bid / per_group;
  const int first_m = g * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int r = bid % per_group;
  return {first_m + r % gsize, r / gsize};
}

// Work item of a persistent walk: a tile, or one row sub-tile of a tile.
struct Item {
  TileCoord tc;
  int sub;   // row sub-tile, -1 for the whole tile
};

// Tail split of a persistent walk over `tiles` tiles by G workgroups: the
// tiles past the last whole round (all of them when tiles < G) are cut along
// M into 8 (or 4) row sub-tiles when that many of each fit in one round, so
// the last round takes a fraction of a tile's time.  1: no split.
__host__ __device__ inline int tail_split(int tiles, int G) {
  const int rem = tiles % G;
  return rem == 0 ? 1 : rem * 8 <= G ? 8 : rem * 4 <= G ? 4 : 1;
}

// Global operand access through buffer resources: a lane whose element lies
// outside the operand gets an offset beyond the descriptor's range and reads
// zeros, so ragged M / N / K tails need no branches.
constexpr uint32_t kOob = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

typedef __attribute__((address_space(3))) void lds_void;

// Direct HBM -> LDS loads of one operand stage (ROWS rows of RB bytes, CPR =
// RB/16 chunks per row).  LDS chunk p of the stage is row p/CPR, physical
// chunk p%CPR, whose logical chunk is (p%CPR) ^ swz(row): the CPR lanes of a
// row read one contiguous RB-byte piece of it in a permuted order.
template <int WAVES, int ROWS, typename T, int RB>
struct SliceLoader {
  static constexpr int E = 16 / (int)sizeof(T);          // elements per chunk
  static constexpr int CPR = RB / 16;                    // chunks per row
  static constexpr int LQ = ROWS * CPR / (64 * WAVES);   // loads per thread per stage
  static_assert(LQ * 64 * WAVES == ROWS * CPR, "stage must split evenly over the loads");
  // A lane's successive loads are RSTEP = 64*WAVES/CPR rows apart.  When that
  // is a multiple of 64 both swizzles repeat and one logical chunk serves all
  // of them; four waves with 128-byte rows (RSTEP 32) alternate between two
  // chunks, which only the whole-stage form (issue_full: K a multiple of the
  // stage depth, so no lane needs a K bound) accepts.
  static constexpr int RSTEP = 64 * WAVES / CPR;
  static constexpr bool kRepeat = RSTEP % 64 == 0;
  static_assert(kRepeat || (RB == 128 && RSTEP == 32), "unsupported load geometry");
  __amdgpu_buffer_rsrc_t src;
  uint32_t voff[LQ];   // byte offset at k0 = 0, kOob if the row is out of range
  uint32_t range;      // bytes covered by src
  int lchunk;          // logical 16-byte chunk of this lane's loads (of load 0)
  int wid;             // this wave's index (wave-uniform)

  __device__ __forceinline__ int first_row() const {
    return ((threadIdx.x >> 6) * 64 + (threadIdx.x & 63)) / CPR;
  }
  __device__ __forceinline__ void set_chunk() {
    const int p = (threadIdx.x >> 6) * 64 + (threadIdx.x & 63);
    lchunk = (p % CPR) ^ swz<RB>(p / CPR);
    wid = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  }
  // logical chunk of load q (its row is first_row() + q * RSTEP)
  __device__ __forceinline__ int chunk_of(int q) const {
    if constexpr (kRepeat) return lchunk;
    const int p = (threadIdx.x >> 6) * 64 + (threadIdx.x & 63);
    return (p % CPR) ^ swz<RB>(p / CPR + q * RSTEP);
  }

  __device__ __forceinline__ void init(const T* base, int64_t rows, int64_t ld, int64_t r0) {
    range = (uint32_t)(rows * ld * (int64_t)sizeof(T));
    src = make_rsrc(base, rows * ld * (int64_t)sizeof(T));
    set_chunk();
#pragma unroll
    for (int q = 0; q < LQ; ++q) {
      const int64_t g = r0 + first_row() + q * RSTEP;
      voff[q] = g < rows ? (uint32_t)(g * ld * (int64_t)sizeof(T) + chunk_of(q) * 16) : kOob;
    }
  }

  // Loads Q0 .. Q1-1 of a whole stage into `dst` (this operand's slot), with
  // the stage's uniform byte offset along K: every lane is inside K, and a
  // stage past the last one passes soff = range, which puts every lane out of
  // the descriptor's range (zeros; voff < 2^31 + 2^31 never wraps since the
  // range is below 2 GB).
  template <int Q0, int Q1>
  __device__ __forceinline__ void issue_full(char* dst, uint32_t soff) const {
#pragma unroll
    for (int q = Q0; q < Q1; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * WAVES + wid) * 1024),
                                               16, (int)voff[q], (int)soff, 0, 0);
  }

  // Load q of a whole stage (as issue_full).
  __device__ __forceinline__ void issue_q(char* dst, uint32_t soff, int q) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * WAVES + wid) * 1024), 16,
                                             (int)voff[q], (int)soff, 0, 0);
  }

  // Rows gathered from arbitrary byte offsets (implicit-GEMM conv: output
  // position m -> its window origin in the padded NHWC input).
  template <typename RowOff>
  __device__ __forceinline__ void init_gather(const T* base, int64_t bytes, int64_t rows,
                                              int64_t r0, RowOff rowoff) {
    static_assert(kRepeat, "gathered rows need one chunk per lane");
    range = (uint32_t)bytes;
    src = make_rsrc(base, bytes);
    set_chunk();
#pragma unroll
    for (int q = 0; q < LQ; ++q) {
      const int64_t g = r0 + first_row() + q * RSTEP;
      voff[q] = g < rows ? (uint32_t)(rowoff(g) + lchunk * 16) : kOob;
    }
  }

  // Issue the loads of the stage starting at k0 into `dst` (this operand's
  // part of a stage); `soff` is the stage's byte offset along K.  For load q
  // of wave w, lane i fills LDS chunk p = (q*WAVES + w)*64 + i, i.e. row
  // p/CPR, physical chunk p%CPR.
  __device__ __forceinline__ void issue(char* dst, int64_t k0, int64_t K, uint32_t soff) const {
    static_assert(kRepeat, "a K bound per lane needs one chunk per lane");
    const int w = threadIdx.x >> 6;
    const bool in_k = lchunk * E < K - k0;
#pragma unroll
    for (int q = 0; q < LQ; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * WAVES + w) * 1024),
                                               16, (int)(in_k ? voff[q] : kOob), (int)soff, 0,
                                               0);
  }
  __device__ __forceinline__ void issue(char* dst, int64_t k0, int64_t K) const {
    issue(dst, k0, K, (uint32_t)(k0 * (int64_t)sizeof(T)));
  }
  // Loads Q0 .. Q1-1 of the stage (plain rows): a stage's loads may be spread.
  template <int Q0, int Q1>
  __device__ __forceinline__ void issue_part(char* dst, int64_t k0, int64_t K) const {
    static_assert(kRepeat, "a K bound per lane needs one chunk per lane");
    const int w = threadIdx.x >> 6;
    const bool in_k = lchunk * E < K - k0;
    const uint32_t soff = (uint32_t)(k0 * (int64_t)sizeof(T));
#pragma unroll
    for (int q = Q0; q < Q1; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * WAVES + w) * 1024),
                                               16, (int)(in_k ? voff[q] : kOob), (int)soff, 0,
                                               0);
  }
};

// Direct HBM -> LDS loads of one stage of a [K, N] bf16 operand for the
// four-wave form: 64 k-rows of the tile's 256 columns, 512 bytes per row.
// Row r of the stage sits at r * 512 in the slot with its 16-byte chunks
// XOR-swizzled by 2 g(r), g(r) = (r & 3) | ((r >> 3) & 1) << 2: the 8 rows
// that half a wave's transposing fragment reads touch together (rows 0..3
// and 8..11 of a 16-row group) then lie in 8 distinct 32-byte bank windows.
// Load q of wave w fills rows 8q + 2w and 8q + 2w + 1 (lanes 0..31, 32..63):
// lane i writes LDS chunk i % 32 of its row, the row's logical chunk
// (i % 32) ^ 2 g(row).  Columns past N read zeros (offset out of range); K
// is a multiple of the stage depth.
struct KNLoader {
  __amdgpu_buffer_rsrc_t src;
  uint32_t voff[8];   // byte offset of load q at k0 = 0 (kOob past N)
  uint32_t range;     // bytes covered by src
  uint32_t kstep;     // bytes per stage along K (64 rows)
  int wid;

  __device__ __forceinline__ void init(const bf16* base, int64_t K, int64_t ld, int64_t n0,
                                       int64_t N) {
    range = (uint32_t)(K * ld * 2);
    kstep = (uint32_t)(64 * ld * 2);
    src = make_rsrc(base, K * ld * 2);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    wid = __builtin_amdgcn_readfirstlane(w);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = 8 * q + 2 * w + (lane >> 5);
      const int g = (r & 3) | (((r >> 3) & 1) << 2);
      const int64_t n = n0 + (int64_t)(((lane & 31) ^ (2 * g)) * 8);
      voff[q] = n < N ? (uint32_t)(r * ld * 2 + n * 2) : kOob;
    }
  }
  template <int Q0, int Q1>
  __device__ __forceinline__ void issue_full(char* dst, uint32_t soff) const {
#pragma unroll
    for (int q = Q0; q < Q1; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * 4 + wid) * 1024), 16,
                                               (int)voff[q], (int)soff, 0, 0);
  }
  __device__ __forceinline__ void issue_q(char* dst, uint32_t soff, int q) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * 4 + wid) * 1024), 16,
                                             (int)voff[q], (int)soff, 0, 0);
  }
};

// MFMA operand fragments of one sub-step (chunks 2kk, 2kk+1) for this wave:
// 4 row tiles of A and NJ column tiles of B; lane (lr, lh) holds the 16-byte
// chunk 2kk+lh of row / column lr of each tile.
template <int NJ, typename T>
struct Frags {
  typename MfmaType<T>::frag a[4], b[NJ];
};

template <int NJ, typename T, int RB>
__device__ __forceinline__ void load_frags(const char* la, const char* lb, int kk, int rowbase,
                                           int colbase, int lr, int lh, Frags<NJ, T>& f) {
  typedef typename MfmaType<T>::frag F;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    f.a[i] = *(const F*)(la + lds_off<RB>(rowbase + i * 32 + lr, kk * 2 + lh));
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    f.b[j] = *(const F*)(lb + lds_off<RB>(colbase + j * 32 + lr, kk * 2 + lh));
}

// bf16: one 32x32x16 MFMA per tile pair (the lane's 8 k values are the
// instruction's k = 8*lh .. 8*lh+7).  fp32: the lane's 4 k values feed four
// 32x32x2 MFMAs, instruction t taking k = 4*lh + t of the chunk pair; A and B
// use the same assignment, so the sum over k is unchanged.
// TR: operands swapped, so tile (i, j) accumulates the transpose (a lane
// holds one row of A's tile i and 16 of B's tile j).
template <int NJ, typename T, bool TR = false>
__device__ __forceinline__ void mfma_step(const Frags<NJ, T>& f, f32x16 (&acc)[4][NJ]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const auto& x = TR ? f.b[j] : f.a[i];
      const auto& y = TR ? f.a[i] : f.b[j];
      if constexpr (sizeof(T) == 2) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, acc[i][j], 0, 0, 0);
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(x[t], y[t], acc[i][j], 0, 0, 0);
      }
    }
}

// One 32 x 32 tile update from a sub-step's fragment pair (as in mfma_step).
template <typename T>
__device__ __forceinline__ f32x16 mfma1(const typename MfmaType<T>::frag& x,
                                        const typename MfmaType<T>::frag& y, f32x16 c) {
  if constexpr (sizeof(T) == 2) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c, 0, 0, 0);
  } else {
#pragma unroll
    for (int t = 0; t < 4; ++t) c = __builtin_amdgcn_mfma_f32_32x32x2f32(x[t], y[t], c, 0, 0, 0);
    return c;
  }
}

// 16 x 16 x 32 MFMA with the accumulator tied to the result in AGPRs (the
// builtin leaves the compiler free to put them apart, and it then copies
// accumulators between every use).  The compiler does not see it as an MFMA:
// the code keeps the distances to readers of the result itself.
__device__ __forceinline__ void mfma16(f32x4& c, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

// vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// Epilogue staging.  In the 32 x 32 MFMA layout a lane holds, for column
// j*32 + lr, the four consecutive rows (r/4)*8 + lh*4 + 0..3 in acc[r .. r+3]
// (r a multiple of 4).  A wave's 32-row slab is stored as [8 row groups of 4
// rows][kSlabU 16-byte units], unit (g, col) holding rows 4g .. 4g+3 of that
// column, so each of those quads is one 16-byte write.  kSlabU = 64 + 1: the
// 8 lanes reading one column unit of 8 consecutive row groups hit distinct
// bank groups.
constexpr int kSlabU = 65;

// Copy acc[I][J0], acc[I][J0+1] (rows I*32 .. I*32+31 of 64 of this wave's
// columns) into the slab.
template <int I, int NJ, int J0 = 0>
__device__ __forceinline__ void stage_slab(const f32x16 (&acc)[4][NJ], float* slab, int lh,
                                           int lr) {
  static_assert(J0 + 2 <= NJ, "a slab holds two column tiles");
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int g = 2 * r4 + lh;
      *(f32x4*)(slab + (g * kSlabU + j * 32 + lr) * 4) =
          f32x4{acc[I][J0 + j][4 * r4], acc[I][J0 + j][4 * r4 + 1], acc[I][J0 + j][4 * r4 + 2],
                acc[I][J0 + j][4 * r4 + 3]};
    }
}

// The same slab from the four-wave form's 16 x 16 tiles: acc16[i][j] holds,
// for column j*16 + l16, the rows i*16 + lq*4 + 0..3 (l16 = lane % 16,
// lq = lane / 16), which is one 16-byte quad of the slab.
template <int I, int J0>
__device__ __forceinline__ void stage_slab16(const f32x4 (&acc16)[8][8], float* slab, int lq,
                                             int l16) {
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      *(f32x4*)(slab + ((4 * h + lq) * kSlabU + jj * 16 + l16) * 4) = acc16[2 * I + h][2 * J0 + jj];
}

// Channel-bias values of one row tile for this lane: rows rb + (r/4)*8 +
// lh*4 + r%4, r = 0..15, of p (zero at rows rb + mrem and beyond).
template <typename T>
__device__ __forceinline__ void load_row_bias(const T* p, int mrem, int lh, float (&b)[16]) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = (r >> 2) * 8 + lh * 4 + (r & 3);
    b[r] = row < mrem ? ld<T>(p, row) : 0.f;
  }
}

// The conv chain on the 16 values of one accumulator tile: rows rb + (r/4)*8
// + lh*4 + r%4 (mrem = M - rb), at position col of image img.  One copy of
// each step's code: the loop over the chain's steps is not unrolled.
template <typename T>
__device__ __forceinline__ void conv_chain16(const GemmArgs& a, float (&v)[16], int64_t rb,
                                             int mrem, int lh, const float (&bc)[16], int pre,
                                             bool ok, int64_t col, int64_t img, int64_t PQ) {
#pragma unroll 1
  for (int s = 0; s < a.epi.n; ++s) {
    const T* p = (const T*)a.epi.ptr[s];
    switch (a.epi.code[s]) {
      case EPI_BIAS_CH:
        if (s == pre) {
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] += bc[r];
        } else {
          float b[16];
          load_row_bias<T>(p + rb, mrem, lh, b);
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] += b[r];
        }
        break;
      case EPI_RELU:
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = fmaxf(v[r], 0.0f);
        break;
      case EPI_GELU_ERF:
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = gelu_erf(v[r]);
        break;
      case EPI_GELU_TANH:
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = gelu_tanh(v[r]);
        break;
      case EPI_GELU_SIGMOID:
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = v[r] / (1.0f + __expf(-1.702f * v[r]));
        break;
      case EPI_SCALE: {
        const float sc = a.epi.s[s];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] *= sc;
        break;
      }
      case EPI_ADD: {   // NCHW operand: (image, channel, position in image)
        const T* q = p + (img * a.M + rb) * PQ + (col - img * PQ);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = (r >> 2) * 8 + lh * 4 + (r & 3);
          if (ok && row < mrem) v[r] += ld<T>(q, (int64_t)row * PQ);
        }
        break;
      }
      default:
        break;
    }
  }
}

// Global pooling of a conv tile straight from the accumulators, without
// staging them in LDS.  Rows are channels, columns positions; lane (lr, lh)
// holds, of row tile i, rows rowbase + i*32 + (r/4)*8 + lh*4 + r%4 (r = 0..15)
// at columns colbase + j*32 + lr.  Per row tile: the chain on every value,
// the pool input, its combination over the lane's NJ columns into the slot of
// the column's image (a tile spans at most two images), and a halving
// butterfly over the 32 lanes lr: at the step across lane bit b a lane keeps
// the half of its values selected by that bit and adds in the partner's copy
// of it, so after bits 4..0 lane lr holds value lr = slot*16 + r.  Results go
// to red[wn][row][slot].  rbias: the tile's values of chain step `pre` (a
// channel bias) in LDS, by tile row.  kBiasReluSum: the chain is exactly
// (channel bias, ReLU) and the pool a sum (GAP), in straight-line code; the
// general form interprets the chain and the pool kind, which costs several
// times the time of the rest of the epilogue.
template <typename T, int NJ, bool kBiasReluSum>
__device__ __forceinline__ void gap_from_acc(const GemmArgs& a, const f32x16 (&acc)[4][NJ],
                                             int64_t m0, int64_t n0, int rowbase, int colbase,
                                             int wn, int lr, int lh, int pre,
                                             const float* rbias, float* red, int ni = 4) {
  const int kind = a.pool;
  const float pp = a.pool_p, idv = pool_id(kind);
  const int64_t PQ = a.cv_P * a.cv_Q;
  const int64_t img0 = n0 / PQ;
  // columns of this lane relative to the tile, against N and the image bound
  const int c_end = (int)min<int64_t>(a.N - n0, 1 << 30);
  const int c_bnd = (int)min<int64_t>((img0 + 1) * PQ - n0, 1 << 30);
  if constexpr (kBiasReluSum) {
    // Transposed tiles: lane lr of tile (i, j) holds channel rowbase+i*32+lr
    // at the 16 positions j*32 + (r/4)*8 + lh*4 + r%4 of the wave's columns,
    // so each sum is lane-local; the two lane halves then combine.  Waves
    // whose columns are all in range and in one image take the plain sum.
    const float alpha = a.alpha;
    const bool plain = colbase + NJ * 32 <= c_end && colbase + NJ * 32 <= c_bnd;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i >= ni) break;
      const int lrow = rowbase + i * 32 + lr;
      const float b = pre >= 0 ? rbias[lrow] : 0.f;
      float x0 = 0.f, x1 = 0.f;
      if (plain) {
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) x0 += fmaxf(fmaf(acc[i][j][r], alpha, b), 0.f);
      } else {
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int p = colbase + j * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
            const float c = p < c_end ? fmaxf(fmaf(acc[i][j][r], alpha, b), 0.f) : 0.f;
            x0 += p < c_bnd ? c : 0.f;
            x1 += p < c_bnd ? 0.f : c;
          }
      }
      x0 += lane_xor<32>(x0);
      x1 += lane_xor<32>(x1);
      if (lh == 0) {
        red[(wn * 256 + lrow) * 2] = x0;
        red[(wn * 256 + lrow) * 2 + 1] = x1;
      }
    }
    return;
  }
#pragma unroll 1
  for (int i = 0; i < ni; ++i) {
    const int64_t rb = m0 + rowbase + i * 32;
    const int mrem = (int)min<int64_t>(a.M - rb, 1 << 30);
    float bc[16];
    if (pre >= 0) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 q4 = *(const f32x4*)(rbias + rowbase + i * 32 + g * 8 + lh * 4);
#pragma unroll
        for (int t = 0; t < 4; ++t) bc[g * 4 + t] = q4[t];
      }
    }
    float x[32];   // x[slot * 16 + r]: this lane's columns, per image slot
#pragma unroll
    for (int k = 0; k < 32; ++k) x[k] = idv;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int cl = colbase + j * 32 + lr;
      const bool ok = cl < c_end, s1 = cl >= c_bnd;
      float v[16];
      switch (i) {   // static accumulator indices
        case 0:
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] = acc[0][j][r];
          break;
        case 1:
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] = acc[1][j][r];
          break;
        case 2:
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] = acc[2][j][r];
          break;
        default:
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] = acc[3][j][r];
          break;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] *= a.alpha;
      if constexpr (kBiasReluSum) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float c = ok ? fmaxf(v[r] + bc[r], 0.f) : 0.f;
          x[r] += s1 ? 0.f : c;
          x[16 + r] += s1 ? c : 0.f;
        }
      } else {
        conv_chain16<T>(a, v, rb, mrem, lh, bc, pre, ok, n0 + cl, s1 ? img0 + 1 : img0, PQ);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float c = ok ? pool_in(kind, pp, v[r]) : idv;
          x[r] = s1 ? x[r] : pool_comb(kind, x[r], c);
          x[16 + r] = s1 ? pool_comb(kind, x[16 + r], c) : x[16 + r];
        }
      }
    }
    // Halving butterfly over lane bits 4..0 (ds_swizzle xor within 32 lanes).
#define MK_GAP_STEP(O, H)                                                        \
  {                                                                              \
    const bool up = (lr & (O)) != 0;                                             \
    _Pragma("unroll") for (int k = 0; k < (H); ++k) {                            \
      const float keep = up ? x[k + (H)] : x[k];                                 \
      const float send = up ? x[k] : x[k + (H)];                                 \
      const float got = __int_as_float(                                          \
          __builtin_amdgcn_ds_swizzle(__float_as_int(send), ((O) << 10) | 0x1F)); \
      x[k] = kBiasReluSum ? keep + got : pool_comb(kind, keep, got);             \
    }                                                                            \
  }
    MK_GAP_STEP(16, 16)
    MK_GAP_STEP(8, 8)
    MK_GAP_STEP(4, 4)
    MK_GAP_STEP(2, 2)
    MK_GAP_STEP(1, 1)
#undef MK_GAP_STEP
    const int r = lr & 15, slot = lr >> 4;
    const int lrow = rowbase + i * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
    red[(wn * 256 + lrow) * 2 + slot] = x[0];
  }
}

// B is [N, K] (K contiguous) here; a [K, N] weight arrives pre-transposed.
// Byte offset along K of implicit-GEMM slice k0 (k = (r*S + s)*C + c, and a
// slice never crosses an (r, s) boundary since C is a multiple of its depth).
template <typename T>
__device__ __forceinline__ uint32_t conv_koff(const GemmArgs& a, int64_t k0) {
  // 32-bit: K = C*R*S and the window's extent in the padded input fit.
  const uint32_t k = (uint32_t)k0, C = (uint32_t)a.cv_C, S = (uint32_t)a.cv_S;
  const uint32_t rs = k / C, c0 = k - rs * C;
  const uint32_t r = rs / S, s = rs - r * S;
  return ((r * (uint32_t)a.cv_Wp + s) * C + c0) * (uint32_t)sizeof(T);
}

// LDS bytes of the epilogue: per wave SL 32-row slabs (8 row groups of
// kSlabU 16-byte units), then the row-reduction exchange [WN][256 rows][2]
// floats.
template <int WN, int BN, int SL = 1>
constexpr int epi_bytes() {
  return SL * 2 * WN * 8 * kSlabU * 16 + WN * BM * 2 * 4;
}

// Variants: WN waves along N (2 rows of waves), BN columns per tile, STG
// stages of RB-byte LDS rows, PIPE main-loop form.
//  <4, 256, 2, 0, 2, 128>: eight waves share one 256 x 256 tile (one
//    workgroup per CU); the stages live in five 32 KB slots, three for A and
//    two for B ([A0 | B0 | A1 | A2 | B1]), so the A loads of a stage can be
//    spread over the stage two ahead of it.  The workgroup is persistent: it
//    walks the tiles v = blockIdx.x, blockIdx.x + gridDim.x, ..., so a tile's
//    epilogue stores drain while the next tile's first stages load.  (Loads
//    issued before the epilogue queued ahead of its stores and slowed it.)
//  <2, 128, 3, 1, 0, 64> (conv): four waves on a 256 x 128 tile in 72 KB of
//    LDS, so two independent workgroups share each CU; one tile per workgroup.
// SIG selects an epilogue compiled for one chain (kSigGeneric: any chain,
// interpreted step by step).
template <typename T, int WN, int BN, int STG, int CONV, int PIPE, int RB, int SIG>
__global__ __launch_bounds__(128 * WN, (BN == 128 ? 2 : 1)) void gemm_mfma_kernel(GemmArgs a) {
  constexpr int BK = RB / (int)sizeof(T);   // K depth of a stage
  constexpr int KSUB = RB / 32;             // 16-byte chunk pairs (MFMA sub-steps) per stage
  constexpr int WAVES = 2 * WN, THREADS = 64 * WAVES;
  constexpr int kStages = STG;
  constexpr int kABytes = BM * RB;          // A part of a stage
  constexpr int kBBytes = BN * RB;          // B part of a stage
  constexpr int kStageBytes = kABytes + kBBytes;
  constexpr int WTN = BN / WN;        // wave tile columns
  constexpr int NJ = WTN / 32;        // 32-wide column tiles per wave
  constexpr bool kPersist = PIPE != 0;
  // Conv bias+ReLU+GAP: transposed accumulators (a lane holds one channel),
  // so the pooling sums are lane-local.
  constexpr bool kTr = SIG == kSigConvBiasReluGap;
  static_assert(PIPE == 0 || (KSUB == 4 && kABytes == 32768 && kBBytes == 32768),
                "the pipelined loop is k64 stages of a 256 x 256 tile");
  // Pipelined slots: A0 0, B0 32K, A1 64K, A2 96K, B1 128K; the epilogue
  // reuses the top of the LDS (clear of A0 and B0, which take the next tile's
  // stage 0 meanwhile).  Ring form: stage slots back to back, the epilogue
  // from 0.
  static_assert(WTN == 64 || (PIPE >= 3 && WTN == 128),
                "the epilogue maps 8 row groups x 8 column groups onto 64 columns of a wave");
  static_assert(PIPE < 3 || (!CONV && WN == 2 && BN == 256 && RB == 128 && sizeof(T) == 2 &&
                              sig_plain(SIG)),
                "the four-wave form runs plain bf16 GEMMs with a compiled chain, no terminal");
  constexpr int kRing = PIPE ? 5 * 32768 : kStages * kStageBytes;
  // (the four-wave epilogue alternates between two slabs per wave)
  constexpr int kSlabs = PIPE >= 3 ? 2 : 1;
  constexpr int kEpiOff = PIPE ? ((kRing - epi_bytes<WN, BN, kSlabs>()) & ~1023) : 0;
  static_assert(PIPE == 0 || kEpiOff >= 65536, "the epilogue must leave A0 and B0 free");
  constexpr int kEpiEnd = kEpiOff + epi_bytes<WN, BN, kSlabs>();
  constexpr int kSmemMain = kEpiEnd > kRing ? kEpiEnd : kRing;
  // Conv: the tile's channel-bias values (first BIAS_CH step) after the ring.
  // Conv: the tile's channel-bias values (first BIAS_CH step): after the
  // ring, or (pipelined form, whose slots fill the LDS) at the start of the
  // epilogue region, unused by the pooling epilogue.
  constexpr int kSmem = kSmemMain + (CONV && !PIPE ? BM * 4 : 0);
  static_assert(kSmem <= 163840, "LDS is 160 KB");
  __shared__ __attribute__((aligned(1024))) char smem[kSmem];
  float* rbias = (float*)(smem + (PIPE ? kEpiOff : kSmemMain));
  const int tiles_m = (int)((a.M + BM - 1) / BM), tiles_n = (int)((a.N + BN - 1) / BN);
  const int tiles = tiles_m * tiles_n;
  // Work items: whole tiles, then (pipelined conv) the row sub-tiles of SR
  // rows of the tiles left after the last whole round.
  const int G = (int)gridDim.x;
  const int tsplit = (CONV && PIPE) ? tail_split(tiles, G) : 1;
  const int tfirst = tsplit > 1 ? tiles - tiles % G : tiles;
  const int trem = tiles - tfirst;
  const int items = tfirst + trem * tsplit;
  const int SR = BM / tsplit;
  auto item_of = [&](int u) -> Item {
    if (u < tfirst) return {tile_of(u, tiles_m, tiles_n), -1};
    const int k = u - tfirst;
    return {tile_of(tfirst + k % trem, tiles_m, tiles_n), k / trem};
  };
  auto row0_of = [&](const Item& it) -> int64_t {
    return (int64_t)it.tc.tm * BM + (it.sub < 0 ? 0 : it.sub * SR);
  };
  // This workgroup's next item from u on (sub-tiles starting past M skipped).
  auto next_item = [&](int u) {
    while (u < items && u >= tfirst && row0_of(item_of(u)) >= a.M) u += G;
    return u;
  };
  const int64_t z = blockIdx.y, bb = z / a.heads, hh = z % a.heads;
  const T* A = (const T*)a.A + a.a_off + bb * a.a_sb + hh * a.a_sh;
  const T* B = (const T*)a.B + a.b_off + bb * a.b_sb + hh * a.b_sh;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / WN, wn = w % WN;
  const int lr = lane & 31, lh = lane >> 5;
  const int rowbase = wm * 128, colbase = wn * WTN;
  const int nk = (int)((a.K + BK - 1) / BK);
  const int64_t PQ = a.cv_P * a.cv_Q;

  SliceLoader<WAVES, BM, T, RB> la;
  std::conditional_t<PIPE == 4, KNLoader, SliceLoader<WAVES, BN, T, RB>> lb;
  auto init_loaders = [&](const Item& it) {
    const int64_t m0 = row0_of(it), n0 = (int64_t)it.tc.tn * BN;
    la.init(A, it.sub < 0 ? a.M : min<int64_t>(a.M, m0 + SR), a.lda, m0);
    if constexpr (CONV) {
      const int64_t bytes = a.cv_Hp * a.cv_Wp * a.cv_C * (int64_t)sizeof(T) *
                            ((uint32_t)a.N / (uint32_t)PQ);
      // 32-bit: positions and byte offsets in the padded input stay below
      // 2^31 (64-bit divisions here cost more than a stage of MFMAs).
      const uint32_t PQu = (uint32_t)PQ, Qu = (uint32_t)a.cv_Q, st = (uint32_t)a.cv_stride;
      const uint32_t Hpu = (uint32_t)a.cv_Hp, Wpu = (uint32_t)a.cv_Wp, Cu = (uint32_t)a.cv_C;
      lb.init_gather(B, bytes, a.N, n0, [&](int64_t m) {
        const uint32_t mu = (uint32_t)m, n = mu / PQu, pq = mu - n * PQu;
        const uint32_t p = pq / Qu, q = pq - p * Qu;
        return ((n * Hpu + p * st) * Wpu + q * st) * Cu * (uint32_t)sizeof(T);
      });
    } else if constexpr (PIPE == 4) {
      lb.init((const bf16*)B, a.K, a.ldb, n0, a.N);
    } else {
      lb.init(B, a.N, a.ldb, n0);
    }
  };
  // Slot addresses.  Pipelined: A of stage ks in A slot ks % 3, B in B slot
  // ks % 2.  Ring: stage ks in slot ks % STG (A part, then B part).
  auto a_slot = [&](int ks) -> char* {
    if (PIPE) {
      const int i = ks % 3;
      return smem + (i == 0 ? 0 : i == 1 ? 65536 : 98304);
    }
    return smem + (ks % kStages) * kStageBytes;
  };
  auto b_slot = [&](int ks) -> char* {
    if (PIPE) return smem + ((ks & 1) ? 131072 : 32768);
    return smem + (ks % kStages) * kStageBytes + kABytes;
  };
  // Loads of stage ks (stages past the last read zeros: every lane's K bound
  // fails).
  auto issue_a = [&](int ks) {
    if constexpr (PIPE < 3) la.issue(a_slot(ks), (int64_t)ks * BK, a.K);
  };
  auto issue_b = [&](int ks) {
    if constexpr (PIPE < 3) {
      const int64_t k0 = (int64_t)ks * BK;
      if (CONV)
        lb.issue(b_slot(ks), k0, a.K, conv_koff<T>(a, k0));
      else
        lb.issue(b_slot(ks), k0, a.K);
    }
  };
  // Sub-tile stages: A (its first 64 rows: one load per thread) in four 8 KB
  // slots at 0, B in four 32 KB slots from 32 KB, so stage 0 sits where a
  // whole tile's does (clear of the epilogue's LDS).
  auto a_slot_s = [&](int ks) -> char* { return smem + (ks & 3) * 8192; };
  auto b_slot_s = [&](int ks) -> char* { return smem + 32768 + (ks & 3) * 32768; };
  auto issue_sub = [&](int ks) {
    if constexpr (PIPE < 3) {
      const int64_t k0 = (int64_t)ks * BK;
      la.template issue_part<0, 1>(a_slot_s(ks), k0, a.K);
      if (CONV)
        lb.issue(b_slot_s(ks), k0, a.K, conv_koff<T>(a, k0));
      else
        lb.issue(b_slot_s(ks), k0, a.K);
    }
  };

  int v = next_item((int)blockIdx.x);
  if (v >= items) return;
  Item it = item_of(v);
  TileCoord tc = it.tc;
  init_loaders(it);
  if constexpr (!PIPE) {
#pragma unroll
    for (int s = 0; s < kStages - 1; ++s)
      if (s < nk) {
        issue_a(s);
        issue_b(s);
      }
  }
  // Conv: the first channel-bias step of the chain (its values for the
  // tile's rows are staged in LDS while the first stages load; conv
  // workgroups take one tile each).
  int pre_ch = -1;
  if (CONV) {
#pragma unroll
    for (int s = 0; s < kMaxEpi; ++s)
      if (s < a.epi.n && pre_ch < 0 && a.epi.code[s] == EPI_BIAS_CH) pre_ch = s;
  }
  if (CONV && !PIPE && pre_ch >= 0) {
    const T* pb = (const T*)a.epi.ptr[pre_ch];
    const int64_t m0 = (int64_t)tc.tm * BM;
    for (int r = threadIdx.x; r < BM; r += THREADS) rbias[r] = m0 + r < a.M ? ld<T>(pb, m0 + r) : 0.f;
  }

  constexpr int LA = SliceLoader<WAVES, BM, T, RB>::LQ, LB = SliceLoader<WAVES, BN, T, RB>::LQ;
  constexpr int LPS = LA + LB;
  // Wait until at most `later` stages issued after the one needed are still
  // in flight (each stage is LPS loads of this wave, issued in order).
  auto wait_slices = [](int later) {
    if (later >= 3)
      wait_vm<3 * LPS>();
    else if (later == 2)
      wait_vm<2 * LPS>();
    else if (later == 1)
      wait_vm<LPS>();
    else
      wait_vm<0>();
  };
  // Per sub-step and wave: MFMAs issued and fragment-read pairs.
  constexpr int kMfmaSub = 4 * NJ * (sizeof(T) == 2 ? 1 : 4);
  constexpr int kReadPairs = (4 + NJ) / 2;
  // A loads: half in sub-step 0, half in sub-step 1; B loads in sub-step 3.
  constexpr int kA0 = (LA + 1) / 2, kA1 = LA - kA0;
  static_assert(PIPE == 0 || kMfmaSub >= kReadPairs + LB + 1, "interleave needs more MFMAs");

  // Row-reduction exchange [WN column groups][256 rows][2], after the slabs
  // (each wave's 32-row slab: 8 row groups of kSlabU 16-byte units).
  float* red = (float*)(smem + kEpiOff) + kSlabs * WAVES * 8 * kSlabU * 4;
  const int64_t cbase = a.c_off + bb * a.c_sb + hh * a.c_sh;
  T* C = (T*)a.C + cbase;
  constexpr int kTerm = sig_terminal(SIG);
  const int term = kTerm >= 0 ? kTerm : a.terminal;
  const bool softmax = term == TERM_SOFTMAX;
  // 16-byte accesses to C and to residual operands need 8-aligned offsets.
  const bool vec_ok = ((a.ldc | cbase) & 7) == 0;

  // Pipelined conv: this thread's channel-bias value of the tile (rows
  // threadIdx.x < BM), loaded with the tile's first stages and written to LDS
  // once the main loop has released it.
  auto load_bias_reg = [&](const Item& t) -> float {
    if (!(CONV && PIPE) || pre_ch < 0 || (int)threadIdx.x >= BM) return 0.f;
    const int64_t r = row0_of(t) + threadIdx.x;
    return r < a.M ? ld<T>((const T*)a.epi.ptr[pre_ch], r) : 0.f;
  };
  float bias_reg = load_bias_reg(it);
  bool staged0 = false;   // this tile's stage 0 was issued during the last epilogue
  constexpr int kEpiVmem = sig_plain(SIG) ? 16 * (NJ / 2) : 0;
  // Four-wave form: LDS byte offsets of the A slots (stage ks in ks % 3) and
  // B slots (ks % 2).
  constexpr int kSlotA3[3] = {0, 65536, 98304};
  constexpr int kSlotB3[2] = {32768, 131072};
  // 16 x 16 x 32 fragments: lane (l16, lq) = (lane % 16, lane / 16) of
  // fragment (t, i) reads row rowbase + i*16 + l16, logical chunk 4t + lq.
  // With X0 = swz(l16) (i*16 and rowbase move the swizzle by 2(i&3) only) its
  // physical chunk is lq ^ X0 ^ 2(2t ^ (i&3)): offset va16[2t ^ (i&3)] +
  // i*2048 within the slot (likewise B with j).
  uint32_t va16[4], vb16[4];
  const int l16 = lane & 15, lq = lane >> 4;
  // [K, N] B (PIPE 4): B fragment j of step t (k = 32t + 8lq .. +7, column
  // colbase + 16j + l16) is two transposing reads of four k-rows each: in a
  // 16-lane group, lane l16 addresses row 8lq + (l16 >> 2) (+4 for the second
  // read), columns 16j + 4 (l16 & 3) .. +3, and receives column 16j + l16 of
  // the four rows.  The row's swizzle term g depends on the lane alone
  // (row & 3 = l16 >> 2, (row >> 3) & 1 = lq & 1); the LDS byte address per
  // (slot, j), the step and the second read as immediate offsets.
  uint32_t vbk[2][8];
  if constexpr (PIPE == 4) {
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
    const int g = (l16 >> 2) | ((lq & 1) << 2);
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        vbk[sb][j] = lds0 + (uint32_t)(sb ? 131072 : 32768) +
                     (uint32_t)((8 * lq + (l16 >> 2)) * 512 +
                                (colbase / 8 + 2 * (j ^ g) + ((l16 & 3) >> 1)) * 16 + (l16 & 1) * 8);
  }
  if constexpr (PIPE >= 3) {
    const int X0 = swz<RB>(l16);
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      va16[d] = (uint32_t)(rowbase * RB + l16 * RB + ((lq ^ X0 ^ (2 * d)) << 4));
      vb16[d] = (uint32_t)(colbase * RB + l16 * RB + ((lq ^ X0 ^ (2 * d)) << 4));
    }
  }
  for (;;) {
    const int64_t m0 = row0_of(it), n0 = (int64_t)tc.tn * BN;
    const bool subt = CONV && PIPE && it.sub >= 0;
    const int rows_it = subt ? SR : BM;
    f32x16 acc[4][NJ];
    f32x4 acc16[8][8];   // the four-wave form's 16 x 16 tiles
    if constexpr (PIPE >= 3) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc16[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    }

    if constexpr (PIPE >= 3) {
      // Four waves, one per SIMD, each a 128 x 128 quarter of the tile (8 x 8
      // tiles of 16 x 16); K a multiple of the 64-deep stage, taken as two
      // 32-deep steps of 64 MFMAs.  A of stage ks sits in slot ks % 3, B in
      // ks % 2.  Step 0 runs on fragments read during the previous step and
      // reads step 1's while A(ks+2) is issued into the slot stage ks-1 held;
      // then the stage barrier (stage ks+1 landed, this stage's reads done),
      // and step 1 reads stage ks+1's first fragments while B(ks+2) refills
      // B slot ks % 2.  The stage loop is unrolled by 6 so every slot offset
      // is a constant: no address arithmetic per fragment read, no K-bound
      // select per load (stages past the last read zeros via the stage
      // offset).
      auto soff3 = [&](int ks, uint32_t range, uint32_t kstep) __attribute__((always_inline))
          -> uint32_t { return ks < nk ? (uint32_t)ks * kstep : range; };
      uint32_t kstep_b = RB;   // B's stage step along K ([K, N]: 64 rows)
      if constexpr (PIPE == 4) kstep_b = lb.kstep;
      struct F16 {
        bf16x8 a[8], b[8];
      };
      auto rd_a = [&](auto SA_, auto T_, int i, bf16x8& d) __attribute__((always_inline)) {
        constexpr int SA = decltype(SA_)::value, TT = decltype(T_)::value;
        d = *(const bf16x8*)(smem + kSlotA3[SA] + i * 2048 + va16[(2 * TT) ^ (i & 3)]);
      };
      auto rd_b = [&](auto SB_, auto T_, int j, bf16x8& d) __attribute__((always_inline)) {
        constexpr int SB = decltype(SB_)::value, TT = decltype(T_)::value;
        if constexpr (PIPE == 4) {
          // (asm: the compiler would wait for every direct-to-LDS load in
          // flight before a transposing read; its results are waited for and
          // redefined at the stage barrier and the stage end)
          u32x2 lo, hi;
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                       : "=v"(lo) : "v"(vbk[SB == 0 ? 0 : 1][j]), "i"(TT * 16384));
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                       : "=v"(hi) : "v"(vbk[SB == 0 ? 0 : 1][j]), "i"(TT * 16384 + 2048));
          d = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3));
        } else {
          d = *(const bf16x8*)(smem + kSlotB3[SB] + j * 2048 + vb16[(2 * TT) ^ (j & 3)]);
        }
      };
      // The transposing reads' results exist after an LDS wait only: redefine
      // them there so that no use is placed before it.
      auto pin_b = [&](F16& f) __attribute__((always_inline)) {
        if constexpr (PIPE == 4) {
#pragma unroll
          for (int j = 0; j < 8; ++j) asm volatile("" : "+v"(f.b[j]));
        }
      };
      // One 32-deep step: 64 MFMAs on `cur`, row by row (A fragment i with
      // the 8 B fragments), in program order with the reads of the next
      // step's 16 fragments into `nxt` (step TN of the stage in slots SA /
      // SB) after every other MFMA of rows 0 .. 3, so that they have returned
      // long before the end of the step, where the stage barrier waits for
      // them, and the 8 operand loads `ld(q)` one per row, in the middle of
      // each (same box, MLP block per step: loads two per row in rows 0 .. 3,
      // +0.8%; reads in rows 0 .. 1, +4%; reads two per row, +0.15%).
      auto step16 = [&](const F16& cur, F16& nxt, auto SA_, auto SB_, auto TN_, auto ld)
          __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            mfma16(acc16[i][j], cur.a[i], cur.b[j]);
            if (i < 4 && (j & 1)) {
              const int r = i * 4 + (j >> 1);
              if (r < 8)
                rd_b(SB_, TN_, r, nxt.b[r]);
              else
                rd_a(SA_, TN_, r - 8, nxt.a[r - 8]);
            }
            if (j == 4) ld(i);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      static_assert(LA == 8 && LB == 8, "eight operand loads per wave and step");
      F16 f0, f1;
      auto stage3 = [&](auto S6_, int ks) __attribute__((always_inline)) {
        constexpr int S6 = decltype(S6_)::value;
        constexpr int SA = S6 % 3, SB = S6 % 2, SA1 = (S6 + 1) % 3, SB1 = (S6 + 1) % 2,
                      SA2 = (S6 + 2) % 3;
        using I0 = std::integral_constant<int, 0>;
        using I1 = std::integral_constant<int, 1>;
        const uint32_t sa2 = soff3(ks + 2, la.range, RB), sb2 = soff3(ks + 2, lb.range, kstep_b);
        // step 0: reads of step 1, A(ks+2) into the slot stage ks-1 held
        step16(f0, f1, std::integral_constant<int, SA>{}, std::integral_constant<int, SB>{}, I1{},
               [&](int q) __attribute__((always_inline)) {
                 la.issue_q(smem + kSlotA3[SA2], sa2, q);
               });
        // stage ks+1 landed (only A(ks+2) may remain) and this wave's reads
        // of stage ks are done; the barrier makes both hold for every wave
        wait_vm<LA>();
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        pin_b(f1);
        // step 1: reads of stage ks+1's step 0, B(ks+2) into B slot ks % 2
        step16(f1, f0, std::integral_constant<int, SA1>{}, std::integral_constant<int, SB1>{},
               I0{}, [&](int q) __attribute__((always_inline)) {
                 lb.issue_q(smem + kSlotB3[SB], sb2, q);
               });
        if constexpr (PIPE == 4) {
          __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): next stage's B fragments
          pin_b(f0);
        }
      };
      if (!staged0) {
        la.template issue_full<0, LA>(smem + kSlotA3[0], 0u);
        lb.template issue_full<0, LB>(smem + kSlotB3[0], 0u);
      }
      la.template issue_full<0, LA>(smem + kSlotA3[1], soff3(1, la.range, RB));
      lb.template issue_full<0, LB>(smem + kSlotB3[1], soff3(1, lb.range, kstep_b));
      if (staged0)
        wait_vm<LA + LB + kEpiVmem>();
      else
        wait_vm<LA + LB>();
      __builtin_amdgcn_s_barrier();
#pragma unroll
      for (int j = 0; j < 8; ++j)
        rd_b(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, j, f0.b[j]);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        rd_a(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, i, f0.a[i]);
      if constexpr (PIPE == 4) {
        __builtin_amdgcn_s_waitcnt(0xc07f);
        pin_b(f0);
      }
      int ks = 0;
      for (; ks + 6 <= nk; ks += 6) {
        stage3(std::integral_constant<int, 0>{}, ks);
        stage3(std::integral_constant<int, 1>{}, ks + 1);
        stage3(std::integral_constant<int, 2>{}, ks + 2);
        stage3(std::integral_constant<int, 3>{}, ks + 3);
        stage3(std::integral_constant<int, 4>{}, ks + 4);
        stage3(std::integral_constant<int, 5>{}, ks + 5);
      }
      if (ks < nk) stage3(std::integral_constant<int, 0>{}, ks);
      if (ks + 1 < nk) stage3(std::integral_constant<int, 1>{}, ks + 1);
      if (ks + 2 < nk) stage3(std::integral_constant<int, 2>{}, ks + 2);
      if (ks + 3 < nk) stage3(std::integral_constant<int, 3>{}, ks + 3);
      if (ks + 4 < nk) stage3(std::integral_constant<int, 4>{}, ks + 4);
      // the last MFMAs finish before the epilogue reads their results
      asm volatile("s_nop 15\n\ts_nop 15" ::: "memory");
    } else if (PIPE && subt) {
      // Row sub-tile: waves wm with wm*32 < SR compute rows wm*32 .. +31 of
      // it into acc[0]; every wave loads.  Three stages in flight; one
      // barrier per stage (it also orders the refill of the slot read in the
      // previous stage after every wave's reads of it).
      const bool cw = wm * 32 < SR;
      if (!staged0) issue_sub(0);
      issue_sub(1);
      issue_sub(2);
      for (int ks = 0; ks < nk; ++ks) {
        wait_vm<2 * (1 + LB)>();
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        issue_sub(ks + 3);
        if (cw) {
          typedef typename MfmaType<T>::frag F;
          const char* ca = a_slot_s(ks);
          const char* cb = b_slot_s(ks);
#pragma unroll
          for (int kk = 0; kk < KSUB; ++kk) {
            F fb[NJ];
            const F fa = *(const F*)(ca + lds_off<RB>(wm * 32 + lr, kk * 2 + lh));
#pragma unroll
            for (int j = 0; j < NJ; ++j)
              fb[j] = *(const F*)(cb + lds_off<RB>(colbase + j * 32 + lr, kk * 2 + lh));
#pragma unroll
            for (int j = 0; j < NJ; ++j)
              acc[0][j] = kTr ? mfma1<T>(fb[j], fa, acc[0][j]) : mfma1<T>(fa, fb[j], acc[0][j]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else if (PIPE) {
      // Stages 0 and 1 go now.  Stage s: sub-steps 0..3,
      // fragments one sub-step ahead of the MFMAs that use them; A(s+2) is
      // issued over sub-steps 0 and 1 (its slot held stage s-1, released by
      // the barrier of stage s-1).  Before sub-step 3 the wave waits for its
      // loads of stage s+1 (only A(s+2) may remain) and for its reads of
      // stage s (lgkmcnt(0)); one barrier makes both hold for every wave,
      // after which stage s+1 is read and B(s+2) refills B slot s % 2.  The
      // body is branch-free: past the last stage every lane's K bound fails
      // and the loads only write zeros into slots never read again.
      // After a prefetched stage 0 the last epilogue's memory operations sit
      // between the two stages: kEpiVmem of them at least (each of its 16
      // rows issues a store in the buffer-store forms), so that many may stay
      // outstanding with stage 1 (otherwise the wait covers them too).
      if (!staged0) {
        issue_a(0);
        issue_b(0);
      }
      issue_a(1);
      issue_b(1);
      if (staged0)
        wait_vm<LA + LB + kEpiVmem>();
      else
        wait_vm<LA + LB>();
      __builtin_amdgcn_s_barrier();
      Frags<NJ, T> f0, f1;
      load_frags<NJ, T, RB>(a_slot(0), b_slot(0), 0, rowbase, colbase, lr, lh, f0);
      for (int ks = 0; ks < nk; ++ks) {
        const char* ca = a_slot(ks);
        const char* cb = b_slot(ks);
        // sub-steps 0..2: MFMAs on the fragments of `sub`, reads of sub+1
        auto sub_step = [&](auto SUB) {
          constexpr int sub = decltype(SUB)::value;
          Frags<NJ, T>& use = (sub & 1) ? f1 : f0;
          Frags<NJ, T>& fill = (sub & 1) ? f0 : f1;
          load_frags<NJ, T, RB>(ca, cb, sub + 1, rowbase, colbase, lr, lh, fill);
          if constexpr (sub == 0)
            la.template issue_part<0, kA0>(a_slot(ks + 2), (int64_t)(ks + 2) * BK, a.K);
          if constexpr (sub == 1)
            la.template issue_part<kA0, LA>(a_slot(ks + 2), (int64_t)(ks + 2) * BK, a.K);
          mfma_step<NJ, T, kTr>(use, acc);
#pragma unroll
          for (int g = 0; g < kReadPairs; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS read
          }
          constexpr int nv = sub == 0 ? kA0 : sub == 1 ? kA1 : 0;
#pragma unroll
          for (int g = 0; g < nv; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
          }
          __builtin_amdgcn_sched_group_barrier(0x008, kMfmaSub - kReadPairs - nv, 0);
          __builtin_amdgcn_sched_barrier(0);
        };
        sub_step(std::integral_constant<int, 0>{});
        sub_step(std::integral_constant<int, 1>{});
        sub_step(std::integral_constant<int, 2>{});
        // last sub-step (fragments in f1)
        wait_vm<LA>();
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        load_frags<NJ, T, RB>(a_slot(ks + 1), b_slot(ks + 1), 0, rowbase, colbase, lr, lh, f0);
        issue_b(ks + 2);
        mfma_step<NJ, T, kTr>(f1, acc);
#pragma unroll
        for (int g = 0; g < kReadPairs; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS read
        }
#pragma unroll
        for (int g = 0; g < LB; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, kMfmaSub - kReadPairs - LB, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      for (int kt = 0; kt < nk; ++kt) {
        // Stage kt has landed once at most the loads of the later stages are
        // outstanding.
        wait_slices(min(kStages - 2, nk - 1 - kt));
        // A bare barrier: __syncthreads() would also drain every outstanding
        // load (its fence), which defeats the ring.  The stage's own loads are
        // complete (vmcnt above), and fragment reads of the slot about to be
        // refilled were consumed by MFMAs before this point.
        __builtin_amdgcn_s_barrier();
        const int nxt = kt + kStages - 1;
        if (nxt < nk) {
          issue_a(nxt);
          issue_b(nxt);
        }
        Frags<NJ, T> f[KSUB];
#pragma unroll
        for (int sub = 0; sub < KSUB; ++sub)
          load_frags<NJ, T, RB>(a_slot(kt), b_slot(kt), sub, rowbase, colbase, lr, lh, f[sub]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int sub = 0; sub < KSUB; ++sub) {
          mfma_step<NJ, T, kTr>(f[sub], acc);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }

    // Every slot is consumed and every refill (zeros past the last stage)
    // has landed before the epilogue reuses the LDS.
    wait_vm<0>();
    __syncthreads();
    if (CONV && PIPE && pre_ch >= 0) {
      int tb = (int)threadIdx.x;   // opaque copy: the address is not kept live
      asm volatile("" : "+v"(tb));
      if (tb < BM) rbias[tb] = bias_reg;
      __syncthreads();
    }
    const int vn = next_item(v + G);
    const bool more = kPersist && vn < items;
    // The next tile's stage 0 loads while this epilogue runs (its LDS is
    // clear of slots A0 and B0; every read of the last stages is done).
    Item it_next = it;
    if (PIPE && more) {
      it_next = item_of(vn);
      init_loaders(it_next);
      if constexpr (PIPE >= 3) {
        la.template issue_full<0, LA>(smem + kSlotA3[0], 0u);
        lb.template issue_full<0, LB>(smem + kSlotB3[0], 0u);
      } else if (CONV && it_next.sub >= 0) {
        issue_sub(0);
      } else {
        issue_a(0);
        issue_b(0);
      }
      bias_reg = load_bias_reg(it_next);
    }
    staged0 = PIPE && more;
    // Lane-derived values of the epilogue, recomputed here from an opaque
    // copy of the thread index: otherwise they are hoisted out of the tile
    // loop, live across the main loop and spill (each reload then waits for
    // every store before it).  lr, lh, rowbase, colbase and wn shadow the
    // kernel-wide ones.
    int tid_e = (int)threadIdx.x;
    asm volatile("" : "+v"(tid_e));
    const int lane_e = tid_e & 63, w_e = tid_e >> 6;
    const int wn_e = w_e % WN;
    const int lr = lane_e & 31, lh = lane_e >> 5;
    const int l16e = lane_e & 15, lqe = lane_e >> 4;
    const int rowbase = (w_e / WN) * (subt ? 32 : 128), colbase = wn_e * WTN;
    // 32-row slab I of 64 columns J0*32 .. J0*32+63 of this wave's tile from
    // the accumulators, in either MFMA layout.
    auto stage_any = [&](auto I_, auto J0_, float* sl) __attribute__((always_inline)) {
      constexpr int I = decltype(I_)::value, J0 = decltype(J0_)::value;
      if constexpr (PIPE >= 3)
        stage_slab16<I, J0>(acc16, sl, lqe, l16e);
      else
        stage_slab<I, NJ, J0>(acc, sl, lh, lr);
    };
    // Epilogue lane roles: 8-column group q and row group rg of the slab;
    // the 8 lanes of a row (same rg) are lanes rg, rg+8, ..., rg+56.
    const int q = lane_e >> 3, rg = lane_e & 7;
    const int wn = wn_e;
    float* slab = (float*)(smem + kEpiOff) + w_e * (kSlabs * 8 * kSlabU * 4);

    // ---------------------------------------------------------------- epilogue
    // acc[i][j][r] is C[row, col] with
    //   row = m0 + rowbase + i*32 + (r/4)*8 + lh*4 + r%4,  col = n0 + colbase + j*32 + lr
    // (four-wave form: acc16[i][j][r] with row = m0 + rowbase + i*16 + lq*4 + r,
    // col = n0 + colbase + j*16 + l16).
    // Each wave stages one 32-row slab at a time in its own LDS region; lane
    // (q, rg) then reads rows 4rg .. 4rg+3 of columns 8q .. 8q+7, applies the
    // chain to each row's 8 values and writes them with one 16-byte store.
    // (the four-wave form finishes its 128 columns as two 64-column halves,
    // moving col0 between them)
    int64_t col0 = n0 + colbase + q * 8;
    int valid = (int)min<int64_t>(8, max<int64_t>(0, a.N - col0));
    // Conv: this lane's 8 positions lie in one image (PQ % 8 == 0).
    const int64_t img = CONV ? (int64_t)((uint32_t)col0 / (uint32_t)PQ) : 0;   // positions < 2^31

    // Compiled TERM_NONE chains store through a buffer resource over C.
    constexpr bool kBufStore = sig_plain(SIG);
    const __amdgpu_buffer_rsrc_t rcst =
        make_rsrc(C, kBufStore ? a.M * a.ldc * (int64_t)sizeof(T) : 0);
    // Residual operand (laid out as C; range checked by signature selection).
    const __amdgpu_buffer_rsrc_t rres =
        make_rsrc(SIG == kSigAdd ? (const T*)a.epi.ptr[0] + cbase : (const T*)a.C,
                  SIG == kSigAdd ? a.M * a.ldc * (int64_t)sizeof(T) : 0);
    // Column bias of this lane's 8 columns, once per tile.
    float bcol[8];
    if constexpr (sig_bias(SIG))
      ld8<T>((const T*)a.epi.ptr[0] + col0, valid == 8 && vec_ok, valid, bcol);

    // One row of the lane: values v of columns col0 .. col0+7 of tile row
    // lrow; `res` is its residual piece (kSigAdd, full pieces), `bt` the conv
    // channel bias of the row.
    auto finish_row = [&](int lrow, float (&v)[8], const u32x4& res, float bt) __attribute__((always_inline)) {
      const int64_t row = m0 + lrow;
      const bool row_ok = row < a.M;
      // Offset of (row, col0) in the output: row-major, or NCHW for a conv
      // (row = channel, col = position).
      const int64_t obase = CONV ? (img * a.M + row) * PQ + (col0 - img * PQ)
                                 : cbase + row * a.ldc + col0;
      if constexpr (SIG == kSigGeluErf) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = sizeof(T) == 2 ? gelu_erf_bf16out(v[e]) : gelu_erf(v[e]);
      } else if constexpr (SIG == kSigAdd) {
        float t8[8];
        if (valid == 8 && vec_ok) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {   // bf16 pairs, low half first
            t8[2 * k] = __uint_as_float(res[k] << 16);
            t8[2 * k + 1] = __uint_as_float(res[k] & 0xFFFF0000u);
          }
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) t8[k] = 0.f;
          if (row_ok && valid > 0) ld8<T>((const T*)a.epi.ptr[0] + obase, false, valid, t8);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += (row_ok && e < valid) ? t8[e] : 0.f;
      } else if constexpr (SIG == kSigBiasGeluTanhScaleSoftmax || SIG == kSigBiasGeluTanhScale) {
        // (v arrives without alpha: alpha * acc + bias is one FMA)
        const float sc = a.epi.s[2];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = gelu_tanh(fmaf(v[e], a.alpha, bcol[e])) * sc;
      } else if constexpr (SIG == kSigBias) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = fmaf(v[e], a.alpha, bcol[e]);
      } else if constexpr (SIG == kSigGeneric || SIG == kSigConvBiasReluGap) {
        if (a.epi.n && row_ok && valid > 0)
          epi_apply8<T>(a.epi, v, row, col0, row, valid, obase, valid == 8 && (CONV || vec_ok),
                        CONV ? pre_ch : -1, bt);
      }
      // Stored values are rounded to the storage type; reductions that need
      // the whole row read them back as stored.  Below, lanes past N take
      // part through selects, not branches.
      if (term == TERM_NONE || term == TERM_SOFTMAX || term == TERM_LAYERNORM)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = rnd<T>(v[e]);
      if constexpr (kBufStore) {
        // 32-bit offsets into C (range checked at selection); rows past M and
        // columns past N get offsets beyond the range and are dropped.
        const int r32 = (int)m0 + lrow;
        const uint32_t roff = row_ok ? (uint32_t)((r32 * (int)a.ldc + (int)col0) * 2) : kOob;
        if (valid == 8 && vec_ok) {
          u32x4 o;
#pragma unroll
          for (int k = 0; k < 4; ++k)
            o[k] = pack2_bf16(v[2 * k], v[2 * k + 1]);
          __builtin_amdgcn_raw_buffer_store_b128(o, rcst, (int)roff, 0, 0);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            __builtin_amdgcn_raw_buffer_store_b16(f2bf(v[e]), rcst,
                                                  (int)(e < valid ? roff + 2 * e : kOob), 0, 0);
        }
      } else if (term != TERM_ROWSUM && row_ok) {
        // NCHW conv output is always 8-aligned (PQ % 8 == 0); a row-major
        // output needs ldc and the batch offset 8-aligned for the vector store.
        const int64_t off = CONV ? obase : row * a.ldc + col0;
        if (valid == 8 && (CONV || vec_ok)) {
          st8<T>(C + off, v);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e < valid) st<T>(C, off + e, v[e]);
        }
      }
      if (term == TERM_LAYERNORM) {
        // moments of this wave's columns of the row: mean, then the squared
        // deviations, over the lane's valid values; lanes then merge
        float sv = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sv += e < valid ? v[e] : 0.f;
        const float n = (float)max(valid, 0);
        const float mean = valid > 0 ? sv / n : 0.f;
        float m2 = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = v[e] - mean;
          m2 += e < valid ? d * d : 0.f;
        }
        Moments mo{n, mean, m2};
#pragma unroll
        for (int o = 8; o < 64; o <<= 1) mo = mom_comb(mo, mom_shfl_xor(mo, o));
        if (q == 0) {
          red[(wn * 256 + lrow) * 2] = mo.mean;
          red[(wn * 256 + lrow) * 2 + 1] = mo.m2;
        }
      } else if (term != TERM_NONE) {
        // reduce over the 8 lanes that share this row (this wave's columns)
        float m = -INFINITY, sum = 0.f;
        if (softmax) {
#pragma unroll
          for (int e = 0; e < 8; ++e) m = fmaxf(m, e < valid ? v[e] : -INFINITY);
          m = fmaxf(m, lane_xor<8>(m));
          m = fmaxf(m, lane_xor<16>(m));
          m = fmaxf(m, lane_xor<32>(m));
          const bool any = m != -INFINITY;
          // exp(v - m) = 2^(v log2 e - m log2 e): one FMA and exp2
          const float ml = any ? m * 1.4426950408889634f : 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x = __builtin_amdgcn_exp2f(fmaf(v[e], 1.4426950408889634f, -ml));
            sum += (e < valid && any) ? x : 0.f;
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) sum += e < valid ? v[e] : 0.f;
        }
        sum += lane_xor<8>(sum);
        sum += lane_xor<16>(sum);
        sum += lane_xor<32>(sum);
        if (q == 0) {
          red[(wn * 256 + lrow) * 2] = m;
          red[(wn * 256 + lrow) * 2 + 1] = sum;
        }
      }
    };

    // Generic form: one slab at a time, rows in a loop that is not unrolled.
    auto finish_slab = [&](int i) {
      __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): slab writes done (wave-private)
      __builtin_amdgcn_wave_barrier();
      f32x4 u[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) u[k] = *(const f32x4*)(slab + (rg * kSlabU + q * 8 + k) * 4);
      // Conv: the channel bias of this lane's 4 rows.
      f32x4 bq = {0.f, 0.f, 0.f, 0.f};
      if (CONV && pre_ch >= 0) bq = *(const f32x4*)(rbias + rowbase + i * 32 + rg * 4);
      // The slab is rewritten next: every lane's reads of it must be done.
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_wave_barrier();
      if constexpr (SIG == kSigBiasGeluTanhScaleSoftmax) {
        // Rows unrolled (static quad indices, no rotation); alpha enters the
        // chain's first FMA.
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          float v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = u[e][t];
          finish_row(rowbase + i * 32 + rg * 4 + t, v, u32x4{0, 0, 0, 0}, 0.f);
        }
      } else {
        // Row t of the quad is element 0 after t rotations (static indices
        // in a loop that is not unrolled).
#pragma unroll 1
        for (int t = 0; t < 4; ++t) {
          float v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            v[e] = u[e][0] * a.alpha;
            u[e] = f32x4{u[e][1], u[e][2], u[e][3], u[e][0]};
          }
          const float bt = bq[0];
          bq = f32x4{bq[1], bq[2], bq[3], bq[0]};
          finish_row(rowbase + i * 32 + rg * 4 + t, v, u32x4{0, 0, 0, 0}, bt);
        }
      }
    };

    // Residual pieces of this lane's 4 rows of slab i, as buffer loads (a
    // lane without a full piece reads zeros, with no branch to wait at).
    auto load_res = [&](int i, u32x4 (&dst)[4]) __attribute__((always_inline)) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int64_t row = m0 + rowbase + i * 32 + rg * 4 + t;
        const bool full = row < a.M && valid == 8 && vec_ok;
        const uint32_t off = full ? (uint32_t)((row * a.ldc + col0) * (int64_t)sizeof(T)) : kOob;
        dst[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rres, (int)off, 0, 0));
      }
    };
    // Compiled chains: slabs and rows unrolled (static indices).  The
    // residual pieces of slab I+1 are requested before slab I's stores: loads
    // and stores share one in-order counter, so a load issued after a store
    // could only be waited for together with that store.
    auto finish_slab_sig = [&](auto I_, u32x4 (&cur)[4], u32x4 (&nxt)[4]) __attribute__((always_inline)) {
      constexpr int I = decltype(I_)::value;
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_wave_barrier();
      f32x4 u[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) u[k] = *(const f32x4*)(slab + (rg * kSlabU + q * 8 + k) * 4);
      if constexpr (SIG == kSigAdd && I < 3) load_res(I + 1, nxt);
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[e] = SIG == kSigBiasGeluTanhScale || SIG == kSigBias ? u[e][t] : u[e][t] * a.alpha;
        finish_row(rowbase + I * 32 + rg * 4 + t, v, cur[t], 0.f);
      }
    };
    if (SIG == kSigConvBiasReluGap || (CONV && term == TERM_GAP)) {
      gap_from_acc<T, NJ, SIG == kSigConvBiasReluGap>(a, acc, m0, n0, rowbase, colbase, wn, lr, lh,
                                                       pre_ch, rbias, red,
                                                       subt ? (rowbase < SR ? 1 : 0) : 4);
    } else if (PIPE >= 3 && m0 + BM <= a.M && n0 + BN <= a.N && vec_ok) {
      // Four-wave form, whole tile: the 8 passes (32-row slab I, 64-column
      // half H) alternate between the wave's two slabs; a pass reads its
      // slab back and then stages the next pass into the other one, so the
      // reads wait for nothing behind them and the staging overlaps this
      // pass's arithmetic and stores (LDS operations of a wave run in order,
      // so only the compiler's ordering needs a fence; the next staging into
      // this slab comes after these reads).  A lane finishes rows rowbase +
      // I*32 + rg*4 + t of columns colbase + H*64 + q*8 .. +7.  No row or
      // column bounds, 32-bit offsets stepping by rows, one 16-byte store per
      // row; residual pieces are requested two passes ahead.  The passes
      // exist twice, with and without the alpha multiply (alpha is 1 in most
      // modules: one VALU operation per value less).
      if constexpr (PIPE >= 3) {
        const float alpha = a.alpha;
        const uint32_t ldc2 = (uint32_t)a.ldc * 2u;
        const uint32_t base0 =
            (uint32_t)((((int)m0 + rowbase + rg * 4) * (int)a.ldc + (int)n0 + colbase + q * 8) * 2);
        float* slab1 = slab + 8 * kSlabU * 4;
        float bc[2][8];
        if constexpr (SIG == kSigBiasGeluTanhScale || SIG == kSigBias) {
#pragma unroll
          for (int h = 0; h < 2; ++h)
            ld8<T>((const T*)a.epi.ptr[0] + n0 + colbase + h * 64 + q * 8, true, 8, bc[h]);
        }
        u32x4 res[3][4];
        auto pass_off = [&](int P, int t) __attribute__((always_inline)) -> uint32_t {
          return base0 + (uint32_t)((P >> 1) * 32 + t) * ldc2 + (uint32_t)(P & 1) * 128u;
        };
        auto load_res3 = [&](auto P_) __attribute__((always_inline)) {
          constexpr int P = decltype(P_)::value;
          if constexpr (SIG == kSigAdd && P < 8) {
#pragma unroll
            for (int t = 0; t < 4; ++t)
              res[P % 3][t] = __builtin_bit_cast(
                  u32x4, __builtin_amdgcn_raw_buffer_load_b128(rres, (int)pass_off(P, t), 0, 0));
          }
        };
        auto stage3 = [&](auto P_) __attribute__((always_inline)) {
          constexpr int P = decltype(P_)::value;
          if constexpr (P < 8) {
            float* sl = (P & 1) ? slab1 : slab;
            stage_any(std::integral_constant<int, P / 2>{},
                      std::integral_constant<int, (P & 1) ? 2 : 0>{}, sl);
          }
          __builtin_amdgcn_wave_barrier();
        };
        auto pass3 = [&](auto P_, auto UA_) __attribute__((always_inline)) {
          constexpr int P = decltype(P_)::value;
          constexpr bool UA = decltype(UA_)::value;   // alpha == 1
          const float* sl = (P & 1) ? slab1 : slab;
          f32x4 u[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) u[k] = *(const f32x4*)(sl + (rg * kSlabU + q * 8 + k) * 4);
          __builtin_amdgcn_wave_barrier();
          stage3(std::integral_constant<int, P + 1>{});
          load_res3(std::integral_constant<int, P + 2>{});
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float x = u[e][t];
              if constexpr (SIG == kSigBiasGeluTanhScale)
                v[e] = gelu_tanh(UA ? x + bc[P & 1][e] : fmaf(x, alpha, bc[P & 1][e])) * a.epi.s[2];
              else if constexpr (SIG == kSigBias)
                v[e] = UA ? x + bc[P & 1][e] : fmaf(x, alpha, bc[P & 1][e]);
              else if constexpr (SIG == kSigGeluErf)
                v[e] = gelu_erf_bf16out(UA ? x : x * alpha);
              else
                v[e] = UA ? x : x * alpha;
            }
            if constexpr (SIG == kSigAdd) {
              const u32x4 r = res[P % 3][t];
#pragma unroll
              for (int k = 0; k < 4; ++k) {
                v[2 * k] += __uint_as_float(r[k] << 16);
                v[2 * k + 1] += __uint_as_float(r[k] & 0xFFFF0000u);
              }
            }
            u32x4 o;
#pragma unroll
            for (int k = 0; k < 4; ++k) o[k] = pack2_bf16(v[2 * k], v[2 * k + 1]);
            __builtin_amdgcn_raw_buffer_store_b128(o, rcst, (int)pass_off(P, t), 0, 0);
          }
        };
        stage3(std::integral_constant<int, 0>{});
        load_res3(std::integral_constant<int, 0>{});
        load_res3(std::integral_constant<int, 1>{});
        auto passes = [&](auto UA) __attribute__((always_inline)) {
          pass3(std::integral_constant<int, 0>{}, UA);
          pass3(std::integral_constant<int, 1>{}, UA);
          pass3(std::integral_constant<int, 2>{}, UA);
          pass3(std::integral_constant<int, 3>{}, UA);
          pass3(std::integral_constant<int, 4>{}, UA);
          pass3(std::integral_constant<int, 5>{}, UA);
          pass3(std::integral_constant<int, 6>{}, UA);
          pass3(std::integral_constant<int, 7>{}, UA);
        };
        if (alpha == 1.f)
          passes(std::true_type{});
        else
          passes(std::false_type{});
      }
    } else if constexpr (sig_plain(SIG)) {
      // (The softmax-partial chain keeps the rolled loop: unrolled, its
      // live values spill.)
      auto half = [&](auto H_) __attribute__((always_inline)) {
        constexpr int H = decltype(H_)::value;
        if constexpr (H > 0) {
          col0 = n0 + colbase + H * 64 + q * 8;
          valid = (int)min<int64_t>(8, max<int64_t>(0, a.N - col0));
          if constexpr (SIG == kSigBiasGeluTanhScale || SIG == kSigBias)
            ld8<T>((const T*)a.epi.ptr[0] + col0, valid == 8 && vec_ok, valid, bcol);
        }
        u32x4 ra[4], rb[4];
        if constexpr (SIG == kSigAdd) load_res(0, ra);
        using J = std::integral_constant<int, 2 * H>;
        stage_any(std::integral_constant<int, 0>{}, J{}, slab);
        finish_slab_sig(std::integral_constant<int, 0>{}, ra, rb);
        stage_any(std::integral_constant<int, 1>{}, J{}, slab);
        finish_slab_sig(std::integral_constant<int, 1>{}, rb, ra);
        stage_any(std::integral_constant<int, 2>{}, J{}, slab);
        finish_slab_sig(std::integral_constant<int, 2>{}, ra, rb);
        stage_any(std::integral_constant<int, 3>{}, J{}, slab);
        finish_slab_sig(std::integral_constant<int, 3>{}, rb, ra);
      };
      half(std::integral_constant<int, 0>{});
      if constexpr (NJ == 4) half(std::integral_constant<int, 1>{});
    } else {
      // A switch keeps every acc index static while the finishing code
      // exists once (the loop itself is not unrolled).
      for (int i = 0; i < 4; ++i) {
        switch (i) {
          case 0: stage_slab<0, NJ>(acc, slab, lh, lr); break;
          case 1: stage_slab<1, NJ>(acc, slab, lh, lr); break;
          case 2: stage_slab<2, NJ>(acc, slab, lh, lr); break;
          default: stage_slab<3, NJ>(acc, slab, lh, lr); break;
        }
        finish_slab(i);
      }
    }
    if (term != TERM_NONE) {
      __syncthreads();
      for (int lrow = threadIdx.x; lrow < rows_it; lrow += THREADS) {
        const int64_t row = m0 + lrow;
        if (row >= a.M) break;
        if (CONV) {   // GAP partials of this position tile, per image slot
#pragma unroll
          for (int slot = 0; slot < 2; ++slot) {
            float ss = pool_id(a.pool);
#pragma unroll
            for (int g = 0; g < WN; ++g)
              ss = pool_comb(a.pool, ss, red[(g * 256 + lrow) * 2 + slot]);
            a.partial[((int64_t)tc.tn * 2 + slot) * a.M + row] = ss;
          }
          continue;
        }
        float* part = a.partial + (row * a.n_tiles + tc.tn) *
                                      (softmax || term == TERM_LAYERNORM ? 2 : 1);
        if (term == TERM_LAYERNORM) {
          // combine the WN waves' column ranges (their counts follow from N)
          Moments mo{0.f, 0.f, 0.f};
#pragma unroll
          for (int g = 0; g < WN; ++g) {
            const int64_t c0 = n0 + g * WTN;
            const float cnt = (float)min<int64_t>(WTN, max<int64_t>(0, a.N - c0));
            mo = mom_comb(mo, Moments{cnt, red[(g * 256 + lrow) * 2], red[(g * 256 + lrow) * 2 + 1]});
          }
          part[0] = mo.mean;
          part[1] = mo.m2;
        } else if (softmax) {
          float mm = -INFINITY;
#pragma unroll
          for (int g = 0; g < WN; ++g) mm = fmaxf(mm, red[(g * 256 + lrow) * 2]);
          float ss = 0.f;
          if (mm != -INFINITY) {
#pragma unroll
            for (int g = 0; g < WN; ++g) {
              const float mg = red[(g * 256 + lrow) * 2];
              if (mg != -INFINITY) ss += red[(g * 256 + lrow) * 2 + 1] * __expf(mg - mm);
            }
          }
          part[0] = mm;
          part[1] = ss;
        } else {
          float ss = 0.f;
#pragma unroll
          for (int g = 0; g < WN; ++g) ss += red[(g * 256 + lrow) * 2 + 1];
          part[0] = ss;
        }
      }
    }
    if (!more) break;
    // The epilogue's LDS accesses are done before any wave loads the next
    // tile's stage 1 (slot A1 overlaps the epilogue's LDS).
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();
    v = vn;
    it = it_next;
    tc = it.tc;
  }
}

// B(k, n) of a [K, N] operand (batched) -> dst[z][n][k], K contiguous (K and
// N are multiples of the 16-byte chunk of E elements).  No LDS: a lane moves
// one E x E block, E 16-byte loads along n transposed in registers into E
// 16-byte stores along k.  Lane (kb, nb) = (lane % 8, lane / 8) of wave w
// takes k-block 8*blockIdx.y + kb and n-block 8*(4*blockIdx.x + w) + nb, so
// every load and every store instruction covers eight 128-byte runs.
template <typename T>
__global__ __launch_bounds__(256) void transpose_b_kernel(GemmArgs a, T* dst) {
  constexpr int E = 16 / (int)sizeof(T);    // elements per chunk
  const int64_t z = blockIdx.z, bb = z / a.heads, hh = z % a.heads;
  const T* src = (const T*)a.B + a.b_off + bb * a.b_sb + hh * a.b_sh;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t k0 = ((int64_t)blockIdx.y * 8 + (lane & 7)) * E;
  const int64_t n0 = (((int64_t)blockIdx.x * 4 + w) * 8 + (lane >> 3)) * E;
  if (k0 >= a.K || n0 >= a.N) return;
  union Chunk {
    uint4 u;
    T e[E];
  } v[E], o;
#pragma unroll
  for (int u = 0; u < E; ++u) v[u].u = *(const uint4*)(src + (k0 + u) * a.ldb + n0);
  T* out = dst + z * a.N * a.K + n0 * a.K + k0;
#pragma unroll
  for (int q = 0; q < E; ++q) {
#pragma unroll
    for (int u = 0; u < E; ++u) o.e[u] = v[u].e[q];
    *(uint4*)(out + q * a.K) = o.u;
  }
}

}  // namespace

int gemm_mfma_limit(int dtype, const GemmArgs& a) {
  if (dtype != MK_BF16 && dtype != MK_F32) return MK_LIMIT_DTYPE;
  const int64_t es = dtype == MK_BF16 ? 2 : 4, E = 16 / es;
  if (a.M < 1 || a.N < 1 || a.K < 1) return MK_LIMIT_SHAPE;
  // 16-byte operand chunks: K (and N for a [K, N] weight), leading dimensions
  // and batch offsets must be multiples of the chunk.
  if (a.K % E || a.lda % E || a.ldb % E) return MK_LIMIT_ALIGN;
  if (a.layout == 1 && a.N % E) return MK_LIMIT_ALIGN;
  const int64_t offs[] = {a.a_off, a.a_sb, a.a_sh, a.b_off, a.b_sb, a.b_sh};
  for (int64_t o : offs)
    if (o % E) return MK_LIMIT_ALIGN;
  // a row terminal (ROWSUM / SOFTMAX / LAYERNORM) is finished over one matrix
  if (a.terminal != TERM_NONE && a.batch * a.heads != 1) return MK_LIMIT_SHAPE;
  // Buffer-resource ranges are 32-bit: every operand slice must stay below 2 GB.
  const int64_t lim = (int64_t)1 << 31;
  if (a.M * a.lda * es >= lim || a.N * (a.layout == 0 ? a.ldb : a.K) * es >= lim)
    return MK_LIMIT_RANGE;
  const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + 127) / 128);
  return tiles < (1ll << 31) && a.batch * a.heads <= 65535 ? MK_LIMIT_NONE : MK_LIMIT_RANGE;
}

bool gemm_mfma_supported(int dtype, const GemmArgs& a) {
  return gemm_mfma_limit(dtype, a) == MK_LIMIT_NONE;
}

int64_t gemm_mfma_bt_bytes(int dtype, const GemmArgs& a) {
  return a.layout == 1 ? (int64_t)a.batch * a.heads * a.N * a.K * (dtype == MK_BF16 ? 2 : 4) : 0;
}

hipError_t launch_transpose_b(int dtype, const GemmArgs& a, void* dst, hipStream_t st) {
  const int64_t E = dtype == MK_BF16 ? 8 : 4;
  dim3 grid((unsigned)((a.N + 32 * E - 1) / (32 * E)), (unsigned)((a.K + 8 * E - 1) / (8 * E)),
            (unsigned)(a.batch * a.heads));
  if (dtype == MK_BF16)
    hipLaunchKernelGGL(transpose_b_kernel<bf16>, grid, dim3(256), 0, st, a, (bf16*)dst);
  else
    hipLaunchKernelGGL(transpose_b_kernel<float>, grid, dim3(256), 0, st, a, (float*)dst);
  return hipGetLastError();
}

GemmArgs gemm_with_bt(const GemmArgs& a, const void* bt) {
  GemmArgs g = a;
  g.B = bt;
  g.layout = 0;
  g.ldb = a.K;
  g.b_off = 0;
  g.b_sh = a.N * a.K;
  g.b_sb = (int64_t)a.heads * a.N * a.K;
  return g;
}

// Compute units of the current device (cached per device).
static int cu_count() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cache[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

// The compiled epilogue for a plain GEMM's chain and terminal (kSigGeneric if
// none matches).
static int gemm_signature(const GemmArgs& a) {
  const EpiDev& e = a.epi;
  // (C and a residual are addressed through buffer resources: one batch,
  // 32-bit byte range)
  const bool buf = a.batch * a.heads == 1 && a.M * a.ldc * 2 < ((int64_t)1 << 31);
  // (a column bias is read with 16-byte loads)
  const bool bias_ok = e.n > 0 && e.code[0] == EPI_BIAS_COL && (uintptr_t)e.ptr[0] % 16 == 0;
  if (a.terminal == TERM_NONE && buf) {
    if (e.n == 0) return kSigNone;
    if (e.n == 1 && e.code[0] == EPI_GELU_ERF) return kSigGeluErf;
    if (e.n == 1 && e.code[0] == EPI_ADD) return kSigAdd;
    if (e.n == 1 && bias_ok) return kSigBias;
    if (e.n == 3 && bias_ok && e.code[1] == EPI_GELU_TANH && e.code[2] == EPI_SCALE)
      return kSigBiasGeluTanhScale;
  } else if (a.terminal == TERM_SOFTMAX && e.n == 3 && bias_ok && e.code[1] == EPI_GELU_TANH &&
             e.code[2] == EPI_SCALE) {
    return kSigBiasGeluTanhScaleSoftmax;
  }
  return kSigGeneric;
}

// The conv chain (channel bias, ReLU) ending in an average pool.
static bool conv_bias_relu_gap(const EpiDev& epi, bool gap, int pool) {
  return gap && pool == MK_OP_GAP && epi.n == 2 && epi.code[0] == EPI_BIAS_CH &&
         epi.code[1] == EPI_RELU;
}

bool conv_bias_relu_gap_wide(int dtype, int64_t C, int64_t PQ, const EpiDev& epi, bool gap,
                             int pool) {
  // bf16 only (fp32 MFMAs run four times longer per tile, and the ring form
  // with two workgroups per CU measured faster there); 128-byte rows of
  // channels; a 256-position tile spans at most two images (PQ >= 256).
  return dtype == MK_BF16 && conv_bias_relu_gap(epi, gap, pool) && C % 64 == 0 && PQ >= 256;
}

int64_t conv_gemm_tile_n(int dtype, int64_t C, int64_t PQ, const EpiDev& epi, bool gap,
                         int pool) {
  return conv_bias_relu_gap_wide(dtype, C, PQ, epi, gap, pool) ? 256 : kConvTileN;
}

static bool conv_wide(int dtype, const GemmArgs& a) {
  return a.conv && conv_bias_relu_gap_wide(dtype, a.cv_C, a.cv_P * a.cv_Q, a.epi,
                                           a.terminal == TERM_GAP, a.pool);
}

// The four-wave form (one wave per SIMD, 128 x 128 per wave) runs the
// compiled chains without a terminal when K is a multiple of the 64-deep
// stage.  MK_GEMM_WAVES=8 in the environment keeps the eight-wave form (for
// side-by-side measurement).
static bool four_wave_form(const GemmArgs& a, int sig) {
  static const int forced = [] {
    const char* e = getenv("MK_GEMM_WAVES");
    return e ? atoi(e) : 0;
  }();
  if (forced == 8) return false;
  return a.K % 64 == 0 && sig_plain(sig);
}

template <typename T>
static void launch_gemm_t(const GemmArgs& a, dim3 grid, hipStream_t st) {
  // Conv GEMMs: the bf16 (channel bias, ReLU, average pool) chain on the
  // persistent 256 x 256 kernel; the rest keep 64-byte rows and the
  // three-stage ring (two workgroups per CU; a slice of 32 bf16 channels stays
  // in one tap), with that chain compiled in where it applies.
  if (a.conv) {
    if (conv_wide(sizeof(T) == 2 ? MK_BF16 : MK_F32, a))
      hipLaunchKernelGGL((gemm_mfma_kernel<T, 4, 256, 2, 1, 2, 128, kSigConvBiasReluGap>), grid,
                         dim3(512), 0, st, a);
    else if (conv_bias_relu_gap(a.epi, a.terminal == TERM_GAP, a.pool))
      hipLaunchKernelGGL((gemm_mfma_kernel<T, 2, kConvTileN, 3, 1, 0, 64, kSigConvBiasReluGap>),
                         grid, dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((gemm_mfma_kernel<T, 2, kConvTileN, 3, 1, 0, 64, kSigGeneric>), grid,
                         dim3(256), 0, st, a);
  } else if constexpr (sizeof(T) != 2) {
    hipLaunchKernelGGL((gemm_mfma_kernel<T, 4, kGemmTileN, 2, 0, 2, 128, kSigGeneric>), grid,
                       dim3(512), 0, st, a);
  } else {
    const int sig = gemm_signature(a);
    if (four_wave_form(a, sig) && a.layout == 1) {
      if constexpr (sizeof(T) == 2) {
        switch (sig) {
#define MK_GEMM_SIG4KN(SIG)                                                                   \
  case SIG:                                                                                   \
    hipLaunchKernelGGL((gemm_mfma_kernel<T, 2, kGemmTileN, 2, 0, 4, 128, SIG>), grid, dim3(256), \
                       0, st, a);                                                             \
    break;
          MK_GEMM_SIG4KN(kSigNone)
          MK_GEMM_SIG4KN(kSigGeluErf)
          MK_GEMM_SIG4KN(kSigAdd)
          MK_GEMM_SIG4KN(kSigBias)
          default:
            MK_GEMM_SIG4KN(kSigBiasGeluTanhScale)
#undef MK_GEMM_SIG4KN
        }
      }
      return;
    }
    if (four_wave_form(a, sig)) {
      switch (sig) {
#define MK_GEMM_SIG4(SIG)                                                                     \
  case SIG:                                                                                   \
    hipLaunchKernelGGL((gemm_mfma_kernel<T, 2, kGemmTileN, 2, 0, 3, 128, SIG>), grid, dim3(256), \
                       0, st, a);                                                             \
    break;
        MK_GEMM_SIG4(kSigNone)
        MK_GEMM_SIG4(kSigGeluErf)
        MK_GEMM_SIG4(kSigAdd)
        MK_GEMM_SIG4(kSigBias)
        default:
          MK_GEMM_SIG4(kSigBiasGeluTanhScale)
#undef MK_GEMM_SIG4
      }
      return;
    }
    switch (sig) {
#define MK_GEMM_SIG(SIG)                                                                      \
  case SIG:                                                                                   \
    hipLaunchKernelGGL((gemm_mfma_kernel<T, 4, kGemmTileN, 2, 0, 2, 128, SIG>), grid, dim3(512), \
                       0, st, a);                                                             \
    break;
      MK_GEMM_SIG(kSigNone)
      MK_GEMM_SIG(kSigGeluErf)
      MK_GEMM_SIG(kSigAdd)
      MK_GEMM_SIG(kSigBiasGeluTanhScaleSoftmax)
      MK_GEMM_SIG(kSigBiasGeluTanhScale)
      MK_GEMM_SIG(kSigBias)
      default:
        MK_GEMM_SIG(kSigGeneric)
#undef MK_GEMM_SIG
    }
  }
}

// A [K, N] weight read in place by the four-wave form (no transpose): bf16,
// one matrix, 256-wide tiles, K a multiple of the stage, a compiled chain.
bool gemm_mfma_native_kn(int dtype, const GemmArgs& a) {
  return dtype == MK_BF16 && a.layout == 1 && !a.conv && a.batch * a.heads == 1 &&
         gemm_mfma_supported(dtype, a) && gemm_mfma_tile_n(dtype, a) == kGemmTileN &&
         four_wave_form(a, gemm_signature(a));
}

int64_t gemm_mfma_tile_n(int dtype, const GemmArgs& a) {
  if (a.conv) return conv_wide(dtype, a) ? 256 : kConvTileN;
  const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + kGemmTileN - 1) / kGemmTileN) *
                        (int64_t)a.batch * a.heads;
  return tiles < kSmallGemmTiles ? 64 : kGemmTileN;
}

hipError_t launch_gemm_mfma(int dtype, const GemmArgs& a, hipStream_t st) {
  const int E = dtype == MK_BF16 ? 8 : 4;
  if (a.conv) {
    const int BKe = (dtype == MK_BF16 ? 32 : 16) * (conv_wide(dtype, a) ? 2 : 1);   // slice depth
    if ((dtype != MK_BF16 && dtype != MK_F32) || a.cv_C % BKe || (a.cv_P * a.cv_Q) % 8 ||
        a.lda % E || a.K % BKe)
      return hipErrorInvalidValue;
  } else if (!gemm_mfma_supported(dtype, a) || (a.layout != 0 && !gemm_mfma_native_kn(dtype, a))) {
    return hipErrorInvalidValue;
  }
  if (((uintptr_t)a.A | (uintptr_t)a.B) % 16) return hipErrorInvalidValue;
  if (!a.conv && gemm_mfma_tile_n(dtype, a) == 64) return launch_gemm_small(dtype, a, st);
  const int64_t bn = gemm_mfma_tile_n(dtype, a);
  const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + bn - 1) / bn);
  // The 256 x 256 kernels run persistent workgroups, one per CU across the
  // batch; the ring conv kernel one workgroup per tile.  Conv: fewer tiles
  // than CUs are all cut into row sub-tiles (as the kernel's tail split
  // does for the last round), one workgroup each.
  int64_t gx = tiles;
  if (bn == 256) {
    const int64_t z = (int64_t)a.batch * a.heads;
    const int64_t g = std::max<int64_t>(1, (cu_count() + z - 1) / z);
    gx = std::min<int64_t>(tiles, g);
    if (a.conv && tiles < g) gx = tiles * tail_split((int)tiles, (int)g);
  }
  dim3 grid((unsigned)gx, (unsigned)(a.batch * a.heads));
  if (dtype == MK_BF16)
    launch_gemm_t<bf16>(a, grid, st);
  else
    launch_gemm_t<float>(a, grid, st);
  return hipGetLastError();
}

}  // namespace mk
