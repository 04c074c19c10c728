// Fused (flash) attention forward on gfx950 matrix cores, bf16 in, fp32
// accumulate:  o_i = sum_j softmax_j(q_i . k_j * scale  [j <= i]) v_j.
//
// This is the single-subkernel form of QK^T -> scale -> causal mask ->
// softmax -> PV: the paper's guidance fuses attention into one submodule when
// online softmax is possible (App. I.1), and its CvT attention kernel walks key
// blocks with a running max and sum (App. H.2).  Here:
//  * Each wave owns 64 queries (two 32-query tiles), so every K and V
//    fragment read from LDS feeds two MFMAs; a workgroup of NW waves shares
//    the K / V blocks, which arrive by direct HBM -> LDS loads in their
//    natural [key][dh] layout.  One wave per SIMD (512 registers).
//  * Scores are computed transposed, S^T = K Q^T, so each lane owns one query
//    and the softmax bookkeeping is lane-local (one exchange between the two
//    lane halves for the final row sum).  K's rows are read in a permuted
//    order (bits 2 and 3 of the key index swapped inside each 32-key tile) so
//    that the accumulator registers of S^T are, after exp, exactly the P^T
//    operand of the next MFMA with keys in natural order.
//  * O is accumulated transposed, O^T = V^T P^T; the V^T operand is read with
//    the transposing LDS load (ds_read_b64_tr_b16).
//  * exp is exp2 with log2(e) folded into the score scale; key blocks above
//    a wave's diagonal are skipped; the query blocks run heaviest first.
#include <type_traits>

#include "dev.hpp"

namespace mk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) char lds_char;

namespace {

constexpr int BKV = 64;              // keys per block
constexpr int kXcds = 8;
constexpr uint32_t kOob = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}

// Key row read by lane-row i of a 32-key tile: bits 2 and 3 swapped (an
// involution, so sigma(kt*32 + sigma(l)) & 7 == l & 7).
__device__ __forceinline__ int sigma(int i) {
  return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1);
}


template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// ---------------------------------------------------------------------------
// The kernel: 64 queries per wave (two 32-query tiles sharing every K and V
// fragment read, so the LDS traffic per MFMA is half that of a 32-query
// wave), one wave per SIMD (512 registers: scores, P and fragments in VGPRs;
// O and Q in AGPRs), NW waves per workgroup sharing the K and V blocks.
// Iteration j is software-pipelined:
//   region 1: S(j+1) = K(j+1) Q^T on the matrix cores, one MFMA at a time,
//             each followed by the exponentials, packing and row sums of
//             two of block j's probabilities;
//   region 2: O^T += V(j)^T P(j)^T, each MFMA followed by the scaling of
//             two of S(j+1)'s scores to log2 units relative to the
//             reference (and, spread over the slots, the loads of K(j+2)
//             and V(j+1)); then (wave's last block only) the mask of S(j+1).
// K blocks and V blocks have two LDS slots each; a barrier at the top of
// each iteration makes block j+1's K and block j's V visible to every wave
// and frees the slots the iteration's loads overwrite.
//
// Softmax reference: the max of each query's first key block.  It is never
// moved, so O and l never need rescaling (a rescale is a VALU pass over the
// AGPR-resident O, which this loop avoids): later scores above the reference
// give p > 1, which fp32 / bf16 hold up to 2^127, and the final O / l is the
// same quotient.  A key block whose probabilities sum past 2^38 (a score at
// least 2^32 above the reference) sets a flag, and the wave then recomputes
// its queries exactly on the slow path after the loop.
//
// Only a wave's last key block has masked entries (causal diagonal, sequence
// end).
constexpr int QW = 64;
// V chunk swizzle (16-byte chunks of a [key][dh] row, dh 128): the rows that
// one transposing read touches together differ in bits 0, 1 and 3; XOR-ing
// the chunk's bits 2-3 with g(r) spreads them over the four 64-byte bank
// groups (unswizzled, the rows lie 256 bytes apart and share one group).
template <int DH>
__device__ __forceinline__ int vswz(int r) {
  return DH >= 128 ? 4 * ((r & 3) ^ (((r >> 3) & 1) << 1)) : 0;
}
constexpr float kOverflowSum = 274877906944.0f;   // 2^38

// Matrix-core products with the register file of every operand fixed.  The
// compiler does not model these as MFMAs, so the code keeps the required
// distance between an MFMA and a VALU read of its result itself (other MFMAs
// in between, or mfma_drain()).  Nor does it keep the two wait states an MFMA
// needs after a VALU write of one of its sources: where it moves O between
// accumulator registers (a block whose register assignment differs from the
// loop's) the move can sit right before the product, so the O product starts
// with those two wait states itself.
__device__ __forceinline__ void mma_s0(f32x16& d, const bf16x8& k, const bf16x8& q) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(k), "a"(q));
}
__device__ __forceinline__ void mma_s(f32x16& d, const bf16x8& k, const bf16x8& q) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(k), "a"(q));
}
__device__ __forceinline__ void mma_o(f32x16& o, const bf16x8& v, const bf16x8& p) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(o) : "v"(v), "v"(p));
}
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15" ::: "memory"); }
// Transposing LDS read issued as asm: the compiler would otherwise wait for
// every outstanding direct-to-LDS load before it (it cannot tell that they
// fill other slots).  Its result is waited for with lds_wait<N>() and then
// redefined by an empty asm, so that the compiler reads it only after the
// wait.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <int OFF>
__device__ __forceinline__ void ld_tr_asm(u32x2& d, uint32_t addr) {
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(d) : "v"(addr), "i"(OFF));
}
template <int N>
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(%0)" :: "i"(N)); }
__device__ __forceinline__ void fence() { __builtin_amdgcn_sched_barrier(0); }

// Combine a value of lanes l and l ^ 32 (the two halves of one query's keys).
__device__ __forceinline__ float swap_max(float m) { return fmaxf(m, __shfl_xor(m, 32, 64)); }
__device__ __forceinline__ float swap_sum(float m) { return m + __shfl_xor(m, 32, 64); }

// Exact attention of one query row (one lane), fp32: the max over all kept
// keys first, then O = sum_j exp2(s_j - max) v_j / sum_j exp2(s_j - max), 32
// dh columns at a time.  Only reached when the pipelined loop's fixed
// reference could not hold a block's probabilities.
template <int DH>
__device__ void attn_row_exact(const bf16* q, const bf16* k, const bf16* v, int64_t ld3,
                               int jend, float sl2, bf16* o) {
  auto score = [&](int j) {
    float s = 0.f;
    for (int e = 0; e < DH; ++e) s = fmaf(bf2f(q[e]), bf2f(k[(int64_t)j * ld3 + e]), s);
    return s * sl2;
  };
  float mx = -INFINITY;
  for (int j = 0; j < jend; ++j) mx = fmaxf(mx, score(j));
  for (int c = 0; c < DH; c += 32) {
    float acc[32];
    for (int d = 0; d < 32; ++d) acc[d] = 0.f;
    float l = 0.f;
    for (int j = 0; j < jend; ++j) {
      const float p = exp2f(score(j) - mx);
      l += p;
      for (int d = 0; d < 32; ++d) acc[d] = fmaf(p, bf2f(v[(int64_t)j * ld3 + c + d]), acc[d]);
    }
    const float inv = l > 0.f ? 1.0f / l : 0.f;
    for (int d = 0; d < 32; ++d) o[c + d] = f2bf(acc[d] * inv);
  }
}

template <int DH, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW, 1) void attn_fwd_pipe_kernel(AttnArgs a) {
  constexpr int NKS = DH / 16;              // 16-deep k steps of S^T over dh
  constexpr int NDT = DH / 32;              // 32-row dh tiles of O^T
  constexpr int KROW = DH * 2;              // bytes per K / V row in LDS
  constexpr int KB = BKV * KROW;            // one K (or V) block
  constexpr int NT = 64 * NW;
  constexpr int BQW = QW * NW;              // queries per workgroup
  constexpr int LD = KB / 16 / NT;          // 16-byte loads per thread per block
  constexpr int R1 = NKS * 4;               // MFMAs of region 1 (S of a block)
  constexpr int R2 = 4 * NDT * 2;           // MFMAs of region 2 (PV of a block)
  constexpr int EPS = 32 / R1;              // exp pairs per region-1 slot
  static_assert(LD * 16 * NT == KB, "block must split evenly over the threads");
  static_assert(EPS * R1 == 32 && 64 % R2 == 0 && R1 % (2 * LD) == 0, "slot counts");
  __shared__ __attribute__((aligned(1024))) char smem[4 * KB];   // K0 K1 V0 V1

  const int64_t S = a.S, H = a.H;
  const int64_t ld3 = 3 * H * DH;
  const int nqb = (int)((S + BQW - 1) / BQW);
  // Work order: the hardware deals workgroups round-robin over the 8 XCDs
  // and, within one, to whichever CU frees up.  When the (batch, head) count
  // divides by 8, each XCD gets whole heads (their K and V fetched into one
  // L2) and takes its query blocks heaviest first across all of its heads
  // (longest-processing-time order: the causal blocks differ in length up to
  // nqb-fold); otherwise heads in order, heaviest block first within each.
  const int64_t total = (int64_t)gridDim.x;
  const int64_t zn = total / nqb;                          // (batch, head) count
  int64_t z;
  int qb;
  if (zn % kXcds == 0) {
    const int64_t zx = zn / kXcds;                         // heads per XCD
    const int64_t x = blockIdx.x % kXcds, i = blockIdx.x / kXcds;
    z = x * zx + i % zx;
    qb = nqb - 1 - (int)(i / zx);
  } else {
    z = blockIdx.x / nqb;
    qb = nqb - 1 - (int)(blockIdx.x % nqb);
  }
  const int64_t b = z / H, h = z % H;
  const int q0 = qb * BQW;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int Si = (int)S;
  const int qf = q0 + w * QW;                             // first query of the wave

  const bf16* qkv = (const bf16*)a.qkv;
  const bf16* Qb = qkv + b * S * ld3 + h * DH;
  const bf16* Kb = qkv + b * S * ld3 + H * DH + h * DH;
  const bf16* Vb = qkv + b * S * ld3 + 2 * H * DH + h * DH;
  const int64_t span = S * ld3 * 2;
  const __amdgpu_buffer_rsrc_t qsrc = make_rsrc(Qb, span);
  const __amdgpu_buffer_rsrc_t ksrc = make_rsrc(Kb, span);
  const __amdgpu_buffer_rsrc_t vsrc = make_rsrc(Vb, span);
  const uint32_t rowb = (uint32_t)(ld3 * 2);

  // Key blocks: the workgroup walks n_kv of them; this wave computes the
  // first nb_w, of which only the last can have masked entries.
  const int nkb = (Si + BKV - 1) / BKV;
  const int n_kv = CAUSAL ? min(nkb, q0 / BKV + NW) : nkb;
  int nb_w = qf >= Si ? 0 : CAUSAL ? qf / BKV + 1 : nkb;
  nb_w = __builtin_amdgcn_readfirstlane(nb_w);

  // Q^T operands (B of S^T = K Q^T): lane holds q[qf + 32 qt + lr][ks*16 + lh*8 .. +7].
  bf16x8 qfr[2][NKS];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int qi = qf + qt * 32 + lr;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t qoff = qi < Si ? (uint32_t)qi * rowb + (uint32_t)(ks * 16 + lh * 8) * 2 : kOob;
      qfr[qt][ks] = __builtin_bit_cast(bf16x8, bload(qsrc, qoff, 0));
    }
  }

  // K / V block loads (direct to LDS, [key][dh]); K chunks swizzled by
  // sigma(row) & 7 for conflict-free fragment reads.
  int lrow[LD];
  uint32_t koff[LD], voff[LD];
#pragma unroll
  for (int q = 0; q < LD; ++q) {
    const int p = (q * NW + w) * 64 + lane;
    lrow[q] = p / (DH / 8);
    const int pch = p % (DH / 8);
    koff[q] = (uint32_t)lrow[q] * rowb + (uint32_t)((pch ^ (sigma(lrow[q]) & 7)) * 16);
    voff[q] = (uint32_t)lrow[q] * rowb + (uint32_t)((pch ^ vswz<DH>(lrow[q])) * 16);
  }
  const int wu = __builtin_amdgcn_readfirstlane(w);
  // Load q (of LD) of this thread's share of key block j into dst.  The
  // block's row offset is the scalar offset; rows past the sequence lie past
  // the buffer's range and read zeros.  Blocks past the workgroup's last are
  // clamped to it (a reload into a slot nobody reads again).
  auto issue1 = [&](__amdgpu_buffer_rsrc_t src, const uint32_t (&off0)[LD], int j, char* dst,
                    int q) {
    const uint32_t soff = (uint32_t)min(j, n_kv - 1) * BKV * rowb;
    // The wave's 1 KB offset, re-derived at every load so the destination is
    // one scalar add from it (a table of every destination, hoisted out of
    // the loop, spills the scalar registers into vector lanes).
    uint32_t wo = (uint32_t)wu * 1024u;
    asm volatile("" : "+s"(wo));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        src, (lds_void*)((lds_char*)dst + wo + q * NW * 1024), 16, (int)off0[q], (int)soff, 0, 0);
  };
  auto issue = [&](__amdgpu_buffer_rsrc_t src, const uint32_t (&off0)[LD], int j, char* dst) {
#pragma unroll
    for (int q = 0; q < LD; ++q) issue1(src, off0, j, dst, q);
  };
  const int krd = sigma(lr) * KROW;
  const int kch = lr & 7;
  // Transposed V reads: in each 16-lane group lane i receives element i%4 of
  // the 8-byte pieces addressed by lanes i/4 + 4e, so lane j addresses key
  // row 8*(g/2) + j/4 and dh column 16*(g%2) + 4*(j%4) of a 16-key step
  // (g = lane/16), and every lane gets 4 consecutive keys of one dh column.
  uint32_t vaddr[NDT];
  {
    const int tj = lane & 15, tg = lane >> 4;
    const int vrow = (tg >> 1) * 8 + (tj >> 2);
    const int vcol = (tg & 1) * 16 + 4 * (tj & 3);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
#pragma unroll
    for (int t = 0; t < NDT; ++t) {
      const int e = t * 32 + vcol;                          // dh element
      vaddr[t] = lds0 + (uint32_t)(vrow * KROW + (((e / 8) ^ vswz<DH>(vrow)) * 16) + (e % 8) * 2);
    }
  }

  f32x16 o[NDT][2];
#pragma unroll
  for (int t = 0; t < NDT; ++t)
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][qt][r] = 0.f;
      asm volatile("" : "+a"(o[t][qt]));
    }
  f32x16 sc[2][4];                                        // [buffer][kt*2 + qt]
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 pk[2][4];                                         // P of a block: [qt][k step]
  float l_run[2] = {0.f, 0.f}, mneg[2] = {0.f, 0.f};
  bool over = false;
  const float sl2 = a.scale * 1.4426950408889634f;

  auto kfrag = [&](int slot, int ks, int kt) -> bf16x8 {
    return *(const bf16x8*)(smem + slot * KB + krd + kt * 32 * KROW + (((ks * 2 + lh) ^ kch) * 16));
  };
  // Pair e of 32 (qt = e/16, kt = e/8 % 2, registers 2(e%8), +1) of a block
  // whose scores already hold s * scale * log2(e) - m: exp2, packed into P.
  auto exp_pair = [&](int C, int e, float (&d)[2]) {
    const int qt = e >> 4, kt = (e >> 3) & 1, rp = e & 7;
    d[0] = __builtin_amdgcn_exp2f(sc[C][kt * 2 + qt][2 * rp]);
    d[1] = __builtin_amdgcn_exp2f(sc[C][kt * 2 + qt][2 * rp + 1]);
  };
  auto pack_pair = [&](int e, const float (&d)[2]) {
    const int qt = e >> 4, kt = (e >> 3) & 1, rp = e & 7;
    pk[qt][kt * 2 + (rp >> 2)][rp & 3] = pack2_bf16(d[0], d[1]);
  };
  // Scores of tile m of block B_ to s * scale * log2(e) - m (registers r0 .. r0+n-1).
  auto to_log2 = [&](int B_, int m, int r0, int n) {
#pragma unroll
    for (int r = r0; r < r0 + n; ++r) sc[B_][m][r] = fmaf(sc[B_][m][r], sl2, mneg[m & 1]);
  };
  // Mask of key block j in sc[B_], tile m: key kv0 + k is dropped for query q
  // when k > lim (causal: past q, or for the off-by-one mutant at q; past the
  // sequence end).  Blocks wholly below the wave's queries get lim >= 63.
  auto mask_tile = [&](int B_, int j, int m) {
    const int kt = m >> 1, qt = m & 1;
    const int kv0 = j * BKV;
    const int kmax = min(BKV, Si - kv0);
    const int qrel = qf + qt * 32 + lr - kv0;
    const int lim = CAUSAL ? min(a.causal == 2 ? qrel - 1 : qrel, kmax - 1) : kmax - 1;
    // All-ones when k > lim, from the sign of lim - k, kept in a vector
    // register (a compare per register would hold 64 lane masks in scalar
    // register pairs and spill the loop's scalars).
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int k = kt * 32 + (r >> 3) * 16 + lh * 8 + (r & 7);
      uint32_t drop = (uint32_t)((lim - k) >> 31);
      asm volatile("" : "+v"(drop));
      const uint32_t v = __float_as_uint(sc[B_][m][r]);
      sc[B_][m][r] = __uint_as_float((v & ~drop) | (0xff800000u & drop));
    }
  };

  // Prologue: K(0) into slot 0, then K(1) and V(0); S(0), its mask and the
  // reference (the block max).
  issue(ksrc, koff, 0, smem);
  issue(ksrc, koff, 1, smem + KB);
  issue(vsrc, voff, 0, smem + 2 * KB);
  wait_vm<2 * LD>();
  __builtin_amdgcn_s_barrier();
  if (nb_w > 0) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const bf16x8 k0 = kfrag(0, ks, 0), k1 = kfrag(0, ks, 1);
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        if (ks == 0) mma_s0(sc[0][m], (m >> 1) ? k1 : k0, qfr[m & 1][ks]);
        else mma_s(sc[0][m], (m >> 1) ? k1 : k0, qfr[m & 1][ks]);
      }
    }
    mfma_drain();
    if (nb_w == 1) {   // block 0 is masked only when it is the wave's last
#pragma unroll
      for (int m = 0; m < 4; ++m) mask_tile(0, 0, m);
    }
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 32; ++i) mx = fmaxf(mx, sc[0][(i >> 4) * 2 + qt][i & 15]);
      const float m = swap_max(mx) * sl2;
      mneg[qt] = m == -INFINITY ? 0.f : -m;
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) to_log2(0, m, 0, 16);
  }

  // Iteration j (C = j % 2): S(j) in sc[C], K(j+1) in K slot 1-C, V(j) in V
  // slot C.  On a wave's last block (LAST) there is no S(j+1): region 1 is
  // the exponentials alone, region 2 the PV products alone, and the wave's
  // share of the workgroup's next loads goes out at the top.
  auto iter = [&](int j, auto PAR, auto LAST_) {
    constexpr int C = decltype(PAR)::value, N = 1 - C;
    constexpr bool LAST = decltype(LAST_)::value;
    if constexpr (LAST) {
      issue(ksrc, koff, j + 2, smem + C * KB);
      issue(vsrc, voff, j + 1, smem + (2 + N) * KB);
    }
    fence();
    // V^T fragments of one k step of region 2: 2 transposing reads per dh
    // tile, issued one k step ahead; lds_wait<2*NDT> before a step's MFMAs
    // leaves only the next step's reads in flight.
    u32x2 vr[2][NDT][2];
    auto vreads = [&](auto KS) {
      constexpr int ks = decltype(KS)::value;
      constexpr int base = (2 + C) * KB + ks * 16 * KROW;   // < 64 KB: an immediate offset
      ld_tr_asm<base>(vr[ks & 1][0][0], vaddr[0]);
      ld_tr_asm<base + 4 * KROW>(vr[ks & 1][0][1], vaddr[0]);
      ld_tr_asm<base>(vr[ks & 1][1][0], vaddr[1]);
      ld_tr_asm<base + 4 * KROW>(vr[ks & 1][1][1], vaddr[1]);
      if constexpr (NDT > 2) {
        ld_tr_asm<base>(vr[ks & 1][2 % NDT][0], vaddr[2 % NDT]);
        ld_tr_asm<base + 4 * KROW>(vr[ks & 1][2 % NDT][1], vaddr[2 % NDT]);
        ld_tr_asm<base>(vr[ks & 1][3 % NDT][0], vaddr[3 % NDT]);
        ld_tr_asm<base + 4 * KROW>(vr[ks & 1][3 % NDT][1], vaddr[3 % NDT]);
      }
    };
    float ls[2][2] = {{0.f, 0.f}, {0.f, 0.f}};   // row sums of P(j): [qt][parity]
    // Region 1: K fragments three k steps ahead; after the MFMA of slot e,
    // the exponentials of pair e and the pack and row sum of pair e-1 (so no
    // VALU op waits on the one before it).
    {
      bf16x8 kf[4][2];
      if constexpr (!LAST) {
#pragma unroll
        for (int ks = 0; ks < 3; ++ks) {
          kf[ks][0] = kfrag(N, ks, 0);
          kf[ks][1] = kfrag(N, ks, 1);
        }
      }
      float pv[2][2];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        if (!LAST && ks + 3 < NKS) {
          kf[(ks + 3) & 3][0] = kfrag(N, ks + 3, 0);
          kf[(ks + 3) & 3][1] = kfrag(N, ks + 3, 1);
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          if constexpr (!LAST) {
            if (ks == 0) mma_s0(sc[N][m], kf[ks & 3][m >> 1], qfr[m & 1][ks]);
            else mma_s(sc[N][m], kf[ks & 3][m >> 1], qfr[m & 1][ks]);
          }
          // The first V^T reads of region 2 (V(j) has been in LDS since the
          // top of this iteration), two slots before the region ends: after
          // the compiler's wait for the last K fragment, which would
          // otherwise also wait for these reads.
          if (ks * 4 + m == R1 - 2) vreads(std::integral_constant<int, 0>{});
          {
            const int slot = ks * 4 + m;
            // Next blocks' loads, one every R1 / (2 LD) slots: K(j+2) into K
            // slot C (K(j) was read in the previous iteration), V(j+1) into V
            // slot N (V(j-1) likewise); the barrier at the top of this
            // iteration ordered those reads before these writes.
            constexpr int every = R1 / (2 * LD);
            if (!LAST && slot % every == 0) {
              const int q = slot / every;
              if (q < LD) issue1(ksrc, koff, j + 2, smem + C * KB, q);
              else issue1(vsrc, voff, j + 1, smem + (2 + N) * KB, q - LD);
            }
          }
#pragma unroll
          for (int i = 0; i < EPS; ++i) {
            const int e = (ks * 4 + m) * EPS + i;          // pair 0..31
            exp_pair(C, e, pv[e & 1]);
            if (e >= 1) {
              pack_pair(e - 1, pv[(e - 1) & 1]);
              float& l = ls[(e - 1) >> 4][(e - 1) & 1];
              l += pv[(e - 1) & 1][0] + pv[(e - 1) & 1][1];
              asm volatile("" : "+v"(l));   // keep the add in this slot
            }
          }
          fence();
        }
      }
      pack_pair(31, pv[1]);
      ls[1][1] += pv[1][0] + pv[1][1];
    }
    // Region 2.
    {
      auto kstep = [&](auto KS) {
        constexpr int ks = decltype(KS)::value;
        if constexpr (ks + 1 < 4) {
          vreads(std::integral_constant<int, ks + 1>{});
          lds_wait<2 * NDT>();
        } else {
          lds_wait<0>();
        }
        // The asm reads' results exist only from here on: redefine them after
        // the wait so that no copy of them is placed before it.
#pragma unroll
        for (int t = 0; t < NDT; ++t)
          asm volatile("" : "+v"(vr[ks & 1][t][0]), "+v"(vr[ks & 1][t][1]));
#pragma unroll
        for (int m = 0; m < 2 * NDT; ++m) {
          const int slot = ks * 2 * NDT + m;
          const int t = m >> 1, qt = m & 1;
          const bf16x8 vf = __builtin_bit_cast(
              bf16x8, __builtin_shufflevector(vr[ks & 1][t][0], vr[ks & 1][t][1], 0, 1, 2, 3));
          mma_o(o[t][qt], vf, __builtin_bit_cast(bf16x8, pk[qt][ks]));
          // S(j+1) to log2 units, 64 / R2 registers per slot, tile by tile in
          // the order its MFMA chains finished (tile 0 three MFMAs before the
          // end of region 1); pinned here (the compiler would otherwise sink
          // them to their use in the next iteration).
          if constexpr (!LAST) {
            constexpr int per = 64 / R2;
            const int t0 = (slot * per) >> 4, r0 = (slot * per) & 15;
            to_log2(N, t0, r0, per);
            if (r0 + per == 16) asm volatile("" : "+v"(sc[N][t0]));
          }
          fence();
        }
      };
      kstep(std::integral_constant<int, 0>{});
      kstep(std::integral_constant<int, 1>{});
      kstep(std::integral_constant<int, 2>{});
      kstep(std::integral_constant<int, 3>{});
      // Mask of S(j+1) when block j+1 is the wave's last (causal diagonal /
      // sequence end); 32 MFMAs after its last product.
      if (!LAST && j + 2 >= nb_w) {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) mask_tile(N, j + 1, mt);
      }
      if constexpr (LAST) {
        // O's last products: the compiler does not see these MFMAs and
        // would copy O out of the AGPRs right behind them; drain first, then
        // redefine O so that every copy comes after the drain.
        mfma_drain();
#pragma unroll
        for (int t = 0; t < NDT; ++t)
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) asm volatile("" : "+a"(o[t][qt]));
      }
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const float lb = ls[qt][0] + ls[qt][1];
        over |= !(lb <= kOverflowSum);
        l_run[qt] += lb;
      }
    }
  };
  // Top of iteration j: block j+1's K and block j's V (issued during
  // iteration j-1) have landed for every wave, and every wave is done with
  // the slots the loads of this iteration overwrite.  A wave past its own
  // blocks still issues its share of the loads.
  auto top = [&](int j) {
    wait_vm<0>();
    __builtin_amdgcn_s_barrier();
  };
  auto top_idle = [&](int j, int par) {
    top(j);
    issue(ksrc, koff, j + 2, smem + par * KB);
    issue(vsrc, voff, j + 1, smem + (3 - par) * KB);
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  using Full = std::integral_constant<bool, false>;
  using Last = std::integral_constant<bool, true>;
  int j = 0;
  for (; j + 2 < nb_w; j += 2) {
    top(j);
    iter(j, P0{}, Full{});
    top(j + 1);
    iter(j + 1, P1{}, Full{});
  }
  if (nb_w - j == 2) {
    top(j);
    iter(j, P0{}, Full{});
    top(j + 1);
    iter(j + 1, P1{}, Last{});
    j += 2;
  } else if (nb_w - j == 1) {
    top(j);
    iter(j, P0{}, Last{});
    ++j;
  }
  for (; j < n_kv; ++j) top_idle(j, j & 1);
  wait_vm<0>();   // no direct-to-LDS load may land after the workgroup ends
  mfma_drain();

  bf16* O = (bf16*)a.o + b * S * H * DH + h * DH;
  if (__builtin_amdgcn_ballot_w64(over) != 0) {
    // Slow path: one lane per query of the wave.
    const int q = qf + lane;
    if (q < Si) {
      const int jend = CAUSAL ? (a.causal == 2 ? q : q + 1) : Si;
      attn_row_exact<DH>(Qb + (int64_t)q * ld3, Kb, Vb, ld3, jend, sl2, O + (int64_t)q * H * DH);
    }
    return;
  }
  // Normalise and store O[b, q, h*DH + d]: lane (lr, lh) holds, per dh tile,
  // rows 8g + 4 lh + 0..3 of query qf + 32 qt + lr (8-byte stores).
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const float l_tot = swap_sum(l_run[qt]);
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    const int q = qf + qt * 32 + lr;
    if (q < Si) {
      bf16* orow = O + (int64_t)q * H * DH;
#pragma unroll
      for (int t = 0; t < NDT; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint2 v;
          v.x = pack2_bf16(o[t][qt][g * 4 + 0] * inv, o[t][qt][g * 4 + 1] * inv);
          v.y = pack2_bf16(o[t][qt][g * 4 + 2] * inv, o[t][qt][g * 4 + 3] * inv);
          *(uint2*)(orow + t * 32 + g * 8 + lh * 4) = v;
        }
    }
  }
}

}  // namespace

int attn_fused_limit(int dtype, const AttnArgs& a) {
  if (dtype != MK_BF16) return MK_LIMIT_DTYPE;
  if (a.dh != 64 && a.dh != 128) return MK_LIMIT_SHAPE;
  const int64_t ld3 = 3 * a.H * a.dh;
  return a.S * ld3 * 2 < ((int64_t)1 << 31) && a.B * a.H * ((a.S + 2 * QW - 1) / (2 * QW)) < (1ll << 31)
             ? MK_LIMIT_NONE
             : MK_LIMIT_RANGE;
}

bool attn_fused_supported(int dtype, const AttnArgs& a) {
  return attn_fused_limit(dtype, a) == MK_LIMIT_NONE;
}

hipError_t launch_attn_fused(int dtype, const AttnArgs& a, hipStream_t st) {
  if (!attn_fused_supported(dtype, a)) return hipErrorInvalidValue;
  if ((uintptr_t)a.qkv % 16 || (uintptr_t)a.o % 16) return hipErrorInvalidValue;
  // Two waves (128 queries) per workgroup, two workgroups per CU.
  constexpr int NW = 2;
  const unsigned grid = (unsigned)(a.B * a.H * ((a.S + QW * NW - 1) / (QW * NW)));
  if (a.dh == 128) {
    if (a.causal)
      hipLaunchKernelGGL((attn_fwd_pipe_kernel<128, true, NW>), dim3(grid), dim3(64 * NW), 0, st, a);
    else
      hipLaunchKernelGGL((attn_fwd_pipe_kernel<128, false, NW>), dim3(grid), dim3(64 * NW), 0, st, a);
  } else {
    if (a.causal)
      hipLaunchKernelGGL((attn_fwd_pipe_kernel<64, true, NW>), dim3(grid), dim3(64 * NW), 0, st, a);
    else
      hipLaunchKernelGGL((attn_fwd_pipe_kernel<64, false, NW>), dim3(grid), dim3(64 * NW), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace mk
