// Fused (flash) attention forward on gfx950 matrix cores, bf16 in, fp32
// accumulate:  o_i = sum_j softmax_j(q_i . k_j * scale  [j <= i]) v_j.
//
// This is the single-subkernel form of QK^T -> scale -> causal mask ->
// softmax -> PV: the paper's guidance fuses attention into one submodule when
// online softmax is possible (App. I.1), and its CvT attention kernel walks key
// blocks with a running max and sum (App. H.2).  Here:
//  * One workgroup (4 waves) per (batch, head, 128-query block); each wave
//    owns 32 queries.  Query blocks are issued heaviest-first (causal).
//  * Scores are computed transposed, S^T = K Q^T, so each lane owns one query
//    and the running max / sum are lane-local (one cross-half exchange per
//    key block).  K's rows are read in a permuted order (bits 2 and 3 of the
//    key index swapped inside each 32-key tile) so that the accumulator
//    registers of S^T are, after exp, exactly the P^T operand of the next
//    MFMA with keys in natural order; no lane shuffles are needed.
//  * O is accumulated transposed, O^T = V^T P^T, so the per-query rescale
//    exp(m_old - m_new) is lane-local as well.  K and V both arrive by direct
//    HBM -> LDS loads in their natural [key][dh] layout; the V^T operand is
//    read with the transposing LDS load (ds_read_b64_tr_b16): within each
//    16-lane group, lane i receives element i%4 of the 8-byte chunks addressed
//    by lanes i/4, i/4+4, i/4+8, i/4+12, so lane j addressing key k0 + j/4,
//    dh d0 + 4*(j%4) hands every lane 4 consecutive keys of one dh column.
//  * exp is exp2 with log2(e) folded into the score scale; key blocks above
//    a wave's diagonal are skipped.
#include <type_traits>

#include "dev.hpp"

namespace mk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

namespace {

constexpr int BQ = 128, BKV = 64, kThreads = 256;
constexpr float kLazy = 8.0f;   // log2 headroom of the running softmax reference
constexpr int kXcds = 8;
constexpr uint32_t kOob = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// Four 16-bit values by the transposing LDS read (see the header comment).
__device__ __forceinline__ v4i16 ld_tr(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
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

template <int DH, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  constexpr int NKS = DH / 16;              // 16-deep k steps of S^T over dh
  constexpr int NDT = DH / 32;              // 32-row dh tiles of O^T
  constexpr int KROW = DH * 2;              // bytes per K row in LDS
  constexpr int KBYTES = BKV * KROW;        // K block
  constexpr int STAGE = 2 * KBYTES;         // K block + V block, both [key][dh]
  constexpr int KCH = BKV * DH / 8;         // 16-byte chunks of a K block
  constexpr int KLOADS = KCH / kThreads;    // per thread
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int64_t S = a.S, H = a.H;
  const int64_t ld3 = 3 * H * DH;
  const int nqb = (int)((S + BQ - 1) / BQ);
  // The hardware deals workgroups round-robin over the 8 XCDs.  When the
  // grid divides evenly, the query blocks of one (batch, head) are all sent
  // to one XCD (heaviest first), so that head's K and V are fetched into one
  // L2 instead of eight.
  int64_t bid = blockIdx.x;
  const int64_t total = (int64_t)gridDim.x;
  if (total % kXcds == 0) bid = (bid % kXcds) * (total / kXcds) + bid / kXcds;
  const int64_t z = bid / nqb;
  const int qb = nqb - 1 - (int)(bid % nqb);              // heaviest first
  const int64_t b = z / H, h = z % H;
  const int64_t q0 = (int64_t)qb * BQ;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int64_t wq0 = q0 + w * 32;
  const int64_t qi = wq0 + lr;                            // this lane's query

  const bf16* qkv = (const bf16*)a.qkv;
  const bf16* Qb = qkv + b * S * ld3 + h * DH;
  const bf16* Kb = qkv + b * S * ld3 + H * DH + h * DH;
  const bf16* Vb = qkv + b * S * ld3 + 2 * H * DH + h * DH;
  const int64_t span = S * ld3 * 2;                       // bytes of one sequence's rows
  const __amdgpu_buffer_rsrc_t qsrc = make_rsrc(Qb, span);
  const __amdgpu_buffer_rsrc_t ksrc = make_rsrc(Kb, span);
  const __amdgpu_buffer_rsrc_t vsrc = make_rsrc(Vb, span);

  // Q^T operand (B of S^T = K Q^T): lane holds q[qi][ks*16 + lh*8 .. +7].
  bf16x8 qf[NKS];
  // Row offsets that can leave the sequence live in the per-lane offset (the
  // range check covers it) with out-of-range rows mapped past the end.
  {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t qoff = qi < S ? (uint32_t)(qi * ld3 * 2 + (ks * 16 + lh * 8) * 2) : kOob;
      qf[ks] = __builtin_bit_cast(bf16x8, bload(qsrc, qoff, 0));
    }
  }

  const int Si = (int)S, wq0i = (int)wq0, qii = (int)qi;
  const int nkb = (int)((S + BKV - 1) / BKV);
  const int n_kv = CAUSAL ? min(nkb, (int)((q0 + BQ + BKV - 1) / BKV)) : nkb;

  // K and V: direct loads into LDS as [key][dh].  Load q of wave w, lane i
  // fills LDS chunk p = (q*4 + w)*64 + i: row p / (DH/8), physical chunk
  // p % (DH/8).  K's chunks are XOR-swizzled by sigma(row) & 7 so that the 32
  // rows of a fragment read (row sigma(lane)) fall in distinct banks; V is
  // read with transposing loads, which are conflict-free unswizzled.
  int krow_of[KLOADS], kchunk[KLOADS], vchunk[KLOADS];
#pragma unroll
  for (int q = 0; q < KLOADS; ++q) {
    const int p = (q * 4 + w) * 64 + lane;
    krow_of[q] = p / (DH / 8);
    vchunk[q] = p % (DH / 8);
    kchunk[q] = vchunk[q] ^ (sigma(krow_of[q]) & 7);
  }
  // Byte offsets of this lane's rows within a block (32-bit: the sequence's
  // rows span less than 2 GB) and the wave's LDS chunks (wave-uniform).
  const uint32_t rowb = (uint32_t)(ld3 * 2);
  uint32_t koff[KLOADS], voff[KLOADS];
#pragma unroll
  for (int q = 0; q < KLOADS; ++q) {
    koff[q] = (uint32_t)krow_of[q] * rowb + kchunk[q] * 16;
    voff[q] = (uint32_t)krow_of[q] * rowb + vchunk[q] * 16;
  }
  const int wu = __builtin_amdgcn_readfirstlane(w);
  // One block of K or V into dst (rows past the sequence read zeros).
  auto issue = [&](__amdgpu_buffer_rsrc_t src, const uint32_t (&off0)[KLOADS], int j, char* dst) {
    const int krem = (int)min<int64_t>(S - (int64_t)j * BKV, BKV);   // keys left in the block
    const uint32_t jb = (uint32_t)j * BKV * rowb;
#pragma unroll
    for (int q = 0; q < KLOADS; ++q) {
      const uint32_t off = krow_of[q] < krem ? off0[q] + jb : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (q * 4 + wu) * 1024), 16,
                                               (int)off, 0, 0, 0);
    }
  };
  // Per-lane part of the transposed V read: key row j/4 of 4, dh column
  // 16*(group%2) + 4*(j%4) (+ 32 t); group = lane/16 also selects the key half.
  const int tj = lane & 15, tg = lane >> 4;
  const int vtr_off = ((tg >> 1) * 8 + (tj >> 2)) * KROW + ((tg & 1) * 16 + 4 * (tj & 3)) * 2;

  f32x16 oacc[NDT];
#pragma unroll
  for (int t = 0; t < NDT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;   // scale * log2(e)

  issue(ksrc, koff, 0, smem);
  issue(vsrc, voff, 0, smem + KBYTES);

  // Block j uses stage j % 2; the loop body is instantiated for both
  // parities so that the stage base is a constant offset of the LDS reads.
  auto block = [&](int j, auto PAR) {
    constexpr int par = decltype(PAR)::value;
    char* cur = smem + par * STAGE;
    char* nxt = smem + (1 - par) * STAGE;
    // Block j has landed (this wave's loads); the barrier makes every wave's
    // loads visible and guarantees block j-1's slot is no longer read.
    wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    if (j + 1 < n_kv) {
      issue(ksrc, koff, j + 1, nxt);
      issue(vsrc, voff, j + 1, nxt + KBYTES);
    }
    const int kv0 = j * BKV;                       // (sequences are below 2^31 rows)
    const bool active = !CAUSAL || kv0 <= wq0i + 31;
    if (active) {
      // S^T for the block: two 32-key tiles, their MFMA chains interleaved
      // (each MFMA's successor on the same accumulator waits for it).
      f32x16 sacc[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kt][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const char* krow = cur + (kt * 32 + sigma(lr)) * KROW;
          const bf16x8 kf = *(const bf16x8*)(krow + (((ks * 2 + lh) ^ (lr & 7)) * 16));
          sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sacc[kt], 0, 0, 0);
        }
      // Scores, mask, running max, in units of log2: s * scale * log2(e).
      // Register r of tile kt holds key kv0 + kt*32 + (r/8)*16 + lh*8 + r%8
      // for query qi.  Only blocks that cross the wave's diagonal or the end
      // of the sequence need the mask.
      const bool need_mask = (CAUSAL && kv0 + BKV - 1 > wq0i) || kv0 + BKV > Si;
      if (need_mask) {
        const int qrel = qii - kv0;                 // keys kv0 + k with k > qrel are masked
        const int kmax = min(BKV, Si - kv0);
        const int lim = CAUSAL ? min(a.causal == 2 ? qrel - 1 : qrel, kmax - 1) : kmax - 1;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int k = kt * 32 + (r >> 3) * 16 + lh * 8 + (r & 7);
            if (k > lim) sacc[kt][r] = -INFINITY;
          }
      }
      float mloc = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sacc[kt][r]);
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * sl2;
      // The reference m_run moves only when the block's max exceeds it by
      // more than kLazy (log2 units): probabilities stay below 2^kLazy, and
      // the rescale of O and l (exact either way: both carry the same
      // reference) is skipped for most blocks.
      const float m_new = mloc > m_run + kLazy ? mloc : m_run;
      const float mneg = m_new == -INFINITY ? 0.f : -m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run + mneg);   // 0 on the first block
      float lsum = 0.f;
      uint32_t pp[2][8];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[kt][r], sl2, mneg));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[kt][r + 1], sl2, mneg));
          lsum += p0 + p1;
          pp[kt][r >> 1] = pack2_bf16(p0, p1);
        }
      l_run = l_run * alpha + lsum;
      m_run = m_new;
      if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {
#pragma unroll
        for (int t = 0; t < NDT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[t][r] *= alpha;
      }
      // O^T += V^T P^T over the block's 4 key steps.
      const char* vb = cur + KBYTES + vtr_off;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        uint4 praw;
        praw.x = pp[ks >> 1][(ks & 1) * 4 + 0];
        praw.y = pp[ks >> 1][(ks & 1) * 4 + 1];
        praw.z = pp[ks >> 1][(ks & 1) * 4 + 2];
        praw.w = pp[ks >> 1][(ks & 1) * 4 + 3];
        const bf16x8 pf = __builtin_bit_cast(bf16x8, praw);
#pragma unroll
        for (int t = 0; t < NDT; ++t) {
          const char* p = vb + ks * 16 * KROW + t * 32 * 2;
          const v4i16 lo = ld_tr(p), hi = ld_tr(p + 4 * KROW);
          const bf16x8 vf = __builtin_bit_cast(
              bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, oacc[t], 0, 0, 0);
        }
      }
    }
  };
  for (int j = 0; j < n_kv; j += 2) {
    block(j, std::integral_constant<int, 0>{});
    if (j + 1 < n_kv) block(j + 1, std::integral_constant<int, 1>{});
  }
  wait_vm<0>();
  __syncthreads();

  // Normalise and write O[b, q, h*DH + d] through LDS for 16-byte stores.
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  bf16* ot = (bf16*)smem + w * 32 * (DH + 8);             // [32 queries][DH] per wave
#pragma unroll
  for (int t = 0; t < NDT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int d = t * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
      ot[lr * (DH + 8) + d] = f2bf(oacc[t][r] * inv);
    }
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_wave_barrier();
  bf16* O = (bf16*)a.o + b * S * H * DH + h * DH;
  constexpr int CPR = DH / 8;                                // 16-byte chunks per row
  for (int c = lane; c < 32 * CPR; c += 64) {
    const int ql = c / CPR, ch = c % CPR;
    const int64_t q = wq0 + ql;
    if (q < S) *(uint4*)(O + q * H * DH + ch * 8) = *(const uint4*)(ot + ql * (DH + 8) + ch * 8);
  }
}

}  // namespace

int attn_fused_limit(int dtype, const AttnArgs& a) {
  if (dtype != MK_BF16) return MK_LIMIT_DTYPE;
  if (a.dh != 64 && a.dh != 128) return MK_LIMIT_SHAPE;
  const int64_t ld3 = 3 * a.H * a.dh;
  return a.S * ld3 * 2 < ((int64_t)1 << 31) && a.B * a.H * ((a.S + BQ - 1) / BQ) < (1ll << 31)
             ? MK_LIMIT_NONE
             : MK_LIMIT_RANGE;
}

bool attn_fused_supported(int dtype, const AttnArgs& a) {
  return attn_fused_limit(dtype, a) == MK_LIMIT_NONE;
}

hipError_t launch_attn_fused(int dtype, const AttnArgs& a, hipStream_t st) {
  if (!attn_fused_supported(dtype, a)) return hipErrorInvalidValue;
  if ((uintptr_t)a.qkv % 16 || (uintptr_t)a.o % 16) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)(a.B * a.H * ((a.S + BQ - 1) / BQ));
  if (a.dh == 128) {
    if (a.causal)
      hipLaunchKernelGGL((attn_fwd_kernel<128, true>), dim3(grid), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<128, false>), dim3(grid), dim3(kThreads), 0, st, a);
  } else {
    if (a.causal)
      hipLaunchKernelGGL((attn_fwd_kernel<64, true>), dim3(grid), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<64, false>), dim3(grid), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace mk
