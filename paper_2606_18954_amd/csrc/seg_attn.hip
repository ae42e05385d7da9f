// Grouped segment attention (gfx950): one work item = (segment, page chunk, row block, kv-head).
//
// All branches that share a segment (B(s), from the scheduler) attend over its tokens together:
// their queries for the kv-head's q-head group form a tile of R = |B(s)| * (Hq/Hkv) rows, so the
// segment's K/V are read from HBM once per kv-head and used by every row.  That turns the
// memory-bound decode step into a dense contraction per segment:
//
//   S^T = K Q^T   (16 tokens x 16 rows per MFMA tile, contraction over head_dim)
//   O^T += V^T P^T (contraction over tokens)
//
// Computing the transposed products keeps every row's state in one lane column: lane l owns row
// l % 16 of a tile, holds scores of tokens 4*(l/16)..+3, and holds output columns
// 16n + 4*(l/16)..+3.  The softmax scores come out of the first MFMA in exactly the register
// layout the second MFMA takes as its B operand, so no shuffles are needed between them.
//
// Data movement: K/V pages of one kv-head are 16 x D contiguous blocks in HBM.  They are copied
// straight into LDS with the gfx950 direct-to-LDS load (global_load_lds_dwordx4: every lane moves
// 16 bytes, a wave instruction fills 1 KiB of LDS), so no VGPRs stage the data and several stages
// stay in flight: a ring of NBUF 16 KiB stages, NBUF-1 of them loading while one is consumed.
// The global side of each wave instruction is a contiguous 1 KiB run of the page block, with the
// 16-byte chunks of every token row permuted (XOR with the token index) so that the MFMA
// operand reads from LDS are free of bank conflicts.  K operands are 16-byte LDS reads; V
// operands use the gfx950 transposing LDS read (ds_read_b64_tr_b16), which hands each lane 4
// tokens of one column.  Slots past the end of a segment are filled from its last valid token
// (finite data whose scores are masked to -inf), so NaN in unused slots never reaches an MFMA.
//
// Online softmax (per row, in the log2 domain): m <- max(m, max_j s_j); alpha = 2^(m_old - m);
// l <- alpha * l + sum_j 2^(s_j - m); O <- alpha * O + P V.  The row maximum is reduced across
// the four lane groups of the wave; l is kept as per-lane partial sums and reduced once at the
// end.  Each work item writes normalised partials o = O / l and lambda = m + log2(l) for every
// row (fp16 with a per-row power-of-two scale for bf16 inputs, fp32 otherwise); the merge kernel
// folds them along each branch's path.
#include "ga_internal.hpp"

#include <hip/hip_ext.h>

#include <type_traits>

#ifndef GA_STAGE_BYTES
#define GA_STAGE_BYTES 16384
#endif
#ifndef GA_RING_STAGES
#define GA_RING_STAGES 4
#endif

namespace ga {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Workgroups per CU and ring depth: two workgroups with four stages for decode; the bf16
// multi-query variant runs three workgroups per CU (its 128-row units are bound by each wave's
// issue and compute, so more waves per CU pay more than a deeper ring) with three stages each,
// and so does bf16 decode on a step with few pages per workgroup (each workgroup then has one
// or two units, whose fixed costs more workgroups overlap better).  (The fp32 variants keep
// two: at three their 32 query registers per tile would spill.)
__host__ __device__ constexpr int attn_wgs_per_cu(bool causal, bool bf16, bool few_pages) {
  return bf16 && (causal || few_pages) ? 3 : 2;
}

template <int D, bool BF16, int WPC = 2>
struct Cfg {
  static constexpr int ELT = BF16 ? 2 : 4;
  static constexpr int ROW = D * ELT;               // bytes of one token row of K or V
  static constexpr int CPR = ROW / 16;              // 16-byte chunks per token row
  static constexpr int KVB = 16 * ROW;              // bytes of a page's K (or V) block
  static constexpr int PB = 2 * KVB;                // bytes of one page of one kv-head
  static constexpr int STAGE = GA_STAGE_BYTES >= PB ? GA_STAGE_BYTES : PB;   // bytes per stage
  static constexpr int SP = STAGE / PB;             // pages per stage
  static constexpr int NBUF = WPC == 3 ? 3 : GA_RING_STAGES;   // stages
  static constexpr int IPP = PB / 1024;             // 1 KiB DMA wave instructions per page
  static constexpr int IPW = IPP / (kAttnThreads / 64);   // ... issued by each wave per page
  static constexpr int NB = D / 16;                 // 16-wide output column blocks
  static constexpr int QR = BF16 ? D / 32 : D / 4;  // Q operand registers per tile
  static_assert(SP >= 1 && IPW >= 1 && STAGE % PB == 0, "stage must hold whole pages");
  static_assert((NBUF - 2) * SP * IPW <= 63, "pending DMA count must fit the wait helper");
};

// Direct-to-LDS copy of 16 bytes per lane: LDS[lds_base + 16 * lane] <- global[base + off].
// base (the page block) and lds_base are wave-uniform SGPR values, off a per-lane VGPR.  Issued
// as inline assembly so that the compiler's wait-count pass does not treat every later LDS read
// as a possible alias of the copy (it would drain the whole pipeline before each stage);
// ordering is explicit instead: wait_vmcnt() before the barrier that publishes a stage.  M0
// holds the LDS base; the kernel keeps no other value in M0.  The copies are non-temporal (nt):
// every K/V byte is read once per step, and streaming it through the caches at normal priority
// would evict the partial rows this kernel writes and the merge kernel reads back.
// The multi-query (causal) variant copies with the normal cache policy instead: there the row
// blocks of one chunk read the same pages, and the later ones find them in the caches.
// (tests/test_isa_invariants.py checks in the built assembly that every M0 write is one of these.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(unsigned off, const void* base, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt"
               :: "v"(off), "s"(base), "s"(lds_base) : "memory", "m0");
}
__device__ __forceinline__ void dma16_cached(unsigned off, const void* base, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(base), "s"(lds_base) : "memory", "m0");
}
// Partial-row stores with device scope (sc1): the L2 writes them through to the memory side at
// once instead of holding them dirty and writing them back later, in the middle of the K/V read
// stream.  (Same bytes; the merged-DAG attention measured 376 -> 370.5 us.)
// A store of more than 64 bits reads its data registers one cycle after issue, and the
// compiler's hazard checks do not look inside inline assembly: the 16-byte store carries its own
// wait states, or the next instruction may overwrite the data before it is read.
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_dev16(f16x8* p, f16x8 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" :: "v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store_dev8(f32x2* p, f32x2 v) {
  asm volatile("global_store_dwordx2 %0, %1, off sc1" :: "v"(p), "v"(v) : "memory");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(n) for a runtime n in [0, 63] (expcnt and lgkmcnt left alone).  The gfx9
// encoding splits vmcnt into bits [3:0] and [15:14].
#define GA_VMCNT(k) (((k) & 15) | (7 << 4) | (15 << 8) | (((k) >> 4) << 14))
__device__ __forceinline__ void wait_vmcnt(int n) {
  // Loads placed before the wait in the source must be issued before it: the s_waitcnt builtin
  // alone does not order ordinary loads, and a load sunk below it would be waited for later,
  // inside the stage loop, draining the copy ring.
  asm volatile("" ::: "memory");
#define GA_VMW(k) case k: __builtin_amdgcn_s_waitcnt(GA_VMCNT(k)); break;
#define GA_VMW8(b) GA_VMW(b) GA_VMW(b + 1) GA_VMW(b + 2) GA_VMW(b + 3) GA_VMW(b + 4) \
                   GA_VMW(b + 5) GA_VMW(b + 6) GA_VMW(b + 7)
  switch (n) {
    GA_VMW8(0) GA_VMW8(8) GA_VMW8(16) GA_VMW8(24) GA_VMW8(32) GA_VMW8(40) GA_VMW8(48) GA_VMW8(56)
    default: __builtin_amdgcn_s_waitcnt(GA_VMCNT(0)); break;
  }
#undef GA_VMW8
#undef GA_VMW
}

template <int N>
__device__ __forceinline__ void wait_vmcnt_const() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(GA_VMCNT(N));
}

// Workgroup barrier without a memory fence: LDS-DMA completion is ordered by the explicit
// vmcnt wait before it; the empty asm statements keep the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Barrier for data exchanged through LDS by ordinary LDS writes: waits for this wave's LDS
// operations only (lgkmcnt(0)), not for its global stores.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Byte offset of 16-byte chunk `ch` of token `tok` inside a K or V block in LDS.
template <int D, bool BF16>
__device__ __forceinline__ int swz(int tok, int ch) {
  using C = Cfg<D, BF16>;
  return tok * C::ROW + ((ch ^ (tok & (C::CPR - 1))) << 4);
}

__device__ __forceinline__ float xmax(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float xsum(float v) {
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}
__device__ __forceinline__ float exp2_(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_(float x) { return __builtin_amdgcn_logf(x); }

template <bool BF16> struct QOp;
template <> struct QOp<true> { bf16x8 v; };
template <> struct QOp<false> { float v; };

__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const int lo = __builtin_amdgcn_readfirstlane((int)(uint32_t)(uint64_t)v);
  const int hi = __builtin_amdgcn_readfirstlane((int)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Scores more than 2^kTau above a row's running reference trigger a reference update; below
// that the stale reference is kept (probabilities up to 2^kTau are exact in fp32 and bf16).
constexpr float kTau = 8.0f;

// Online softmax (log2 domain) over NPG pages of 16 tokens for each of the wave's NT tiles
// (S[g][t]: page g's scores): masks tokens past each page's valid tokens, and moves a row's
// reference m only when some score exceeds it by more than 2^kTau, so the common page needs no
// cross-lane reduction and no rescale of O.
// CAUSAL (multi-query units): when cm is set, the lane's score i of tile t on page g is also
// masked for i > thr[g][t] (the row's last visible token, relative to token 4 kg of the page).
// A row may then have seen no token yet (m = -inf, l = 0, O = 0); the guards keep it at exactly
// that.
template <int NPG, int NT, int NBW, int NBT, bool CAUSAL>
__device__ __forceinline__ void softmax_pages(f32x4 (&S)[NPG][NT], float (&p)[NPG][NT][4],
                                              float (&m)[NT], float (&l)[NT],
                                              f32x4 (&O)[NT][NBT], const bool (&last)[NPG],
                                              const int (&last_valid)[NPG], bool cm,
                                              const int (&thr)[NPG][NT], int kg, float sl2) {
  const float NEG_INF = -__builtin_huge_valf();
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    float lm = NEG_INF;
#pragma unroll
    for (int g = 0; g < NPG; ++g) {
      if (last[g]) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * kg + i >= last_valid[g]) S[g][t][i] = NEG_INF;
      }
      if constexpr (CAUSAL) {
        if (cm) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (i > thr[g][t]) S[g][t][i] = NEG_INF;
        }
      }
      lm = fmaxf(lm, fmaxf(fmaxf(S[g][t][0], S[g][t][1]), fmaxf(S[g][t][2], S[g][t][3])));
    }
    lm *= sl2;
    if (__any(lm > m[t] + kTau)) {
      const float mn = fmaxf(m[t], xmax(lm));
      float alpha = exp2_(m[t] - mn);
      if constexpr (CAUSAL) alpha = mn == NEG_INF ? 1.f : alpha;
      m[t] = mn;
      l[t] *= alpha;
#pragma unroll
      for (int i = 0; i < NBW; ++i) O[t][i] *= alpha;
    }
    float nm = -m[t];
    if constexpr (CAUSAL) nm = m[t] == NEG_INF ? 0.f : nm;
#pragma unroll
    for (int g = 0; g < NPG; ++g) {
#pragma unroll
      for (int i = 0; i < 4; ++i) p[g][t][i] = exp2_(fmaf(S[g][t][i], sl2, nm));
      l[t] += (p[g][t][0] + p[g][t][1]) + (p[g][t][2] + p[g][t][3]);
    }
  }
}

// NPG consecutive pages (p0, p0 + 1, ... of the stage at sb) for one wave: NT row tiles (qop[0 .. NT-1])
// producing NBW output column blocks (O[t][i] holds column block n0 + i); for CAUSAL units,
// cl[t] is the lane's row limit relative to the stage's first page.  All LDS operand reads of
// the first column blocks are issued before the first MFMA, so they overlap S = K Q^T and the
// softmax.
// bf16, two pages: the PV product contracts both pages' 32 tokens in one K = 32 instruction.
// The lane's eight K slots are tokens 4 kg .. 4 kg + 3 of the first page, then the same tokens
// of the second: the slots of V^T (two transposing reads) and of P (the lane's own
// probabilities) are ordered alike, and a contraction does not depend on the order of its
// terms.
template <int D, bool BF16, int NPG, int NT, int NBW, bool CAUSAL>
__device__ __forceinline__ void kv_pages(const unsigned char* sb, const int* pwords, int p0,
                                         float sl2, int r16, int kg,
                                         int n0, bool cm, const int (&cl)[NT],
                                         const QOp<BF16> (&qop)[NT][Cfg<D, BF16>::QR],
                                         float (&m)[NT], float (&l)[NT],
                                         f32x4 (&O)[NT][Cfg<D, BF16>::NB]) {
  using C = Cfg<D, BF16>;
  static_assert(BF16 || NPG == 1, "fp32 pages are taken one at a time");
  const unsigned char* kb[NPG];
  const unsigned char* vb[NPG];
  bool last[NPG];
  int last_valid[NPG];
  int thr[NPG][NT];
#pragma unroll
  for (int g = 0; g < NPG; ++g) {
    kb[g] = sb + p0 * C::PB + g * C::PB;
    vb[g] = kb[g] + C::KVB;
    // Valid tokens of the page (a segment of the chain may end inside it): from its page word.
    const int vm1 = (int)((unsigned)__builtin_amdgcn_readfirstlane(pwords[p0 + g]) >>
                          kPageValidShift);
    last[g] = vm1 < kPageTokens - 1;
    last_valid[g] = vm1 + 1;
#pragma unroll
    for (int t = 0; t < NT; ++t) thr[g][t] = CAUSAL ? cl[t] - kPageTokens * (p0 + g) : 0;
  }
  f32x4 S[NPG][NT];
#pragma unroll
  for (int g = 0; g < NPG; ++g)
#pragma unroll
    for (int t = 0; t < NT; ++t) S[g][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float p[NPG][NT][4];
  if constexpr (BF16) {
    // V^T operand of column block n: lane reads 4 tokens (4 kg + r16 / 4 supplies the row) of
    // 4 columns through the transposing read; the chunk index is permuted like the writes.
    // The V operands are read in batches of VB column blocks (register budget).
    constexpr int VB = NT * NPG == 4 ? (NBW >= 8 ? NBW / 8 : 1) : NT * NPG == 2 ? NBW / 2 : NBW;
    static_assert(NBW % VB == 0, "column blocks come in whole batches");
    // The lane's 32-byte piece of block n is chunk 2 n + c (c = (r16 & 3) / 2) of token row tv,
    // XOR-permuted by x = tv mod CPR; (2 n + c) ^ x = (2 n ^ (x & ~1)) + (c ^ (x & 1)), so its
    // offset is the one of block 0 with 32 n XORed in.
    const int tv = 4 * kg + (r16 >> 2);
    const int xv = tv & (C::CPR - 1);
    const int voff = tv * C::ROW + (((xv & ~1) | (((r16 & 3) >> 1) ^ (xv & 1))) << 4) +
                     (r16 & 1) * 8;
    auto vread = [&](int g, int n) {
      return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vb[g] + (voff ^ (n << 5))));
    };
    s16x4 va[VB][NPG];
#pragma unroll
    for (int i = 0; i < VB; ++i)
#pragma unroll
      for (int g = 0; g < NPG; ++g) va[i][g] = vread(g, n0 + i);
#pragma unroll
    for (int g = 0; g < NPG; ++g) {
      // (the second page's K is read once the first page's products are issued: register
      // budget)
      if (g > 0) asm volatile("" ::: "memory");
      bf16x8 ka[C::QR];
#pragma unroll
      for (int jj = 0; jj < C::QR; ++jj)
        ka[jj] = *reinterpret_cast<const bf16x8*>(kb[g] + swz<D, BF16>(r16, 4 * jj + kg));
#pragma unroll
      for (int jj = 0; jj < C::QR; ++jj)
#pragma unroll
        for (int t = 0; t < NT; ++t)
          S[g][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[jj], qop[t][jj].v, S[g][t], 0, 0,
                                                            0);
    }
    softmax_pages<NPG, NT, NBW, C::NB, CAUSAL>(S, p, m, l, O, last, last_valid, cm, thr, kg,
                                               sl2);
    s16x4 pb[NT][NPG];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int g = 0; g < NPG; ++g)
#pragma unroll
        for (int i = 0; i < 4; ++i) pb[t][g][i] = __builtin_bit_cast(short, (__bf16)p[g][t][i]);
#pragma unroll
    for (int i0 = 0; i0 < NBW; i0 += VB) {
      if (i0 > 0) {
#pragma unroll
        for (int i = 0; i < VB; ++i)
#pragma unroll
          for (int g = 0; g < NPG; ++g) va[i][g] = vread(g, n0 + i0 + i);
      }
#pragma unroll
      for (int i = 0; i < VB; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if constexpr (NPG == 2) {
            const bf16x8 av = __builtin_bit_cast(
                bf16x8, __builtin_shufflevector(va[i][0], va[i][1], 0, 1, 2, 3, 4, 5, 6, 7));
            const bf16x8 bp = __builtin_bit_cast(
                bf16x8, __builtin_shufflevector(pb[t][0], pb[t][1], 0, 1, 2, 3, 4, 5, 6, 7));
            O[t][i0 + i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bp, O[t][i0 + i], 0, 0, 0);
          } else {
            O[t][i0 + i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va[i][0], pb[t][0],
                                                                     O[t][i0 + i], 0, 0, 0);
          }
        }
    }
  } else {
#pragma unroll
    for (int jj = 0; jj < C::QR; ++jj) {
      const float ka = *reinterpret_cast<const float*>(kb[0] + swz<D, BF16>(r16, jj) + kg * 4);
#pragma unroll
      for (int t = 0; t < NT; ++t)
        S[0][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ka, qop[t][jj].v, S[0][t], 0, 0, 0);
    }
    softmax_pages<1, NT, NBW, C::NB, CAUSAL>(S, p, m, l, O, last, last_valid, cm, thr, kg, sl2);
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
      const int n = n0 + i;
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int tv = 4 * kg + i4;
        const float va = *reinterpret_cast<const float*>(
            vb[0] + swz<D, BF16>(tv, 4 * n + (r16 >> 2)) + (r16 & 3) * 4);
#pragma unroll
        for (int t = 0; t < NT; ++t)
          O[t][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(va, p[0][t][i4], O[t][i], 0, 0, 0);
      }
    }
  }
}

// One K/V stage for one wave: pages p0, p0 + pstep, ... below npst of the stage; consecutive
// ones (pstep = 1) in pairs where two are left (bf16), the others one at a time.
template <int D, bool BF16, int NT, int NBW, bool CAUSAL>
__device__ __forceinline__ void kv_stage(const unsigned char* sb, const int* pwords, int p0,
                                         int pstep, int npst, float sl2,
                                         int r16, int kg, int n0, bool cm, const int (&cl)[NT],
                                         const QOp<BF16> (&qop)[NT][Cfg<D, BF16>::QR],
                                         float (&m)[NT], float (&l)[NT],
                                         f32x4 (&O)[NT][Cfg<D, BF16>::NB]) {
  asm volatile("" : "+v"(r16), "+v"(kg));   // per-lane offsets recomputed per call, not hoisted
  int pis = p0;
  if constexpr (BF16) {
    if (pstep == 1)
      for (; pis + 1 < npst; pis += 2)
        kv_pages<D, BF16, 2, NT, NBW, CAUSAL>(sb, pwords, pis, sl2, r16, kg, n0, cm, cl, qop, m,
                                              l, O);
  }
  for (; pis < npst; pis += pstep)
    kv_pages<D, BF16, 1, NT, NBW, CAUSAL>(sb, pwords, pis, sl2, r16, kg, n0, cm, cl, qop, m, l, O);
}

// CAUSAL: the multi-query variant.  A unit whose descriptor carries a causal word c (word 1;
// kNoCausal otherwise) lets the row of group rank j see token t of the chunk (t counted as
// 16 x page index + slot) only for t <= c + j.
template <int D, bool BF16, bool CAUSAL, int WPC>
__global__ __launch_bounds__(kAttnThreads, WPC)
void k_seg_attn(AttnArgs a) {
  using C = Cfg<D, BF16, WPC>;
  using T = typename std::conditional<BF16, __bf16, float>::type;
  constexpr int NI = C::SP * C::IPW;                // copies per wave per full stage
  __shared__ __align__(1024) unsigned char smem[C::NBUF * C::STAGE];
  // Descriptors of the current and the next work unit (double buffer) and the next unit's id.
  __shared__ __align__(1024) int s_desc[2][kDescMaxBytes / 4];
  __shared__ float s_ml[4][2][64];
  __shared__ int s_next[2];
  // Waves that split one tile's pages hand their (m, l, O) to the tile's split-0 wave through the
  // last ring slot: at most MAXW hand-overs of NB KiB each.
  constexpr int MAXW = (C::SP < 4 ? C::SP : 4) - 1 > 2 * ((C::SP < 2 ? C::SP : 2) - 1)
                           ? (C::SP < 4 ? C::SP : 4) - 1
                           : 2 * ((C::SP < 2 ? C::SP : 2) - 1);
  static_assert(MAXW <= 4 && MAXW * C::NB * 1024 <= C::STAGE, "hand-over must fit one stage");

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, kg = lane >> 4;
  const int n_work = (int)(a.counters[0] * a.Hkv);
  const float NEG_INF = -__builtin_huge_valf();
  const unsigned char* pool = static_cast<const unsigned char*>(a.pool);
  const T* qbase = static_cast<const T*>(a.q);
  const unsigned lds_ring =
      (unsigned)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
  const unsigned lds_desc =
      (unsigned)(uintptr_t)(__attribute__((address_space(3))) int*)&s_desc[0][0];
  const int dins = (a.desc_words * 4 + 1023) / 1024;      // copy instructions per descriptor
  const int br_word = kDescHead + a.chunk_pages;          // first branch id in a descriptor

  // Wave 0 copies the descriptor of unit v (if v < n_work) into buffer nb and publishes v (or
  // -1: queue exhausted) there; the copy is waited for before the next end-of-unit barrier.
  auto fetch_desc = [&](int v, int nb) {
    const bool ok = v < n_work;
    if (lane == 0) s_next[nb] = ok ? v : -1;
    if (ok) {
      const int* src = a.desc + (int64_t)(v / a.Hkv) * a.desc_words;
      const unsigned dst = lds_desc + nb * kDescMaxBytes;
      for (int i = 0; i < dins; ++i)
        dma16(1024 * i + 16 * lane, src, __builtin_amdgcn_readfirstlane(dst + 1024 * i));
    }
  };

  // Per-lane source offsets inside a page block for this wave's copies: copy i of a stage covers
  // bytes [1024 j, 1024 j + 1024) with j = wave + 4 i, i.e. page i / IPW of the stage, piece
  // j % IPP of that page.  Chunks are XOR-permuted by token so the LDS layout is swizzled.
  int c_tok[NI], c_rest[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int o = ((wave + 4 * i) % C::IPP) * 1024 + lane * 16;   // byte offset in the page
    const int kv = o / C::KVB;
    const int tok = (o % C::KVB) / C::ROW;
    const int pc = (o % C::ROW) >> 4;
    c_tok[i] = tok;
    c_rest[i] = kv * C::KVB + ((pc ^ (tok & (C::CPR - 1))) << 4);
  }

  // Work streams: stream s holds the units of the kv heads h = s mod ns in item order (its unit
  // j is unit (j / per) Hkv + (j mod per) ns + s) and is owned by the gs(s) workgroups with
  // blockIdx = s mod ns.  The owner of rank r takes stream units r and r + gs(s) without a
  // claim: the whole grid claiming at once serialises on the counters for several microseconds,
  // and the first claim then comes during the second unit, when the workgroups are out of step.
  // Later units are claimed through the stream's head, which counts claims past its first
  // 2 gs(s) units; a workgroup whose stream is exhausted claims from the next streams.
  const int ns = a.streams;
  const int per = a.Hkv / ns;
  const int n_str = (int)(a.counters[0] * per);
  int* heads = reinterpret_cast<int*>(a.counters + 4);
  auto gs = [&](int st) { return ((int)gridDim.x - st + ns - 1) / ns; };
  auto unit_of = [&](int j, int st) {
    return j < n_str ? (j / per) * a.Hkv + (j % per) * ns + st : n_work;
  };
  int cs = (int)blockIdx.x % ns;           // the stream claimed from
  const int rank = (int)blockIdx.x / ns;
  if (wave == 0) {
    fetch_desc(unit_of(rank, cs), 0);
    wait_vmcnt(0);
  }
  __syncthreads();

  bool first = true;                       // the first unit (its successor needs no claim)
  for (int b = 0;; b ^= 1) {
    // Unit fields from its descriptor (the scheduler's record, then the chunk's page words and
    // the row block's branch ids; each page word carries the page's valid tokens).
    const int w = __builtin_amdgcn_readfirstlane(s_next[b]);
    if (w < 0) break;
    const int* dsc = &s_desc[b][0];
    const int kvh = w % a.Hkv;
    const int np = __builtin_amdgcn_readfirstlane(dsc[0]);
    const int cnt = __builtin_amdgcn_readfirstlane(dsc[3]);
    const int rb = __builtin_amdgcn_readfirstlane(dsc[4]);
    const int prow_base = __builtin_amdgcn_readfirstlane(dsc[7]);
    const int row0 = rb * kRowsPerBlock;
    const int R = min(kRowsPerBlock, cnt * a.group - row0);
    const int nrt = (R + 15) >> 4;

    // Wave roles: with >= 3 row tiles the waves split the tiles (tiles wave and wave + 4), and
    // so they do with fewer at two workgroups per CU (the tile owners take every page: there the
    // hand-over below costs more than the idle waves); at three workgroups per CU (steps with
    // few pages per workgroup) waves sharing a tile split the stage's pages and are combined at
    // the end.
    int ks, split, t0, ntile;
    if (nrt >= 4) { ks = 1; split = 0; t0 = wave; ntile = (wave + 4 < nrt) ? 2 : 1; }
    else if (nrt == 3 || WPC == 2) { ks = 1; split = 0; t0 = wave; ntile = wave < nrt ? 1 : 0; }
    else if (nrt == 2) {
      ks = C::SP < 2 ? C::SP : 2; split = wave >> 1; t0 = wave & 1; ntile = split < ks;
    } else {
      ks = C::SP < 4 ? C::SP : 4; split = wave; t0 = 0; ntile = split < ks;
    }

    // The rest of the unit, specialised on the number of row tiles this wave owns (the
    // second tile's registers exist only where they are used).
    auto run_unit = [&](auto nt_tag) {
      constexpr int NT = decltype(nt_tag)::value;
      // Q operand (B of S^T = K Q^T): lane holds row r16 of the tile, head_dim slice by kg.
      auto load_q = [&](QOp<BF16> (&qop)[NT][C::QR]) {
  #pragma unroll
      for (int k = 0; k < NT; ++k) {
        const int r = (t0 + 4 * k) * 16 + r16;
        const bool live = k < ntile && r < R;
        const T* qp = qbase;
        if (live) {
          const int gr = row0 + r;
          const int j = gr / a.group;
          const int h = kvh * a.group + (gr - j * a.group);
          const int br = dsc[br_word + j - row0 / a.group];
          qp = qbase + ((int64_t)br * a.Hq + h) * D;
        }
  #pragma unroll
        for (int jj = 0; jj < C::QR; ++jj) {
          if constexpr (BF16) {
            bf16x8 v = {};
            if (live) v = *reinterpret_cast<const bf16x8*>(qp + 32 * jj + 8 * kg);
            qop[k][jj].v = v;
          } else {
            qop[k][jj].v = live ? qp[4 * jj + kg] : 0.f;
          }
        }
      }
      };
  
      // Causal limits: the lane's row (group rank j) sees chunk token t for t <= cw + j; cl[k]
      // holds that bound relative to token 4 kg of the chunk's first page.
      bool cm = false;
      int cl[NT];
  #pragma unroll
      for (int k = 0; k < NT; ++k) cl[k] = 0;
      if constexpr (CAUSAL) {
        const int cw = __builtin_amdgcn_readfirstlane(dsc[1]);
        cm = cw != kNoCausal;
  #pragma unroll
        for (int k = 0; k < NT; ++k)
          cl[k] = cw + (row0 + (t0 + 4 * k) * 16 + r16) / a.group - 4 * kg;
      }

      float m[NT], l[NT];
      f32x4 O[NT][C::NB];
  #pragma unroll
      for (int k = 0; k < NT; ++k) {
        m[k] = NEG_INF;
        l[k] = 0.f;
  #pragma unroll
        for (int n = 0; n < C::NB; ++n) O[k][n] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
  
      const int64_t blk_stride = (int64_t)a.Hkv * 2 * C::KVB;
      const unsigned char* pool_h = (const unsigned char*)uniform64(
          (int64_t)(uintptr_t)(pool + (int64_t)kvh * 2 * C::KVB));
  
      // With one work stream, the row blocks of one chunk (which workgroups on every XCD stream
      // at about the same time) start at different pages: the full stages are taken in rotated
      // order (a partial last stage stays last), so that they do not all ask for the same page
      // at once.  With several streams they share the L2s of few XCDs, and taking the pages in
      // the same order lets the later ones find what the first fetched.  Issue order st, ring
      // slot st mod NBUF; stage_of(st) is the stage of the chunk it holds.
      const int nfull = np / C::SP;
      const int nrb_c = (cnt * a.group + kRowsPerBlock - 1) / kRowsPerBlock;
      const int rot = ns == 1 && nfull > 1 ? (rb * nfull) / nrb_c : 0;
      auto stage_of = [&](int st) {
        int x = st + rot;
        if (x >= nfull) x -= nfull;
        return st < nfull ? x : st;
      };
      auto issue = [&](int st) {
        const unsigned dst = lds_ring + (st % C::NBUF) * C::STAGE + wave * 1024;
        const int sg = stage_of(st);
        const int npst = min(C::SP, np - sg * C::SP);
        // All page ids of the stage are read before the first copy: one LDS round trip (the
        // copies' memory clobber would otherwise force a re-read before each of them).  Ids past
        // the chunk are read but unused.
        int pw[C::SP];
  #pragma unroll
        for (int q = 0; q < C::SP; ++q)
          pw[q] = __builtin_amdgcn_readfirstlane(s_desc[b][kDescHead + sg * C::SP + q]);
  #pragma unroll
        for (int i = 0; i < NI; ++i) {
          const int pis = i / C::IPW;
          if (pis < npst) {
            // Token rows past the page's valid tokens re-read its last valid token (finite
            // data; their scores are masked).
            const int pid = pw[pis] & kPageIdMask;
            const int vm1 = (int)((unsigned)pw[pis] >> kPageValidShift);
            const unsigned char* base = pool_h + (int64_t)pid * blk_stride;
            if constexpr (CAUSAL)
              dma16_cached(min(c_tok[i], vm1) * C::ROW + c_rest[i], base,
                     __builtin_amdgcn_readfirstlane(dst + i * 4096));
            else
              dma16(min(c_tok[i], vm1) * C::ROW + c_rest[i], base,
                    __builtin_amdgcn_readfirstlane(dst + i * 4096));
          }
        }
      };
  
      // The first stages are issued right away; the queries and the next unit's claim are loaded
      // behind them, and one wait covers all three (the compiler cannot see the copies, so a wait
      // it placed for its own loads inside the stage loop would also drain them).
      const int nst = (np + C::SP - 1) / C::SP;
      for (int st = 0; st < C::NBUF - 1 && st < nst; ++st) issue(st);
      QOp<BF16> qop[NT][C::QR];
      load_q(qop);
      int claim = 0;
      if (!first && wave == 0 && lane == 0) claim = atomicAdd(&heads[cs], 1);
      wait_vmcnt(0);
      // (the claim is consumed only here, after the wait, so that no use of it before the wait
      // makes the compiler wait for it, and with it for every copy in flight)
      asm volatile("" : "+v"(claim));
      // Wave 0 fetches the next unit's descriptor while this one streams.
      if (wave == 0) {
        int v;
        if (first) {
          v = unit_of(rank + gs(cs), cs);
        } else {
          int j = 2 * gs(cs) + __builtin_amdgcn_readfirstlane(claim);
          // (a stream found exhausted stays so: each claim tries every stream at most once)
          for (int t = 1; j >= n_str && t < ns; ++t) {
            cs = cs + 1 == ns ? 0 : cs + 1;
            int c = 0;
            if (lane == 0) c = atomicAdd(&heads[cs], 1);
            j = 2 * gs(cs) + __builtin_amdgcn_readfirstlane(c);
          }
          v = unit_of(j, cs);
        }
        fetch_desc(v, b ^ 1);
      }
      first = false;
      for (int st = 0; st < nst; ++st) {
        // Wait until this wave's copies of stage st have landed (copies of later stages may stay
        // in flight), then make every wave's copies visible.
        const int ahead = min(nst - 1 - st, C::NBUF - 2);
        const int pend = C::IPW * (min(np, (st + 1 + ahead) * C::SP) - (st + 1) * C::SP);
        if (pend == (C::NBUF - 2) * NI) wait_vmcnt_const<(C::NBUF - 2) * NI>();
        else wait_vmcnt(pend);
        wg_barrier();
        // All waves are done with stage st - 1, so its buffer can be refilled.
        if (st + C::NBUF - 1 < nst) issue(st + C::NBUF - 1);
        const int buf = st % C::NBUF;
        const int sg = stage_of(st);
        const int npst = min(C::SP, np - sg * C::SP);
        if (ntile > 0) {
          const unsigned char* sb = smem + buf * C::STAGE;
          int cls[NT];
  #pragma unroll
          for (int k = 0; k < NT; ++k) cls[k] = cl[k] - kPageTokens * C::SP * sg;
          kv_stage<D, BF16, NT, C::NB, CAUSAL>(sb, &s_desc[b][kDescHead + sg * C::SP], split, ks,
                                               npst, a.scale_log2, r16, kg, 0, cm, cls, qop, m,
                                               l, O);
        }
      }
      // Every wave is done with the ring; wave 0's copy of the next descriptor has landed (the
      // partial stores of earlier units need not have).
      if (wave == 0) wait_vmcnt(0);
      lds_barrier();
  
      // Fresh copies of the lane and its lane group: the epilogue's per-lane addresses are then
      // formed here, once per unit, instead of being hoisted out of the unit loop and kept live
      // (or spilled) through every stage.
      int lane_e = lane, kg_e = kg;
      asm volatile("" : "+v"(lane_e), "+v"(kg_e));
      // Row sums: reduce the per-lane_e partials across the four lane_e groups.
      float L[NT];
  #pragma unroll
      for (int k = 0; k < NT; ++k) L[k] = xsum(l[k]);
  
      if (ks > 1) {
        // Waves that split one tile's pages hand (m, l, O) to the tile's split-0 wave through
        // the last ring slot: the next unit's first stages go to the other slots, and this one
        // is refilled only after that unit's first barrier.
        constexpr int NV = C::NB * 4;
        float* cb = reinterpret_cast<float*>(smem + (C::NBUF - 1) * C::STAGE);
        if (split > 0 && ntile > 0) {
          const int wi = (split - 1) * nrt + t0;
          float* mine = cb + wi * NV * 64;
          s_ml[wi][0][lane_e] = m[0];
          s_ml[wi][1][lane_e] = L[0];
  #pragma unroll
          for (int n = 0; n < C::NB; ++n)
  #pragma unroll
            for (int i = 0; i < 4; ++i) mine[(4 * n + i) * 64 + lane_e] = O[0][n][i];
        }
        lds_barrier();
        if (split == 0 && ntile > 0) {
          float M = m[0];
          for (int sp = 1; sp < ks; ++sp) M = fmaxf(M, s_ml[(sp - 1) * nrt + t0][0][lane_e]);
          // (a causal row that saw no token in any split has M = -inf and stays empty)
          const float Ms = CAUSAL && M == NEG_INF ? 0.f : M;
          const float w0 = exp2_(m[0] - Ms);
          float Lc = w0 * L[0];
          f32x4 Oc[C::NB];
  #pragma unroll
          for (int n = 0; n < C::NB; ++n) Oc[n] = O[0][n] * w0;
          for (int sp = 1; sp < ks; ++sp) {
            const int wi = (sp - 1) * nrt + t0;
            const float* o = cb + wi * NV * 64;
            const float wgt = exp2_(s_ml[wi][0][lane_e] - Ms);
            Lc += wgt * s_ml[wi][1][lane_e];
  #pragma unroll
            for (int n = 0; n < C::NB; ++n)
  #pragma unroll
              for (int i = 0; i < 4; ++i) Oc[n][i] += wgt * o[(4 * n + i) * 64 + lane_e];
          }
          m[0] = M;
          L[0] = Lc;
  #pragma unroll
          for (int n = 0; n < C::NB; ++n) O[0][n] = Oc[n];
        }
      }
  
      if (split == 0) {
  #pragma unroll
        for (int k = 0; k < NT; ++k) {
          if (k >= ntile) break;
          const int r = (t0 + 4 * k) * 16 + r16;
          // A causal row that saw no token of the chunk (L = 0) stores o = 0, lambda = -inf.
          const float inv = CAUSAL && !(L[k] > 0.f) ? 0.f : 1.f / L[k];
          if constexpr (BF16) {
            // fp16 partial in lane_e order, scaled so the row's largest |o| is below 2^15 (the
            // four lanes of a row agree on the scale; L >= 1, so |o| <= max |V|).
            float amax = 0.f;
  #pragma unroll
            for (int n = 0; n < C::NB; ++n)
  #pragma unroll
              for (int i = 0; i < 4; ++i) amax = fmaxf(amax, fabsf(O[k][n][i]));
            amax = xmax(amax) * inv;
            const int e = max(__builtin_amdgcn_frexp_expf(amax), -100);
            const float up = __builtin_amdgcn_ldexpf(inv, kPartScaleBits - e);
            if (r < R) {
              const int gr = row0 + r;
              const int j = gr / a.group;
              const int h = kvh * a.group + (gr - j * a.group);
              const int64_t row = ((int64_t)prow_base + j) * a.Hq + h;
              f16x8* dst = reinterpret_cast<f16x8*>(static_cast<_Float16*>(a.po) + row * D +
                                                    8 * kg_e);
  #pragma unroll
              for (int c = 0; c < C::NB / 2; ++c) {
                f16x8 v;
  #pragma unroll
                for (int i = 0; i < 4; ++i) {
                  v[i] = (_Float16)(O[k][2 * c][i] * up);
                  v[4 + i] = (_Float16)(O[k][2 * c + 1][i] * up);
                }
                store_dev16(dst + 4 * c, v);   // the row's four lanes fill 64 contiguous bytes
              }
              if (kg_e == 0)
                store_dev8(reinterpret_cast<f32x2*>(a.plse + 2 * row),
                           f32x2{m[k] + log2_(L[k]), __builtin_amdgcn_ldexpf(1.f, e - kPartScaleBits)});
            }
          } else {
            if (r < R) {
              const int gr = row0 + r;
              const int j = gr / a.group;
              const int h = kvh * a.group + (gr - j * a.group);
              const int64_t row = ((int64_t)prow_base + j) * a.Hq + h;
              float* dst = static_cast<float*>(a.po) + row * D + 4 * kg_e;
  #pragma unroll
              for (int n = 0; n < C::NB; ++n)
                *reinterpret_cast<f32x4*>(dst + 16 * n) = O[k][n] * inv;
              if (kg_e == 0) a.plse[row] = m[k] + log2_(L[k]);
            }
          }
        }
      }
    };
    // No barrier here: the next unit's first copies go to slots every wave is done with (the
    // barrier after the stage loop), its descriptor was published by that barrier, and nothing
    // reads this unit's descriptor buffer after the unit's start.
    if (ntile == 2) run_unit(std::integral_constant<int, 2>{});
    else run_unit(std::integral_constant<int, 1>{});
  }
}

template <int D, bool BF16>
hipError_t launch_t(const AttnArgs& a, bool causal, bool few_pages, int grid,
                    hipStream_t stream, hipEvent_t t0, hipEvent_t t1) {
  constexpr int W_CAUSAL = attn_wgs_per_cu(true, BF16, false);
  constexpr int W_WIDE = attn_wgs_per_cu(false, BF16, true);
  constexpr int W_DECODE = attn_wgs_per_cu(false, BF16, false);
  auto go = [&](auto kernel) {
    if (t0 || t1)
      hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(kAttnThreads), 0, stream, t0, t1, 0, a);
    else
      hipLaunchKernelGGL(kernel, dim3(grid), dim3(kAttnThreads), 0, stream, a);
  };
  if (causal) go(k_seg_attn<D, BF16, true, W_CAUSAL>);
  else if (few_pages && W_WIDE != W_DECODE) go(k_seg_attn<D, BF16, false, W_WIDE>);
  else go(k_seg_attn<D, BF16, false, W_DECODE>);
  return hipGetLastError();
}

}  // namespace

int seg_attn_grid(int head_dim, bool bf16, bool causal, bool few_pages, int num_cus) {
  (void)head_dim;
  // 256-thread workgroups (LDS-bound)
  return num_cus * attn_wgs_per_cu(causal, bf16, few_pages);
}

hipError_t launch_seg_attn(const AttnArgs& a, int head_dim, bool bf16, bool causal,
                           bool few_pages, int grid, hipStream_t stream, hipEvent_t t0,
                           hipEvent_t t1) {
  if (bf16) {
    if (head_dim == 64) return launch_t<64, true>(a, causal, few_pages, grid, stream, t0, t1);
    if (head_dim == 128) return launch_t<128, true>(a, causal, few_pages, grid, stream, t0, t1);
  } else {
    if (head_dim == 64) return launch_t<64, false>(a, causal, few_pages, grid, stream, t0, t1);
    if (head_dim == 128) return launch_t<128, false>(a, causal, few_pages, grid, stream, t0, t1);
  }
  return hipErrorInvalidValue;
}

}  // namespace ga
