// Equivalence detection over rollout states and the graph suffix (Sec. 3.2, "Graph
// Construction"; Alg. S.1, Stage 1).
//
// Two states of one prompt's graph that are neither ancestor nor descendant of each other are
// compared by the cosine of their embeddings; pairs at or above kappa are linked, and the
// classes Q(v) are the connected components of the links.  The similarity is a dense
// contraction over the embedding width, so it runs on bf16 MFMA: one workgroup per 64 x 64
// tile (row states i0.., column states j0.., both of one prompt, i0 <= j0), the width streamed
// through LDS in 64-wide stages, each wave holding a 32 x 32 quadrant as 2 x 2 MFMA tiles.  The
// epilogue tests every pair of the quadrant (u < v, same prompt, not ancestor-related by the
// Euler intervals of the generation tree, z_u.z_v >= kappa |z_u| |z_v|) and links the qualifying
// ones at once with a lock-free union-find on a global parent array: the larger root is hooked
// under the smaller with a compare-and-swap, so every class's final root is its smallest state
// (a deterministic label, whatever order the links land in).
//
// Graph suffix: C_g(u) is u's direct successors plus those of the other members of Q(u) that lie
// deeper than u (shared edges only point deeper, so the graph stays acyclic).  One thread per
// state counts them over its prompt's states, a scan gives the CSR offsets, and a second pass
// writes them in ascending state order.
#include "ga_internal.hpp"

namespace ga {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 64;       // states per tile side
constexpr int kKC = 64;         // embedding components per LDS stage (128 bytes per state row)

__device__ __forceinline__ int load_rep(const int* rep, int x) {
  return __hip_atomic_load(rep + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int find_root(const int* rep, int x) {
  int p = load_rep(rep, x);
  while (p != x) {
    x = p;
    p = load_rep(rep, x);
  }
  return x;
}

// Links the classes of a and b: the larger root is hooked under the smaller one.  A failed
// compare-and-swap means another link changed that root first; the roots are looked up again.
__device__ void unite(int* rep, int a, int b) {
  while (true) {
    a = find_root(rep, a);
    b = find_root(rep, b);
    if (a == b) return;
    if (a > b) {
      const int t = a;
      a = b;
      b = t;
    }
    if (atomicCAS(rep + b, b, a) == b) return;
  }
}

// Prompts of more than 256 states: inverse norm of each of their embeddings (NaN for a zero
// vector, which is then never linked) and the union-find parent reset to a singleton.  One wave
// per state of the list a.big.
__global__ __launch_bounds__(256) void k_norms(EquivArgs a) {
  const int64_t wi = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wi >= a.n_big) return;
  const int64_t w = a.big[wi];
  const bf16x8* row = reinterpret_cast<const bf16x8*>(a.z + w * a.dim);
  float s = 0.f;
  for (int c = lane; c < a.dim / 8; c += 64) {
    const bf16x8 v = row[c];
#pragma unroll
    for (int i = 0; i < 8; ++i) s = fmaf((float)v[i], (float)v[i], s);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) {
    a.inv_norm[w] = s > 0.f ? 1.f / sqrtf(s) : __builtin_nanf("");
    a.rep[w] = (int)w;
  }
}

__global__ __launch_bounds__(256) void k_sim_union(EquivArgs a) {
  __shared__ __align__(16) unsigned char sA[kTile * kKC * 2];
  __shared__ __align__(16) unsigned char sB[kTile * kKC * 2];
  const int4 it = a.items[blockIdx.x];        // (first row state, first column state, prompt end)
  const int i0 = it.x, j0 = it.y, pend = it.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  // Global -> LDS: thread t moves 16-byte chunk t % 8 of state rows t / 8 and t / 8 + 32 of both
  // tiles; chunks are XOR-permuted by row so the MFMA operand reads are conflict-free.
  const int lr = tid >> 3, lc = tid & 7;
  auto gload = [&](int s0, int r, int kc) {
    const int s = s0 + r;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (s < pend) v = *reinterpret_cast<const uint4*>(a.z + (int64_t)s * a.dim + kc * kKC + lc * 8);
    return v;
  };
  auto lds_off = [](int row, int chunk) { return row * (kKC * 2) + ((chunk ^ (row & 7)) << 4); };
  uint4 ra0 = gload(i0, lr, 0), ra1 = gload(i0, lr + 32, 0);
  uint4 rb0 = gload(j0, lr, 0), rb1 = gload(j0, lr + 32, 0);
  f32x4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nk = a.dim / kKC;
  for (int kc = 0; kc < nk; ++kc) {
    __syncthreads();                            // every wave is done with the previous stage
    *reinterpret_cast<uint4*>(sA + lds_off(lr, lc)) = ra0;
    *reinterpret_cast<uint4*>(sA + lds_off(lr + 32, lc)) = ra1;
    *reinterpret_cast<uint4*>(sB + lds_off(lr, lc)) = rb0;
    *reinterpret_cast<uint4*>(sB + lds_off(lr + 32, lc)) = rb1;
    __syncthreads();
    if (kc + 1 < nk) {                          // next stage's loads overlap this stage's MFMAs
      ra0 = gload(i0, lr, kc + 1);
      ra1 = gload(i0, lr + 32, kc + 1);
      rb0 = gload(j0, lr, kc + 1);
      rb1 = gload(j0, lr + 32, kc + 1);
    }
#pragma unroll
    for (int ks = 0; ks < kKC / 32; ++ks) {
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        av[t] = *reinterpret_cast<const bf16x8*>(sA + lds_off(wm * 32 + t * 16 + r16, ks * 4 + kg));
        bv[t] = *reinterpret_cast<const bf16x8*>(sB + lds_off(wn * 32 + t * 16 + r16, ks * 4 + kg));
      }
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[x], bv[y], acc[x][y], 0, 0, 0);
    }
  }
  // acc[x][y][i] = z_u . z_v with u the row state (4 kg + i of row tile x), v the column state
  // (r16 of column tile y).
#pragma unroll
  for (int y = 0; y < 2; ++y) {
    const int v = j0 + wn * 32 + y * 16 + r16;
    if (v >= pend) continue;
    const int tin_v = a.tin[v], tout_v = a.tout[v];
    const float nv = a.inv_norm[v];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int u = i0 + wm * 32 + x * 16 + 4 * kg + i;
        if (u >= v) continue;
        const int tin_u = a.tin[u], tout_u = a.tout[u];
        const bool related = (tin_u <= tin_v && tin_v < tout_u) || (tin_v <= tin_u && tin_u < tout_v);
        const float cs = acc[x][y][i] * a.inv_norm[u] * nv;
        if (!related && cs >= a.kappa) unite(a.rep, u, v);
        if (a.edge_sim && a.parent[v] == u) a.edge_sim[v] = cs;
      }
  }
}

// One prompt of at most 256 states in one workgroup (8 waves).  The prompt's embeddings stream
// through an LDS ring of 4 stages of 32 components (256 rows x 64 bytes each), 3 stages in
// flight, copied straight from HBM into LDS (global_load_lds_dwordx4: each lane moves 16 bytes,
// one wave instruction fills 1 KiB = 16 rows; 16-byte chunks are XOR-permuted by row pair so the
// MFMA operand reads are conflict-free).  The upper triangle of the 16 x 16 grid of 16 x 16
// tiles (136 tiles) is dealt out as strips: wave w owns row strips w and 15 - w, i.e. the 16 - w
// tiles (w, w..15) and the w + 1 tiles (15 - w, 15 - w..15), 17 per wave.  The squared norms
// are the diagonals of the diagonal tiles (the same fp32 sums as the dot products).  Links are
// made with a union-find in LDS and the labels written at the end.
constexpr int kPromptMax = 256;
constexpr int kPKC = 32;                        // components per stage: one MFMA k-step
constexpr int kPRow = kPKC * 2;                 // bytes of one state row in a stage
constexpr int kPStage = kPromptMax * kPRow;     // 16 KiB
constexpr int kPRing = 4;

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// LDS[lds_base + 16 * lane] <- global[base + off] (16 bytes per lane).  M0 holds the LDS base;
// the kernel keeps no other value in M0, and completion is awaited with explicit vmcnt waits.
__device__ __forceinline__ void dma16(unsigned off, const void* base, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(base), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(n) for a runtime n in [0, 15] (expcnt and lgkmcnt left alone).
#define EQ_VMCNT(k) (((k) & 15) | (7 << 4) | (15 << 8))
__device__ __forceinline__ void wait_vm(int n) {
  asm volatile("" ::: "memory");
  switch (n) {
    case 0: __builtin_amdgcn_s_waitcnt(EQ_VMCNT(0)); break;
    case 1: __builtin_amdgcn_s_waitcnt(EQ_VMCNT(1)); break;
    case 2: __builtin_amdgcn_s_waitcnt(EQ_VMCNT(2)); break;
    case 3: __builtin_amdgcn_s_waitcnt(EQ_VMCNT(3)); break;
    default: __builtin_amdgcn_s_waitcnt(EQ_VMCNT(4)); break;
  }
}

__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A wave-uniform pointer held in scalar registers (both halves read from the first lane as
// unsigned 32-bit values, so the low half is not sign-extended into the high one).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return reinterpret_cast<const void*>((uintptr_t)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ int poff(int row, int chunk) {
  return row * kPRow + ((chunk ^ ((row >> 1) & 3)) << 4);
}

__device__ __forceinline__ int lds_find(int* r, int x) {
  int p = __hip_atomic_load(r + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  while (p != x) {
    x = p;
    p = __hip_atomic_load(r + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  return x;
}

__device__ void lds_unite(int* r, int a, int b) {
  while (true) {
    a = lds_find(r, a);
    b = lds_find(r, b);
    if (a == b) return;
    if (a > b) {
      const int t = a;
      a = b;
      b = t;
    }
    if (atomicCAS(r + b, b, a) == b) return;
  }
}

__global__ __launch_bounds__(512, 2) void k_prompt_classes(EquivArgs a) {
  __shared__ __align__(1024) unsigned char ring[kPRing * kPStage];
  __shared__ float s_inv[kPromptMax];
  __shared__ int s_tin[kPromptMax], s_tout[kPromptMax], s_rep[kPromptMax], s_par[kPromptMax];
  const int2 pr = a.prompts[blockIdx.x];          // (first state, states)
  const int s0 = pr.x, n = pr.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, kg = lane >> 4;
  const int nt = (n + 15) >> 4;                   // 16-row tiles holding states
  if (tid < kPromptMax) {
    s_rep[tid] = tid;
    s_tin[tid] = tid < n ? a.tin[s0 + tid] : 0;
    s_tout[tid] = tid < n ? a.tout[s0 + tid] : 0;
    s_par[tid] = tid < n ? a.parent[s0 + tid] - s0 : -1;   // prompt-local (< 0 for the root)
  }
  __syncthreads();

  // Copies: wave w issues instructions q = 2w and 2w + 1 of every stage; instruction q fills rows
  // 16q .. 16q + 15, lane l the LDS chunk l % 4 of row 16q + l / 4 with the global chunk that
  // the permutation puts there.  Rows past the prompt re-read its last state (valid memory;
  // their products are never used).
  const void* pbase = uniform_ptr(a.z + (int64_t)s0 * a.dim);
  unsigned coff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 16 * (2 * wave + j) + (lane >> 2);
    const int chunk = (lane & 3) ^ ((row >> 1) & 3);
    coff[j] = (unsigned)(min(row, n - 1) * a.dim * 2 + chunk * 16);
  }
  const unsigned lds_ring = (unsigned)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)ring;
  const int nst = a.dim / kPKC;
  auto issue = [&](int st) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
      dma16(coff[j] + (unsigned)(st * kPRow), pbase,
            __builtin_amdgcn_readfirstlane(lds_ring + (st % kPRing) * kPStage + (2 * wave + j) * 1024));
  };
  // Strips of this wave and the 17 tiles (strip, column) it owns.
  const int sa = wave, sb = 15 - wave;
  auto tile_strip = [&](int k) { return k < 16 - sa ? sa : sb; };
  auto tile_col = [&](int k) { return k < 16 - sa ? sa + k : k - 1; };
  f32x4 acc[17];
#pragma unroll
  for (int k = 0; k < 17; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int st = 0; st < kPRing - 1 && st < nst; ++st) issue(st);
  for (int st = 0; st < nst; ++st) {
    wait_vm(2 * min(nst - 1 - st, kPRing - 2));   // this wave's copies of stage st have landed
    ring_barrier();                               // ... and every wave's; stage st - 1 is done
    if (st + kPRing - 1 < nst) issue(st + kPRing - 1);
    const unsigned char* stg = ring + (st % kPRing) * kPStage;
    const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(stg + poff(sa * 16 + r16, kg));
    const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(stg + poff(sb * 16 + r16, kg));
#pragma unroll
    for (int k = 0; k < 17; ++k) {
      const int srow = tile_strip(k), col = tile_col(k);
      if (srow < nt && col < nt) {
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(stg + poff(col * 16 + r16, kg));
        acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(srow == sa ? a0 : a1, b, acc[k], 0, 0, 0);
      }
    }
  }
  // Squared norms from the diagonal tiles (strip, strip): row 16 strip + m sits in lane
  // (r16 = m, kg = m / 4), element m % 4.
#pragma unroll
  for (int k = 0; k < 17; ++k) {
    const int srow = tile_strip(k), col = tile_col(k);
    if (srow != col || srow >= nt) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * kg + i == r16) {
        const float q = acc[k][i];
        s_inv[srow * 16 + r16] = q > 0.f ? 1.f / sqrtf(q) : __builtin_nanf("");
      }
  }
  __syncthreads();
  // acc[k][i] = z_u . z_v, u = 16 strip + 4 kg + i, v = 16 col + r16 (prompt-local).
#pragma unroll
  for (int k = 0; k < 17; ++k) {
    const int srow = tile_strip(k), col = tile_col(k);
    if (srow >= nt || col >= nt) continue;
    const int v = col * 16 + r16;
    if (v >= n) continue;
    const int tin_v = s_tin[v], tout_v = s_tout[v];
    const float nv = s_inv[v];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = srow * 16 + 4 * kg + i;
      if (u >= v) continue;
      const int tin_u = s_tin[u], tout_u = s_tout[u];
      const bool related = (tin_u <= tin_v && tin_v < tout_u) || (tin_v <= tin_u && tin_u < tout_v);
      const float cs = acc[k][i] * s_inv[u] * nv;
      if (!related && cs >= a.kappa) lds_unite(s_rep, u, v);
      if (a.edge_sim && s_par[v] == u) a.edge_sim[s0 + v] = cs;
    }
  }
  __syncthreads();
  if (tid < n) {
    a.labels[s0 + tid] = s0 + lds_find(s_rep, tid);
    if (a.edge_sim && s_par[tid] < 0) a.edge_sim[s0 + tid] = 0.f;
  }
}

// Final labels: every state's root (all links have landed: kernel boundary).
__global__ void k_labels(EquivArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.n_big) return;
  const int v = a.big[i];
  a.labels[v] = find_root(a.rep, v);
  if (a.edge_sim && a.parent[v] < 0) a.edge_sim[v] = 0.f;
}

// Graph suffix, pass 1 (count into cnt[u]) or pass 2 (write from off[u]).
// The block's 256 states lie in consecutive prompts, so every state they scan lies between the
// first state's prompt start and the last state's prompt end: with prompts of up to 256 states
// that span (at most 768 states) is staged in LDS once, and each thread scans it there; longer
// spans are scanned in global memory.  Same scan, same order, either way.
constexpr int kSufStage = 1024;

template <bool FILL>
__global__ __launch_bounds__(256) void k_suffix(SuffixArgs a) {
  __shared__ int s_par[kSufStage], s_lab[kSufStage], s_dep[kSufStage];
  const int64_t base = (int64_t)blockIdx.x * 256;
  const int64_t last = min(base + 255, a.N - 1);
  const int lo = a.pstart[base], hi = a.pend[last];
  const bool staged = hi - lo <= kSufStage;
  if (staged) {
    for (int i = threadIdx.x; i < hi - lo; i += 256) {
      s_par[i] = a.parent[lo + i];
      s_lab[i] = a.labels[lo + i];
      s_dep[i] = a.depth[lo + i];
    }
  }
  __syncthreads();
  const int64_t u = base + threadIdx.x;
  if (u >= a.N) return;
  const int lu = a.labels[u], du = a.depth[u];
  int64_t k = FILL ? a.off[u] : 0;
  const int c0 = a.pstart[u], c1 = a.pend[u];
  if (staged) {
    for (int c = c0; c < c1; ++c) {
      const int p = s_par[c - lo];           // p lies in u's prompt: p >= c0 >= lo
      if (p < 0) continue;
      if (p == (int)u || (s_lab[p - lo] == lu && s_dep[c - lo] > du)) {
        if (FILL) a.states[k] = c;
        ++k;
      }
    }
  } else {
    for (int c = c0; c < c1; ++c) {
      const int p = a.parent[c];
      if (p < 0) continue;
      if (p == (int)u || (a.labels[p] == lu && a.depth[c] > du)) {
        if (FILL) a.states[k] = c;
        ++k;
      }
    }
  }
  if (!FILL) a.cnt[u] = k;
}

// Exclusive scan of cnt[0..N) into off[0..N] (off[N] = total) over many workgroups.
__global__ __launch_bounds__(1024) void k_scan_sums(SuffixArgs a) {
  __shared__ int64_t red[16];
  const int64_t i = (int64_t)blockIdx.x * 1024 + threadIdx.x;
  int64_t v = i < a.N ? a.cnt[i] : 0;
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t t = 0;
    for (int w = 0; w < 16; ++w) t += red[w];
    a.blk[blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(1024) void k_scan_apply(SuffixArgs a) {
  __shared__ int64_t red[16], wsum[16];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int64_t pre = 0;
  for (int k = t; k < (int)blockIdx.x; k += 1024) pre += a.blk[k];
  for (int o = 32; o > 0; o >>= 1) pre += __shfl_xor(pre, o);
  if (lane == 0) red[w] = pre;
  __syncthreads();
  int64_t base = 0;
  for (int k = 0; k < 16; ++k) base += red[k];
  const int64_t i = (int64_t)blockIdx.x * 1024 + t;
  const int64_t v = i < a.N ? a.cnt[i] : 0;
  int64_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int64_t before = 0;
  for (int k = 0; k < w; ++k) before += wsum[k];
  if (i < a.N) a.off[i] = base + before + x - v;
  if (i == a.N - 1) a.off[a.N] = base + before + x;
}

}  // namespace

hipError_t launch_equivalence(const EquivArgs& a, hipStream_t stream) {
  if (a.n_prompts > 0)
    hipLaunchKernelGGL(k_prompt_classes, dim3((unsigned)a.n_prompts), dim3(512), 0, stream, a);
  if (a.n_big > 0) {
    hipLaunchKernelGGL(k_norms, dim3((unsigned)((a.n_big * 64 + 255) / 256)), dim3(256), 0, stream,
                       a);
    if (a.n_items > 0)
      hipLaunchKernelGGL(k_sim_union, dim3((unsigned)a.n_items), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(k_labels, dim3((unsigned)((a.n_big + 255) / 256)), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_suffix_count(const SuffixArgs& a, hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  const unsigned g = (unsigned)((a.N + 255) / 256);
  hipLaunchKernelGGL(k_suffix<false>, dim3(g), dim3(256), 0, stream, a);
  const unsigned sb = (unsigned)((a.N + 1023) / 1024);
  hipLaunchKernelGGL(k_scan_sums, dim3(sb), dim3(1024), 0, stream, a);
  hipLaunchKernelGGL(k_scan_apply, dim3(sb), dim3(1024), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_suffix_fill(const SuffixArgs& a, hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  hipLaunchKernelGGL(k_suffix<true>, dim3((unsigned)((a.N + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ga
