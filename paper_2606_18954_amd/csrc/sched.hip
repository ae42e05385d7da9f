// Segment scheduler (GPU): groups the branches that share each segment and emits the work list.
//
// Input: the rollout graph as branch -> segment-list CSR (a branch's context is the
// concatenation of the edge tokens on its root path; Sec. 3.2 and Alg. S.1 Stage 1).
// Output:
//   B(s)          branches whose path contains s, ascending (CSR grp_off / grp_br)
//   entry_rank    for each path entry (b, s): the position of b inside B(s)
//   seg_nchunk    page chunks of each referenced segment (chunk_pages pages per chunk)
//   items         (segment, chunk, row block) work items, grouped by segment; segments in
//                 descending order of per-item cost (pages x (2 + row tiles)), ties by id
//   seg_prow_off  first partial row of each segment; partial row of (s, chunk c, rank j) is
//                 seg_prow_off[s] + c * |B(s)| + j
// Every output is a pure function of the graph: group order comes from ranking, not from the
// order in which atomics land, so two schedules of one graph are bit-identical.
#include "ga_internal.hpp"

namespace ga {
namespace {

constexpr int kT = 256;

__global__ void k_init(DevGraph g, DevSchedule sc) {
  int s = blockIdx.x * kT + threadIdx.x;
  if (s < g.S) {
    sc.grp_cnt[s] = 0;
    sc.grp_fill[s] = 0;
  }
  if (s < 4) sc.counters[s] = 0;
}

// Branch of each path entry (binary search in path_off) and |B(s)| histogram.
__global__ void k_count(DevGraph g, DevSchedule sc) {
  int e = blockIdx.x * kT + threadIdx.x;
  if (e >= g.E) return;
  int lo = 0, hi = g.B;                 // invariant: path_off[lo] <= e < path_off[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (g.path_off[mid] <= e) lo = mid; else hi = mid;
  }
  sc.entry_branch[e] = lo;
  atomicAdd(&sc.grp_cnt[g.path_segs[e]], 1);
}

// Cost of one work item of segment s (pages of a chunk x per-page work), used to order the
// work list longest first so the persistent grid does not end on a long item.
__device__ __forceinline__ uint32_t item_cost(int npg, int cnt, int group, int chunk_pages) {
  const int rows = min(cnt * group, kRowsPerBlock);
  const int tiles = (rows + 15) / 16;
  return (uint32_t)(min(npg, chunk_pages) * (2 + tiles));
}

constexpr int kSortCap = 8192;   // segments sorted in LDS; larger graphs keep segment order

// Exclusive scans over segments (one workgroup; each thread owns a contiguous range):
// group offsets and partial-row offsets in segment order, item offsets in work-list order.
__global__ __launch_bounds__(1024) void k_scan(DevGraph g, DevSchedule sc, int32_t group,
                                               int32_t chunk_pages) {
  __shared__ int64_t sh[3][1024];
  __shared__ uint64_t keys[kSortCap];
  const int t = threadIdx.x;
  const int S = g.S;
  const int per = (S + 1023) / 1024;
  const int s0 = min(S, t * per), s1 = min(S, s0 + per);
  auto seg_info = [&](int s, int& cnt, int& nch, int& nrb, int& npg) {
    cnt = sc.grp_cnt[s];
    npg = (g.seg_len[s] + kPageTokens - 1) / kPageTokens;
    nch = cnt > 0 ? (npg + chunk_pages - 1) / chunk_pages : 0;
    nrb = (int)(((int64_t)cnt * group + kRowsPerBlock - 1) / kRowsPerBlock);
  };
  auto block_scan = [&](int64_t a, int64_t b, int64_t c) {
    sh[0][t] = a; sh[1][t] = b; sh[2][t] = c;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {   // Hillis-Steele inclusive scan
      int64_t x0 = 0, x1 = 0, x2 = 0;
      if (t >= off) { x0 = sh[0][t - off]; x1 = sh[1][t - off]; x2 = sh[2][t - off]; }
      __syncthreads();
      sh[0][t] += x0; sh[1][t] += x1; sh[2][t] += x2;
      __syncthreads();
    }
  };

  // 1. Group and partial-row offsets in segment order.
  int64_t a = 0, c = 0;
  for (int s = s0; s < s1; ++s) {
    int cnt, nch, nrb, npg;
    seg_info(s, cnt, nch, nrb, npg);
    a += cnt;
    c += (int64_t)nch * cnt;
  }
  block_scan(a, 0, c);
  int64_t ra = t ? sh[0][t - 1] : 0, rc = t ? sh[2][t - 1] : 0;
  for (int s = s0; s < s1; ++s) {
    int cnt, nch, nrb, npg;
    seg_info(s, cnt, nch, nrb, npg);
    sc.grp_off[s] = ra;
    sc.seg_prow_off[s] = rc;
    sc.seg_nchunk[s] = nch;
    ra += cnt;
    rc += (int64_t)nch * cnt;
  }
  if (t == 1023) {
    sc.grp_off[S] = sh[0][1023];
    sc.seg_prow_off[S] = sh[2][1023];
    sc.counters[1] = sh[2][1023];
  }
  __syncthreads();

  // 2. Work-list order: segments by descending item cost, ties by segment id (bitonic sort of
  //    unique 64-bit keys, so the order is a pure function of the graph).
  const bool sorted = S <= kSortCap;
  int n = 1;
  if (sorted) {
    while (n < S) n <<= 1;
    for (int i = t; i < n; i += 1024) {
      uint64_t key = ~0ull;
      if (i < S) {
        int cnt, nch, nrb, npg;
        seg_info(i, cnt, nch, nrb, npg);
        const uint32_t cost = cnt > 0 ? item_cost(npg, cnt, group, chunk_pages) : 0u;
        key = ((uint64_t)(0xffffffffu - cost) << 32) | (uint32_t)i;
      }
      keys[i] = key;
    }
    __syncthreads();
    for (int k = 2; k <= n; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = t; i < n; i += 1024) {
          const int l = i ^ j;
          if (l > i) {
            const uint64_t x = keys[i], y = keys[l];
            const bool up = (i & k) == 0;
            if ((x > y) == up) { keys[i] = y; keys[l] = x; }
          }
        }
        __syncthreads();
      }
    }
  }
  // 3. Item offsets in work-list order.
  int64_t b = 0;
  for (int i = s0; i < s1; ++i) {
    const int s = sorted ? (int)(uint32_t)keys[i] : i;
    int cnt, nch, nrb, npg;
    seg_info(s, cnt, nch, nrb, npg);
    b += (int64_t)nch * nrb;
  }
  block_scan(0, b, 0);
  int64_t rb = t ? sh[1][t - 1] : 0;
  for (int i = s0; i < s1; ++i) {
    const int s = sorted ? (int)(uint32_t)keys[i] : i;
    int cnt, nch, nrb, npg;
    seg_info(s, cnt, nch, nrb, npg);
    sc.seg_item_off[s] = rb;
    rb += (int64_t)nch * nrb;
  }
  if (t == 1023) {
    sc.seg_item_off[S] = sh[1][1023];
    sc.counters[0] = sh[1][1023];
  }
}

__global__ void k_scatter(DevGraph g, DevSchedule sc) {
  int e = blockIdx.x * kT + threadIdx.x;
  if (e >= g.E) return;
  const int s = g.path_segs[e];
  const int pos = atomicAdd(&sc.grp_fill[s], 1);
  sc.grp_tmp[sc.grp_off[s] + pos] = sc.entry_branch[e];
}

// Rank of each entry's branch inside B(s) (branch ids within a group are distinct because a
// path visits a segment at most once), placement into ascending order, and the work items.
__global__ void k_rank_items(DevGraph g, DevSchedule sc, int32_t group) {
  int i = blockIdx.x * kT + threadIdx.x;
  if (i < g.E) {
    const int s = g.path_segs[i];
    const int b = sc.entry_branch[i];
    const int64_t off = sc.grp_off[s];
    const int cnt = sc.grp_cnt[s];
    int r = 0;
    for (int k = 0; k < cnt; ++k) r += sc.grp_tmp[off + k] < b;
    sc.grp_br[off + r] = b;
    sc.entry_rank[i] = r;
  }
  if (i < g.S) {
    const int nch = sc.seg_nchunk[i];
    const int nrb = (int)(((int64_t)sc.grp_cnt[i] * group + kRowsPerBlock - 1) / kRowsPerBlock);
    int64_t w = sc.seg_item_off[i];
    for (int c = 0; c < nch; ++c)
      for (int rbk = 0; rbk < nrb; ++rbk) sc.items[w++] = make_int4(i, c, rbk, 0);
  }
}

inline int blocks(int64_t n) { return (int)((n + kT - 1) / kT); }

}  // namespace

hipError_t launch_schedule(const DevGraph& g, const DevSchedule& sc, int32_t group,
                           int32_t chunk_pages, hipStream_t stream) {
  hipLaunchKernelGGL(k_init, dim3(blocks(g.S > 4 ? g.S : 4)), dim3(kT), 0, stream, g, sc);
  if (g.E > 0)
    hipLaunchKernelGGL(k_count, dim3(blocks(g.E)), dim3(kT), 0, stream, g, sc);
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, stream, g, sc, group, chunk_pages);
  if (g.E > 0)
    hipLaunchKernelGGL(k_scatter, dim3(blocks(g.E)), dim3(kT), 0, stream, g, sc);
  const int64_t n = g.E > g.S ? g.E : g.S;
  if (n > 0)
    hipLaunchKernelGGL(k_rank_items, dim3(blocks(n)), dim3(kT), 0, stream, g, sc, group);
  return hipGetLastError();
}

}  // namespace ga
