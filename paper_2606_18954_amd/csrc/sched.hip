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
//   bpart         each branch's partial rows as CSR (bpart_off), in path order then chunk
//                 order: the merge folds them in exactly this order
// Every output is a pure function of the graph: group order comes from ranking, not from the
// order in which atomics land, so two schedules of one graph are bit-identical.
#include "ga_internal.hpp"

namespace ga {
namespace {

constexpr int kT = 256;

// Workgroup barrier for LDS data only: waits for this wave's LDS operations, not for its global
// stores (no phase of the single-workgroup scheduler reads global data another thread wrote).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);            // lgkmcnt(0); vmcnt and expcnt not waited on
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__global__ void k_init(DevGraph g, DevSchedule sc, int32_t reuse) {
  int s = blockIdx.x * kT + threadIdx.x;
  if (s < g.S && !reuse) {
    sc.grp_cnt[s] = 0;
    sc.grp_fill[s] = 0;
  }
  if (s < kNumCounters) sc.counters[s] = 0;
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

// Chunk c of a segment of npg pages cut into nch chunks: pages [c npg / nch, (c + 1) npg / nch),
// so the chunks of one segment differ by at most a page (each at most chunk_pages, since
// nch = ceil(npg / chunk_pages)) instead of ending on a short remainder.
__device__ __forceinline__ int chunk_first_page(int c, int npg, int nch) {
  return (int)(((int64_t)c * npg) / nch);
}

// Cost of one work item of segment s (pages of its longest chunk x per-page work), used to
// order the work list longest first so the persistent grid does not end on a long item.
__device__ __forceinline__ uint32_t item_cost(int npg, int cnt, int group, int chunk_pages) {
  const int rows = min(cnt * group, kRowsPerBlock);
  const int tiles = (rows + 15) / 16;
  const int nch = (npg + chunk_pages - 1) / chunk_pages;
  return (uint32_t)(((npg + nch - 1) / max(nch, 1)) * (2 + tiles));
}

// Cost class of a work item: half-octave bins of item_cost (0 for a segment without items).
// The work list is ordered by descending class, ties by segment id: longest first, to within a
// factor of 1.5, and a pure function of the graph.
constexpr int kCostClasses = 32;
__device__ __forceinline__ int cost_class(uint32_t cost) {
  if (cost == 0) return 0;
  const int e = 31 - __builtin_clz(cost);
  const int m = e > 0 ? (int)((cost >> (e - 1)) & 1u) : 0;
  return min(kCostClasses - 1, 1 + 2 * e + m);
}

// Inclusive scan of one int over the 64 lanes of a wave with DPP: row shifts by 1, 2, 4 and 8
// scan each row of 16 lanes (lanes shifted in from outside the row read 0), then the last lane
// of row 0 is added to row 1 and of row 2 to row 3 (row_bcast:15), and the last lane of row 1 to
// rows 2 and 3 (row_bcast:31).  Rows left out by the row mask keep their value.
__device__ __forceinline__ int wave_scan_incl(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

#ifndef GA_SORT_CAP
#define GA_SORT_CAP 8192
#endif
constexpr int kSortCap = GA_SORT_CAP;   // segments sorted in LDS; larger graphs keep segment order

// Per-segment scans (run by one 1024-thread workgroup; each thread owns a contiguous range of
// segments): group offsets and partial-row offsets in segment order, then item offsets in
// work-list order.  cnt_of(s) returns |B(s)|; keys is LDS scratch of kSortCap entries.
template <typename CntOf>
__device__ void scan_segments(const DevGraph& g, const DevSchedule& sc, int32_t group,
                              int32_t chunk_pages, CntOf cnt_of, int64_t (*sh)[1024],
                              uint64_t* keys) {
  const int t = threadIdx.x;
  const int S = g.S;
  const int per = (S + 1023) / 1024;
  const int s0 = min(S, t * per), s1 = min(S, s0 + per);
  auto seg_info = [&](int s, int& cnt, int& nch, int& nrb, int& npg) {
    cnt = cnt_of(s);
    npg = (g.seg_len[s] + kPageTokens - 1) / kPageTokens;
    nch = cnt > 0 ? (npg + chunk_pages - 1) / chunk_pages : 0;
    nrb = (int)(((int64_t)cnt * group + kRowsPerBlock - 1) / kRowsPerBlock);
  };
  // Inclusive block scan of three values into sh[0..2][t]: DPP wave scans, then the totals of
  // the waves before (group offsets are at most E, partial rows and items at most the int32
  // counts the plan was sized for, so every sum fits an int).
  auto block_scan = [&](int64_t a, int64_t b, int64_t c) {
    const int lane = t & 63, wv = t >> 6;
    int v[3] = {(int)a, (int)b, (int)c};
#pragma unroll
    for (int k = 0; k < 3; ++k) v[k] = wave_scan_incl(v[k]);
    __syncthreads();                               // readers of sh from before are done
    int* ws = reinterpret_cast<int*>(&sh[0][0]);   // [3][16] wave totals
    if (lane == 63) {
#pragma unroll
      for (int k = 0; k < 3; ++k) ws[k * 16 + wv] = v[k];
    }
    __syncthreads();
    int64_t r[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      int base = 0;
      for (int w = 0; w < wv; ++w) base += ws[k * 16 + w];
      r[k] = (int64_t)(v[k] + base);
    }
    __syncthreads();                               // every wave has read the totals
    sh[0][t] = r[0]; sh[1][t] = r[1]; sh[2][t] = r[2];
    __syncthreads();
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

  // 2. Work-list order: segments by descending cost class, ties by segment id, so the order is
  //    a pure function of the graph.  Up to 4096 segments: a stable counting sort by class
  //    (segment s = 1024 u + t sits in slot u; lanes of a wave with equal classes are matched
  //    by five bit ballots, and the per-(slot, wave) counts of each class are prefix-summed by
  //    one wave per class); beyond, a bitonic sort of unique 64-bit keys.  keys[i] ends up
  //    holding the segment at work-list position i.
  const bool sorted = S <= kSortCap;
  if (S <= 4096) {
    constexpr int NBK = kCostClasses;
    const int lane = t & 63, wv = t >> 6;
    const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
    const int nslots = (S + 1023) >> 10;
    int* cw = reinterpret_cast<int*>(&sh[0][0]);   // [class * 64 + slot * 16 + wave]
    int* tot = reinterpret_cast<int*>(&sh[2][0]);  // [class] totals, then [NBK + class] offsets
    __syncthreads();                               // readers of the last scan are done
    for (int i = t; i < 4 * 16 * NBK; i += 1024) cw[i] = 0;
    __syncthreads();
    int bk[4], wr[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      bk[u] = 0;
      wr[u] = 0;
      if (u < nslots) {
        const int sg = 1024 * u + t;
        const bool valid = sg < S;
        int bucket = 0;
        if (valid) {
          int cnt, nch, nrb, npg;
          seg_info(sg, cnt, nch, nrb, npg);
          const uint32_t cost = cnt > 0 ? item_cost(npg, cnt, group, chunk_pages) : 0u;
          bucket = kCostClasses - 1 - cost_class(cost);
        }
        uint64_t m = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 5; ++bit) {
          const bool on = (bucket >> bit) & 1;
          const uint64_t bb = __ballot(valid && on);
          m &= on ? bb : ~bb;
        }
        bk[u] = bucket;
        wr[u] = __popcll(m & lt);
        if (valid && (m & lt) == 0) cw[bucket * 64 + u * 16 + wv] = __popcll(m);
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {                  // wave wv: classes wv and wv + 16
      const int c = wv + 16 * h;
      const int v = cw[c * 64 + lane];
      int x = v;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (lane >= off) x += y;
      }
      cw[c * 64 + lane] = x - v;
      if (lane == 63) tot[c] = x;
    }
    __syncthreads();
    if (t < 64) {
      const int v = t < NBK ? tot[t] : 0;
      int x = v;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (t >= off) x += y;
      }
      if (t < NBK) tot[NBK + t] = x - v;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int sg = 1024 * u + t;
      if (u < nslots && sg < S)
        keys[tot[NBK + bk[u]] + cw[bk[u] * 64 + u * 16 + wv] + wr[u]] = (uint64_t)sg;
    }
    __syncthreads();
  } else if (sorted) {
    int n = 1;
    while (n < S) n <<= 1;
    for (int i = t; i < n; i += 1024) {
      uint64_t key = ~0ull;
      if (i < S) {
        int cnt, nch, nrb, npg;
        seg_info(i, cnt, nch, nrb, npg);
        const uint32_t cost = cnt > 0 ? item_cost(npg, cnt, group, chunk_pages) : 0u;
        key = ((uint64_t)(kCostClasses - cost_class(cost)) << 32) | (uint32_t)i;
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

__global__ __launch_bounds__(1024) void k_scan(DevGraph g, DevSchedule sc, int32_t group,
                                               int32_t chunk_pages) {
  __shared__ int64_t sh[3][1024];
  __shared__ uint64_t keys[kSortCap];
  // (a rescheduled plan skips k_init, whose only work then is this)
  if (threadIdx.x < kNumCounters) sc.counters[threadIdx.x] = 0;
  scan_segments(g, sc, group, chunk_pages, [&](int s) { return sc.grp_cnt[s]; }, sh, keys);
}

// Exclusive scan over path entries of their chunk counts (one 1024-thread workgroup): the slot
// of each entry's first partial in the flat per-branch lists, and the branch CSR offsets.
// Exclusive scan of the partial rows of every path entry (its segment's chunk count), in entry
// order, over many workgroups: k_entry_sums totals each block of kScanBlock entries, and
// k_entry_scan gives each block the sum of the blocks before it, scans inside the block and
// writes each branch's first slot at its first entry (k_bpart_off does that last part for a
// graph without entries).
constexpr int kScanBlock = 1024;

__device__ __forceinline__ int64_t block_sum_1024(int64_t v, int64_t* red) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) red[w] = v;
  __syncthreads();
  int64_t tot = 0;
  for (int i = 0; i < kScanBlock / 64; ++i) tot += red[i];
  __syncthreads();
  return tot;
}

__global__ __launch_bounds__(kScanBlock) void k_entry_sums(DevGraph g, DevSchedule sc) {
  __shared__ int64_t red[kScanBlock / 64];
  const int64_t e = (int64_t)blockIdx.x * kScanBlock + threadIdx.x;
  const int64_t v = e < g.E ? sc.seg_nchunk[g.path_segs[e]] : 0;
  const int64_t tot = block_sum_1024(v, red);
  if (threadIdx.x == 0) sc.blk_sum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kScanBlock) void k_entry_scan(DevGraph g, DevSchedule sc) {
  __shared__ int64_t red[kScanBlock / 64];
  __shared__ int64_t wsum[kScanBlock / 64];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  // Offset of this block: the sum of the block totals before it.
  int64_t pre = 0;
  for (int k = t; k < (int)blockIdx.x; k += kScanBlock) pre += sc.blk_sum[k];
  const int64_t base = block_sum_1024(pre, red);
  const int64_t e = (int64_t)blockIdx.x * kScanBlock + t;
  const int64_t v = e < g.E ? sc.seg_nchunk[g.path_segs[e]] : 0;
  int64_t x = v;                                   // inclusive scan inside the wave
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int64_t before = 0;
  for (int i = 0; i < w; ++i) before += wsum[i];
  if (e < g.E) {
    const int64_t slot = base + before + x - v;
    sc.entry_part[e] = slot;
    const int b = sc.entry_branch[e];
    if (e == g.path_off[b]) sc.bpart_off[b] = slot;
    if (e == g.E - 1) sc.bpart_off[g.B] = slot + v;
  }
}

__global__ void k_bpart_off(DevGraph g, DevSchedule sc) {
  const int64_t b = (int64_t)blockIdx.x * kT + threadIdx.x;
  if (b > g.B) return;
  if (b < g.B) {
    sc.bpart_off[b] = sc.entry_part[g.path_off[b]];
  } else {
    sc.bpart_off[b] =
        g.E > 0 ? sc.entry_part[g.E - 1] + sc.seg_nchunk[g.path_segs[g.E - 1]] : 0;
  }
}

// Descriptor causal word of the chunk of segment s that starts at page p0.
__device__ __forceinline__ int causal_word(const DevGraph& g, int s, int p0) {
  const int c = g.seg_causal[s];
  return c == kNoCausal ? kNoCausal : c - p0 * kPageTokens;
}

// Partial rows of path entry e (its segment's chunks, in order) into the branch list.
__device__ __forceinline__ void write_entry_parts(const DevGraph& g, const DevSchedule& sc,
                                                  int e, int rank, int cnt) {
  const int s = g.path_segs[e];
  const int nch = sc.seg_nchunk[s];
  const int64_t base = sc.seg_prow_off[s] + rank;
  const int64_t slot = sc.entry_part[e];
  for (int c = 0; c < nch; ++c) sc.bpart[slot + c] = (int32_t)(base + (int64_t)c * cnt);
}

// Emits the work items of segment s at work-list offset w (chunk-major, then row block): the
// (segment, chunk, row block) triple and the head of the item's descriptor.
__device__ __forceinline__ void emit_items(const DevGraph& g, const DevSchedule& sc, int s,
                                           int cnt, int group, int chunk_pages, int64_t w,
                                           int64_t goff, int64_t prow_off) {
  const int len = g.seg_len[s];
  const int npg = (len + kPageTokens - 1) / kPageTokens;
  const int nch = cnt > 0 ? (npg + chunk_pages - 1) / chunk_pages : 0;
  const int nrb = (int)(((int64_t)cnt * group + kRowsPerBlock - 1) / kRowsPerBlock);
  const int64_t poff = g.seg_page_off[s];
  const int last_valid = len - (npg - 1) * kPageTokens;
  for (int c = 0; c < nch; ++c) {
    const int p0 = chunk_first_page(c, npg, nch);
    const int np = chunk_first_page(c + 1, npg, nch) - p0;
    for (int rbk = 0; rbk < nrb; ++rbk, ++w) {
      sc.items[w] = make_int4(s, c, rbk, 0);
      int4* d = reinterpret_cast<int4*>(sc.desc + w * sc.desc_words);
      d[0] = make_int4(np, causal_word(g, s, p0), last_valid, cnt);
      d[1] = make_int4(rbk, (int)goff, (int)(poff + p0), (int)(prow_off + (int64_t)c * cnt));
    }
  }
}

// The whole scheduler in one workgroup for graphs that fit in LDS (<= kSmallSegs segments,
// <= kSmallEntries path entries, < kSmallBranches branches): the graph is read once into LDS and
// every phase works there between workgroup barriers; only outputs go to global memory.  Thread t
// owns a contiguous run of at most four segments (for the per-segment scans, in segment order and
// in work-list order) and a contiguous run of at most four branches (for the per-entry work).
constexpr int kSmallSegs = 4096;
constexpr int kSmallEntries = 8192;
constexpr int kSmallBranches = 4096;

// reuse: the plan's groups are already in place from an earlier schedule (B(s), |B(s)|, the
// group offsets, each entry's branch and rank, each group's branches in ascending order: they
// follow the paths alone, which a plan keeps); only what the lengths decide is recomputed.
__global__ __launch_bounds__(1024) void k_sched_one(DevGraph g, DevSchedule sc, int32_t group,
                                                    int32_t chunk_pages, int32_t reuse) {
  constexpr int NBK = kCostClasses;
  constexpr int SPT = kSmallSegs / 1024;
  __shared__ unsigned short l_segs[kSmallEntries];        // path_segs
  __shared__ unsigned short l_tmp[kSmallEntries];         // B(s) in arrival order
  __shared__ unsigned short l_poff[kSmallBranches + 1];   // path_off
  __shared__ int l_npg[kSmallSegs];                       // pages in use per segment
  __shared__ int l_nch[kSmallSegs];                       // chunks per segment
  __shared__ int l_part[kSmallEntries];                   // each entry's first partial slot
  __shared__ int l_cnt[kSmallSegs];                       // |B(s)|
  __shared__ int l_cur[kSmallSegs];                       // scatter cursors, then work-list order
  __shared__ int l_cw[NBK * 4 * 16];                      // sort: counts per (class, slot, wave)
  __shared__ int l_boff[NBK];                             // sort: first position of each class
  __shared__ int l_wsum[2][3][16];                        // wave totals of the two block scans
  int* const l_order = l_cur;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int S = g.S, E = g.E, B = g.B;
  const int per = (S + 1023) >> 10;
  const int s0 = min(S, t * per), s1 = min(S, s0 + per);
  const int pb = (B + 1023) >> 10;
  const int b0 = min(B, t * pb), b1 = min(B, b0 + pb);
  // pages in use and chunks of a segment on some path (its count is positive), computed once
  auto npg_of = [&](int s) { return l_npg[s]; };
  auto nch_len = [&](int s) { return l_nch[s]; };
  auto nrb_of = [&](int s) {
    return (int)(((int64_t)l_cnt[s] * group + kRowsPerBlock - 1) / kRowsPerBlock);
  };
  // Inclusive block scan of three ints (wave scans, then the totals of the waves before);
  // returns the inclusive values and, in tot, the block totals.
  auto block_scan3 = [&](int (&v)[3], int (*ws)[16], int (&tot)[3]) {
#pragma unroll
    for (int k = 0; k < 3; ++k) v[k] = wave_scan_incl(v[k]);
    if (lane == 63) {
#pragma unroll
      for (int k = 0; k < 3; ++k) ws[k][wv] = v[k];
    }
    lds_barrier();
#pragma unroll
    for (int k = 0; k < 3; ++k) tot[k] = 0;
    for (int w = 0; w < 16; ++w) {
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        const int x = ws[k][w];
        if (w < wv) v[k] += x;
        tot[k] += x;
      }
    }
  };

  // 0. Read the graph (all loads issued before any is used); clear the counts and the sort's
  //    bins.
  {
    int vs[kSmallEntries / 1024], vp[kSmallBranches / 1024], vl[SPT];
#pragma unroll
    for (int u = 0; u < kSmallEntries / 1024; ++u)
      vs[u] = t + 1024 * u < E ? g.path_segs[t + 1024 * u] : 0;
#pragma unroll
    for (int u = 0; u < kSmallBranches / 1024; ++u)
      vp[u] = t + 1024 * u <= B ? (int)g.path_off[t + 1024 * u] : 0;
#pragma unroll
    for (int u = 0; u < SPT; ++u) vl[u] = t + 1024 * u < S ? g.seg_len[t + 1024 * u] : 0;
#pragma unroll
    for (int u = 0; u < kSmallEntries / 1024; ++u)
      if (t + 1024 * u < E) l_segs[t + 1024 * u] = (unsigned short)vs[u];
#pragma unroll
    for (int u = 0; u < kSmallBranches / 1024; ++u)
      if (t + 1024 * u <= B) l_poff[t + 1024 * u] = (unsigned short)vp[u];
#pragma unroll
    for (int u = 0; u < SPT; ++u)
      if (t + 1024 * u < S) {
        const int npg = (vl[u] + kPageTokens - 1) / kPageTokens;
        l_npg[t + 1024 * u] = npg;
        l_nch[t + 1024 * u] = (npg + chunk_pages - 1) / chunk_pages;
      }
    if (reuse) {
#pragma unroll
      for (int u = 0; u < SPT; ++u)
        if (t + 1024 * u < S) l_cnt[t + 1024 * u] = sc.grp_cnt[t + 1024 * u];
    } else {
#pragma unroll
      for (int u = 0; u < SPT; ++u)
        if (t + 1024 * u < S) l_cnt[t + 1024 * u] = 0;
    }
    for (int i = t; i < 4 * 16 * NBK; i += 1024) l_cw[i] = 0;
  }
  if (t < kNumCounters) sc.counters[t] = 0;
  lds_barrier();

  // 1. |B(s)|, and the chunks of the entries of this thread's branches (one partial row per
  //    chunk in each branch's list).
  if (!reuse)
    for (int e = t; e < E; e += 1024) atomicAdd(&l_cnt[l_segs[e]], 1);
  int ne = 0;
  for (int e = l_poff[b0]; e < l_poff[b1]; ++e) ne += nch_len(l_segs[e]);
  lds_barrier();

  // 2. One scan in segment order (group offsets, partial-row offsets) and over this thread's
  //    branches (each branch's first slot in the partial lists); per-segment outputs; the
  //    sort's class counts.
  int slot0;
  {
    int v[3] = {0, ne, 0}, tot[3];
    for (int s = s0; s < s1; ++s) {
      const int cnt = l_cnt[s];
      v[0] += cnt;
      v[2] += cnt > 0 ? nch_len(s) * cnt : 0;
    }
    const int own0 = v[0], own2 = v[2];
    block_scan3(v, l_wsum[0], tot);
    int ra = v[0] - own0, rc = v[2] - own2;
    slot0 = v[1] - ne;
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      const int s = s0 + u;
      if (s < s1) {
        const int cnt = l_cnt[s];
        const int nch = cnt > 0 ? nch_len(s) : 0;
        if (!reuse) {
          l_cur[s] = ra;
          sc.grp_cnt[s] = cnt;
          sc.grp_off[s] = ra;
        }
        sc.seg_prow_off[s] = rc;
        sc.seg_nchunk[s] = nch;
        ra += cnt;
        rc += nch * cnt;
      }
    }
    if (t == 1023) {
      if (!reuse) sc.grp_off[S] = tot[0];
      sc.seg_prow_off[S] = tot[2];
      sc.counters[1] = tot[2];
      sc.bpart_off[B] = tot[1];
    }
  }
  // Work-list order: a stable counting sort of the segments by class (bin 0 = the costliest),
  // ties by segment id.  Segment 1024 u + t sits in slot u; lanes of a wave in the same bin are
  // matched by five bit ballots, and each first lane of a bin records the count.
  int bk[SPT], wr[SPT];
  const int nslots = (S + 1023) >> 10;
  {
    const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      bk[u] = 0;
      wr[u] = 0;
      if (u < nslots) {
        const int sg = 1024 * u + t;
        const bool valid = sg < S;
        int bin = 0;
        if (valid) {
          const int cnt = l_cnt[sg];
          const uint32_t cost = cnt > 0 ? item_cost(npg_of(sg), cnt, group, chunk_pages) : 0u;
          bin = NBK - 1 - cost_class(cost);
        }
        uint64_t m = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 5; ++bit) {
          const bool on = (bin >> bit) & 1;
          const uint64_t bb = __ballot(valid && on);
          m &= on ? bb : ~bb;
        }
        bk[u] = bin;
        wr[u] = __popcll(m & lt);
        if (valid && (m & lt) == 0) l_cw[bin * 64 + u * 16 + wv] = __popcll(m);
      }
    }
  }
  lds_barrier();                                   // cursors and class counts are complete

  // 3. Scatter each branch into its groups (arrival order); exclusive prefix of each class's
  //    counts over the (slot, wave) pairs (wave wv takes classes wv and wv + 16, lane = pair).
  if (!reuse)
    for (int b = b0; b < b1; ++b)
      for (int e = l_poff[b]; e < l_poff[b + 1]; ++e)
        l_tmp[atomicAdd(&l_cur[l_segs[e]], 1)] = (unsigned short)b;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = wv + 16 * h;
    const int v = l_cw[c * 64 + lane];           // (class-major: one contiguous row per class)
    const int x = wave_scan_incl(v);
    l_cw[c * 64 + lane] = x - v;
    if (lane == 63) l_boff[c] = x;                 // class total, made an offset below
  }
  lds_barrier();

  // 4. Per path entry of this thread's branches (a contiguous run of entries): its branch and
  //    its first slot in the branch's partial list, and each branch's first slot; B(s) in
  //    arrival order.  Ranks, groups in ascending order and the lists are written by k_emit.
  //    Wave 0 turns the class totals into offsets.
  {
    int slot = slot0;
    for (int b = b0; b < b1; ++b) {
      sc.bpart_off[b] = slot;
      for (int e = l_poff[b]; e < l_poff[b + 1]; ++e) {
        if (!reuse) sc.entry_branch[e] = b;
        l_part[e] = slot;                          // (written out coalesced after the barrier)
        slot += nch_len(l_segs[e]);
      }
    }
    if (!reuse)
      for (int e = t; e < E; e += 1024) sc.grp_tmp[e] = l_tmp[e];
  }
  if (wv == 0) {
    const int v = lane < NBK ? l_boff[lane] : 0;
    const int x = wave_scan_incl(v);
    if (lane < NBK) l_boff[lane] = x - v;
  }
  lds_barrier();

  // 5. Place each segment at its work-list position; the entries' first partial slots.
  for (int e = t; e < E; e += 1024) sc.entry_part[e] = l_part[e];
#pragma unroll
  for (int u = 0; u < SPT; ++u) {
    const int sg = 1024 * u + t;
    if (u < nslots && sg < S) l_order[l_boff[bk[u]] + l_cw[bk[u] * 64 + u * 16 + wv] + wr[u]] = sg;
  }
  lds_barrier();

  // 6. Item offsets in work-list order (this thread's positions s0 .. s1).
  {
    int v[3] = {0, 0, 0}, tot[3];
    for (int i = s0; i < s1; ++i) {
      const int s = l_order[i];
      v[0] += l_cnt[s] > 0 ? nch_len(s) * nrb_of(s) : 0;
    }
    const int own = v[0];
    block_scan3(v, l_wsum[1], tot);
    int w = v[0] - own;
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      const int i = s0 + u;
      if (i < s1) {
        const int s = l_order[i];
        sc.seg_item_off[s] = w;
        sc.seg_order[i] = s;
        sc.order_item_off[i] = w;
        // The segment's items (chunk-major, then row block), which k_emit then reads directly.
        const int nrb = nrb_of(s);
        const int nit = l_cnt[s] > 0 ? nch_len(s) * nrb : 0;
        for (int k = 0; k < nit; ++k) sc.items[w + k] = make_int4(s, k / nrb, k % nrb, 0);
        w += nit;
      }
    }
    if (t == 1023) {
      sc.seg_item_off[S] = tot[0];
      sc.order_item_off[S] = tot[0];
      sc.counters[0] = tot[0];
    }
  }
}

// Outputs of the single-workgroup scheduler that are independent per path entry and per item,
// written in parallel.
//   Blocks [0, eblocks), one thread per path entry (b, s): the rank r of b inside B(s) (count
//   of smaller branch ids in B(s) as scattered), B(s) in ascending order, the entry's rank, its
//   partial rows (one per chunk of s, in chunk order) and b's place in the branch list of every
//   descriptor whose row block holds b's rows.
//   Later blocks, one wave per work item (the items written by k_sched_one): the head of its
//   descriptor and the chunk's page ids.
__global__ __launch_bounds__(kT) void k_emit(DevGraph g, DevSchedule sc, int32_t group,
                                             int32_t chunk_pages, int32_t eblocks, int32_t reuse) {
  if ((int)blockIdx.x < eblocks) {
    const int e = blockIdx.x * kT + threadIdx.x;
    if (e >= g.E) return;
    const int s = g.path_segs[e];
    const int b = sc.entry_branch[e];
    const int off = (int)sc.grp_off[s];
    const int cnt = sc.grp_cnt[s];
    int r = 0;
    if (reuse) {
      r = sc.entry_rank[e];
    } else {
      int k = 0;
      for (; k + 4 <= cnt; k += 4)
        r += (sc.grp_tmp[off + k] < b) + (sc.grp_tmp[off + k + 1] < b) +
             (sc.grp_tmp[off + k + 2] < b) + (sc.grp_tmp[off + k + 3] < b);
      for (; k < cnt; ++k) r += sc.grp_tmp[off + k] < b;
      sc.grp_br[off + r] = b;
      sc.entry_rank[e] = r;
    }
    const int nch = sc.seg_nchunk[s];
    const int slot = (int)sc.entry_part[e];
    const int prow = (int)sc.seg_prow_off[s] + r;
    for (int c = 0; c < nch; ++c) sc.bpart[slot + c] = prow + c * cnt;
    const int nrb = (cnt * group + kRowsPerBlock - 1) / kRowsPerBlock;
    const int rb_lo = (r * group) / kRowsPerBlock;
    const int rb_hi = (r * group + group - 1) / kRowsPerBlock;
    const int w0 = (int)sc.seg_item_off[s];
    for (int c = 0; c < nch; ++c)
      for (int rb = rb_lo; rb <= rb_hi; ++rb) {
        const int64_t w = w0 + c * nrb + rb;
        const int j0 = (rb * kRowsPerBlock) / group;
        sc.desc[w * sc.desc_words + kDescHead + chunk_pages + (r - j0)] = b;
      }
    return;
  }
  const int64_t w = (int64_t)(blockIdx.x - eblocks) * (kT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= sc.counters[0]) return;
  const int4 it = sc.items[w];
  const int s = it.x, c = it.y, rb = it.z;
  const int cnt = sc.grp_cnt[s], len = g.seg_len[s];
  const int npg = (len + kPageTokens - 1) / kPageTokens;
  const int nch = (npg + chunk_pages - 1) / chunk_pages;
  const int p0 = chunk_first_page(c, npg, nch);
  const int np = chunk_first_page(c + 1, npg, nch) - p0;
  const int poff = (int)g.seg_page_off[s] + p0;
  int32_t* d = sc.desc + w * sc.desc_words;
  if (lane == 0) {
    reinterpret_cast<int4*>(d)[0] =
        make_int4(np, causal_word(g, s, p0), len - (npg - 1) * kPageTokens, cnt);
    reinterpret_cast<int4*>(d)[1] =
        make_int4(rb, (int)sc.grp_off[s], poff, (int)sc.seg_prow_off[s] + c * cnt);
  }
  for (int i = lane; i < np; i += 64) d[kDescHead + i] = g.seg_pages[poff + i];
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
__global__ void k_rank_items(DevGraph g, DevSchedule sc, int32_t group, int32_t chunk_pages,
                             int32_t reuse) {
  int i = blockIdx.x * kT + threadIdx.x;
  if (i < g.E && reuse) {
    const int s = g.path_segs[i];
    write_entry_parts(g, sc, i, sc.entry_rank[i], sc.grp_cnt[s]);
  } else if (i < g.E) {
    const int s = g.path_segs[i];
    const int b = sc.entry_branch[i];
    const int64_t off = sc.grp_off[s];
    const int cnt = sc.grp_cnt[s];
    // rank of b in B(s) = branches of the group below b (eight independent loads in flight)
    const int32_t* grp = sc.grp_tmp + off;
    int r0 = 0, r1 = 0, r2 = 0, r3 = 0, r4 = 0, r5 = 0, r6 = 0, r7 = 0, k = 0;
    for (; k + 8 <= cnt; k += 8) {
      r0 += grp[k] < b;
      r1 += grp[k + 1] < b;
      r2 += grp[k + 2] < b;
      r3 += grp[k + 3] < b;
      r4 += grp[k + 4] < b;
      r5 += grp[k + 5] < b;
      r6 += grp[k + 6] < b;
      r7 += grp[k + 7] < b;
    }
    for (; k < cnt; ++k) r0 += grp[k] < b;
    const int r = r0 + r1 + r2 + r3 + r4 + r5 + r6 + r7;
    sc.grp_br[off + r] = b;
    sc.entry_rank[i] = r;
    write_entry_parts(g, sc, i, r, cnt);
  }
  if (i < g.S)
    emit_items(g, sc, i, sc.grp_cnt[i], group, chunk_pages, sc.seg_item_off[i], sc.grp_off[i],
               sc.seg_prow_off[i]);
}

// Completes each item's descriptor after its head is written: the chunk's physical page ids and
// the branch ids of its row block (one wave per item).
__global__ void k_fill_desc(DevGraph g, DevSchedule sc, int32_t group, int32_t chunk_pages) {
  const int64_t w = (int64_t)blockIdx.x * (kT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= sc.counters[0]) return;
  int32_t* d = sc.desc + w * sc.desc_words;
  const int4 h0 = reinterpret_cast<const int4*>(d)[0];
  const int4 h1 = reinterpret_cast<const int4*>(d)[1];
  const int np = h0.x, cnt = h0.w, rb = h1.x, goff = h1.y, poff = h1.z;
  for (int i = lane; i < np; i += 64) d[kDescHead + i] = g.seg_pages[poff + i];
  const int row0 = rb * kRowsPerBlock;
  const int R = min(kRowsPerBlock, cnt * group - row0);
  const int j0 = row0 / group, nbj = (row0 + R - 1) / group - j0 + 1;
  for (int i = lane; i < nbj; i += 64) d[kDescHead + chunk_pages + i] = sc.grp_br[goff + j0 + i];
}

inline int blocks(int64_t n) { return (int)((n + kT - 1) / kT); }

}  // namespace

// One wave per chain: its segments in path order, each with its pages in order (the lanes copy a
// segment's pages together), the last page of a segment carrying its valid token count; the
// chain's length counts the token positions of that page list ((pages - 1) x 16 + valid tokens
// of the last page).
__global__ void k_chain_pages(LengthArgs a) {
  const int v = blockIdx.x * (kT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (v >= a.chains) return;
  int32_t* dst = a.chain_pages + a.chain_page_off[v];
  int pos = 0, last_valid = kPageTokens;
  for (int k = a.chain_seg_off[v]; k < a.chain_seg_off[v + 1]; ++k) {
    const int x = a.chain_segs[k];
    const int len = a.new_len[x];
    const int n = (len + kPageTokens - 1) / kPageTokens;
    const int32_t* src = a.src_pages + a.src_page_off[x];
    if (lane == 0) a.seg_pos[x] = pos;
    for (int i = lane; i < n; i += 64) {
      const int valid = i == n - 1 ? len - (n - 1) * kPageTokens : kPageTokens;
      dst[pos + i] = src[i] | ((valid - 1) << kPageValidShift);
    }
    pos += n;
    last_valid = len - (n - 1) * kPageTokens;
  }
  if (lane == 0) a.chain_len[v] = (pos - 1) * kPageTokens + last_valid;
}

// One thread per branch of a multi-query plan: its newest segment closes its chain, so query i of
// the branch sits at chain token 16 x (chain pages before the segment) + len - n + i.
__global__ void k_chain_causal(LengthArgs a) {
  const int b = blockIdx.x * kT + threadIdx.x;
  if (b >= a.branches) return;
  const int x = a.br_last[b];
  a.chain_causal[a.seg_chain[x]] = a.seg_pos[x] * kPageTokens + a.new_len[x] - a.br_count[b];
}

hipError_t launch_set_lengths(const LengthArgs& a, hipStream_t stream) {
  if (a.chains > 0)
    hipLaunchKernelGGL(k_chain_pages, dim3((unsigned)((a.chains + kT / 64 - 1) / (kT / 64))),
                       dim3(kT), 0, stream, a);
  if (a.branches > 0)
    hipLaunchKernelGGL(k_chain_causal, dim3((unsigned)((a.branches + kT - 1) / kT)), dim3(kT), 0,
                       stream, a);
  return hipGetLastError();
}

hipError_t launch_schedule(const DevGraph& g, const DevSchedule& sc, int32_t group,
                           int32_t chunk_pages, int64_t max_items, bool reuse,
                           hipStream_t stream) {
  const int fill_blocks = (int)((max_items + kT / 64 - 1) / (kT / 64));
  if (g.S <= kSmallSegs && g.E <= kSmallEntries && g.B < kSmallBranches) {
    hipLaunchKernelGGL(k_sched_one, dim3(1), dim3(1024), 0, stream, g, sc, group, chunk_pages,
                       (int32_t)reuse);
    const int eblocks = blocks(g.E);
    if (eblocks + fill_blocks > 0)
      hipLaunchKernelGGL(k_emit, dim3(eblocks + fill_blocks), dim3(kT), 0, stream, g, sc, group,
                         chunk_pages, eblocks, (int32_t)reuse);
    return hipGetLastError();
  }
  // (with reuse, the entry branches, |B(s)| and the groups in arrival order are not rebuilt,
  // and k_scan clears the counters)
  if (!reuse)
    hipLaunchKernelGGL(k_init, dim3(blocks(g.S > 4 ? g.S : 4)), dim3(kT), 0, stream, g, sc,
                       (int32_t)reuse);
  if (g.E > 0 && !reuse)
    hipLaunchKernelGGL(k_count, dim3(blocks(g.E)), dim3(kT), 0, stream, g, sc);
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, stream, g, sc, group, chunk_pages);
  const int64_t sblocks = ((int64_t)g.E + kScanBlock - 1) / kScanBlock;
  if (sblocks > 0) {
    hipLaunchKernelGGL(k_entry_sums, dim3((unsigned)sblocks), dim3(kScanBlock), 0, stream, g, sc);
    hipLaunchKernelGGL(k_entry_scan, dim3((unsigned)sblocks), dim3(kScanBlock), 0, stream, g, sc);
  } else {
    hipLaunchKernelGGL(k_bpart_off, dim3(blocks((int64_t)g.B + 1)), dim3(kT), 0, stream, g, sc);
  }
  if (g.E > 0 && !reuse)
    hipLaunchKernelGGL(k_scatter, dim3(blocks(g.E)), dim3(kT), 0, stream, g, sc);
  const int64_t n = g.E > g.S ? g.E : g.S;
  if (n > 0)
    hipLaunchKernelGGL(k_rank_items, dim3(blocks(n)), dim3(kT), 0, stream, g, sc, group,
                       chunk_pages, (int32_t)reuse);
  if (fill_blocks > 0)
    hipLaunchKernelGGL(k_fill_desc, dim3(fill_blocks), dim3(kT), 0, stream, g, sc, group,
                       chunk_pages);
  return hipGetLastError();
}

}  // namespace ga
