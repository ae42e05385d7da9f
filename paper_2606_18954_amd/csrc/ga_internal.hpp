// Internal declarations shared by the host runtime (api.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace ga {

constexpr int kPageTokens = 16;
// Page-table words: page id in bits [0, 27), valid tokens of the page minus one above.
constexpr int kPageValidShift = 27;
constexpr int32_t kPageIdMask = (1 << kPageValidShift) - 1;
// Query rows (branch x q-head-in-group) handled by one work item: 8 MFMA row tiles of 16.
constexpr int kRowsPerBlock = 128;
// Upper bound on pages per work item (the chunk's page ids are staged in LDS).
constexpr int kMaxChunkPages = 128;
constexpr int kAttnThreads = 256;        // 4 wave64 per workgroup

// Work-item descriptor (int32 words, one per item, fixed stride), written by the scheduler and
// copied whole into LDS by the attention kernel:
//   [0..3]  pages in the chunk, causal word (kNoCausal, or for a multi-query segment c such that
//           the row of group rank j sees chunk token 16 x page + slot only up to c + j), valid
//           tokens of the segment's last page, |B(s)|
//   [4..7]  row block, group offset of B(s), page-table offset of the chunk, first partial row
//   [8 .. 8 + chunk_pages)            page words of the chunk (page id | (valid tokens - 1) << 27)
//   [8 + chunk_pages .. + branches)   branch ids of the row block's rows (B(s) from row0/group)
constexpr int kDescHead = 8;
constexpr int32_t kNoCausal = 0x40000000;
constexpr int kDescMaxBytes = 1024;      // LDS slot per descriptor (one 1 KiB copy)
__host__ __device__ inline int desc_branch_max(int group) {
  const int n = (kRowsPerBlock + group - 1) / group + 1;
  return n < kRowsPerBlock ? n : kRowsPerBlock;
}
__host__ __device__ inline int desc_words(int chunk_pages, int group) {
  return (kDescHead + chunk_pages + desc_branch_max(group) + 3) & ~3;
}
// Most pages a chunk may have so that its descriptor fits one slot (the chunk size is capped
// at this by the plan, so that no chunk's descriptor outgrows the slot).
__host__ __device__ inline int max_chunk_pages(int group) {
  const int fit = kDescMaxBytes / 4 - kDescHead - desc_branch_max(group);
  return fit < kMaxChunkPages ? fit : kMaxChunkPages;
}
static_assert(kDescMaxBytes / 4 - kDescHead - kRowsPerBlock >= 64,
              "a descriptor slot must hold a useful chunk at every group size");

// Device copy of the rollout graph (chains as segments), written by plan_create's upload; the
// lengths, page lists and causal origins are rewritten in place by a length update.
struct DevGraph {
  int32_t S, B, E;
  const int32_t* seg_len;        // [S]
  const int64_t* seg_page_off;   // [S+1] start of each list (room for all owned pages)
  const int32_t* seg_pages;      // [P]   the first ceil(seg_len / 16) entries of each list used
  const int64_t* path_off;       // [B+1]
  const int32_t* path_segs;      // [E]
  const int32_t* seg_causal;     // [S]  causal origin of a multi-query segment, else kNoCausal:
                                 //      the row of group rank j sees token 16 x page + slot of
                                 //      the segment's page list only up to seg_causal + j
};

// Scheduler outputs (device memory owned by the plan).
struct DevSchedule {
  int32_t* grp_cnt;        // [S]   |B(s)|
  int32_t* grp_fill;       // [S]   scatter cursors
  int64_t* grp_off;        // [S+1] CSR offsets of B(s)
  int32_t* grp_tmp;        // [E]   B(s) in arrival order
  int32_t* grp_br;         // [E]   B(s), ascending branch ids
  int32_t* entry_branch;   // [E]   branch of each path entry
  int32_t* entry_rank;     // [E]   position of the entry's branch inside B(s)
  int32_t* seg_nchunk;     // [S]   page chunks of each segment
  int64_t* seg_item_off;   // [S+1] first work item of each segment
  int64_t* seg_prow_off;   // [S+1] first partial row (per q-head) of each segment
  int32_t* seg_order;      // [S]   segments in work-list order
  int64_t* order_item_off; // [S+1] first work item of the segment at each work-list position
  int4* items;             // [max_items] (segment, chunk, row block, unused)
  int32_t* desc;           // [max_items * desc_words (+ kDescMaxBytes of padding)] descriptors
  int32_t desc_words;      // descriptor stride in int32 words (a multiple of 4)
  int64_t* counters;       // [8]: items, partial rows, spare, spare, then kMaxStreams int32
                           //      work-stream heads (the attention kernel's claim counters)
  int64_t* entry_part;     // [E]   first slot of each path entry in the branch partial lists
  int64_t* bpart_off;      // [B+1] CSR offsets of each branch's partial rows
  int32_t* bpart;          // [partial rows] partial rows of each branch: path order, then chunk
  int64_t* blk_sum;        // [ceil(E / 1024)] per-block totals of the entry scan
};

// Partial rows (one per partial row and q-head), in one of two formats:
// * fp32 inputs: po [rows][Hq][D] fp32, the normalised partial output o in column order;
//   plse [rows][Hq] fp32, its log2-domain log-sum-exp lambda.
// * bf16 inputs: po [rows][Hq][D] fp16, o scaled by 2^(15 - e) (e: the binary exponent of the
//   row's largest |o|, so every value is below 2^15) and stored in lane order: column
//   16 n + 4 g + i (n < D/16, g < 4, i < 4) at position 32 (n / 2) + 8 g + 4 (n % 2) + i, so
//   the four lanes that hold a tile row write 64 contiguous bytes per store; plse [rows][Hq][2]
//   fp32, (lambda, 2^(e - 15)), the second being the factor that undoes the scaling.
constexpr int kPartScaleBits = 15;

// The attention kernel's work streams: the units of kv heads h with h mod streams == s form
// stream s, owned by the workgroups with blockIdx mod streams == s.  Workgroups are dispatched
// to the eight XCDs round robin, so a stream is served by 8 / streams of them, and the row
// blocks of one (chunk, kv head) share those XCDs' L2s.
constexpr int kMaxStreams = 8;
constexpr int kNumCounters = 4 + kMaxStreams / 2;   // int64 words of the counters array

struct AttnArgs {
  const void* q;
  const void* pool;
  const int32_t* desc;     // work-item descriptors (layout above)
  int64_t* counters;       // [0] items; from [4], kMaxStreams int32 work-stream heads (units
                           //     of each stream claimed past its first two rounds)
  void* po;                // partial outputs (format above)
  float* plse;             // partial log-sum-exps (format above)
  int32_t Hq, Hkv, group, chunk_pages;
  int32_t desc_words;      // descriptor stride (int32 words)
  int32_t streams;         // work streams: divides Hkv and kMaxStreams
  float scale_log2;        // softmax scale * log2(e)
};

struct MergeArgs {
  const int64_t* bpart_off;
  const int32_t* bpart;
  const void* po;          // partial outputs (format above)
  const float* plse;
  void* out;
  float* lse;
  int64_t* counters;       // the attention kernel's work-stream heads are re-armed here
  int32_t B, Hq;
};

// Page-pool writes (kv_write.hip): token j goes to slot word dst_words[j] (page * 16 + slot),
// from k_new / v_new [n][Hkv][D] (append, src_words == nullptr) or from the pool slot
// src_words[j] (copy).  Tokens whose words fall outside [0, num_slots) are skipped.
struct KvWriteArgs {
  unsigned char* pool;
  const unsigned char* k_new;
  const unsigned char* v_new;
  const int32_t* src_words;
  const int32_t* dst_words;
  int64_t num_slots;       // num_pages * 16
  int32_t n, Hkv, row_bytes;
};

// Equivalence detection (equiv.hip).  z [N][dim] bf16 bits; items: (first row state, first
// column state, end of their prompt's states, unused) per 64 x 64 tile, row tile <= column tile.
struct EquivArgs {
  const unsigned short* z;
  float* inv_norm;         // [N]
  int* rep;                // [N]  union-find parents
  const int32_t* tin;      // [N]  Euler interval of each state in its generation tree
  const int32_t* tout;     // [N]
  const int4* items;       // [n_items] tiles of the prompts of more than 256 states
  const int2* prompts;     // [n_prompts] (first state, states) of the prompts of <= 256 states
  const int32_t* big;      // [n_big] the states of the larger prompts
  int32_t* labels;         // [N]  output: smallest state of the class
  const int32_t* parent;   // [N]
  float* edge_sim;         // [N]  optional output: sim(p(v), v), 0 for a root
  int64_t N, n_items, n_prompts, n_big;
  int32_t dim;
  float kappa;
};

struct SuffixArgs {
  const int32_t* labels;   // [N]
  const int32_t* parent;   // [N]
  const int32_t* depth;    // [N]
  const int32_t* pstart;   // [N]  first state of the state's prompt
  const int32_t* pend;     // [N]  one past its last state
  int64_t* cnt;            // [N]  |C_g(u)|
  int64_t* off;            // [N + 1] CSR offsets
  int64_t* blk;            // [ceil(N / 1024)] scan block totals
  int32_t* states;         // [total] output
  int64_t N;
};

// Graph reward and dual-group advantage (reward.hip).  Device arrays of N states unless noted.
struct RewardArgs {
  const int32_t* labels;   // class labels (smallest member)
  const int32_t* reward;   // R(v) >= 0 for a terminal state, negative otherwise
  const float* edge_sim;   // sim(p(v), v)
  const int32_t *parent, *depth, *tin, *tout, *pstart, *pend;
  int32_t* lab;            // labels, sanitised
  int64_t* euler;          // packed (R, 1) of terminal states in Euler order
  int64_t* pre;            // [N + 1] its exclusive prefix sums
  int64_t* blk;            // scan block totals
  int64_t* own;            // packed (c_own, t_own)
  int64_t* ctot;           // packed class totals, by label
  int32_t* anchor;         // a_Q of each member of a class of two or more, else -1
  double* aeff_node;       // A_eff(v) of each such member
  double *gmean, *gstd;    // correctness-group statistics of each source state
  double *score, *step, *a_cor, *a_eff, *a_dual;   // outputs
  const int2* prompts;     // [n_prompts] (first state, states) of every prompt
  int64_t N, n_prompts;
  int64_t n_big;           // states in prompts of more than 512 states (0: one launch per batch)
  double w, lambda_eff;
};

// Launchers (each returns the launch status).
// New segment lengths applied on the device: each chain's page list (laid out at a fixed offset
// with room for every page its segments own), its length and, for multi-query plans, its causal
// origin are rebuilt from the lengths of the segments as given.
struct LengthArgs {
  int32_t chains, branches;        // chains; branches as given (multi-query plans, else 0)
  const int32_t* new_len;          // [S0] lengths of the segments as given
  const int64_t* src_page_off;     // [S0+1] page table as given
  const int32_t* src_pages;        // [P0]
  const int32_t* chain_seg_off;    // [chains+1] CSR of each chain's segments, in path order
  const int32_t* chain_segs;
  const int32_t* seg_chain;        // [S0] chain of each segment (-1: on no path)
  const int32_t* br_last;          // [branches] newest segment of each branch
  const int32_t* br_count;         // [branches] its query count
  int32_t* seg_pos;                // [S0] written: pages of its chain before the segment
  int32_t* chain_len;              // [chains] written (DevGraph::seg_len)
  const int64_t* chain_page_off;   // [chains+1] (DevGraph::seg_page_off)
  int32_t* chain_pages;            // written (DevGraph::seg_pages)
  int32_t* chain_causal;           // [chains] written for multi-query plans (DevGraph::seg_causal)
};
hipError_t launch_set_lengths(const LengthArgs& a, hipStream_t stream);

// reuse: the groups (B(s), |B(s)|, entry branches and ranks, ascending group lists) written by
// an earlier schedule of the same plan are still in place, and only what the lengths decide is
// recomputed.
hipError_t launch_schedule(const DevGraph& g, const DevSchedule& sc, int32_t group,
                           int32_t chunk_pages, int64_t max_items, bool reuse,
                           hipStream_t stream);
// few_pages: a decode step with under 64 pages (times kv-heads) per workgroup at two per CU.
// t0 / t1 (optional, timing events): bound to the kernel's own dispatch (hipExtLaunchKernel), so
// that their elapsed time is the kernel's execution, without the queue's gaps around it.
hipError_t launch_seg_attn(const AttnArgs& a, int head_dim, bool bf16, bool causal,
                           bool few_pages, int grid, hipStream_t stream,
                           hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
// t0 / t1 as for launch_seg_attn; no kernel (and no event) when there are no rows.
hipError_t launch_merge(const MergeArgs& a, int head_dim, bool out_bf16, bool part_f16,
                        hipStream_t stream, hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
hipError_t launch_kv_write(const KvWriteArgs& a, hipStream_t stream);
hipError_t launch_equivalence(const EquivArgs& a, hipStream_t stream);
hipError_t launch_suffix_count(const SuffixArgs& a, hipStream_t stream);
hipError_t launch_suffix_fill(const SuffixArgs& a, hipStream_t stream);
hipError_t launch_advantages(const RewardArgs& a, hipStream_t stream);
// Number of co-resident attention workgroups the persistent grid uses on this device.
int seg_attn_grid(int head_dim, bool bf16, bool causal, bool few_pages, int num_cus);
// Work streams of an attention launch (the largest power of two dividing Hkv and
// kMaxStreams): multi-query units split a shared chunk into many row blocks, each of which
// reads the chunk, so they are kept on few XCDs.  Decode units mostly hold one row block per
// chunk and keep one stream.
inline int attn_streams(int Hkv, bool causal) {
  if (!causal) return 1;
  int s = kMaxStreams;
  while (Hkv % s) s >>= 1;
  return s;
}

}  // namespace ga
