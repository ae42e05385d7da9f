// Host runtime of the graph-segment decode attention library: validation, plans, workspace,
// launches and the C entry points declared in include/graphattn.h.
#include "../../include/graphattn.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "ga_internal.hpp"

namespace {

thread_local std::string g_err;

ga_status fail(ga_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

ga_status hip_fail(hipError_t e, const char* what) {
  return fail(GA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define GA_HIP(call, what)                       \
  do {                                           \
    hipError_t e_ = (call);                      \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Attention workgroups kept resident per device (persistent grid).
int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    return 256;
  return n;
}

// The graph as uploaded.  Consecutive segments whose branch sets are identical (every branch
// through s continues with s', and |B(s)| = |B(s')|) form a chain; attention over a chain's
// concatenated tokens equals the log-sum-exp merge of its segments, so each chain is scheduled
// as one segment: one partial per branch and chunk, and longer work items.  A chain's page list
// concatenates the pages its segments' lengths use, in path order; every page id carries its
// valid token count in the bits from ga::kPageValidShift up, so the pages where a segment ends
// mid-page are masked.  Each chain's list starts at a fixed offset with room for every page its
// segments own in the page table, so new lengths (graphattn_plan_set_lengths) rewrite it in
// place.
struct CGraph {
  int32_t S0 = 0;                  // segments and path entries as given
  int64_t E0 = 0;
  std::vector<int32_t> seg_len, seg_pages, path_segs, npg;
  std::vector<int64_t> seg_page_off, path_off;
  std::vector<int32_t> vid;        // [S0] chain of each segment (-1: on no path)
  std::vector<int32_t> ventry;     // [E0] uploaded entry of the chain the path entry belongs to
  std::vector<int32_t> head;       // [chains] first segment of each chain
  std::vector<char> first;         // [S0] the segment starts its chain
  std::vector<int32_t> causal;     // [chains] causal origin (multi-query plans), else kNoCausal
  std::vector<int32_t> chain_seg_off, chain_segs;   // CSR: each chain's segments in path order
};

struct Sizes {
  int32_t S = 0, B = 0, E = 0;
  int64_t P = 0;               // entries of seg_pages in use
  // Length updates (graphattn_plan_set_lengths): the graph as given and the chains' segments.
  int32_t S0 = 0, B0q = 0, CS = 0;   // segments; branches of a multi-query plan; chain entries
  int64_t P0 = 0;                    // entries of the page table as given
  int32_t chunk_pages = 0;
  bool few_pages = false;      // under 64 pages (x kv-heads) per workgroup at two per CU
  int64_t max_items = 0;       // upper bound on work items per kv-head
  int32_t desc_words = 0;      // work-item descriptor stride (int32 words)
  int64_t prows = 0;           // partial rows per q-head
};

}  // namespace

namespace ga {
// Error reporting for the other host source files (equiv_api.cpp).
ga_status host_fail(ga_status st, const char* msg) { return fail(st, "%s", msg); }
ga_status host_hip_fail(hipError_t e, const char* what) { return hip_fail(e, what); }
void host_clear_error() { g_err.clear(); }
}  // namespace ga

struct ga_plan {
  ga_params p{};
  Sizes z;
  // One device allocation carved into the graph copy, the schedule and the partial buffers.
  void* dev = nullptr;
  size_t dev_bytes = 0;
  void* pin = nullptr;         // pinned host staging of the graph upload
  size_t pin_bytes = 0;
  bool owns_memory = true;
  bool scheduled = false;
  bool grouped = false;        // the groups of an earlier schedule are in the workspace
  bool causal = false;         // a multi-query plan (graphattn_plan_create_extend)
  int32_t B0 = 0;              // branches as given (z.B counts query rows)
  int num_cus = 256;
  CGraph cg;                   // the uploaded (chain) graph and its map to the given one
  // Length updates (graphattn_plan_set_lengths): the page table's offsets and, for multi-query
  // plans, each branch's newest segment and query count, for validation on the host; the device
  // side rebuilds the chains' page lists from arrays uploaded with the graph (la).
  bool updatable = false;
  std::vector<int64_t> h_page_off;
  std::vector<int32_t> h_pages;    // (kept until the first upload has packed it)
  std::vector<int32_t> h_last, h_counts;
  ga::LengthArgs la{};
  size_t len_off = 0;              // byte offset of the device copy of the lengths
  // Pinned slots for the lengths of successive updates, each reused only after its copy has
  // left it, so the host may run a few updates ahead of the device.
  static constexpr int kLenSlots = 4;
  int32_t* len_pin = nullptr;
  hipEvent_t len_ev[kLenSlots] = {};
  int64_t len_calls = 0;
  hipEvent_t uploaded = nullptr;   // recorded after the graph upload from the pinned staging
  ga::DevGraph g{};
  ga::DevSchedule sc{};
  void* po = nullptr;
  float* plse = nullptr;
  // Kernel timing (graphattn_plan_profile): events for up to prof_cap schedule / run calls.
  int32_t prof_cap = 0, prof_sched = 0, prof_runs = 0;
  std::vector<hipEvent_t> ev_sched;   // 2 per recorded schedule call
  std::vector<hipEvent_t> ev_run;     // 4 per recorded run: attention start and end, merge start
                                      // and end
  hipEvent_t ev_last = nullptr;
};

namespace {

// ----------------------------------------------------------------------------------------------
// Validation (host, before any device work)
// ----------------------------------------------------------------------------------------------

ga_status validate_params(const ga_params* p) {
  if (!p) return fail(GA_EINVAL, "params is NULL");
  if (p->num_q_heads <= 0 || p->num_kv_heads <= 0)
    return fail(GA_EINVAL, "head counts must be positive (Hq=%d, Hkv=%d)", p->num_q_heads,
                p->num_kv_heads);
  if (p->num_q_heads % p->num_kv_heads)
    return fail(GA_EINVAL, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)",
                p->num_q_heads, p->num_kv_heads);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(GA_EUNSUPPORTED, "head_dim %d unsupported (64 or 128)", p->head_dim);
  if (p->page_size != ga::kPageTokens)
    return fail(GA_EUNSUPPORTED, "page_size %d unsupported (16)", p->page_size);
  if (p->dtype != GA_F32 && p->dtype != GA_BF16)
    return fail(GA_EUNSUPPORTED, "dtype %d unsupported", p->dtype);
  if (p->num_pages < 0) return fail(GA_EINVAL, "num_pages is negative");
  if (p->num_pages > (1LL << ga::kPageValidShift))
    return fail(GA_EUNSUPPORTED, "num_pages %lld exceeds 2^%d", (long long)p->num_pages,
                ga::kPageValidShift);
  if (!std::isfinite(p->softmax_scale) || p->softmax_scale < 0.f)
    return fail(GA_EINVAL, "softmax_scale must be finite and >= 0");
  if (p->out_f32 != 0 && p->out_f32 != 1) return fail(GA_EINVAL, "out_f32 must be 0 or 1");
  return GA_OK;
}

ga_status validate_graph(const ga_segment_table* st, const ga_branch_paths* bp,
                         const ga_params* p, Sizes* z, std::vector<int32_t>* seg_npages) {
  if (!st) return fail(GA_EINVAL, "segment_table is NULL");
  if (!bp) return fail(GA_EINVAL, "branch_paths is NULL");
  const int32_t S = st->num_segments, B = bp->num_branches;
  if (S < 0) return fail(GA_EINVAL, "num_segments is negative");
  if (B < 0) return fail(GA_EINVAL, "num_branches is negative");
  if (!st->seg_page_offsets) return fail(GA_EINVAL, "seg_page_offsets is NULL");
  if (S > 0 && !st->seg_len) return fail(GA_EINVAL, "seg_len is NULL");
  if (st->seg_page_offsets[0] != 0) return fail(GA_EINVAL, "seg_page_offsets[0] must be 0");
  seg_npages->assign(S, 0);
  for (int32_t s = 0; s < S; ++s) {
    const int32_t len = st->seg_len[s];
    if (len < 1) return fail(GA_EINVAL, "segment %d has length %d (< 1)", s, len);
    const int64_t a = st->seg_page_offsets[s], b = st->seg_page_offsets[s + 1];
    if (b < a) return fail(GA_EINVAL, "seg_page_offsets decreases at segment %d", s);
    const int64_t need = (len + ga::kPageTokens - 1) / ga::kPageTokens;
    if (b - a < need)
      return fail(GA_EINVAL, "segment %d has %lld tokens but only %lld pages", s, (long long)len,
                  (long long)(b - a));
    (*seg_npages)[s] = (int32_t)need;
  }
  const int64_t P = st->seg_page_offsets[S];
  if (P > 0 && !st->seg_pages) return fail(GA_EINVAL, "seg_pages is NULL");
  for (int64_t i = 0; i < P; ++i) {
    const int32_t pg = st->seg_pages[i];
    if (pg < 0 || pg >= p->num_pages)
      return fail(GA_ERANGE, "seg_pages[%lld] = %d outside [0, %lld)", (long long)i, pg,
                  (long long)p->num_pages);
  }
  if (!bp->path_offsets) return fail(GA_EINVAL, "path_offsets is NULL");
  if (bp->path_offsets[0] != 0) return fail(GA_EINVAL, "path_offsets[0] must be 0");
  const int64_t E = bp->path_offsets[B];
  if (E > 0x7fffffffLL) return fail(GA_EINVAL, "too many path entries (%lld)", (long long)E);
  if (E > 0 && !bp->path_segs) return fail(GA_EINVAL, "path_segs is NULL");
  std::vector<int32_t> stamp(S, -1);
  for (int32_t b = 0; b < B; ++b) {
    const int64_t a = bp->path_offsets[b], e1 = bp->path_offsets[b + 1];
    if (e1 < a) return fail(GA_EINVAL, "path_offsets decreases at branch %d", b);
    if (e1 == a) return fail(GA_EINVAL, "branch %d has an empty path", b);
    for (int64_t e = a; e < e1; ++e) {
      const int32_t s = bp->path_segs[e];
      if (s < 0 || s >= S)
        return fail(GA_ERANGE, "branch %d names segment %d outside [0, %d)", b, s, S);
      if (stamp[s] == b) return fail(GA_EINVAL, "branch %d visits segment %d twice", b, s);
      stamp[s] = b;
    }
  }
  z->S = S;
  z->B = B;
  z->E = (int32_t)E;
  z->P = P;
  return GA_OK;
}

// Builds the chain graph (CGraph above) from a validated graph; npg0 = pages of each segment.
ga_status compress_chains(const ga_segment_table* st, const ga_branch_paths* bp,
                          const std::vector<int32_t>& npg0, CGraph* c) {
  const int32_t S = st->num_segments, B = bp->num_branches;
  const int64_t E = bp->path_offsets[B];
  c->S0 = S;
  c->E0 = E;
  // succ[s]: the segment every path continues with after s (-1: none or not unique).
  std::vector<int32_t> cnt(S, 0), succ(S, -2), link(S, -1);
  std::vector<char> haspred(S, 0);
  for (int32_t b = 0; b < B; ++b)
    for (int64_t e = bp->path_offsets[b]; e < bp->path_offsets[b + 1]; ++e) {
      const int32_t s = bp->path_segs[e];
      const int32_t n = e + 1 < bp->path_offsets[b + 1] ? bp->path_segs[e + 1] : -1;
      ++cnt[s];
      succ[s] = succ[s] == -2 ? n : (succ[s] == n ? n : -1);
    }
  // s links to s' when every branch through s continues with s' and no other branch enters s',
  // so B(s) = B(s').  Each segment has at most one link in and out, and paths never revisit a
  // segment, so the links form disjoint chains.
  for (int32_t s = 0; s < S; ++s) {
    const int32_t n = succ[s];
    if (cnt[s] > 0 && n >= 0 && cnt[n] == cnt[s]) {
      link[s] = n;
      haspred[n] = 1;
    }
  }
  c->vid.assign(S, -1);
  c->first.assign(S, 0);
  c->head.clear();
  c->causal.clear();
  c->seg_len.clear();
  c->npg.clear();
  c->seg_pages.clear();
  c->seg_page_off.assign(1, 0);
  c->chain_seg_off.assign(1, 0);
  c->chain_segs.clear();
  for (int32_t s = 0; s < S; ++s) {
    if (cnt[s] == 0 || haspred[s]) continue;
    const int32_t v = (int32_t)c->head.size();
    c->head.push_back(s);
    c->first[s] = 1;
    int64_t pages = 0, owned = 0;
    int32_t last_valid = ga::kPageTokens;
    const int64_t base = (int64_t)c->seg_pages.size();
    for (int32_t x = s; x >= 0; x = link[x]) {
      c->vid[x] = v;
      c->chain_segs.push_back(x);
      owned += st->seg_page_offsets[x + 1] - st->seg_page_offsets[x];
      const int32_t len = st->seg_len[x], n = npg0[x];
      const int64_t off = st->seg_page_offsets[x];
      for (int32_t i = 0; i < n; ++i) {
        const int32_t valid = i == n - 1 ? len - (n - 1) * ga::kPageTokens : ga::kPageTokens;
        c->seg_pages.push_back(st->seg_pages[off + i] | ((valid - 1) << ga::kPageValidShift));
      }
      pages += n;
      last_valid = len - (n - 1) * ga::kPageTokens;
    }
    const int64_t tokens = (pages - 1) * ga::kPageTokens + last_valid;
    // Every page the chain's segments own could come into use (graphattn_plan_set_lengths):
    // the page list keeps room for all of them, and the token positions must stay in range.
    if (owned * ga::kPageTokens >= ga::kNoCausal)
      return fail(GA_EUNSUPPORTED, "segment chain from segment %d owns %lld pages", s,
                  (long long)owned);
    c->seg_pages.resize(base + owned, 0);
    c->seg_len.push_back((int32_t)tokens);
    c->npg.push_back((int32_t)pages);
    c->causal.push_back(ga::kNoCausal);
    c->seg_page_off.push_back((int64_t)c->seg_pages.size());
    c->chain_seg_off.push_back((int32_t)c->chain_segs.size());
  }
  // Paths over chains: a chain's first segment stands for the chain; the rest of the chain
  // follows it immediately in every path through it.
  c->path_segs.clear();
  c->path_off.assign(1, 0);
  c->ventry.assign(E, -1);
  for (int32_t b = 0; b < B; ++b) {
    int32_t cur = -1;
    for (int64_t e = bp->path_offsets[b]; e < bp->path_offsets[b + 1]; ++e) {
      const int32_t s = bp->path_segs[e];
      if (c->first[s]) {
        cur = (int32_t)c->path_segs.size();
        c->path_segs.push_back(c->vid[s]);
      }
      c->ventry[e] = cur;
    }
    c->path_off.push_back((int64_t)c->path_segs.size());
  }
  return GA_OK;
}

// Chunking policy: split a segment only when the whole step would otherwise leave the
// persistent grid short of work; every extra chunk costs one more partial per branch row.
// The chunk size follows the pages in use (npg); the bounds on partial rows and work items
// follow the pages each chain owns (npg_cap >= npg), so that any later lengths fit.
void size_schedule(const ga_segment_table* st, const ga_branch_paths* bp, const ga_params* p,
                   const std::vector<int32_t>& npg, const std::vector<int64_t>& npg_cap,
                   int num_cus, Sizes* z) {
  std::vector<char> used(z->S, 0);
  for (int64_t e = 0; e < z->E; ++e) used[bp->path_segs[e]] = 1;
  int64_t ref_pages = 0;
  for (int32_t s = 0; s < z->S; ++s) ref_pages += used[s] ? npg[s] : 0;
  // About 4 work items per resident workgroup, in chunks of at most 128 pages (longer units
  // leave too long a tail once the queue is empty; a little fewer at group size 1, so that the
  // descriptor's list of up to 128 branches still fits its slot), and no chunk shorter than the
  // pages each workgroup has anyway (up to 24): a unit costs about as much as 13 pages before
  // its first page, so short units pay mostly overhead, unless the graph is too small to give
  // every workgroup work (then short chunks spread it; 4 pages at the least).  Fewer, longer
  // chunks also mean fewer partial rows to merge and fewer items to schedule.
  const int64_t wgs = 2LL * num_cus;
  const int64_t target_items = 4 * wgs;
  const int64_t work = ref_pages * p->num_kv_heads;
  int64_t cap = (work + target_items - 1) / target_items;
  const int32_t max_cap = ga::max_chunk_pages(p->num_q_heads / p->num_kv_heads);
  if (cap > max_cap) cap = max_cap;
  const int64_t floor_pages = std::min<int64_t>(24, std::max<int64_t>(4, (work + wgs - 1) / wgs));
  if (cap < floor_pages) cap = floor_pages;
  z->chunk_pages = (int32_t)cap;
  // A step this small gives each workgroup one or two units, whose fixed costs (first pages'
  // latency, partial stores) three workgroups per CU overlap better than two (bf16 decode).
  z->few_pages = work < 64 * wgs;
  const int32_t group = p->num_q_heads / p->num_kv_heads;
  int64_t chunks_ref = 0, prows = 0;
  for (int32_t s = 0; s < z->S; ++s)
    if (used[s]) chunks_ref += (npg_cap[s] + cap - 1) / cap;
  for (int64_t e = 0; e < z->E; ++e) {
    const int32_t s = bp->path_segs[e];
    prows += (npg_cap[s] + cap - 1) / cap;
  }
  z->prows = prows;   // partial rows are stored as int32 in the branch lists (checked by the caller)
  // items(s) = chunks(s) * ceil(|B(s)| g / 128) <= chunks(s) * (|B(s)| g / 128 + 1)
  z->max_items = chunks_ref + (prows * group + ga::kRowsPerBlock - 1) / ga::kRowsPerBlock;
  z->desc_words = ga::desc_words((int)cap, group);
  (void)st;
}

struct Layout {
  size_t off[48];
  size_t total;
};

// Device workspace layout (byte offsets of every array in the single allocation).
enum {
  L_SEG_LEN, L_SEG_PAGE_OFF, L_SEG_PAGES, L_PATH_OFF, L_PATH_SEGS, L_SEG_CAUSAL,  // uploaded
  L_SEG_CHAIN, L_SRC_OFF, L_SRC_PAGES, L_CH_SEG_OFF, L_CH_SEGS, L_BR_LAST, L_BR_COUNT,
  L_NEW_LEN,                                                                      // uploaded
  L_SEG_POS,
  L_GRP_CNT, L_GRP_FILL, L_GRP_OFF, L_GRP_TMP, L_GRP_BR, L_ENTRY_BR, L_ENTRY_RANK, L_SEG_NCH,
  L_SEG_ITEM_OFF, L_SEG_PROW_OFF, L_SEG_ORDER, L_ORDER_ITEM_OFF, L_ITEMS, L_DESC, L_COUNTERS, L_ENTRY_PART, L_BPART_OFF, L_BPART, L_BLK_SUM,
  L_PO, L_PLSE, L_COUNT
};
static_assert(L_COUNT <= 48, "Layout::off must hold every array");

Layout layout(const Sizes& z, const ga_params& p) {
  size_t sz[L_COUNT];
  sz[L_SEG_LEN] = sizeof(int32_t) * z.S;
  sz[L_SEG_PAGE_OFF] = sizeof(int64_t) * (z.S + 1);
  sz[L_SEG_PAGES] = sizeof(int32_t) * z.P;
  sz[L_PATH_OFF] = sizeof(int64_t) * (z.B + 1);
  sz[L_PATH_SEGS] = sizeof(int32_t) * z.E;
  sz[L_SEG_CAUSAL] = sizeof(int32_t) * z.S;
  sz[L_SEG_CHAIN] = sizeof(int32_t) * z.S0;
  sz[L_SRC_OFF] = z.S0 ? sizeof(int64_t) * (z.S0 + 1) : 0;
  sz[L_SRC_PAGES] = sizeof(int32_t) * z.P0;
  sz[L_CH_SEG_OFF] = z.S0 ? sizeof(int32_t) * (z.S + 1) : 0;
  sz[L_CH_SEGS] = sizeof(int32_t) * z.CS;
  sz[L_BR_LAST] = sizeof(int32_t) * z.B0q;
  sz[L_BR_COUNT] = sizeof(int32_t) * z.B0q;
  sz[L_NEW_LEN] = sizeof(int32_t) * z.S0;
  sz[L_SEG_POS] = sizeof(int32_t) * z.S0;
  sz[L_GRP_CNT] = sizeof(int32_t) * z.S;
  sz[L_GRP_FILL] = sizeof(int32_t) * z.S;
  sz[L_GRP_OFF] = sizeof(int64_t) * (z.S + 1);
  sz[L_GRP_TMP] = sizeof(int32_t) * z.E;
  sz[L_GRP_BR] = sizeof(int32_t) * z.E;
  sz[L_ENTRY_BR] = sizeof(int32_t) * z.E;
  sz[L_ENTRY_RANK] = sizeof(int32_t) * z.E;
  sz[L_SEG_NCH] = sizeof(int32_t) * z.S;
  sz[L_SEG_ITEM_OFF] = sizeof(int64_t) * (z.S + 1);
  sz[L_SEG_PROW_OFF] = sizeof(int64_t) * (z.S + 1);
  sz[L_SEG_ORDER] = sizeof(int32_t) * (z.S > 0 ? z.S : 1);
  sz[L_ORDER_ITEM_OFF] = sizeof(int64_t) * (z.S + 1);
  sz[L_ITEMS] = sizeof(int4) * (z.max_items > 0 ? z.max_items : 1);
  // (padded so that whole-slot copies of the last descriptor stay inside the allocation)
  sz[L_DESC] = sizeof(int32_t) * (size_t)z.desc_words * (z.max_items > 0 ? z.max_items : 1) +
               ga::kDescMaxBytes;
  sz[L_COUNTERS] = sizeof(int64_t) * ga::kNumCounters;
  sz[L_ENTRY_PART] = sizeof(int64_t) * z.E;
  sz[L_BPART_OFF] = sizeof(int64_t) * (z.B + 1);
  sz[L_BPART] = sizeof(int32_t) * z.prows;
  sz[L_BLK_SUM] = sizeof(int64_t) * ((z.E + 1023) / 1024 + 1);
  // Partials: fp16 values + (lambda, scale) for bf16 inputs, fp32 values + lambda for fp32.
  const bool f16_parts = p.dtype == GA_BF16;
  sz[L_PO] = (f16_parts ? 2 : 4) * (size_t)z.prows * p.num_q_heads * p.head_dim;
  sz[L_PLSE] = (f16_parts ? 8 : 4) * (size_t)z.prows * p.num_q_heads;
  Layout L{};
  size_t o = 0;
  for (int i = 0; i < L_COUNT; ++i) {
    // The uploaded graph arrays are packed back to back (8-byte aligned) so one copy moves them.
    o = align_up(o, i <= L_NEW_LEN ? 8 : 256);
    L.off[i] = o;
    o += sz[i];
  }
  L.total = align_up(o, 256);
  return L;
}

size_t upload_bytes(const Layout& L) { return L.off[L_SEG_POS]; }

void bind(ga_plan* pl, const Layout& L) {
  char* d = static_cast<char*>(pl->dev);
  const Sizes& z = pl->z;
  pl->g.S = z.S;
  pl->g.B = z.B;
  pl->g.E = z.E;
  pl->g.seg_len = reinterpret_cast<const int32_t*>(d + L.off[L_SEG_LEN]);
  pl->g.seg_page_off = reinterpret_cast<const int64_t*>(d + L.off[L_SEG_PAGE_OFF]);
  pl->g.seg_pages = reinterpret_cast<const int32_t*>(d + L.off[L_SEG_PAGES]);
  pl->g.path_off = reinterpret_cast<const int64_t*>(d + L.off[L_PATH_OFF]);
  pl->g.path_segs = reinterpret_cast<const int32_t*>(d + L.off[L_PATH_SEGS]);
  pl->g.seg_causal = reinterpret_cast<const int32_t*>(d + L.off[L_SEG_CAUSAL]);
  pl->sc.grp_cnt = reinterpret_cast<int32_t*>(d + L.off[L_GRP_CNT]);
  pl->sc.grp_fill = reinterpret_cast<int32_t*>(d + L.off[L_GRP_FILL]);
  pl->sc.grp_off = reinterpret_cast<int64_t*>(d + L.off[L_GRP_OFF]);
  pl->sc.grp_tmp = reinterpret_cast<int32_t*>(d + L.off[L_GRP_TMP]);
  pl->sc.grp_br = reinterpret_cast<int32_t*>(d + L.off[L_GRP_BR]);
  pl->sc.entry_branch = reinterpret_cast<int32_t*>(d + L.off[L_ENTRY_BR]);
  pl->sc.entry_rank = reinterpret_cast<int32_t*>(d + L.off[L_ENTRY_RANK]);
  pl->sc.seg_nchunk = reinterpret_cast<int32_t*>(d + L.off[L_SEG_NCH]);
  pl->sc.seg_item_off = reinterpret_cast<int64_t*>(d + L.off[L_SEG_ITEM_OFF]);
  pl->sc.seg_prow_off = reinterpret_cast<int64_t*>(d + L.off[L_SEG_PROW_OFF]);
  pl->sc.seg_order = reinterpret_cast<int32_t*>(d + L.off[L_SEG_ORDER]);
  pl->sc.order_item_off = reinterpret_cast<int64_t*>(d + L.off[L_ORDER_ITEM_OFF]);
  pl->sc.items = reinterpret_cast<int4*>(d + L.off[L_ITEMS]);
  pl->sc.desc = reinterpret_cast<int32_t*>(d + L.off[L_DESC]);
  pl->sc.desc_words = z.desc_words;
  pl->sc.counters = reinterpret_cast<int64_t*>(d + L.off[L_COUNTERS]);
  pl->sc.entry_part = reinterpret_cast<int64_t*>(d + L.off[L_ENTRY_PART]);
  pl->sc.bpart_off = reinterpret_cast<int64_t*>(d + L.off[L_BPART_OFF]);
  pl->sc.bpart = reinterpret_cast<int32_t*>(d + L.off[L_BPART]);
  pl->sc.blk_sum = reinterpret_cast<int64_t*>(d + L.off[L_BLK_SUM]);
  ga::LengthArgs& la = pl->la;
  la.chains = z.S;
  la.branches = z.B0q;
  la.new_len = reinterpret_cast<const int32_t*>(d + L.off[L_NEW_LEN]);
  la.src_page_off = reinterpret_cast<const int64_t*>(d + L.off[L_SRC_OFF]);
  la.src_pages = reinterpret_cast<const int32_t*>(d + L.off[L_SRC_PAGES]);
  la.chain_seg_off = reinterpret_cast<const int32_t*>(d + L.off[L_CH_SEG_OFF]);
  la.chain_segs = reinterpret_cast<const int32_t*>(d + L.off[L_CH_SEGS]);
  la.seg_chain = reinterpret_cast<const int32_t*>(d + L.off[L_SEG_CHAIN]);
  la.br_last = reinterpret_cast<const int32_t*>(d + L.off[L_BR_LAST]);
  la.br_count = reinterpret_cast<const int32_t*>(d + L.off[L_BR_COUNT]);
  la.seg_pos = reinterpret_cast<int32_t*>(d + L.off[L_SEG_POS]);
  la.chain_len = reinterpret_cast<int32_t*>(d + L.off[L_SEG_LEN]);
  la.chain_page_off = reinterpret_cast<const int64_t*>(d + L.off[L_SEG_PAGE_OFF]);
  la.chain_pages = reinterpret_cast<int32_t*>(d + L.off[L_SEG_PAGES]);
  la.chain_causal = reinterpret_cast<int32_t*>(d + L.off[L_SEG_CAUSAL]);
  pl->len_off = L.off[L_NEW_LEN];
  pl->po = d + L.off[L_PO];
  pl->plse = reinterpret_cast<float*>(d + L.off[L_PLSE]);
}

void pack_upload(const ga_segment_table* st, const ga_branch_paths* bp, const int32_t* causal,
                 const Layout& L, const Sizes& z, char* h) {
  if (z.S) std::memcpy(h + L.off[L_SEG_LEN], st->seg_len, sizeof(int32_t) * z.S);
  std::memcpy(h + L.off[L_SEG_PAGE_OFF], st->seg_page_offsets, sizeof(int64_t) * (z.S + 1));
  if (z.P) std::memcpy(h + L.off[L_SEG_PAGES], st->seg_pages, sizeof(int32_t) * z.P);
  std::memcpy(h + L.off[L_PATH_OFF], bp->path_offsets, sizeof(int64_t) * (z.B + 1));
  if (z.E) std::memcpy(h + L.off[L_PATH_SEGS], bp->path_segs, sizeof(int32_t) * z.E);
  if (z.S) std::memcpy(h + L.off[L_SEG_CAUSAL], causal, sizeof(int32_t) * z.S);
}

// Workspace of graphattn_decode_static: a static device array, so that the call allocates no
// device or pinned memory.  Every call on one device uses that device's copy; calls are ordered
// through the events below (and serialised on the host by the lock), so a later call reuses
// the array only after the earlier one's kernels are done with it.  Nothing in it has to start
// at zero: the scheduler clears its counters, and every other array is written before it is
// read.  The graph upload is staged in pageable host memory.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
constexpr int kStaticDevices = 16;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
struct StaticScratch {
  std::mutex mu;
  void* dev = nullptr;            // the array's device address (hipGetSymbolAddress)
  std::vector<char> stage;        // host staging of the graph upload
  hipEvent_t done = nullptr;      // recorded after the last call's kernels
  hipEvent_t uploaded = nullptr;  // recorded after the last call's upload
};
StaticScratch g_static[kStaticDevices];

// Process-wide workspace reused by graphattn_decode.
struct DecodeCache {
  std::mutex mu;
  void* dev = nullptr;
  size_t dev_bytes = 0;
  void* pin = nullptr;
  size_t pin_bytes = 0;
  int device = -1;
  hipEvent_t done = nullptr;      // recorded after the last decode's kernels
  hipEvent_t uploaded = nullptr;  // recorded after the last decode's upload
};
DecodeCache g_cache;

// Multi-query plans: query row i of branch b becomes a branch of its own with b's path (the rows
// of one branch are consecutive, in query order), so every segment a branch shares is attended
// once for all of the rows that share it.  b's newest segment (its path's last entry) is on no
// other path, so its group is exactly b's rows and a row's rank there is its query index i; the
// causal limit inside that segment is a per-rank token bound (DevGraph::seg_causal).
ga_status expand_queries(const ga_segment_table* st, const ga_branch_paths* bp,
                         const int32_t* counts, std::vector<int64_t>* vpo,
                         std::vector<int32_t>* vps) {
  const int32_t S = st->num_segments, B = bp->num_branches;
  if (B > 0 && !counts) return fail(GA_EINVAL, "query_counts is NULL");
  std::vector<int32_t> occ(S, 0);
  for (int64_t e = 0; e < bp->path_offsets[B]; ++e) ++occ[bp->path_segs[e]];
  int64_t rows = 0, entries = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int64_t a = bp->path_offsets[b], e1 = bp->path_offsets[b + 1];
    const int32_t last = bp->path_segs[e1 - 1];
    if (occ[last] != 1)
      return fail(GA_EINVAL, "query segment %d of branch %d is on another path", last, b);
    if (counts[b] < 1 || counts[b] > st->seg_len[last])
      return fail(GA_EINVAL, "branch %d: query count %d outside [1, %d]", b, counts[b],
                  st->seg_len[last]);
    rows += counts[b];
    entries += (int64_t)counts[b] * (e1 - a);
  }
  if (rows > 0x7fffffffLL || entries > 0x7fffffffLL)
    return fail(GA_EINVAL, "too many query rows (%lld) or row path entries (%lld)",
                (long long)rows, (long long)entries);
  vpo->assign(1, 0);
  vpo->reserve(rows + 1);
  vps->clear();
  vps->reserve(entries);
  for (int32_t b = 0; b < B; ++b)
    for (int32_t i = 0; i < counts[b]; ++i) {
      vps->insert(vps->end(), bp->path_segs + bp->path_offsets[b],
                  bp->path_segs + bp->path_offsets[b + 1]);
      vpo->push_back((int64_t)vps->size());
    }
  return GA_OK;
}

// Multi-query plans: the newest segment of branch b closes its chain (it is the last entry of
// every path through it) and starts on a page of its own, so its token t is chain token
// 16 x (chain pages before it) + t, and query i sits at t = len - n_b + i.
ga_status set_causal(const ga_plan* pl, const int32_t* seg_len, const std::vector<int32_t>& npg,
                     CGraph* c) {
  for (size_t b = 0; b < pl->h_last.size(); ++b) {
    const int32_t last = pl->h_last[b];
    const int32_t v = c->vid[last];
    if (c->seg_len[v] >= ga::kNoCausal)
      return fail(GA_EUNSUPPORTED, "segment chain of branch %d spans %d tokens", (int)b,
                  c->seg_len[v]);
    c->causal[v] = (c->npg[v] - npg[last]) * ga::kPageTokens + seg_len[last] - pl->h_counts[b];
  }
  return GA_OK;
}

ga_status plan_init(const ga_segment_table* st, const ga_branch_paths* bp, const ga_params* p,
                    const int32_t* query_counts, bool updatable, ga_plan* pl, Layout* L) {
  ga_status rc = validate_params(p);
  if (rc) return rc;
  std::vector<int32_t> npg;
  rc = validate_graph(st, bp, p, &pl->z, &npg);
  if (rc) return rc;
  pl->B0 = bp->num_branches;
  std::vector<int64_t> vpo;
  std::vector<int32_t> vps;
  ga_branch_paths vbp{};
  if (query_counts) {
    rc = expand_queries(st, bp, query_counts, &vpo, &vps);
    if (rc) return rc;
    vbp = ga_branch_paths{(int32_t)(vpo.size() - 1), vpo.data(), vps.data()};
    rc = validate_graph(st, &vbp, p, &pl->z, &npg);
    if (rc) return rc;
    pl->causal = true;
  }
  const ga_branch_paths* ebp = query_counts ? &vbp : bp;
  rc = compress_chains(st, ebp, npg, &pl->cg);
  if (rc) return rc;
  // Kept for length updates.
  const int32_t S0 = st->num_segments;
  pl->updatable = updatable;
  if (updatable) {
    pl->h_page_off.assign(st->seg_page_offsets, st->seg_page_offsets + S0 + 1);
    pl->h_pages.assign(st->seg_pages, st->seg_pages + st->seg_page_offsets[S0]);
  }
  if (query_counts) {
    pl->h_last.resize(bp->num_branches);
    for (int32_t b = 0; b < bp->num_branches; ++b)
      pl->h_last[b] = bp->path_segs[bp->path_offsets[b + 1] - 1];
    pl->h_counts.assign(query_counts, query_counts + bp->num_branches);
    rc = set_causal(pl, st->seg_len, npg, &pl->cg);
    if (rc) return rc;
  }
  const CGraph& c = pl->cg;
  pl->z.S = (int32_t)c.head.size();
  pl->z.E = (int32_t)c.path_segs.size();
  pl->z.P = (int64_t)c.seg_pages.size();
  const ga_segment_table cst{pl->z.S, c.seg_len.data(), c.seg_page_off.data(), c.seg_pages.data()};
  const ga_branch_paths cbp{pl->z.B, c.path_off.data(), c.path_segs.data()};
  pl->p = *p;
  if (pl->p.softmax_scale == 0.f) pl->p.softmax_scale = 1.f / std::sqrt((float)p->head_dim);
  pl->num_cus = device_cus();
  std::vector<int64_t> npg_cap(pl->z.S);          // pages each chain owns
  for (int32_t v = 0; v < pl->z.S; ++v) npg_cap[v] = c.seg_page_off[v + 1] - c.seg_page_off[v];
  if (updatable) {
    pl->z.S0 = S0;
    pl->z.P0 = st->seg_page_offsets[S0];
    pl->z.CS = (int32_t)c.chain_segs.size();
    pl->z.B0q = query_counts ? bp->num_branches : 0;
  }
  size_schedule(&cst, &cbp, p, c.npg, npg_cap, pl->num_cus, &pl->z);
  if (pl->z.prows > 0x7fffffffLL)
    return fail(GA_EINVAL, "too many partial rows (%lld)", (long long)pl->z.prows);
  if (pl->z.P > 0x7fffffffLL)
    return fail(GA_EINVAL, "too many page-table entries (%lld)", (long long)pl->z.P);
  // Work units (item x kv-head) are claimed through a 32-bit counter that may overshoot by a
  // few claims per workgroup.
  if (pl->z.max_items * p->num_kv_heads > (1LL << 30))
    return fail(GA_EINVAL, "too many work units (%lld)",
                (long long)(pl->z.max_items * p->num_kv_heads));
  *L = layout(pl->z, pl->p);
  return GA_OK;
}

ga_status upload(ga_plan* pl, const Layout& L, hipStream_t stream) {
  const CGraph& c = pl->cg;
  const ga_segment_table cst{pl->z.S, c.seg_len.data(), c.seg_page_off.data(), c.seg_pages.data()};
  const ga_branch_paths cbp{pl->z.B, c.path_off.data(), c.path_segs.data()};
  char* h = static_cast<char*>(pl->pin);
  pack_upload(&cst, &cbp, c.causal.data(), L, pl->z, h);
  const Sizes& z = pl->z;
  if (z.S0) {
    std::memcpy(h + L.off[L_SEG_CHAIN], c.vid.data(), sizeof(int32_t) * z.S0);
    std::memcpy(h + L.off[L_SRC_OFF], pl->h_page_off.data(), sizeof(int64_t) * (z.S0 + 1));
    if (z.P0) std::memcpy(h + L.off[L_SRC_PAGES], pl->h_pages.data(), sizeof(int32_t) * z.P0);
    std::memcpy(h + L.off[L_CH_SEG_OFF], c.chain_seg_off.data(), sizeof(int32_t) * (z.S + 1));
    if (z.CS) std::memcpy(h + L.off[L_CH_SEGS], c.chain_segs.data(), sizeof(int32_t) * z.CS);
    if (z.B0q) {
      std::memcpy(h + L.off[L_BR_LAST], pl->h_last.data(), sizeof(int32_t) * z.B0q);
      std::memcpy(h + L.off[L_BR_COUNT], pl->h_counts.data(), sizeof(int32_t) * z.B0q);
    }
  }
  pl->h_pages.clear();
  pl->h_pages.shrink_to_fit();
  GA_HIP(hipMemcpyAsync(pl->dev, pl->pin, upload_bytes(L), hipMemcpyHostToDevice, stream),
         "graph upload");
  if (pl->uploaded) GA_HIP(hipEventRecord(pl->uploaded, stream), "record upload");
  return GA_OK;
}

ga_status check_run_ptrs(const ga_plan* pl, const void* q, const void* pool, const void* out,
                         const float* lse) {
  if (pl->z.B == 0) return GA_OK;
  if (!q || !pool || !out || !lse) return fail(GA_EINVAL, "q, kv_page_pool, out and lse must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(pool) |
       reinterpret_cast<uintptr_t>(out)) & 15)
    return fail(GA_EINVAL, "q, kv_page_pool and out must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(lse) & 3) return fail(GA_EINVAL, "lse must be 4-byte aligned");
  return GA_OK;
}

ga_status do_schedule(ga_plan* pl, hipStream_t stream) {
  const bool rec = pl->prof_sched < pl->prof_cap;
  if (rec) GA_HIP(hipEventRecord(pl->ev_sched[2 * pl->prof_sched], stream), "profile event");
  if (pl->z.B > 0 || pl->z.S > 0) {
    // The groups (B(s), their order, the entry ranks) follow the paths alone, which a plan never
    // changes, so after the first schedule only what the lengths decide is recomputed.
    const bool reuse = pl->grouped;
    pl->grouped = false;
    GA_HIP(ga::launch_schedule(pl->g, pl->sc, pl->p.num_q_heads / pl->p.num_kv_heads,
                               pl->z.chunk_pages, pl->z.max_items, reuse, stream),
           "scheduler launch");
    pl->grouped = true;
  }
  if (rec) {
    hipEvent_t e = pl->ev_sched[2 * pl->prof_sched + 1];
    GA_HIP(hipEventRecord(e, stream), "profile event");
    pl->ev_last = e;
    ++pl->prof_sched;
  }
  pl->scheduled = true;
  return GA_OK;
}

ga_status do_run(ga_plan* pl, const void* q, const void* pool, void* out, float* lse,
                 hipStream_t stream) {
  ga_status rc = check_run_ptrs(pl, q, pool, out, lse);
  if (rc) return rc;
  // A plan without a current schedule (new, or given new lengths) is scheduled first.
  if (!pl->scheduled) {
    rc = do_schedule(pl, stream);
    if (rc) return rc;
  }
  if (pl->z.B == 0) return GA_OK;
  // The merge re-arms the attention kernel's work-stream heads; a schedule clears them as
  // well.  If a launch below fails, the plan loses its schedule, so the next run schedules (and
  // so re-arms the heads) before it attends.
  pl->scheduled = false;
  const bool bf16 = pl->p.dtype == GA_BF16;
  ga::AttnArgs a{};
  a.q = q;
  a.pool = pool;
  a.desc = pl->sc.desc;
  a.counters = pl->sc.counters;
  a.po = pl->po;
  a.plse = pl->plse;
  a.Hq = pl->p.num_q_heads;
  a.Hkv = pl->p.num_kv_heads;
  a.group = a.Hq / a.Hkv;
  a.chunk_pages = pl->z.chunk_pages;
  a.desc_words = pl->z.desc_words;
  a.streams = ga::attn_streams(a.Hkv, pl->causal);
  a.scale_log2 = pl->p.softmax_scale * 1.4426950408889634f;
  int64_t grid = (int64_t)ga::seg_attn_grid(pl->p.head_dim, bf16, pl->causal, pl->z.few_pages,
                                            pl->num_cus);
  const int64_t work = pl->z.max_items * pl->p.num_kv_heads;
  if (work < grid) grid = work;
  // Profiled runs bind their events to the attention and merge dispatches themselves (a kernel
  // with no work gets a plain event pair instead).
  const bool rec = pl->prof_runs < pl->prof_cap;
  hipEvent_t* ev = rec ? &pl->ev_run[4 * pl->prof_runs] : nullptr;
  if (grid > 0)
    GA_HIP(ga::launch_seg_attn(a, pl->p.head_dim, bf16, pl->causal, pl->z.few_pages, (int)grid,
                               stream, rec ? ev[0] : nullptr, rec ? ev[1] : nullptr),
           "attention launch");
  else if (rec) {
    GA_HIP(hipEventRecord(ev[0], stream), "profile event");
    GA_HIP(hipEventRecord(ev[1], stream), "profile event");
  }
  ga::MergeArgs m{};
  m.bpart_off = pl->sc.bpart_off;
  m.bpart = pl->sc.bpart;
  m.po = pl->po;
  m.plse = pl->plse;
  m.out = out;
  m.lse = lse;
  m.counters = pl->sc.counters;
  m.B = pl->z.B;
  m.Hq = pl->p.num_q_heads;
  const bool merge_rows = (int64_t)m.B * m.Hq > 0;
  GA_HIP(ga::launch_merge(m, pl->p.head_dim, bf16 && !pl->p.out_f32, bf16, stream,
                          rec && merge_rows ? ev[2] : nullptr,
                          rec && merge_rows ? ev[3] : nullptr),
         "merge launch");
  pl->scheduled = true;
  if (rec) {
    if (!merge_rows) {
      GA_HIP(hipEventRecord(ev[2], stream), "profile event");
      GA_HIP(hipEventRecord(ev[3], stream), "profile event");
    }
    pl->ev_last = ev[3];
    ++pl->prof_runs;
  }
  return GA_OK;
}

void profile_clear(ga_plan* pl) {
  for (hipEvent_t e : pl->ev_sched) (void)hipEventDestroy(e);
  for (hipEvent_t e : pl->ev_run) (void)hipEventDestroy(e);
  pl->ev_sched.clear();
  pl->ev_run.clear();
  pl->prof_cap = pl->prof_sched = pl->prof_runs = 0;
  pl->ev_last = nullptr;
}

}  // namespace

extern "C" {

const char* graphattn_last_error(void) { return g_err.c_str(); }

static ga_status plan_create(const ga_segment_table* segment_table,
                             const ga_branch_paths* branch_paths, const int32_t* query_counts,
                             const ga_params* params, void* hip_stream, ga_plan** plan) {
  g_err.clear();
  if (!plan) return fail(GA_EINVAL, "plan out-pointer is NULL");
  *plan = nullptr;
  ga_plan* pl = new ga_plan();
  Layout L;
  ga_status rc = plan_init(segment_table, branch_paths, params, query_counts, true, pl, &L);
  if (rc) {
    delete pl;
    return rc;
  }
  pl->dev_bytes = L.total;
  pl->pin_bytes = upload_bytes(L);
  if (hipMalloc(&pl->dev, pl->dev_bytes) != hipSuccess) {
    delete pl;
    (void)hipGetLastError();
    return fail(GA_ENOMEM, "device workspace of %zu bytes", L.total);
  }
  if (hipHostMalloc(&pl->pin, pl->pin_bytes > 0 ? pl->pin_bytes : 1) != hipSuccess) {
    (void)hipFree(pl->dev);
    delete pl;
    (void)hipGetLastError();
    return fail(GA_ENOMEM, "pinned staging of %zu bytes", pl->pin_bytes);
  }
  bind(pl, L);
  if (hipEventCreateWithFlags(&pl->uploaded, hipEventDisableTiming) != hipSuccess) {
    pl->uploaded = nullptr;
    graphattn_plan_destroy(pl);
    return hip_fail(hipGetLastError(), "event");
  }
  if (pl->z.S0 > 0) {
    if (hipHostMalloc(reinterpret_cast<void**>(&pl->len_pin),
                      sizeof(int32_t) * pl->z.S0 * ga_plan::kLenSlots) != hipSuccess) {
      pl->len_pin = nullptr;
      graphattn_plan_destroy(pl);
      (void)hipGetLastError();
      return fail(GA_ENOMEM, "pinned staging of the segment lengths");
    }
    for (hipEvent_t& e : pl->len_ev)
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
        e = nullptr;
        graphattn_plan_destroy(pl);
        return hip_fail(hipGetLastError(), "event");
      }
  }
  rc = upload(pl, L, static_cast<hipStream_t>(hip_stream));
  if (rc) {
    graphattn_plan_destroy(pl);
    return rc;
  }
  *plan = pl;
  return GA_OK;
}

ga_status graphattn_plan_create(const ga_segment_table* segment_table,
                                const ga_branch_paths* branch_paths, const ga_params* params,
                                void* hip_stream, ga_plan** plan) {
  return plan_create(segment_table, branch_paths, nullptr, params, hip_stream, plan);
}

ga_status graphattn_plan_create_extend(const ga_segment_table* segment_table,
                                       const ga_branch_paths* branch_paths,
                                       const int32_t* query_counts, const ga_params* params,
                                       void* hip_stream, ga_plan** plan) {
  if (!query_counts && branch_paths && branch_paths->num_branches > 0) {
    g_err.clear();
    if (plan) *plan = nullptr;
    return fail(GA_EINVAL, "query_counts is NULL");
  }
  static const int32_t none = 0;
  return plan_create(segment_table, branch_paths, query_counts ? query_counts : &none, params,
                     hip_stream, plan);
}

ga_status graphattn_plan_set_lengths(ga_plan* plan, const int32_t* seg_len, void* hip_stream) {
  g_err.clear();
  if (!plan) return fail(GA_EINVAL, "plan is NULL");
  if (!plan->updatable) return fail(GA_EINVAL, "plan does not take new lengths");
  const int32_t S = plan->cg.S0;
  if (S > 0 && !seg_len) return fail(GA_EINVAL, "seg_len is NULL");
  for (int32_t s = 0; s < S; ++s) {
    const int32_t len = seg_len[s];
    if (len < 1) return fail(GA_EINVAL, "segment %d has length %d (< 1)", s, len);
    const int64_t owned = plan->h_page_off[s + 1] - plan->h_page_off[s];
    const int64_t need = (len + ga::kPageTokens - 1) / ga::kPageTokens;
    if (need > owned)
      return fail(GA_EINVAL, "segment %d has %d tokens but owns only %lld pages", s, len,
                  (long long)owned);
  }
  for (size_t b = 0; b < plan->h_last.size(); ++b)
    if (plan->h_counts[b] > seg_len[plan->h_last[b]])
      return fail(GA_EINVAL, "branch %d: query count %d exceeds its newest segment's %d tokens",
                  (int)b, plan->h_counts[b], seg_len[plan->h_last[b]]);
  if (S == 0) {
    plan->scheduled = false;
    return GA_OK;
  }
  // The chains (which segments go together) follow the paths only, and each chain's page list
  // has room for every page its segments own: the device rebuilds the page lists, valid token
  // counts, chain lengths and causal origins from the new lengths in place.  The lengths go
  // through a ring of pinned slots; the host waits only if the slot's copy from kLenSlots
  // updates ago has not left it yet.
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  const int slot = (int)(plan->len_calls % ga_plan::kLenSlots);
  if (plan->len_calls >= ga_plan::kLenSlots)
    GA_HIP(hipEventSynchronize(plan->len_ev[slot]), "wait for an earlier length upload");
  int32_t* h = plan->len_pin + (size_t)slot * S;
  std::memcpy(h, seg_len, sizeof(int32_t) * S);
  GA_HIP(hipMemcpyAsync(static_cast<char*>(plan->dev) + plan->len_off, h, sizeof(int32_t) * S,
                        hipMemcpyHostToDevice, stream), "length upload");
  GA_HIP(hipEventRecord(plan->len_ev[slot], stream), "record length upload");
  ++plan->len_calls;
  // (if the launch fails, the chains and the schedule stay those of the previous lengths)
  GA_HIP(ga::launch_set_lengths(plan->la, stream), "length update launch");
  plan->scheduled = false;
  return GA_OK;
}

ga_status graphattn_schedule(ga_plan* plan, void* hip_stream) {
  g_err.clear();
  if (!plan) return fail(GA_EINVAL, "plan is NULL");
  return do_schedule(plan, static_cast<hipStream_t>(hip_stream));
}

ga_status graphattn_run(ga_plan* plan, const void* q, const void* kv_page_pool, void* out,
                        float* lse, void* hip_stream) {
  g_err.clear();
  if (!plan) return fail(GA_EINVAL, "plan is NULL");
  return do_run(plan, q, kv_page_pool, out, lse, static_cast<hipStream_t>(hip_stream));
}

ga_status graphattn_plan_info(const ga_plan* plan, ga_plan_info* info) {
  g_err.clear();
  if (!plan || !info) return fail(GA_EINVAL, "plan or info is NULL");
  info->num_segments = plan->cg.S0;
  info->num_branches = plan->B0;
  info->num_query_rows = plan->z.B;
  info->num_entries = (int32_t)plan->cg.E0;
  info->num_chains = plan->z.S;
  info->chunk_pages = plan->z.chunk_pages;
  info->rows_per_block = ga::kRowsPerBlock;
  info->num_items = -1;
  info->num_partial_rows = plan->z.prows;
  info->workgroups_per_cu = ga::seg_attn_grid(plan->p.head_dim, plan->p.dtype == GA_BF16,
                                              plan->causal, plan->z.few_pages, 1);
  info->work_streams = ga::attn_streams(plan->p.num_kv_heads, plan->causal);
  if (plan->scheduled) {
    int64_t n = 0;
    if (hipMemcpy(&n, plan->sc.counters, sizeof n, hipMemcpyDeviceToHost) == hipSuccess)
      info->num_items = n;
  }
  return GA_OK;
}

ga_status graphattn_plan_debug_dump(const ga_plan* plan, void* hip_stream,
                                    int64_t* group_offsets, int32_t* group_branches,
                                    int32_t* entry_ranks, int32_t* items,
                                    int32_t* segment_chunks, int64_t* branch_part_offsets,
                                    int32_t* branch_parts) {
  g_err.clear();
  if (!plan) return fail(GA_EINVAL, "plan is NULL");
  if (!plan->scheduled) return fail(GA_EINVAL, "plan has no schedule");
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  GA_HIP(hipStreamSynchronize(s), "synchronise");
  const Sizes& z = plan->z;
  const CGraph& c = plan->cg;
  // The schedule is over chains; groups, ranks and chunk counts are reported per given segment
  // and path entry (a segment's group is its chain's).
  std::vector<int64_t> vgoff(z.S + 1);
  std::vector<int32_t> vgbr(z.E), vrank(z.E), vnch(z.S);
  GA_HIP(hipMemcpy(vgoff.data(), plan->sc.grp_off, sizeof(int64_t) * (z.S + 1),
                   hipMemcpyDeviceToHost), "dump group offsets");
  if (z.E) {
    GA_HIP(hipMemcpy(vgbr.data(), plan->sc.grp_br, sizeof(int32_t) * z.E, hipMemcpyDeviceToHost),
           "dump groups");
    GA_HIP(hipMemcpy(vrank.data(), plan->sc.entry_rank, sizeof(int32_t) * z.E,
                     hipMemcpyDeviceToHost), "dump ranks");
  }
  if (z.S)
    GA_HIP(hipMemcpy(vnch.data(), plan->sc.seg_nchunk, sizeof(int32_t) * z.S,
                     hipMemcpyDeviceToHost), "dump chunks");
  int64_t off = 0;
  for (int32_t sg = 0; sg < c.S0; ++sg) {
    const int32_t v = c.vid[sg];
    const int64_t n = v >= 0 ? vgoff[v + 1] - vgoff[v] : 0;
    if (group_offsets) group_offsets[sg] = off;
    if (group_branches)
      for (int64_t k = 0; k < n; ++k) group_branches[off + k] = vgbr[vgoff[v] + k];
    if (segment_chunks) segment_chunks[sg] = c.first[sg] ? vnch[v] : 0;
    off += n;
  }
  if (group_offsets) group_offsets[c.S0] = off;
  if (entry_ranks)
    for (int64_t e = 0; e < c.E0; ++e) entry_ranks[e] = vrank[c.ventry[e]];
  if (branch_part_offsets || branch_parts) {
    // Each branch's partial rows (per q-head) as the merge folds them: path order, then chunk
    // order.  The schedule's branches are the dumped ones (query rows for multi-query plans).
    std::vector<int64_t> boff(z.B + 1);
    GA_HIP(hipMemcpy(boff.data(), plan->sc.bpart_off, sizeof(int64_t) * (z.B + 1),
                     hipMemcpyDeviceToHost), "dump partial offsets");
    if (boff[z.B] > z.prows)
      return fail(GA_EINVAL, "schedule overflow (%lld partial rows)", (long long)boff[z.B]);
    if (branch_part_offsets) std::memcpy(branch_part_offsets, boff.data(), sizeof(int64_t) * (z.B + 1));
    if (branch_parts && boff[z.B] > 0)
      GA_HIP(hipMemcpy(branch_parts, plan->sc.bpart, sizeof(int32_t) * boff[z.B],
                       hipMemcpyDeviceToHost), "dump partial rows");
  }
  if (items) {
    int64_t n = 0;
    GA_HIP(hipMemcpy(&n, plan->sc.counters, sizeof n, hipMemcpyDeviceToHost), "dump count");
    if (n > z.max_items) return fail(GA_EINVAL, "schedule overflow (%lld items)", (long long)n);
    std::vector<int4> tmp(n);
    if (n)
      GA_HIP(hipMemcpy(tmp.data(), plan->sc.items, sizeof(int4) * n, hipMemcpyDeviceToHost),
             "dump items");
    for (int64_t i = 0; i < n; ++i) {
      items[3 * i] = c.head[tmp[i].x];
      items[3 * i + 1] = tmp[i].y;
      items[3 * i + 2] = tmp[i].z;
    }
  }
  return GA_OK;
}

ga_status graphattn_plan_profile(ga_plan* plan, int32_t max_calls) {
  g_err.clear();
  if (!plan) return fail(GA_EINVAL, "plan is NULL");
  if (max_calls < 0) return fail(GA_EINVAL, "max_calls is negative");
  if (plan->ev_last) GA_HIP(hipEventSynchronize(plan->ev_last), "profile sync");
  profile_clear(plan);
  plan->ev_sched.resize(2 * (size_t)max_calls);
  plan->ev_run.resize(4 * (size_t)max_calls);
  for (auto* v : {&plan->ev_sched, &plan->ev_run})
    for (hipEvent_t& e : *v)
      if (hipEventCreate(&e) != hipSuccess) {
        e = nullptr;
        profile_clear(plan);
        return fail(GA_EHIP, "profile event creation failed");
      }
  plan->prof_cap = max_calls;
  return GA_OK;
}

ga_status graphattn_plan_profile_read(ga_plan* plan, ga_profile* out) {
  g_err.clear();
  if (!plan || !out) return fail(GA_EINVAL, "plan or out is NULL");
  *out = ga_profile{};
  if (plan->ev_last) GA_HIP(hipEventSynchronize(plan->ev_last), "profile sync");
  for (int32_t i = 0; i < plan->prof_sched; ++i) {
    float ms = 0.f;
    GA_HIP(hipEventElapsedTime(&ms, plan->ev_sched[2 * i], plan->ev_sched[2 * i + 1]), "elapsed");
    out->sched_ms += ms;
  }
  for (int32_t i = 0; i < plan->prof_runs; ++i) {
    float a = 0.f, m = 0.f;
    GA_HIP(hipEventElapsedTime(&a, plan->ev_run[4 * i], plan->ev_run[4 * i + 1]), "elapsed");
    GA_HIP(hipEventElapsedTime(&m, plan->ev_run[4 * i + 2], plan->ev_run[4 * i + 3]), "elapsed");
    out->attn_ms += a;
    out->merge_ms += m;
  }
  out->schedules = plan->prof_sched;
  out->runs = plan->prof_runs;
  return GA_OK;
}

void graphattn_plan_destroy(ga_plan* plan) {
  if (!plan) return;
  profile_clear(plan);
  if (plan->uploaded) (void)hipEventDestroy(plan->uploaded);
  for (hipEvent_t e : plan->len_ev)
    if (e) (void)hipEventDestroy(e);
  if (plan->owns_memory) {
    if (plan->dev) {
      (void)hipDeviceSynchronize();
      (void)hipFree(plan->dev);
    }
    if (plan->pin) (void)hipHostFree(plan->pin);
    if (plan->len_pin) (void)hipHostFree(plan->len_pin);
  }
  delete plan;
}

static ga_status one_shot(const void* q, const void* kv_page_pool,
                          const ga_segment_table* segment_table,
                          const ga_branch_paths* branch_paths, const int32_t* query_counts,
                          void* out, float* lse, const ga_params* params, void* hip_stream) {
  g_err.clear();
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  ga_plan pl;
  Layout L;
  ga_status rc = plan_init(segment_table, branch_paths, params, query_counts, false, &pl, &L);
  if (rc) return rc;
  rc = check_run_ptrs(&pl, q, kv_page_pool, out, lse);
  if (rc) return rc;
  pl.scheduled = false;
  pl.owns_memory = false;
  std::lock_guard<std::mutex> lock(g_cache.mu);
  int dev = 0;
  GA_HIP(hipGetDevice(&dev), "current device");
  if (g_cache.device != dev) {
    // A new device: drop the old cache (its buffers belong to the previous device).
    g_cache.dev = nullptr;
    g_cache.pin = nullptr;
    g_cache.dev_bytes = g_cache.pin_bytes = 0;
    g_cache.done = g_cache.uploaded = nullptr;
    g_cache.device = dev;
  }
  if (!g_cache.done) {
    GA_HIP(hipEventCreateWithFlags(&g_cache.done, hipEventDisableTiming), "event");
    GA_HIP(hipEventCreateWithFlags(&g_cache.uploaded, hipEventDisableTiming), "event");
  }
  // The previous call's upload must have left the staging buffer before it is refilled, and its
  // kernels must be done with the device workspace before this stream reuses it.
  GA_HIP(hipEventSynchronize(g_cache.uploaded), "wait for previous upload");
  if (g_cache.dev_bytes < L.total) {
    GA_HIP(hipEventSynchronize(g_cache.done), "wait for previous decode");
    if (g_cache.dev) (void)hipFree(g_cache.dev);
    g_cache.dev = nullptr;
    g_cache.dev_bytes = 0;
    if (hipMalloc(&g_cache.dev, L.total) != hipSuccess) {
      (void)hipGetLastError();
      return fail(GA_ENOMEM, "device workspace of %zu bytes", L.total);
    }
    g_cache.dev_bytes = L.total;
  }
  const size_t ub = upload_bytes(L);
  if (g_cache.pin_bytes < ub || !g_cache.pin) {
    if (g_cache.pin) (void)hipHostFree(g_cache.pin);
    g_cache.pin = nullptr;
    g_cache.pin_bytes = 0;
    if (hipHostMalloc(&g_cache.pin, ub > 0 ? ub : 1) != hipSuccess) {
      (void)hipGetLastError();
      return fail(GA_ENOMEM, "pinned staging of %zu bytes", ub);
    }
    g_cache.pin_bytes = ub;
  }
  pl.dev = g_cache.dev;
  pl.pin = g_cache.pin;
  bind(&pl, L);
  GA_HIP(hipStreamWaitEvent(stream, g_cache.done, 0), "order after previous decode");
  rc = upload(&pl, L, stream);
  if (rc) return rc;
  GA_HIP(hipEventRecord(g_cache.uploaded, stream), "record upload");
  rc = do_schedule(&pl, stream);
  if (rc) return rc;
  rc = do_run(&pl, q, kv_page_pool, out, lse, stream);
  if (rc) return rc;
  GA_HIP(hipEventRecord(g_cache.done, stream), "record decode");
  return GA_OK;
}

ga_status graphattn_decode(const void* q, const void* kv_page_pool,
                           const ga_segment_table* segment_table,
                           const ga_branch_paths* branch_paths, void* out, float* lse,
                           const ga_params* params, void* hip_stream) {
  return one_shot(q, kv_page_pool, segment_table, branch_paths, nullptr, out, lse, params,
                  hip_stream);
}

ga_status graphattn_decode_static(const void* q, const void* kv_page_pool,
                                  const ga_segment_table* segment_table,
                                  const ga_branch_paths* branch_paths, void* out, float* lse,
                                  const ga_params* params, void* hip_stream) {
  g_err.clear();
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  ga_plan pl;
  Layout L;
  ga_status rc = plan_init(segment_table, branch_paths, params, nullptr, false, &pl, &L);
  if (rc) return rc;
  rc = check_run_ptrs(&pl, q, kv_page_pool, out, lse);
  if (rc) return rc;
  if (L.total > kStaticScratchBytes)
    return fail(GA_ENOMEM, "workspace of %zu bytes exceeds the static scratch of %zu bytes",
                L.total, (size_t)kStaticScratchBytes);
  pl.scheduled = false;
  pl.owns_memory = false;
  int dev = 0;
  GA_HIP(hipGetDevice(&dev), "current device");
  if (dev < 0 || dev >= kStaticDevices)
    return fail(GA_EUNSUPPORTED, "device %d beyond the %d the static scratch serves", dev,
                kStaticDevices);
  StaticScratch& st = g_static[dev];
  std::lock_guard<std::mutex> lock(st.mu);
  if (!st.dev) {
    // Once per device, with the device current: the array's address on this device.  The host
    // name of the array is not a device address; only this pointer is passed on.
    void* ptr = nullptr;
    GA_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "scratch address");
    GA_HIP(hipEventCreateWithFlags(&st.done, hipEventDisableTiming), "event");
    GA_HIP(hipEventCreateWithFlags(&st.uploaded, hipEventDisableTiming), "event");
    st.dev = ptr;
  }
  // The previous call's upload must have left the staging buffer, and its kernels must be done
  // with the scratch before this stream reuses it.
  GA_HIP(hipEventSynchronize(st.uploaded), "wait for previous upload");
  const size_t ub = upload_bytes(L);
  if (st.stage.size() < ub) st.stage.resize(ub);
  pl.dev = st.dev;
  pl.pin = st.stage.data();
  bind(&pl, L);
  GA_HIP(hipStreamWaitEvent(stream, st.done, 0), "order after previous call");
  rc = upload(&pl, L, stream);
  if (rc) return rc;
  GA_HIP(hipEventRecord(st.uploaded, stream), "record upload");
  rc = do_schedule(&pl, stream);
  if (rc) return rc;
  rc = do_run(&pl, q, kv_page_pool, out, lse, stream);
  if (rc) return rc;
  GA_HIP(hipEventRecord(st.done, stream), "record decode");
  return GA_OK;
}

static ga_status kv_write(void* pool, const void* k_new, const void* v_new, const int32_t* src,
                          const int32_t* dst, int32_t n, const ga_params* params,
                          void* hip_stream) {
  g_err.clear();
  ga_status rc = validate_params(params);
  if (rc) return rc;
  if (n < 0) return fail(GA_EINVAL, "num_tokens is negative");
  if (n == 0) return GA_OK;
  if (!pool || !dst || (src == nullptr && (!k_new || !v_new)))
    return fail(GA_EINVAL, "device pointers must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(pool) | reinterpret_cast<uintptr_t>(k_new) |
       reinterpret_cast<uintptr_t>(v_new)) & 15)
    return fail(GA_EINVAL, "kv_page_pool, k_new and v_new must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 3)
    return fail(GA_EINVAL, "slot word arrays must be 4-byte aligned");
  ga::KvWriteArgs a{};
  a.pool = static_cast<unsigned char*>(pool);
  a.k_new = static_cast<const unsigned char*>(k_new);
  a.v_new = static_cast<const unsigned char*>(v_new);
  a.src_words = src;
  a.dst_words = dst;
  a.num_slots = params->num_pages * ga::kPageTokens;
  a.n = n;
  a.Hkv = params->num_kv_heads;
  a.row_bytes = params->head_dim * (params->dtype == GA_BF16 ? 2 : 4);
  if ((int64_t)n * a.Hkv * 2 * (a.row_bytes / 16) > 0x7fffffffLL * 256)
    return fail(GA_EINVAL, "too many tokens (%d)", n);
  GA_HIP(ga::launch_kv_write(a, static_cast<hipStream_t>(hip_stream)), "kv write launch");
  return GA_OK;
}

ga_status graphattn_kv_append(void* kv_page_pool, const void* k_new, const void* v_new,
                              const int32_t* slot_words, int32_t num_tokens,
                              const ga_params* params, void* hip_stream) {
  return kv_write(kv_page_pool, k_new, v_new, nullptr, slot_words, num_tokens, params,
                  hip_stream);
}

ga_status graphattn_kv_copy(void* kv_page_pool, const int32_t* src_slot_words,
                            const int32_t* dst_slot_words, int32_t num_tokens,
                            const ga_params* params, void* hip_stream) {
  if (!src_slot_words && num_tokens > 0) {
    g_err.clear();
    return fail(GA_EINVAL, "src_slot_words is NULL");
  }
  return kv_write(kv_page_pool, nullptr, nullptr, src_slot_words, dst_slot_words, num_tokens,
                  params, hip_stream);
}

ga_status graphattn_extend(const void* q, const void* kv_page_pool,
                           const ga_segment_table* segment_table,
                           const ga_branch_paths* branch_paths, const int32_t* query_counts,
                           void* out, float* lse, const ga_params* params, void* hip_stream) {
  if (!query_counts && branch_paths && branch_paths->num_branches > 0) {
    g_err.clear();
    return fail(GA_EINVAL, "query_counts is NULL");
  }
  static const int32_t none = 0;
  return one_shot(q, kv_page_pool, segment_table, branch_paths,
                  query_counts ? query_counts : &none, out, lse, params, hip_stream);
}

}  // extern "C"
