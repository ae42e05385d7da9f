/*
 * graphattn.h -- C ABI of graph-segment decode attention on MI355X (gfx950).
 *
 * Problem (GraphPO, Sec. 3.2 "Graph Construction" and Alg. S.1 Stage 1): a rollout graph has
 * reasoning steps as edges and the prompt as its root; the generation context of a state is the
 * ordered concatenation of the edge tokens on its path from the root.  Each edge's tokens form
 * a *segment* whose K/V live in fixed-size pages of a shared pool.  Every active *branch* (a
 * state being extended) is a list of segment ids, and at each decode step it issues one query
 * per q-head that attends, with ordinary scaled-dot-product softmax attention, over all tokens
 * of all segments on its path.  Siblings share their parent's prefix segments (Sec. 1) and
 * virtually merged states share the representative's successors (Sec. 3.2, graph suffix C_g),
 * so one segment is usually read by many branches.
 *
 * The library groups the branches that share each segment (a GPU segment scheduler), computes
 * every segment's contribution for all of its branches at once (a grouped dense contraction on
 * bf16 MFMA with a wave-level online softmax), and folds the per-segment partial results of
 * each branch with a log-sum-exp merge.  The result equals the textbook attention over the
 * branch's concatenated context up to floating-point rounding.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Device buffers (q, kv_page_pool, out, lse) are caller-owned device pointers; the library never
 * frees or reallocates them.  Index arrays (segment table, branch paths) are caller-owned HOST
 * arrays, read only during the call that receives them.
 *
 *   q             [B][Hq][D]                 dtype; one decode query per branch and q-head
 *   kv_page_pool  [num_pages][Hkv][2][16][D] dtype; index 0 of the third axis is K, 1 is V
 *   out           [B][Hq][D]                 dtype (same as q), or float32 if params->out_f32
 *   lse           [B][Hq]                    float32, natural log of sum_j exp(scale * q.k_j)
 *
 * Token t of segment s sits in page seg_pages[seg_page_offsets[s] + t / 16], slot t % 16.  Each
 * segment starts at slot 0 of its first page.  The contents of slots >= seg_len in a segment's
 * last page, and of pages no segment references, are unspecified (they may hold NaN) and are
 * never used.  Grouped-query attention: q-head h reads kv-head h / (Hq / Hkv).
 *
 * Errors: all inputs are validated on the host before any device work is enqueued.  On error
 * the call returns a negative ga_status, writes nothing to any caller buffer, and
 * graphattn_last_error() describes the failure (thread-local).  Device work is asynchronous on
 * the given HIP stream (NULL = the default stream).
 */
#ifndef GRAPHATTN_H
#define GRAPHATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GA_OK = 0,
  GA_EINVAL = -1,        /* malformed argument: null pointer, bad CSR, empty or repeating path */
  GA_ERANGE = -2,        /* segment id or page id out of range */
  GA_ENOMEM = -3,        /* device or pinned-host allocation failed */
  GA_EHIP = -4,          /* a HIP runtime call or kernel launch failed */
  GA_EUNSUPPORTED = -5   /* head_dim, page_size or dtype outside what the kernels implement */
} ga_status;

typedef enum { GA_F32 = 0, GA_BF16 = 1 } ga_dtype;

/* The rollout graph's segments: one segment per generated step (edge) plus the prompt (root).
 * seg_len[s] >= 1 tokens; seg_page_offsets is CSR into seg_pages with seg_page_offsets[0] = 0,
 * non-decreasing, and at least ceil(seg_len[s] / 16) pages per segment.  Page ids lie in
 * [0, num_pages), num_pages <= 2^27 (GA_EUNSUPPORTED beyond).  Host memory. */
typedef struct {
  int32_t num_segments;
  const int32_t* seg_len;           /* [S] */
  const int64_t* seg_page_offsets;  /* [S + 1] */
  const int32_t* seg_pages;         /* [seg_page_offsets[S]] */
} ga_segment_table;

/* The active branches: branch b's context is segments path_segs[path_offsets[b] ..
 * path_offsets[b+1]), root first.  Paths are non-empty and visit a segment at most once (paths
 * in a DAG are simple, Sec. 3.2); the order of segments does not change the result.  Host
 * memory. */
typedef struct {
  int32_t num_branches;
  const int64_t* path_offsets;      /* [B + 1], path_offsets[0] = 0, non-decreasing */
  const int32_t* path_segs;         /* [path_offsets[B]] */
} ga_branch_paths;

typedef struct {
  int32_t num_q_heads;     /* Hq, a positive multiple of num_kv_heads */
  int32_t num_kv_heads;    /* Hkv > 0 */
  int32_t head_dim;        /* D: 64 or 128 */
  int32_t page_size;       /* tokens per page: 16 */
  int64_t num_pages;       /* extent of kv_page_pool, for range checks */
  int32_t dtype;           /* ga_dtype of q and kv_page_pool (and of out unless out_f32) */
  float softmax_scale;     /* 0 selects 1/sqrt(head_dim) */
  int32_t out_f32;         /* 0: out has dtype; 1: out is float32 (no final rounding) */
} ga_params;

/* A validated rollout graph uploaded to the device, plus its schedule and workspace. */
typedef struct ga_plan ga_plan;

/* One decode step of graph-segment attention, end to end: validate, upload the graph, group
 * the branches of every segment, run the grouped segment attention and merge each branch's
 * partials.  Equivalent to plan_create + schedule + run + destroy, but reuses a cached device
 * workspace between calls (calls on different streams are ordered through an event).  q,
 * kv_page_pool, out, lse: device pointers as described above; with num_branches = 0 nothing is
 * launched.  Returns GA_OK or a negative ga_status. */
ga_status graphattn_decode(const void* q, const void* kv_page_pool,
                           const ga_segment_table* segment_table,
                           const ga_branch_paths* branch_paths, void* out, float* lse,
                           const ga_params* params, void* hip_stream);

/* Multi-query ("extend") attention: several query tokens per branch, causal inside the branch's
 * newest segment.  A continuation is predicted token by token from prefix(u) (Alg. S.1, Stage 1),
 * so prefilling a new step segment, or checking several drafted tokens at once, gives each of its
 * tokens one query over the path's earlier segments plus the segment's tokens up to itself.
 * Branch b's newest segment is the LAST entry of its path and must be on no other path; its
 * K/V are already in the pool (graphattn_kv_append).  query_counts[b] = n_b in [1, len(last)]
 * (host array): the queries are the segment's last n_b tokens, query i at position
 * len(last) - n_b + i, seeing every token of the other path segments and tokens 0 .. that
 * position of the newest one (itself included).  With n_b = 1 this is graphattn_decode.
 *   q    [R][Hq][D]  R = sum_b n_b query rows, branch-major, ascending i within a branch
 *   out  [R][Hq][D], lse [R][Hq]  (as for decode, per query row)
 * Rows of one branch share its path's segments with each other and with every branch on them,
 * so a segment's K/V are read once per kv-head for all of those rows.  GA_EINVAL for a NULL
 * query_counts with branches, a count outside [1, len(last)] or a newest segment shared with
 * another path.  Otherwise as graphattn_decode. */
ga_status graphattn_extend(const void* q, const void* kv_page_pool,
                           const ga_segment_table* segment_table,
                           const ga_branch_paths* branch_paths, const int32_t* query_counts,
                           void* out, float* lse, const ga_params* params, void* hip_stream);

/* The graph of a rollout (Sec. 3.2 "Graph Construction": step segments as edges, the prompt
 * as root, branches as the active states' paths), prepared once for many decode steps and
 * layers.  Validate the graph and parameters, allocate the plan's device workspace (sized for this
 * graph, with every segment at all the pages the page table gives it, so that lengths set later
 * by graphattn_plan_set_lengths fit) and enqueue the upload of the index arrays on hip_stream.  The host arrays may be
 * released when the call returns.  *plan receives a new plan (NULL on error). */
ga_status graphattn_plan_create(const ga_segment_table* segment_table,
                                const ga_branch_paths* branch_paths, const ga_params* params,
                                void* hip_stream, ga_plan** plan);

/* A plan for graphattn_extend's problem (same arguments and checks): graphattn_schedule and
 * graphattn_run then take q / out / lse with R = sum_b n_b rows.  In the schedule (plan_info,
 * debug dump) every query row is a branch with its branch's path. */
ga_status graphattn_plan_create_extend(const ga_segment_table* segment_table,
                                       const ga_branch_paths* branch_paths,
                                       const int32_t* query_counts, const ga_params* params,
                                       void* hip_stream, ga_plan** plan);

/* New segment lengths for a plan, for the decode loop of Alg. S.1 (Stage 1): each step stores
 * a token per branch in the page slot after its newest segment's last token
 * (graphattn_kv_append) and the segment grows by one; a state that spawns children starts new
 * segments.  seg_len [num_segments of the plan's graph] host, read during the call: every
 * length >= 1 and within the pages the segment owns in the plan's page table (the page table
 * may give a segment more pages than its length uses, reserved for growth); for a multi-query
 * plan each branch's query count must stay <= its newest segment's length.  GA_EINVAL
 * otherwise, and the plan is unchanged.  Paths, page ids and query counts stay as created.  The
 * lengths are copied to the device and the plan's segment chains (page lists with their valid
 * token counts, lengths, causal origins) are rebuilt there in place, asynchronously on
 * hip_stream and ordered after the work already enqueued there (work of this plan on other
 * streams must be complete); the lengths pass through one of four pinned slots in turn, and
 * the host waits only when that slot's copy from four updates earlier is still pending.  No
 * allocation.  The plan must be scheduled again (graphattn_schedule) before
 * its next run. */
ga_status graphattn_plan_set_lengths(ga_plan* plan, const int32_t* seg_len, void* hip_stream);

/* Segment scheduler, on the GPU: transpose branch->segments into segment->branches (B(s) in
 * ascending branch order: the branches that share a segment, i.e. siblings sharing a prefix
 * (Sec. 1) and merged states sharing a suffix (Sec. 3.2, C_g)), give each path entry the
 * branch's position inside B(s), split long segments into page chunks and emit the work list of
 * (segment, chunk, row block) items and each branch's partial-row list.  Enqueued on
 * hip_stream.  graphattn_run schedules by itself when the plan has no current schedule (a new
 * plan, or new lengths); calling this first splits the work for timing or for one schedule
 * serving several runs.  Deterministic: the same graph always yields the same schedule. */
ga_status graphattn_schedule(ga_plan* plan, void* hip_stream);

/* Grouped segment attention and log-sum-exp merge for one layer's q and K/V pool (the
 * attention of every branch over prefix(u), Alg. S.1 Stage 1, grouped per segment as in
 * graphattn_decode), using the plan's schedule (the rollout graph is shared by every layer of a
 * decode step, so a schedule serves any number of runs); a plan without a current schedule is
 * scheduled first, on the same stream.  Device pointers as described above.  Enqueued on
 * hip_stream; runs on one plan must not overlap (they share the partial-result workspace).  If
 * a launch fails (GA_EHIP) the outputs are unspecified and the plan is scheduled again by its
 * next run. */
ga_status graphattn_run(ga_plan* plan, const void* q, const void* kv_page_pool, void* out,
                        float* lse, void* hip_stream);

/* Sizes of the schedule, available after plan_create.  The plan schedules chains: maximal runs
 * of consecutive path segments whose branch sets are identical (every branch through s continues
 * with s', and no other branch enters s') are attended as one segment, which is exact (attention
 * over disjoint token sets merges by log-sum-exp) and leaves one partial per branch and chunk of
 * the chain. */
typedef struct {
  /* S and B as given; E = path entries of the schedule: path_offsets[B] for decode plans,
   * sum_b n_b |path_b| for multi-query plans */
  int32_t num_segments, num_branches, num_entries;
  int32_t chunk_pages;        /* maximum pages per work item */
  int32_t rows_per_block;     /* maximum query rows (branch x q-head-in-group) per work item */
  int64_t num_items;          /* work items per kv-head */
  int64_t num_partial_rows;   /* partial results per q-head the workspace holds: the sum over
                                 path entries of chunks, each segment at all the pages it owns
                                 (equal to the rows in use when segments own no spare pages) */
  int32_t num_chains;         /* chains scheduled (segments on some path, after merging runs) */
  int32_t num_query_rows;     /* rows of q / out / lse: B for decode plans, sum_b n_b for extend */
  int32_t workgroups_per_cu;  /* attention workgroups resident per CU in the persistent grid */
  int32_t work_streams;       /* work streams the attention units are split into (by kv-head) */
} ga_plan_info;
ga_status graphattn_plan_info(const ga_plan* plan, ga_plan_info* info);

/* Inspection of the scheduler's integer output (test infrastructure: the grouping, ranks and
 * partial lists are compared bit for bit with a plain-loop grouping of the paths).  Copies the
 * device schedule back to host arrays (synchronises hip_stream; GA_EINVAL if the plan has no
 * current schedule).  Any pointer may be NULL to skip that array.  Sizes: group_offsets [S+1]
 * and group_branches [E] (B(s) as CSR, ascending ids), entry_ranks [E] (position of each path
 * entry's branch inside its segment's group), items [3 * num_items] as (segment, chunk, row
 * block) triples, segment_chunks [S], branch_part_offsets [num_query_rows + 1] and branch_parts
 * [num_partial_rows] (each branch's partial rows per q-head as CSR, in the order the merge folds
 * them: path order, then chunk order; only branch_part_offsets[num_query_rows] entries are
 * written).  Groups and ranks are per given segment and path entry.  Items, chunk counts and
 * partial rows are per chain: an item names its chain by the chain's first segment,
 * segment_chunks holds a chain's chunk count at its first segment and 0 at the others, a branch
 * lists the partials of each chain on its path at the chain's first segment, and the partial
 * row of (chain v, chunk c, rank j) is prow(v) + c |B(v)| + j with prow the running sum of
 * chunks x |B| over the chains in the order of their first segments. */
ga_status graphattn_plan_debug_dump(const ga_plan* plan, void* hip_stream,
                                    int64_t* group_offsets, int32_t* group_branches,
                                    int32_t* entry_ranks, int32_t* items,
                                    int32_t* segment_chunks, int64_t* branch_part_offsets,
                                    int32_t* branch_parts);

/* Measurement infrastructure.  Kernel timing with HIP events: recorded on the launch stream
 * around each scheduler pass, and bound to each attention and each merge dispatch (their elapsed
 * time is the kernel's own execution, without the gaps of the queue around it).
 * graphattn_plan_profile(plan, n) arms recording for the
 * next n schedule and n run calls (n = 0 disarms and clears); graphattn_plan_profile_read
 * synchronises on the last recorded event and returns the accumulated times in milliseconds
 * and the number of calls recorded.  Timing is for eager calls: do not arm it around calls that
 * a stream capture records into a HIP graph. */
typedef struct {
  int32_t schedules, runs;     /* calls recorded */
  double sched_ms;             /* sum over recorded schedule calls */
  double attn_ms;              /* sum over recorded runs: grouped segment attention kernel */
  double merge_ms;             /* sum over recorded runs: log-sum-exp merge kernel */
} ga_profile;
ga_status graphattn_plan_profile(ga_plan* plan, int32_t max_calls);
ga_status graphattn_plan_profile_read(ga_plan* plan, ga_profile* out);

/* Page-pool writes (Alg. S.1, Stage 1: each decode step extends the newest segment of every
 * active branch by its token; a continuation is split into step segments).  A slot word
 * w = page * 16 + slot names one token slot of kv_page_pool.  Slot words are DEVICE arrays (one
 * mapping serves every layer's pool), so they are range-checked in the kernel: a token whose
 * word lies outside [0, num_pages * 16) is skipped and nothing outside the pool is written
 * (negative words pad a batch).  Only params->num_kv_heads, head_dim, dtype and num_pages are
 * used; the call validates params like the others and is asynchronous on hip_stream.
 *
 * graphattn_kv_append: token j's K and V, k_new / v_new [num_tokens][Hkv][D] (device, the pool's
 * dtype), are stored for every kv-head at slot_words[j].  Destinations must be distinct
 * (otherwise which token lands is unspecified).
 *
 * graphattn_kv_copy: every kv-head's K and V of slot src_slot_words[j] are copied to slot
 * dst_slot_words[j].  Since each segment starts at slot 0 of a page of its own, a fork needs no
 * copy (children open new pages); cutting a generated run into step segments inside a page moves
 * the tokens after the cut to fresh pages with this call.  Destinations must be distinct and
 * disjoint from the sources (otherwise the result is unspecified).
 *
 * Both: pool, k_new and v_new 16-byte aligned; num_tokens >= 0 (0: nothing is launched). */
ga_status graphattn_kv_append(void* kv_page_pool, const void* k_new, const void* v_new,
                              const int32_t* slot_words, int32_t num_tokens,
                              const ga_params* params, void* hip_stream);
ga_status graphattn_kv_copy(void* kv_page_pool, const int32_t* src_slot_words,
                            const int32_t* dst_slot_words, int32_t num_tokens,
                            const ga_params* params, void* hip_stream);

/* Rollout states for equivalence detection: the generation tree of every prompt in a batch.
 * parent[v] = p(v), the state v was generated from (-1 for a prompt's root).  Each prompt's
 * states are consecutive, its root first, and p(v) < v (GA_EINVAL otherwise).  Host memory. */
typedef struct {
  int32_t num_states;
  const int32_t* parent;   /* [N] */
} ga_state_forest;

/* A forest validated and uploaded once (its Euler intervals, depths, prompt ranges and the tile
 * list of the similarity), plus the kernels' scratch; the graph_suffix / equivalence_classes
 * calls below are forest_create + one call + forest_destroy.  Create enqueues the upload on
 * hip_stream (the host arrays may be released on return); destroy waits for the device. */
typedef struct ga_forest ga_forest;
ga_status graphattn_forest_create(const ga_state_forest* forest, void* hip_stream,
                                  ga_forest** out);
/* forest_classes also writes, when edge_sim is not NULL, edge_sim[v] = sim(p(v), v) (device
 * float [N], 0 for a root): the cosine of each state with its predecessor, from the same
 * products (the graph reward's endpoint similarity). */
ga_status graphattn_forest_classes(ga_forest* forest, const void* embeddings, int32_t dim,
                                   int32_t dtype, float kappa, int32_t* labels, float* edge_sim,
                                   void* hip_stream);
ga_status graphattn_forest_suffix(ga_forest* forest, const int32_t* labels,
                                  int64_t* suffix_offsets, int32_t* suffix_states,
                                  int64_t capacity, int64_t* total, void* hip_stream);
void graphattn_forest_destroy(ga_forest* forest);

/* Equivalence classes of rollout states (Sec. 3.2 "Graph Construction"; Alg. S.1, Stage 1).
 * Two states of the same prompt that are neither ancestor nor descendant of each other are
 * compared by the cosine of their embeddings; pairs with cosine >= kappa are joined by
 * union-find, so the classes Q(v) are the connected components of those links.  A state with a
 * zero embedding is never joined.
 *   embeddings  [N][dim] device, bf16 (dtype = GA_BF16; GA_EUNSUPPORTED otherwise), 16-byte
 *               aligned; dim a positive multiple of 64 (GA_EUNSUPPORTED otherwise)
 *   labels      [N] device int32, written: the smallest state id of each state's class
 * The cosine is computed from fp32 sums of the bf16 products (error below 2.5e-4 at
 * dim = 4096), so a pair within that distance of kappa may be decided either way.  Host
 * validation first; returns after the device work (its workspace is freed on return; the
 * forest calls above are asynchronous). */
ga_status graphattn_equivalence_classes(const void* embeddings, int32_t dim, int32_t dtype,
                                        const ga_state_forest* forest, float kappa,
                                        int32_t* labels, void* hip_stream);

/* Graph suffix (Sec. 3.2, the equation of C_g): C_g(u) = u's direct successors plus those of
 * the other members of Q(u) that lie deeper than u (shared edges only point deeper, so the
 * graph stays acyclic).  labels [N] device int32 (as written by graphattn_equivalence_classes).
 * Output as CSR: suffix_offsets [N + 1] device int64, suffix_states [*total] device int32,
 * ascending state ids per state.  The call synchronises hip_stream to learn the size: *total
 * (host) receives it; if it exceeds capacity the call returns GA_ERANGE and writes neither
 * output array (call again with a larger buffer). */
ga_status graphattn_graph_suffix(const int32_t* labels, const ga_state_forest* forest,
                                 int64_t* suffix_offsets, int32_t* suffix_states,
                                 int64_t capacity, int64_t* total, void* hip_stream);

/* Graph reward and dual-group advantage (Sec. 3.3-3.4; Alg. S.1, Stages 2-3) for every
 * state v and the direct edge (p(v), v) into it.  Device inputs of N entries:
 *   labels    classes as written by forest_classes (a label outside [v's prompt's first state,
 *             v] is read as v itself)
 *   reward    R(v) (0 or 1) for a terminal state, any negative value for other states
 *   edge_sim  sim(p(v), v), e.g. from forest_classes (roots ignored)
 * w in [0, 1] pools the outcomes of class partners; lambda_eff >= 0 weighs efficiency.
 * Outputs (device double [N] each):
 *   score        S(v) = (c_own(v) + w sum_{q in Q(v)\v} c_own(q)) / (t_own(v) + w sum t_own(q)),
 *                c_own / t_own = correct / all terminal states in v's subtree; NaN when the
 *                denominator is 0 (no evidence)
 *   step_reward  r(v) = (S(v) - S(p(v))) (1 - max(0, edge_sim(v))); NaN for a root or an
 *                undefined score
 *   a_cor        z-score of r(v) (population std) among the defined rewards of the group
 *                E_cor(p(v)) = edges into C_g(p(v)), when that group has two or more edges and a
 *                spread above 1e-12; 0 otherwise (scores lie in [0, 1], so a smaller spread is
 *                the fp64 rounding of rewards that are equal by the definition)
 *   a_eff        sum, over the classes Q of two or more and their members x whose route from
 *                a_Q (the deepest proper ancestor of all of Q) passes through this edge, of
 *                mean_Q(S) z(-l_x), l_x = d(x) - d(a_Q) (z over Q, population std; 0 if no
 *                spread)
 *   a_dual       a_cor + lambda_eff a_eff
 * Asynchronous on hip_stream; deterministic. */
typedef struct {
  double* score;
  double* step_reward;
  double* a_cor;
  double* a_eff;
  double* a_dual;
} ga_advantages;
ga_status graphattn_forest_advantages(ga_forest* forest, const int32_t* labels,
                                      const int32_t* reward, const float* edge_sim, double w,
                                      double lambda_eff, const ga_advantages* out,
                                      void* hip_stream);

/* graphattn_decode without any device or pinned-host allocation, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, checks, kernels and results (bit for bit) as graphattn_decode;
 * the workspace (uploaded graph, schedule, partial results) lives in a static device array of
 * 64 MiB per device, held from the first call on a device until the process ends.  A graph
 * whose workspace exceeds it is rejected with GA_ENOMEM before any device work (the message
 * gives both sizes); the merged-DAG decode step of 1024 branches needs about 45 MiB.  The graph
 * upload is staged in ordinary (pageable) host memory and host-side validation uses the heap.
 * All calls on one device share its array: each call waits (on the device, through an event)
 * for the previous call's kernels before it reuses the array, and concurrent host calls are
 * serialised by a lock, so calls on several streams do not race but do not overlap either.
 * Devices 0..15. */
ga_status graphattn_decode_static(const void* q, const void* kv_page_pool,
                                  const ga_segment_table* segment_table,
                                  const ga_branch_paths* branch_paths, void* out, float* lse,
                                  const ga_params* params, void* hip_stream);

/* Release the plan and its device workspace (waits for work still using it). */
void graphattn_plan_destroy(ga_plan* plan);

/* Thread-local description of the last failure in this thread ("" if none). */
const char* graphattn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GRAPHATTN_H */
