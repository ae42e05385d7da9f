// Host side of equivalence detection and the graph suffix: forest validation, Euler intervals,
// the tile list, a cached device workspace, launches, and the two C entry points.
#include "../../include/graphattn.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "ga_internal.hpp"

namespace ga {
ga_status host_fail(ga_status st, const char* msg);
ga_status host_hip_fail(hipError_t e, const char* what);
void host_clear_error();
}  // namespace ga

namespace {

ga_status efail(ga_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
ga_status efail(ga_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return ga::host_fail(st, buf);
}

#define EQ_HIP(call, what)                                 \
  do {                                                     \
    hipError_t e_ = (call);                                \
    if (e_ != hipSuccess) return ga::host_hip_fail(e_, what); \
  } while (0)

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// The forest as the kernels need it.
struct Forest {
  int64_t N = 0;
  std::vector<int32_t> parent, depth, tin, tout, pstart, pend;
  std::vector<int4> items;       // 64 x 64 tiles of the prompts of more than 256 states
  std::vector<int2> prompts;     // (first state, states) of the prompts of at most 256 states
  std::vector<int32_t> big;      // the states of the larger prompts
  std::vector<int2> all;         // (first state, states) of every prompt
  int64_t big_reward = 0;        // states in prompts of more than 512 states
};

constexpr int32_t kPromptMax = 256;   // states one workgroup classifies on its own

// Each prompt's states are consecutive, its root first; p(v) < v.  Depths, prompt ranges and
// Euler intervals (tin <= tin' < tout exactly when the state is an ancestor of the other).
ga_status build_forest(const ga_state_forest* f, bool with_items, Forest* fo) {
  if (!f) return efail(GA_EINVAL, "forest is NULL");
  const int32_t N = f->num_states;
  if (N < 0) return efail(GA_EINVAL, "num_states is negative");
  if (N > 0 && !f->parent) return efail(GA_EINVAL, "parent is NULL");
  fo->N = N;
  fo->parent.assign(f->parent, f->parent + N);
  fo->depth.assign(N, 0);
  fo->pstart.assign(N, 0);
  fo->pend.assign(N, 0);
  int32_t root = -1;
  for (int32_t v = 0; v < N; ++v) {
    const int32_t p = f->parent[v];
    if (p < -1 || p >= v)
      return efail(GA_EINVAL, "parent[%d] = %d: a predecessor must precede its state", v, p);
    if (p == -1) {
      root = v;
    } else if (p < root) {
      return efail(GA_EINVAL, "state %d: its prompt's states are not consecutive", v);
    }
    fo->depth[v] = p < 0 ? 0 : fo->depth[p] + 1;
    fo->pstart[v] = root;
  }
  for (int32_t v = N - 1, end = N; v >= 0; --v) {
    fo->pend[v] = end;
    if (f->parent[v] == -1) end = v;
  }
  // Children lists, then an explicit depth-first walk per prompt.
  std::vector<int32_t> coff(N + 1, 0), kids(N > 0 ? N : 1);
  for (int32_t v = 0; v < N; ++v)
    if (f->parent[v] >= 0) ++coff[f->parent[v] + 1];
  for (int32_t v = 0; v < N; ++v) coff[v + 1] += coff[v];
  std::vector<int32_t> fill(coff.begin(), coff.end() - 1);
  for (int32_t v = 0; v < N; ++v)
    if (f->parent[v] >= 0) kids[fill[f->parent[v]]++] = v;
  fo->tin.assign(N, 0);
  fo->tout.assign(N, 0);
  std::vector<std::pair<int32_t, int32_t>> stack;
  int32_t clock = 0;
  for (int32_t r = 0; r < N; ++r) {
    if (f->parent[r] != -1) continue;
    stack.push_back({r, coff[r]});
    fo->tin[r] = clock++;
    while (!stack.empty()) {
      auto& top = stack.back();
      if (top.second < coff[top.first + 1]) {
        const int32_t c = kids[top.second++];
        fo->tin[c] = clock++;
        stack.push_back({c, coff[c]});
      } else {
        fo->tout[top.first] = clock;
        stack.pop_back();
      }
    }
  }
  fo->items.clear();
  fo->prompts.clear();
  fo->big.clear();
  fo->all.clear();
  fo->big_reward = 0;
  for (int32_t r = 0; r < N; r = fo->pend[r]) {
    fo->all.push_back(make_int2(r, fo->pend[r] - r));
    if (fo->pend[r] - r > 512) fo->big_reward += fo->pend[r] - r;
  }
  if (with_items) {
    for (int32_t r = 0; r < N; r = fo->pend[r]) {
      const int32_t e = fo->pend[r];
      if (e - r <= kPromptMax) {
        fo->prompts.push_back(make_int2(r, e - r));
        continue;
      }
      for (int32_t v = r; v < e; ++v) fo->big.push_back(v);
      for (int32_t i0 = r; i0 < e; i0 += 64)
        for (int32_t j0 = i0; j0 < e; j0 += 64) fo->items.push_back(make_int4(i0, j0, e, 0));
    }
  }
  return GA_OK;
}

template <typename T>
void put(char* pin, size_t& o, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(pin + o, v.data(), sizeof(T) * v.size());
  o = align256(o + sizeof(T) * v.size());
}

}  // namespace

// A validated forest on the device: its arrays (uploaded once) and the scratch of the kernels.
struct ga_forest {
  Forest fo;
  void* dev = nullptr;
  void* pin = nullptr;
  int32_t *tin = nullptr, *tout = nullptr, *parent = nullptr, *depth = nullptr;
  int32_t *pstart = nullptr, *pend = nullptr;
  int4* items = nullptr;
  int2* prompts = nullptr;
  int2* all = nullptr;
  int32_t* big = nullptr;
  float* inv_norm = nullptr;
  int* rep = nullptr;
  int64_t *cnt = nullptr, *off = nullptr, *blk = nullptr;
  // graph reward scratch
  int32_t *lab = nullptr, *anchor = nullptr;
  int64_t *euler = nullptr, *pre = nullptr, *own = nullptr, *ctot = nullptr;
  double *aeff_node = nullptr, *gmean = nullptr, *gstd = nullptr;
};

namespace {

void forest_free(ga_forest* f) {
  if (!f) return;
  if (f->dev) {
    (void)hipDeviceSynchronize();
    (void)hipFree(f->dev);
  }
  if (f->pin) (void)hipHostFree(f->pin);
  delete f;
}

ga_status forest_create(const ga_state_forest* forest, hipStream_t stream, ga_forest** out) {
  if (!out) return efail(GA_EINVAL, "forest out-pointer is NULL");
  *out = nullptr;
  ga_forest* f = new ga_forest();
  ga_status rc = build_forest(forest, true, &f->fo);
  if (rc) {
    delete f;
    return rc;
  }
  const Forest& fo = f->fo;
  if ((int64_t)fo.items.size() > 0x7fffffffLL) {
    delete f;
    return efail(GA_EINVAL, "too many tiles");
  }
  const size_t n4 = align256(4 * fo.N), n8 = align256(8 * fo.N);
  const size_t up = 6 * n4 + align256(sizeof(int4) * fo.items.size()) +
                    align256(sizeof(int2) * fo.prompts.size()) + align256(4 * fo.big.size()) +
                    align256(sizeof(int2) * fo.all.size());
  const size_t nblk = (size_t)((fo.N + 1023) / 1024);
  const size_t scan = align256(8 * (fo.N + 1));
  const size_t total = up + 2 * n4 + n8 + scan + align256(8 * (nblk + 1))   // classes, suffix
                       + 2 * n4 + 3 * n8 + scan + 3 * n8;                     // graph reward
  if (hipMalloc(&f->dev, total) != hipSuccess) {
    (void)hipGetLastError();
    f->dev = nullptr;
    forest_free(f);
    return efail(GA_ENOMEM, "device workspace of %zu bytes", total);
  }
  if (hipHostMalloc(&f->pin, up > 0 ? up : 1) != hipSuccess) {
    (void)hipGetLastError();
    f->pin = nullptr;
    forest_free(f);
    return efail(GA_ENOMEM, "pinned staging of %zu bytes", up);
  }
  char* pin = static_cast<char*>(f->pin);
  size_t o = 0;
  put(pin, o, fo.tin);
  put(pin, o, fo.tout);
  put(pin, o, fo.parent);
  put(pin, o, fo.depth);
  put(pin, o, fo.pstart);
  put(pin, o, fo.pend);
  put(pin, o, fo.items);
  put(pin, o, fo.prompts);
  put(pin, o, fo.big);
  put(pin, o, fo.all);
  char* d = static_cast<char*>(f->dev);
  f->tin = reinterpret_cast<int32_t*>(d);
  f->tout = reinterpret_cast<int32_t*>(d + n4);
  f->parent = reinterpret_cast<int32_t*>(d + 2 * n4);
  f->depth = reinterpret_cast<int32_t*>(d + 3 * n4);
  f->pstart = reinterpret_cast<int32_t*>(d + 4 * n4);
  f->pend = reinterpret_cast<int32_t*>(d + 5 * n4);
  f->items = reinterpret_cast<int4*>(d + 6 * n4);
  const size_t oi = 6 * n4 + align256(sizeof(int4) * fo.items.size());
  f->prompts = reinterpret_cast<int2*>(d + oi);
  f->big = reinterpret_cast<int32_t*>(d + oi + align256(sizeof(int2) * fo.prompts.size()));
  f->all = reinterpret_cast<int2*>(d + oi + align256(sizeof(int2) * fo.prompts.size()) +
                                   align256(4 * fo.big.size()));
  f->inv_norm = reinterpret_cast<float*>(d + up);
  f->rep = reinterpret_cast<int*>(d + up + n4);
  f->cnt = reinterpret_cast<int64_t*>(d + up + 2 * n4);
  f->off = reinterpret_cast<int64_t*>(d + up + 2 * n4 + n8);
  f->blk = reinterpret_cast<int64_t*>(d + up + 2 * n4 + n8 + scan);
  char* r = d + up + 2 * n4 + n8 + scan + align256(8 * (nblk + 1));
  f->lab = reinterpret_cast<int32_t*>(r);
  f->anchor = reinterpret_cast<int32_t*>(r + n4);
  f->euler = reinterpret_cast<int64_t*>(r + 2 * n4);
  f->own = reinterpret_cast<int64_t*>(r + 2 * n4 + n8);
  f->ctot = reinterpret_cast<int64_t*>(r + 2 * n4 + 2 * n8);
  f->pre = reinterpret_cast<int64_t*>(r + 2 * n4 + 3 * n8);
  f->aeff_node = reinterpret_cast<double*>(r + 2 * n4 + 3 * n8 + scan);
  f->gmean = reinterpret_cast<double*>(r + 2 * n4 + 4 * n8 + scan);
  f->gstd = reinterpret_cast<double*>(r + 2 * n4 + 5 * n8 + scan);
  if (up > 0) {
    const hipError_t e = hipMemcpyAsync(d, pin, up, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) {
      forest_free(f);
      return ga::host_hip_fail(e, "forest upload");
    }
  }
  *out = f;
  return GA_OK;
}

ga_status forest_classes(ga_forest* f, const void* embeddings, int32_t dim, int32_t dtype,
                         float kappa, int32_t* labels, float* edge_sim, hipStream_t stream) {
  if (!f) return efail(GA_EINVAL, "forest is NULL");
  if (dtype != GA_BF16) return efail(GA_EUNSUPPORTED, "embeddings must be bf16");
  if (dim < 64 || dim % 64) return efail(GA_EUNSUPPORTED, "dim %d unsupported (a multiple of 64)", dim);
  if (!std::isfinite(kappa)) return efail(GA_EINVAL, "kappa must be finite");
  if (f->fo.N == 0) return GA_OK;
  if (!embeddings || !labels) return efail(GA_EINVAL, "embeddings and labels must be non-NULL");
  if (reinterpret_cast<uintptr_t>(embeddings) & 15)
    return efail(GA_EINVAL, "embeddings must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(labels) | reinterpret_cast<uintptr_t>(edge_sim)) & 3)
    return efail(GA_EINVAL, "labels and edge_sim must be 4-byte aligned");
  ga::EquivArgs a{};
  a.parent = f->parent;
  a.edge_sim = edge_sim;
  a.z = static_cast<const unsigned short*>(embeddings);
  a.tin = f->tin;
  a.tout = f->tout;
  a.items = f->items;
  a.prompts = f->prompts;
  a.big = f->big;
  a.n_prompts = (int64_t)f->fo.prompts.size();
  a.n_big = (int64_t)f->fo.big.size();
  a.inv_norm = f->inv_norm;
  a.rep = f->rep;
  a.labels = labels;
  a.N = f->fo.N;
  a.n_items = (int64_t)f->fo.items.size();
  a.dim = dim;
  a.kappa = kappa;
  EQ_HIP(ga::launch_equivalence(a, stream), "equivalence launch");
  return GA_OK;
}

ga_status forest_suffix(ga_forest* f, const int32_t* labels, int64_t* suffix_offsets,
                        int32_t* suffix_states, int64_t capacity, int64_t* total,
                        hipStream_t stream) {
  if (!total) return efail(GA_EINVAL, "total is NULL");
  *total = 0;
  if (!f) return efail(GA_EINVAL, "forest is NULL");
  if (!suffix_offsets) return efail(GA_EINVAL, "suffix_offsets is NULL");
  if (capacity < 0) return efail(GA_EINVAL, "capacity is negative");
  const int64_t N = f->fo.N;
  if (N > 0 && !labels) return efail(GA_EINVAL, "labels is NULL");
  if ((reinterpret_cast<uintptr_t>(suffix_offsets) & 7) ||
      (reinterpret_cast<uintptr_t>(labels) & 3) || (reinterpret_cast<uintptr_t>(suffix_states) & 3))
    return efail(GA_EINVAL, "misaligned output or label array");
  ga::SuffixArgs a{};
  a.labels = labels;
  a.parent = f->parent;
  a.depth = f->depth;
  a.pstart = f->pstart;
  a.pend = f->pend;
  a.cnt = f->cnt;
  a.off = f->off;
  a.blk = f->blk;
  a.states = suffix_states;
  a.N = N;
  int64_t n = 0;
  if (N > 0) {
    EQ_HIP(ga::launch_suffix_count(a, stream), "suffix count launch");
    EQ_HIP(hipMemcpyAsync(&n, a.off + N, sizeof n, hipMemcpyDeviceToHost, stream), "total");
  }
  EQ_HIP(hipStreamSynchronize(stream), "synchronise");
  *total = n;
  if (n > capacity)
    return efail(GA_ERANGE, "graph suffix needs %lld entries, capacity is %lld", (long long)n,
                 (long long)capacity);
  if (n > 0 && !suffix_states) return efail(GA_EINVAL, "suffix_states is NULL");
  if (N == 0) {
    EQ_HIP(hipMemsetAsync(suffix_offsets, 0, sizeof(int64_t), stream), "offsets");
    return GA_OK;
  }
  EQ_HIP(hipMemcpyAsync(suffix_offsets, a.off, sizeof(int64_t) * (N + 1),
                        hipMemcpyDeviceToDevice, stream), "offsets");
  EQ_HIP(ga::launch_suffix_fill(a, stream), "suffix fill launch");
  return GA_OK;
}

}  // namespace

extern "C" {

ga_status graphattn_forest_create(const ga_state_forest* forest, void* hip_stream,
                                  ga_forest** out) {
  ga::host_clear_error();
  return forest_create(forest, static_cast<hipStream_t>(hip_stream), out);
}

ga_status graphattn_forest_classes(ga_forest* forest, const void* embeddings, int32_t dim,
                                   int32_t dtype, float kappa, int32_t* labels, float* edge_sim,
                                   void* hip_stream) {
  ga::host_clear_error();
  return forest_classes(forest, embeddings, dim, dtype, kappa, labels, edge_sim,
                        static_cast<hipStream_t>(hip_stream));
}

ga_status graphattn_forest_advantages(ga_forest* forest, const int32_t* labels,
                                      const int32_t* reward, const float* edge_sim, double w,
                                      double lambda_eff, const ga_advantages* out,
                                      void* hip_stream) {
  ga::host_clear_error();
  if (!forest) return efail(GA_EINVAL, "forest is NULL");
  if (!out) return efail(GA_EINVAL, "out is NULL");
  if (!std::isfinite(w) || w < 0.0 || w > 1.0) return efail(GA_EINVAL, "w must lie in [0, 1]");
  if (!std::isfinite(lambda_eff) || lambda_eff < 0.0)
    return efail(GA_EINVAL, "lambda_eff must be finite and >= 0");
  const int64_t N = forest->fo.N;
  if (N == 0) return GA_OK;
  const void* ptrs[] = {labels, reward, edge_sim, out->score, out->step_reward, out->a_cor,
                        out->a_eff, out->a_dual};
  for (const void* q : ptrs)
    if (!q) return efail(GA_EINVAL, "device arrays must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(labels) | reinterpret_cast<uintptr_t>(reward) |
       reinterpret_cast<uintptr_t>(edge_sim)) & 3)
    return efail(GA_EINVAL, "labels, reward and edge_sim must be 4-byte aligned");
  if ((reinterpret_cast<uintptr_t>(out->score) | reinterpret_cast<uintptr_t>(out->step_reward) |
       reinterpret_cast<uintptr_t>(out->a_cor) | reinterpret_cast<uintptr_t>(out->a_eff) |
       reinterpret_cast<uintptr_t>(out->a_dual)) & 7)
    return efail(GA_EINVAL, "output arrays must be 8-byte aligned");
  ga::RewardArgs a{};
  a.labels = labels;
  a.reward = reward;
  a.edge_sim = edge_sim;
  a.parent = forest->parent;
  a.depth = forest->depth;
  a.tin = forest->tin;
  a.tout = forest->tout;
  a.pstart = forest->pstart;
  a.pend = forest->pend;
  a.lab = forest->lab;
  a.euler = forest->euler;
  a.pre = forest->pre;
  a.blk = forest->blk;
  a.own = forest->own;
  a.ctot = forest->ctot;
  a.anchor = forest->anchor;
  a.aeff_node = forest->aeff_node;
  a.gmean = forest->gmean;
  a.gstd = forest->gstd;
  a.score = out->score;
  a.step = out->step_reward;
  a.a_cor = out->a_cor;
  a.a_eff = out->a_eff;
  a.a_dual = out->a_dual;
  a.N = N;
  a.prompts = forest->all;
  a.n_prompts = (int64_t)forest->fo.all.size();
  a.n_big = forest->fo.big_reward;
  a.w = w;
  a.lambda_eff = lambda_eff;
  EQ_HIP(ga::launch_advantages(a, static_cast<hipStream_t>(hip_stream)), "advantage launch");
  return GA_OK;
}

ga_status graphattn_forest_suffix(ga_forest* forest, const int32_t* labels,
                                  int64_t* suffix_offsets, int32_t* suffix_states,
                                  int64_t capacity, int64_t* total, void* hip_stream) {
  ga::host_clear_error();
  return forest_suffix(forest, labels, suffix_offsets, suffix_states, capacity, total,
                       static_cast<hipStream_t>(hip_stream));
}

void graphattn_forest_destroy(ga_forest* forest) { forest_free(forest); }

ga_status graphattn_equivalence_classes(const void* embeddings, int32_t dim, int32_t dtype,
                                        const ga_state_forest* forest, float kappa,
                                        int32_t* labels, void* hip_stream) {
  ga::host_clear_error();
  if (dtype != GA_BF16) return efail(GA_EUNSUPPORTED, "embeddings must be bf16");
  if (dim < 64 || dim % 64) return efail(GA_EUNSUPPORTED, "dim %d unsupported (a multiple of 64)", dim);
  if (!std::isfinite(kappa)) return efail(GA_EINVAL, "kappa must be finite");
  Forest probe;
  ga_status rc = build_forest(forest, false, &probe);
  if (rc) return rc;
  if (probe.N == 0) return GA_OK;
  if (!embeddings || !labels) return efail(GA_EINVAL, "embeddings and labels must be non-NULL");
  if (reinterpret_cast<uintptr_t>(embeddings) & 15)
    return efail(GA_EINVAL, "embeddings must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(labels) & 3) return efail(GA_EINVAL, "labels must be 4-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  ga_forest* f = nullptr;
  rc = forest_create(forest, stream, &f);
  if (rc) return rc;
  rc = forest_classes(f, embeddings, dim, dtype, kappa, labels, nullptr, stream);
  forest_free(f);
  return rc;
}

ga_status graphattn_graph_suffix(const int32_t* labels, const ga_state_forest* forest,
                                 int64_t* suffix_offsets, int32_t* suffix_states,
                                 int64_t capacity, int64_t* total, void* hip_stream) {
  ga::host_clear_error();
  if (!total) return efail(GA_EINVAL, "total is NULL");
  *total = 0;
  Forest probe;
  ga_status rc = build_forest(forest, false, &probe);
  if (rc) return rc;
  if (!suffix_offsets) return efail(GA_EINVAL, "suffix_offsets is NULL");
  if (capacity < 0) return efail(GA_EINVAL, "capacity is negative");
  if (probe.N > 0 && !labels) return efail(GA_EINVAL, "labels is NULL");
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  ga_forest* f = nullptr;
  rc = forest_create(forest, stream, &f);
  if (rc) return rc;
  rc = forest_suffix(f, labels, suffix_offsets, suffix_states, capacity, total, stream);
  forest_free(f);
  return rc;
}

}  // extern "C"
