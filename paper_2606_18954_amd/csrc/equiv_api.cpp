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
  std::vector<int4> items;
};

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
  if (with_items) {
    for (int32_t r = 0; r < N; r = fo->pend[r]) {
      const int32_t e = fo->pend[r];
      for (int32_t i0 = r; i0 < e; i0 += 64)
        for (int32_t j0 = i0; j0 < e; j0 += 64) fo->items.push_back(make_int4(i0, j0, e, 0));
    }
  }
  return GA_OK;
}

// Process-wide device workspace and pinned staging for these calls (grown on demand; a call
// waits for the previous one's upload and kernels before reusing them).
struct Cache {
  std::mutex mu;
  void* dev = nullptr;
  size_t dev_bytes = 0;
  void* pin = nullptr;
  size_t pin_bytes = 0;
  int device = -1;
  hipEvent_t done = nullptr;
};
Cache g_eq;

ga_status acquire(size_t dev_bytes, size_t pin_bytes, hipStream_t stream) {
  int dev = 0;
  EQ_HIP(hipGetDevice(&dev), "current device");
  if (g_eq.device != dev) {
    g_eq.dev = g_eq.pin = nullptr;
    g_eq.dev_bytes = g_eq.pin_bytes = 0;
    g_eq.done = nullptr;
    g_eq.device = dev;
  }
  if (!g_eq.done) EQ_HIP(hipEventCreateWithFlags(&g_eq.done, hipEventDisableTiming), "event");
  // The staging buffer is refilled on the host, so everything the previous call enqueued
  // (its upload included) must be done.
  EQ_HIP(hipEventSynchronize(g_eq.done), "wait for the previous call");
  if (g_eq.dev_bytes < dev_bytes) {
    if (g_eq.dev) (void)hipFree(g_eq.dev);
    g_eq.dev = nullptr;
    g_eq.dev_bytes = 0;
    if (hipMalloc(&g_eq.dev, dev_bytes) != hipSuccess) {
      (void)hipGetLastError();
      return efail(GA_ENOMEM, "device workspace of %zu bytes", dev_bytes);
    }
    g_eq.dev_bytes = dev_bytes;
  }
  if (g_eq.pin_bytes < pin_bytes || !g_eq.pin) {
    if (g_eq.pin) (void)hipHostFree(g_eq.pin);
    g_eq.pin = nullptr;
    g_eq.pin_bytes = 0;
    if (hipHostMalloc(&g_eq.pin, pin_bytes > 0 ? pin_bytes : 1) != hipSuccess) {
      (void)hipGetLastError();
      return efail(GA_ENOMEM, "pinned staging of %zu bytes", pin_bytes);
    }
    g_eq.pin_bytes = pin_bytes;
  }
  (void)stream;
  return GA_OK;
}

template <typename T>
void put(char* pin, size_t& o, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(pin + o, v.data(), sizeof(T) * v.size());
  o = align256(o + sizeof(T) * v.size());
}

}  // namespace

extern "C" {

ga_status graphattn_equivalence_classes(const void* embeddings, int32_t dim, int32_t dtype,
                                        const ga_state_forest* forest, float kappa,
                                        int32_t* labels, void* hip_stream) {
  ga::host_clear_error();
  if (dtype != GA_BF16) return efail(GA_EUNSUPPORTED, "embeddings must be bf16");
  if (dim < 64 || dim % 64) return efail(GA_EUNSUPPORTED, "dim %d unsupported (a multiple of 64)", dim);
  if (!std::isfinite(kappa)) return efail(GA_EINVAL, "kappa must be finite");
  Forest fo;
  ga_status rc = build_forest(forest, true, &fo);
  if (rc) return rc;
  if (fo.N == 0) return GA_OK;
  if (!embeddings || !labels) return efail(GA_EINVAL, "embeddings and labels must be non-NULL");
  if (reinterpret_cast<uintptr_t>(embeddings) & 15)
    return efail(GA_EINVAL, "embeddings must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(labels) & 3) return efail(GA_EINVAL, "labels must be 4-byte aligned");
  if ((int64_t)fo.items.size() > 0x7fffffffLL) return efail(GA_EINVAL, "too many tiles");
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  std::lock_guard<std::mutex> lock(g_eq.mu);
  // Uploaded (pinned, one copy): tin, tout, items.  Device only: inverse norms, parents.
  const size_t up = align256(4 * fo.N) * 2 + align256(sizeof(int4) * fo.items.size());
  const size_t total = up + align256(4 * fo.N) * 2;
  rc = acquire(total, up, stream);
  if (rc) return rc;
  char* pin = static_cast<char*>(g_eq.pin);
  size_t o = 0;
  put(pin, o, fo.tin);
  put(pin, o, fo.tout);
  put(pin, o, fo.items);
  char* d = static_cast<char*>(g_eq.dev);
  EQ_HIP(hipMemcpyAsync(d, pin, up, hipMemcpyHostToDevice, stream), "forest upload");
  ga::EquivArgs a{};
  a.z = static_cast<const unsigned short*>(embeddings);
  a.tin = reinterpret_cast<const int32_t*>(d);
  a.tout = reinterpret_cast<const int32_t*>(d + align256(4 * fo.N));
  a.items = reinterpret_cast<const int4*>(d + 2 * align256(4 * fo.N));
  a.inv_norm = reinterpret_cast<float*>(d + up);
  a.rep = reinterpret_cast<int*>(d + up + align256(4 * fo.N));
  a.labels = labels;
  a.N = fo.N;
  a.n_items = (int64_t)fo.items.size();
  a.dim = dim;
  a.kappa = kappa;
  EQ_HIP(ga::launch_equivalence(a, stream), "equivalence launch");
  EQ_HIP(hipEventRecord(g_eq.done, stream), "record");
  return GA_OK;
}

ga_status graphattn_graph_suffix(const int32_t* labels, const ga_state_forest* forest,
                                 int64_t* suffix_offsets, int32_t* suffix_states,
                                 int64_t capacity, int64_t* total, void* hip_stream) {
  ga::host_clear_error();
  if (!total) return efail(GA_EINVAL, "total is NULL");
  *total = 0;
  Forest fo;
  ga_status rc = build_forest(forest, false, &fo);
  if (rc) return rc;
  if (!suffix_offsets) return efail(GA_EINVAL, "suffix_offsets is NULL");
  if (capacity < 0) return efail(GA_EINVAL, "capacity is negative");
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  if (fo.N == 0) {
    const int64_t zero = 0;
    EQ_HIP(hipMemcpyAsync(suffix_offsets, &zero, sizeof zero, hipMemcpyHostToDevice, stream),
           "offsets");
    EQ_HIP(hipStreamSynchronize(stream), "synchronise");
    return GA_OK;
  }
  if (!labels) return efail(GA_EINVAL, "labels is NULL");
  if ((reinterpret_cast<uintptr_t>(suffix_offsets) & 7) ||
      (reinterpret_cast<uintptr_t>(labels) & 3) || (reinterpret_cast<uintptr_t>(suffix_states) & 3))
    return efail(GA_EINVAL, "misaligned output or label array");
  std::lock_guard<std::mutex> lock(g_eq.mu);
  const size_t n4 = align256(4 * fo.N);
  const size_t up = 4 * n4;                          // parent, depth, pstart, pend
  const size_t nblk = (size_t)((fo.N + 1023) / 1024);
  const size_t tot = up + align256(8 * fo.N) + align256(8 * (fo.N + 1)) + align256(8 * nblk);
  rc = acquire(tot, up, stream);
  if (rc) return rc;
  char* pin = static_cast<char*>(g_eq.pin);
  size_t o = 0;
  put(pin, o, fo.parent);
  put(pin, o, fo.depth);
  put(pin, o, fo.pstart);
  put(pin, o, fo.pend);
  char* d = static_cast<char*>(g_eq.dev);
  EQ_HIP(hipMemcpyAsync(d, pin, up, hipMemcpyHostToDevice, stream), "forest upload");
  ga::SuffixArgs a{};
  a.labels = labels;
  a.parent = reinterpret_cast<const int32_t*>(d);
  a.depth = reinterpret_cast<const int32_t*>(d + n4);
  a.pstart = reinterpret_cast<const int32_t*>(d + 2 * n4);
  a.pend = reinterpret_cast<const int32_t*>(d + 3 * n4);
  a.cnt = reinterpret_cast<int64_t*>(d + up);
  a.off = reinterpret_cast<int64_t*>(d + up + align256(8 * fo.N));
  a.blk = reinterpret_cast<int64_t*>(d + up + align256(8 * fo.N) + align256(8 * (fo.N + 1)));
  a.states = suffix_states;
  a.N = fo.N;
  EQ_HIP(ga::launch_suffix_count(a, stream), "suffix count launch");
  int64_t n = 0;
  EQ_HIP(hipMemcpyAsync(&n, a.off + fo.N, sizeof n, hipMemcpyDeviceToHost, stream), "total");
  EQ_HIP(hipStreamSynchronize(stream), "synchronise");
  *total = n;
  if (n > capacity) {
    EQ_HIP(hipEventRecord(g_eq.done, stream), "record");
    return efail(GA_ERANGE, "graph suffix needs %lld entries, capacity is %lld", (long long)n,
                 (long long)capacity);
  }
  if (n > 0 && !suffix_states) return efail(GA_EINVAL, "suffix_states is NULL");
  EQ_HIP(hipMemcpyAsync(suffix_offsets, a.off, sizeof(int64_t) * (fo.N + 1),
                        hipMemcpyDeviceToDevice, stream), "offsets");
  EQ_HIP(ga::launch_suffix_fill(a, stream), "suffix fill launch");
  EQ_HIP(hipEventRecord(g_eq.done, stream), "record");
  return GA_OK;
}

}  // extern "C"
