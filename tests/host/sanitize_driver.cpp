// Host-only driver for the sanitizer build of the library's host runtime: random valid and
// invalid rollout graphs, query counts and state forests go through plan creation (validation,
// segment chains, query expansion, schedule sizing) and forest creation (validation, depths,
// Euler intervals, tile lists).  Without a GPU every call stops at its first device allocation,
// after all of that host code has run.  The kernel launchers are stubs: no call reaches them.
#include "graphattn.h"

#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include <hip/hip_runtime.h>
#include "ga_internal.hpp"

namespace ga {
hipError_t launch_schedule(const DevGraph&, const DevSchedule&, int32_t, int32_t, int64_t, bool,
                           hipStream_t) { std::abort(); }
hipError_t launch_seg_attn(const AttnArgs&, int, bool, bool, bool, int, hipStream_t, hipEvent_t,
                           hipEvent_t) { std::abort(); }
hipError_t launch_merge(const MergeArgs&, int, bool, bool, hipStream_t, hipEvent_t, hipEvent_t) {
  std::abort();
}
hipError_t launch_kv_write(const KvWriteArgs&, hipStream_t) { std::abort(); }
hipError_t launch_equivalence(const EquivArgs&, hipStream_t) { std::abort(); }
hipError_t launch_suffix_count(const SuffixArgs&, hipStream_t) { std::abort(); }
hipError_t launch_suffix_fill(const SuffixArgs&, hipStream_t) { std::abort(); }
hipError_t launch_advantages(const RewardArgs&, hipStream_t) { std::abort(); }
hipError_t launch_set_lengths(const LengthArgs&, hipStream_t) { std::abort(); }
int seg_attn_grid(int, bool, bool, bool, int num_cus) { return 2 * num_cus; }
}  // namespace ga

int main(int argc, char** argv) {
  const int trials = argc > 1 ? std::atoi(argv[1]) : 300;
  std::mt19937 rng(12345);
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int statuses[8] = {0};
  for (int t = 0; t < trials; ++t) {
    // A random graph: segments with random lengths and pages, paths over random segment lists.
    const int S = U(1, 40), B = U(1, 30);
    std::vector<int32_t> len(S), pages;
    std::vector<int64_t> off(S + 1, 0);
    for (int s = 0; s < S; ++s) {
      len[s] = U(1, 100);
      const int np = (len[s] + 15) / 16 + (U(0, 9) == 0 ? -1 : 0);   // sometimes too few pages
      for (int i = 0; i < np; ++i) pages.push_back(U(0, 60) == 0 ? -3 : U(0, 499));
      off[s + 1] = (int64_t)pages.size();
    }
    std::vector<int64_t> po(B + 1, 0);
    std::vector<int32_t> ps;
    for (int b = 0; b < B; ++b) {
      const int n = U(U(0, 30) == 0 ? 0 : 1, 7);
      std::vector<char> used(S, 0);
      for (int i = 0; i < n; ++i) {
        int s = U(0, S - 1);
        if (used[s] && U(0, 3)) continue;                          // rarely a repeat
        used[s] = 1;
        ps.push_back(U(0, 80) == 0 ? S + 2 : s);
      }
      po[b + 1] = (int64_t)ps.size();
    }
    ga_segment_table st{S, len.data(), off.data(), pages.data()};
    ga_branch_paths bp{B, po.data(), ps.empty() ? nullptr : ps.data()};
    ga_params p{U(0, 20) == 0 ? 6 : 28, 4, U(0, 20) == 0 ? 96 : 128, 16, 500, GA_BF16, 0.f, 0};
    ga_plan* plan = nullptr;
    const ga_status a = graphattn_plan_create(&st, &bp, &p, nullptr, &plan);
    statuses[-a]++;
    if (plan) graphattn_plan_destroy(plan);
    std::vector<int32_t> counts(B);
    for (int b = 0; b < B; ++b) counts[b] = U(0, 40);
    const ga_status e = graphattn_plan_create_extend(&st, &bp, counts.data(), &p, nullptr, &plan);
    statuses[-e]++;
    if (plan) graphattn_plan_destroy(plan);
    // A random forest (sometimes malformed).
    const int N = U(0, 700);
    std::vector<int32_t> par(N);
    int root = 0;
    for (int v = 0; v < N; ++v) {
      if (v == 0 || U(0, 60) == 0) {
        par[v] = -1;
        root = v;
      } else {
        par[v] = U(root, v - 1);
      }
      if (U(0, 400) == 0) par[v] = U(-3, N + 3);
    }
    ga_state_forest f{N, par.data()};
    ga_forest* fo = nullptr;
    const ga_status c = graphattn_forest_create(&f, nullptr, &fo);
    statuses[-c]++;
    if (fo) graphattn_forest_destroy(fo);
  }
  std::printf("statuses:");
  for (int i = 0; i < 6; ++i) std::printf(" %d", statuses[i]);
  std::printf("\nok\n");
  return 0;
}
