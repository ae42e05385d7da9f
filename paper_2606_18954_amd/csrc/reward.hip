// Graph reward and dual-group advantage over the rollout states (Sec. 3.3-3.4; Alg. S.1,
// Stages 2-3), one pass per step over all states of a batch.
//
//   outcomes   c_own / t_own: sums over the terminal states of each state's subtree.  With the
//              states placed in Euler order (tin), a subtree is the contiguous range
//              [tin(v), tout(v)), so one prefix sum of the packed (R, 1) values of terminal states
//              gives every subtree's sums as a difference (integers: exact).
//   pooling    class totals by integer atomics (exact, so the order they land in is irrelevant);
//              S(v) = (c + w (C_Q - c)) / (t + w (T_Q - t)) in fp64, NaN without evidence.
//   step       r(v) = (S(v) - S(p(v))) (1 - max(0, sim(p(v), v))) on the edge into v.
//   correctness  the group of source u is E_cor(u) = {edges into C_g(u)}: u's successors plus
//              those of its class partners that lie deeper than u, found by one scan over the
//              prompt's states; mean and population std of the defined rewards; the edge into v
//              takes its z-score in the group of p(v) (0 without spread or reward; a spread of
//              at most kSpreadFloor is none: rewards equal by the definition differ by rounding).
//   efficiency per class of two or more (found by its smallest member): the deepest proper
//              ancestor a_Q of all members, route lengths l = d(v) - d(a_Q), z-scores of -l
//              gated by the class's mean defined score; every edge then sums, in ascending
//              state order, the values of the members in its subtree whose anchor lies above it.
//   dual       A_dual = A_cor + lambda A_eff.
// Every value is computed in a fixed order, so the results are deterministic.
#include "ga_internal.hpp"

namespace ga {
namespace {

constexpr int kB = 256;
// Scores lie in [0, 1] and |r| <= 2: rewards equal by the definition differ by fp64 rounding
// (~1e-16) at most, unequal ones by far more, so a correctness group spread at or below this
// is taken as none (its z-scores are 0) rather than rounding blown up to order one.
constexpr double kSpreadFloor = 1e-12;

__device__ __forceinline__ int64_t gid() { return (int64_t)blockIdx.x * kB + threadIdx.x; }

__global__ void k_outcome_vals(RewardArgs a) {
  const int64_t v = gid();
  if (v >= a.N) return;
  // A label must name a state of the same prompt no later than v (the smallest member of v's
  // class); anything else is read as v itself, so no index leaves the prompt.
  const int l = a.labels[v];
  a.lab[v] = (l >= a.pstart[v] && l <= (int)v) ? l : (int)v;
  const int r = a.reward[v];
  a.euler[a.tin[v]] = r >= 0 ? (((int64_t)r << 32) | 1) : 0;
  a.ctot[v] = 0;                                  // class totals, indexed by label
}

// Exclusive scan of euler[0, N) into pre[0, N] over many workgroups (block totals first).
__global__ __launch_bounds__(1024) void k_pre_sums(RewardArgs a) {
  __shared__ int64_t red[16];
  const int64_t i = (int64_t)blockIdx.x * 1024 + threadIdx.x;
  int64_t v = i < a.N ? a.euler[i] : 0;
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t t = 0;
    for (int w = 0; w < 16; ++w) t += red[w];
    a.blk[blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(1024) void k_pre_apply(RewardArgs a) {
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
  const int64_t v = i < a.N ? a.euler[i] : 0;
  int64_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int64_t before = 0;
  for (int k = 0; k < w; ++k) before += wsum[k];
  if (i < a.N) a.pre[i] = base + before + x - v;
  if (i == a.N - 1) a.pre[a.N] = base + before + x;
}

// Own outcomes (packed: correct << 32 | terminal states) and their class totals.
__global__ void k_own(RewardArgs a) {
  const int64_t v = gid();
  if (v >= a.N) return;
  const int64_t own = a.pre[a.tout[v]] - a.pre[a.tin[v]];
  a.own[v] = own;
  atomicAdd(reinterpret_cast<unsigned long long*>(a.ctot + a.lab[v]), (unsigned long long)own);
}

__global__ void k_scores(RewardArgs a) {
  const int64_t v = gid();
  if (v >= a.N) return;
  const int64_t own = a.own[v], tot = a.ctot[a.lab[v]];
  const double c = (double)(own >> 32), t = (double)(own & 0xffffffffLL);
  const double C = (double)(tot >> 32), T = (double)(tot & 0xffffffffLL);
  const double num = c + a.w * (C - c), den = t + a.w * (T - t);
  a.score[v] = den > 0.0 ? num / den : __builtin_nan("");
  a.anchor[v] = -1;                               // set for class members by the next kernel
  a.aeff_node[v] = 0.0;
}

// Step rewards; and, for the smallest member of each class of two or more, the class's
// anchor, its members' efficiency values and their anchors.
__global__ void k_step_and_classes(RewardArgs a) {
  const int64_t v = gid();
  if (v >= a.N) return;
  const int p = a.parent[v];
  double r = __builtin_nan("");
  if (p >= 0) {
    const double s = fmax(0.0, (double)a.edge_sim[v]);
    r = (a.score[v] - a.score[p]) * (1.0 - s);
  }
  a.step[v] = r;
  if (a.lab[v] != (int)v) return;               // not the smallest member of its class
  const int lo = a.pstart[v], hi = a.pend[v];
  int m = 0, lca = -1;
  double ssum = 0.0;
  int sdef = 0;
  for (int x = (int)v; x < hi; ++x) {
    if (a.lab[x] != (int)v) continue;
    ++m;
    if (!isnan(a.score[x])) {
      ssum += a.score[x];
      ++sdef;
    }
    if (lca < 0) {
      lca = x;
      continue;
    }
    int y = x, z = lca;                            // lowest common ancestor by depth walking
    while (a.depth[y] > a.depth[z]) y = a.parent[y];
    while (a.depth[z] > a.depth[y]) z = a.parent[z];
    while (y != z) {
      y = a.parent[y];
      z = a.parent[z];
    }
    lca = y;
  }
  (void)lo;
  if (m < 2) return;
  const int anc = a.lab[lca] == (int)v ? a.parent[lca] : lca;   // a proper ancestor of all
  if (anc < 0) return;                             // a class holding its prompt's root
  const double gate = sdef > 0 ? ssum / sdef : 0.0;
  double lsum = 0.0;
  for (int x = (int)v; x < hi; ++x)
    if (a.lab[x] == (int)v) lsum += -(double)(a.depth[x] - a.depth[anc]);
  const double mean = lsum / m;
  double q = 0.0;
  for (int x = (int)v; x < hi; ++x)
    if (a.lab[x] == (int)v) {
      const double d = -(double)(a.depth[x] - a.depth[anc]) - mean;
      q += d * d;
    }
  const double sd = sqrt(q / m);
  for (int x = (int)v; x < hi; ++x)
    if (a.lab[x] == (int)v) {
      const double l = -(double)(a.depth[x] - a.depth[anc]);
      a.aeff_node[x] = sd > 0.0 ? gate * (l - mean) / sd : 0.0;
      a.anchor[x] = anc;
    }
}

// Correctness-group statistics of every source state u (over E_cor(u)), and the efficiency
// value of the edge into every state.
__global__ void k_groups_and_routes(RewardArgs a) {
  const int64_t u = gid();
  if (u >= a.N) return;
  const int lu = a.lab[u], du = a.depth[u], lo = a.pstart[u], hi = a.pend[u];
  int n = 0, members = 0;
  double s = 0.0;
  for (int c = lo; c < hi; ++c) {
    const int p = a.parent[c];
    if (p < 0 || !(p == (int)u || (a.lab[p] == lu && a.depth[c] > du))) continue;
    ++members;
    if (isnan(a.step[c])) continue;
    s += a.step[c];
    ++n;
  }
  double mean = 0.0, sd = 0.0;
  if (members > 1 && n > 0) {
    mean = s / n;
    double q = 0.0;
    for (int c = lo; c < hi; ++c) {
      const int p = a.parent[c];
      if (p < 0 || !(p == (int)u || (a.lab[p] == lu && a.depth[c] > du))) continue;
      if (isnan(a.step[c])) continue;
      const double d = a.step[c] - mean;
      q += d * d;
    }
    sd = sqrt(q / n);
    if (!(sd > kSpreadFloor)) sd = 0.0;
  }
  a.gmean[u] = mean;
  a.gstd[u] = sd;                                  // 0: no group, or no spread
  double e = 0.0;
  if (a.parent[u] >= 0) {
    const int tin_u = a.tin[u], tout_u = a.tout[u];
    for (int x = lo; x < hi; ++x) {
      const int an = a.anchor[x];
      if (an < 0 || a.tin[x] < tin_u || a.tin[x] >= tout_u) continue;
      if (a.depth[an] < du) e += a.aeff_node[x];
    }
  }
  a.a_eff[u] = e;
}

__global__ void k_dual(RewardArgs a) {
  const int64_t v = gid();
  if (v >= a.N) return;
  const int p = a.parent[v];
  double c = 0.0;
  if (p >= 0 && !isnan(a.step[v]) && a.gstd[p] > 0.0) c = (a.step[v] - a.gmean[p]) / a.gstd[p];
  a.a_cor[v] = c;
  a.a_dual[v] = c + a.lambda_eff * a.a_eff[v];
}

// Every prompt of at most kRPromptMax states in one workgroup, its arrays in LDS, one launch:
//   outcomes   a prefix sum of the packed (R, 1) values in Euler order (subtrees are ranges);
//   pooling    class totals by LDS integer atomics;
//   lists      children and class members as CSR built with LDS atomics and then sorted, so
//              each state's correctness group reads only its class's children and each class's
//              efficiency values only its members;
//   routes     the edge into u sums over u's subtree, read off the Euler order.
// The results equal the multi-kernel path's up to the order of a few fp64 sums.
constexpr int kRPromptMax = 512;

template <typename T>
__device__ void lds_scan_excl(T* v, int n) {          // exclusive scan of v[0, n] in place
  __shared__ T tmp[kRPromptMax + 1];
  for (int i = threadIdx.x; i <= n; i += 256) tmp[i] = v[i];
  __syncthreads();
  for (int off = 1; off <= n; off <<= 1) {
    T add[3] = {0, 0, 0};
    int k = 0;
    for (int i = threadIdx.x; i <= n; i += 256, ++k) add[k] = i >= off ? tmp[i - off] : 0;
    __syncthreads();
    k = 0;
    for (int i = threadIdx.x; i <= n; i += 256, ++k) tmp[i] += add[k];
    __syncthreads();
  }
  for (int i = threadIdx.x; i <= n; i += 256) v[i] = i ? tmp[i - 1] : 0;
  __syncthreads();
}

__device__ void sort_small(int* a, int n) {           // insertion sort of a short list
  for (int i = 1; i < n; ++i) {
    const int x = a[i];
    int j = i - 1;
    while (j >= 0 && a[j] > x) {
      a[j + 1] = a[j];
      --j;
    }
    a[j + 1] = x;
  }
}

__global__ __launch_bounds__(256) void k_prompt_advantages(RewardArgs a) {
  __shared__ int s_par[kRPromptMax], s_lab[kRPromptMax], s_dep[kRPromptMax];
  __shared__ int s_tin[kRPromptMax], s_tout[kRPromptMax], s_eul[kRPromptMax];
  __shared__ int s_anc[kRPromptMax];
  __shared__ int s_coff[kRPromptMax + 1], s_kids[kRPromptMax], s_cfill[kRPromptMax];
  __shared__ int s_moff[kRPromptMax + 1], s_mem[kRPromptMax], s_mfill[kRPromptMax];
  __shared__ long long s_pre[kRPromptMax + 1];
  __shared__ unsigned long long s_ctot[kRPromptMax];
  __shared__ double s_S[kRPromptMax], s_r[kRPromptMax], s_aen[kRPromptMax];
  __shared__ double s_gm[kRPromptMax], s_gs[kRPromptMax];
  const int2 pr = a.prompts[blockIdx.x];
  const int s0 = pr.x, n = pr.y, tid = threadIdx.x;
  const int t0 = a.tin[s0];
  for (int v = tid; v <= n; v += 256) {
    s_coff[v] = 0;
    s_moff[v] = 0;
    s_pre[v] = 0;
  }
  for (int v = tid; v < n; v += 256) {
    s_ctot[v] = 0;
    s_cfill[v] = 0;
    s_mfill[v] = 0;
  }
  __syncthreads();
  for (int v = tid; v < n; v += 256) {               // prompt-local indices throughout
    const int g = s0 + v;
    const int l = a.labels[g];
    const int lab = ((l >= s0 && l <= g) ? l : g) - s0;
    s_lab[v] = lab;
    const int p = a.parent[g];
    s_par[v] = p >= 0 ? p - s0 : -1;
    s_dep[v] = a.depth[g];
    const int tin = a.tin[g] - t0;
    s_tin[v] = tin;
    s_tout[v] = a.tout[g] - t0;
    s_eul[tin] = v;
    const int r = a.reward[g];
    s_pre[tin] = r >= 0 ? (((long long)r << 32) | 1) : 0;
    if (p >= 0) atomicAdd(&s_coff[p - s0], 1);
    atomicAdd(&s_moff[lab], 1);
  }
  __syncthreads();
  // Exclusive scans over [0, n]: s_pre[k] = sum of the outcome values at Euler positions < k (so
  // a subtree's sums are s_pre[tout] - s_pre[tin]); s_coff[p] = where p's children start and
  // s_moff[l] = where the members labelled l start.
  lds_scan_excl(s_pre, n);
  lds_scan_excl(s_coff, n);
  lds_scan_excl(s_moff, n);
  for (int v = tid; v < n; v += 256) {
    const int p = s_par[v];
    if (p >= 0) s_kids[s_coff[p] + atomicAdd(&s_cfill[p], 1)] = v;
    const int l = s_lab[v];
    s_mem[s_moff[l] + atomicAdd(&s_mfill[l], 1)] = v;
  }
  __syncthreads();
  for (int v = tid; v < n; v += 256) {               // lists in ascending order
    sort_small(s_kids + s_coff[v], s_cfill[v]);
    sort_small(s_mem + s_moff[v], s_mfill[v]);
  }
  __syncthreads();
  for (int v = tid; v < n; v += 256) {               // own outcomes -> class totals
    const long long own = s_pre[s_tout[v]] - s_pre[s_tin[v]];
    atomicAdd(&s_ctot[s_lab[v]], (unsigned long long)own);
    s_anc[v] = -1;
    s_aen[v] = 0.0;
  }
  __syncthreads();
  for (int v = tid; v < n; v += 256) {               // pooled scores
    const long long own = s_pre[s_tout[v]] - s_pre[s_tin[v]];
    const long long tot = (long long)s_ctot[s_lab[v]];
    const double c = (double)(own >> 32), t = (double)(own & 0xffffffffLL);
    const double C = (double)(tot >> 32), T = (double)(tot & 0xffffffffLL);
    const double num = c + a.w * (C - c), den = t + a.w * (T - t);
    const double S = den > 0.0 ? num / den : __builtin_nan("");
    s_S[v] = S;
    a.score[s0 + v] = S;
  }
  __syncthreads();
  for (int v = tid; v < n; v += 256) {               // step rewards; class efficiency values
    const int p = s_par[v];
    double r = __builtin_nan("");
    if (p >= 0) r = (s_S[v] - s_S[p]) * (1.0 - fmax(0.0, (double)a.edge_sim[s0 + v]));
    s_r[v] = r;
    a.step[s0 + v] = r;
    if (s_lab[v] != v) continue;
    const int* mem = s_mem + s_moff[v];
    const int m = s_mfill[v];
    if (m < 2) continue;
    int lca = mem[0], sdef = 0;
    double ssum = 0.0;
    for (int k = 0; k < m; ++k) {
      const int x = mem[k];
      if (!isnan(s_S[x])) {
        ssum += s_S[x];
        ++sdef;
      }
      int y = x, z = lca;
      while (s_dep[y] > s_dep[z]) y = s_par[y];
      while (s_dep[z] > s_dep[y]) z = s_par[z];
      while (y != z) {
        y = s_par[y];
        z = s_par[z];
      }
      lca = y;
    }
    const int anc = s_lab[lca] == v ? s_par[lca] : lca;
    if (anc < 0) continue;
    const double gate = sdef > 0 ? ssum / sdef : 0.0;
    double lsum = 0.0;
    for (int k = 0; k < m; ++k) lsum += -(double)(s_dep[mem[k]] - s_dep[anc]);
    const double mean = lsum / m;
    double q = 0.0;
    for (int k = 0; k < m; ++k) {
      const double d = -(double)(s_dep[mem[k]] - s_dep[anc]) - mean;
      q += d * d;
    }
    const double sd = sqrt(q / m);
    for (int k = 0; k < m; ++k) {
      const int x = mem[k];
      const double l = -(double)(s_dep[x] - s_dep[anc]);
      s_aen[x] = sd > 0.0 ? gate * (l - mean) / sd : 0.0;
      s_anc[x] = anc;
    }
  }
  __syncthreads();
  for (int u = tid; u < n; u += 256) {               // correctness groups; efficiency per edge
    const int lu = s_lab[u], du = s_dep[u];
    const int* mem = s_mem + s_moff[lu];
    const int m = s_mfill[lu];
    int cnt = 0, members = 0;
    double sum = 0.0;
    for (int k = 0; k < m; ++k) {
      const int q = mem[k];
      const int* kid = s_kids + s_coff[q];
      for (int j = 0; j < s_cfill[q]; ++j) {
        const int c = kid[j];
        if (q != u && s_dep[c] <= du) continue;
        ++members;
        if (isnan(s_r[c])) continue;
        sum += s_r[c];
        ++cnt;
      }
    }
    double mean = 0.0, sd = 0.0;
    if (members > 1 && cnt > 0) {
      mean = sum / cnt;
      double q2 = 0.0;
      for (int k = 0; k < m; ++k) {
        const int q = mem[k];
        const int* kid = s_kids + s_coff[q];
        for (int j = 0; j < s_cfill[q]; ++j) {
          const int c = kid[j];
          if ((q != u && s_dep[c] <= du) || isnan(s_r[c])) continue;
          const double d = s_r[c] - mean;
          q2 += d * d;
        }
      }
      sd = sqrt(q2 / cnt);
      if (!(sd > kSpreadFloor)) sd = 0.0;
    }
    s_gm[u] = mean;
    s_gs[u] = sd;
    double e = 0.0;
    if (s_par[u] >= 0)
      for (int pos = s_tin[u]; pos < s_tout[u]; ++pos) {
        const int x = s_eul[pos];
        const int an = s_anc[x];
        if (an >= 0 && s_dep[an] < du) e += s_aen[x];
      }
    a.a_eff[s0 + u] = e;
  }
  __syncthreads();
  for (int v = tid; v < n; v += 256) {
    const int p = s_par[v];
    double c = 0.0;
    if (p >= 0 && !isnan(s_r[v]) && s_gs[p] > 0.0) c = (s_r[v] - s_gm[p]) / s_gs[p];
    a.a_cor[s0 + v] = c;
    a.a_dual[s0 + v] = c + a.lambda_eff * a.a_eff[s0 + v];   // written by this thread above
  }
}

}  // namespace

hipError_t launch_advantages(const RewardArgs& a, hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  if (a.n_big == 0) {
    hipLaunchKernelGGL(k_prompt_advantages, dim3((unsigned)a.n_prompts), dim3(256), 0, stream, a);
    return hipGetLastError();
  }
  const unsigned g = (unsigned)((a.N + kB - 1) / kB);
  const unsigned sb = (unsigned)((a.N + 1023) / 1024);
  hipLaunchKernelGGL(k_outcome_vals, dim3(g), dim3(kB), 0, stream, a);
  hipLaunchKernelGGL(k_pre_sums, dim3(sb), dim3(1024), 0, stream, a);
  hipLaunchKernelGGL(k_pre_apply, dim3(sb), dim3(1024), 0, stream, a);
  hipLaunchKernelGGL(k_own, dim3(g), dim3(kB), 0, stream, a);
  hipLaunchKernelGGL(k_scores, dim3(g), dim3(kB), 0, stream, a);
  hipLaunchKernelGGL(k_step_and_classes, dim3(g), dim3(kB), 0, stream, a);
  hipLaunchKernelGGL(k_groups_and_routes, dim3(g), dim3(kB), 0, stream, a);
  hipLaunchKernelGGL(k_dual, dim3(g), dim3(kB), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ga
