// Log-sum-exp merge of per-segment partials along each branch's path.
//
// A branch's context is the disjoint union of its segments' tokens (and of each segment's page
// chunks), so with lambda_i = log2 sum_{j in piece i} 2^(s_j) and o_i the piece's normalised
// output, the exact result over the whole context is
//   Lambda = log2 sum_i 2^(lambda_i),  out = sum_i 2^(lambda_i - Lambda) o_i.
// The scheduler lists each branch's partials in path order, then chunk order; the merge folds them
// in that order in one pass with a running maximum, so the result is deterministic.  The
// natural-log lse is Lambda * ln 2.  Partials of bf16 inputs are fp16 values with a power-of-two
// scale per row (format in ga_internal.hpp); the scale is folded into the row's weight.
#include "ga_internal.hpp"

#include <hip/hip_ext.h>

namespace ga {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int D, bool BF16, bool PF16>
__global__ __launch_bounds__(256) void k_merge(MergeArgs a) {
  // fp16 partials: 16 lanes per row, each lane 8 stored positions (16 bytes) = two groups of 4
  // consecutive columns; fp32 partials: D / 4 lanes per row, 4 columns each.
  constexpr int CPL = PF16 ? 8 : 4;            // values per lane
  constexpr int LPR = D / CPL;                 // lanes per (branch, q-head) row
  constexpr int RPB = 256 / LPR;               // rows per workgroup
  constexpr int PS = PF16 ? 2 : 1;
  // Partials loaded per batch before any is folded.  Two, with the next batch's ids loaded
  // ahead, keep 8 waves per SIMD and two value loads per row in flight; four leave fewer rows
  // resident and are slower.
  constexpr int KB = 2;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0 && tid < kMaxStreams) reinterpret_cast<int*>(a.counters + 4)[tid] = 0;
  const int64_t row = (int64_t)blockIdx.x * RPB + tid / LPR;
  const int sub = tid % LPR;
  if (row >= (int64_t)a.B * a.Hq) return;
  const int b = (int)(row / a.Hq);
  const int h = (int)(row % a.Hq);
  const float NEG_INF = -__builtin_huge_valf();
  const int64_t k0 = a.bpart_off[b], k1 = a.bpart_off[b + 1];
  float M = NEG_INF, W = 0.f;
  float acc[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) acc[i] = 0.f;
  // The next batch's partial-row ids are loaded one batch ahead, so that each batch's values
  // wait for one load round trip instead of two (the id, then the values it names).
  int32_t nid[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) nid[j] = k0 + j < k1 ? a.bpart[k0 + j] : 0;
  for (int64_t kb = k0; kb < k1; kb += KB) {
    const int nk = (int)min((int64_t)KB, k1 - kb);
    int64_t idx[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) idx[j] = j < nk ? (int64_t)nid[j] * a.Hq + h : 0;
#pragma unroll
    for (int j = 0; j < KB; ++j) nid[j] = kb + KB + j < k1 ? a.bpart[kb + KB + j] : 0;
    float lam[KB], sc[KB], o[KB][CPL];
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      if (j >= nk) { lam[j] = NEG_INF; sc[j] = 0.f; continue; }
      if constexpr (PF16) {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const f32x2 ls = *reinterpret_cast<const f32x2*>(a.plse + idx[j] * PS);
        lam[j] = ls[0];
        sc[j] = ls[1];
        typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
        const f16x8 v = *reinterpret_cast<const f16x8*>(static_cast<const _Float16*>(a.po) +
                                                        idx[j] * D + 8 * sub);
#pragma unroll
        for (int i = 0; i < 8; ++i) o[j][i] = (float)v[i];
      } else {
        lam[j] = a.plse[idx[j]];
        sc[j] = 1.f;
        const f32x4 v = *reinterpret_cast<const f32x4*>(static_cast<const float*>(a.po) +
                                                        idx[j] * D + 4 * sub);
#pragma unroll
        for (int i = 0; i < 4; ++i) o[j][i] = v[i];
      }
    }
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      if (j >= nk) break;
      if (lam[j] > M) {
        const float r = __builtin_amdgcn_exp2f(M - lam[j]);
        W *= r;
#pragma unroll
        for (int i = 0; i < CPL; ++i) acc[i] *= r;
        M = lam[j];
      }
      const float wl = __builtin_amdgcn_exp2f(lam[j] - M);
      const float ws = wl * sc[j];
#pragma unroll
      for (int i = 0; i < CPL; ++i) acc[i] += o[j][i] * ws;
      W += wl;
    }
  }
  const float inv = 1.f / W;
  // Columns of this lane: fp16 positions 8 sub .. 8 sub + 7 hold columns 16 n + 4 g + (0..3) and
  // 16 (n + 1) + 4 g + (0..3) with n = 2 (sub / 4), g = sub % 4; fp32 holds 4 sub .. 4 sub + 3.
  auto put4 = [&](int col, int i0) {
    if constexpr (BF16) {
      unsigned short u[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) u[i] = __builtin_bit_cast(unsigned short, (__bf16)(acc[i0 + i] * inv));
      *reinterpret_cast<uint2*>(static_cast<unsigned short*>(a.out) + row * D + col) =
          make_uint2(u[0] | ((unsigned)u[1] << 16), u[2] | ((unsigned)u[3] << 16));
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + row * D + col) =
          f32x4{acc[i0] * inv, acc[i0 + 1] * inv, acc[i0 + 2] * inv, acc[i0 + 3] * inv};
    }
  };
  if constexpr (PF16) {
    const int n = 2 * (sub / 4), g = sub % 4;
    put4(16 * n + 4 * g, 0);
    put4(16 * (n + 1) + 4 * g, 4);
  } else {
    put4(4 * sub, 0);
  }
  if (sub == 0) a.lse[row] = (M + __builtin_amdgcn_logf(W)) * 0.69314718055994531f;
}

template <int D, bool BF16, bool PF16>
hipError_t launch_t(const MergeArgs& a, hipStream_t stream, hipEvent_t t0, hipEvent_t t1) {
  constexpr int RPB = 256 / (D / (PF16 ? 8 : 4));
  const int64_t rows = (int64_t)a.B * a.Hq;
  const int grid = (int)((rows + RPB - 1) / RPB);
  if (grid == 0) return hipSuccess;
  if (t0 || t1)
    hipExtLaunchKernelGGL(k_merge<D, BF16, PF16>, dim3(grid), dim3(256), 0, stream, t0, t1, 0, a);
  else
    hipLaunchKernelGGL((k_merge<D, BF16, PF16>), dim3(grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <bool BF16, bool PF16>
hipError_t launch_d(const MergeArgs& a, int head_dim, hipStream_t stream, hipEvent_t t0,
                    hipEvent_t t1) {
  if (head_dim == 64) return launch_t<64, BF16, PF16>(a, stream, t0, t1);
  if (head_dim == 128) return launch_t<128, BF16, PF16>(a, stream, t0, t1);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int head_dim, bool bf16, bool part_f16,
                        hipStream_t stream, hipEvent_t t0, hipEvent_t t1) {
  if (bf16) return part_f16 ? launch_d<true, true>(a, head_dim, stream, t0, t1)
                            : launch_d<true, false>(a, head_dim, stream, t0, t1);
  return part_f16 ? launch_d<false, true>(a, head_dim, stream, t0, t1)
                  : launch_d<false, false>(a, head_dim, stream, t0, t1);
}

}  // namespace ga
