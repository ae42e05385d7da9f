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

namespace ga {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int D, bool BF16, bool PF16>
__global__ __launch_bounds__(256) void k_merge(MergeArgs a) {
  constexpr int LPR = D / 4;               // lanes per (branch, q-head) row, 4 columns each
  constexpr int RPB = 256 / LPR;           // rows per workgroup
  constexpr int PS = PF16 ? 2 : 1;         // floats per partial log-sum-exp entry
  const int tid = threadIdx.x;
  // The attention kernel has drained its work queue (stream order): re-arm it for the next run.
  if (blockIdx.x == 0 && tid == 0) a.counters[2] = 0;
  const int64_t row = (int64_t)blockIdx.x * RPB + tid / LPR;
  const int sub = tid % LPR;
  if (row >= (int64_t)a.B * a.Hq) return;
  const int b = (int)(row / a.Hq);
  const int h = (int)(row % a.Hq);
  const float NEG_INF = -__builtin_huge_valf();
  const int64_t k0 = a.bpart_off[b], k1 = a.bpart_off[b + 1];
  // This lane's 4 columns 4 sub .. 4 sub + 3 = 16 n + 4 g + (0 .. 3) with n = sub / 4, g = sub % 4;
  // in the fp16 format they sit at position 32 (n / 2) + 8 g + 4 (n % 2) of the row (the lane
  // order of the attention kernel's tiles).
  const int pos = PF16 ? (sub / 8) * 32 + (sub % 4) * 8 + ((sub / 4) % 2) * 4 : 4 * sub;
  // One pass in list order (path order, then chunk order) with a running maximum: when a
  // partial's log-sum-exp exceeds it, the sums so far are rescaled.
  float M = NEG_INF, W = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int64_t k = k0; k < k1; ++k) {
    const int64_t idx = (int64_t)a.bpart[k] * a.Hq + h;
    const float lam = a.plse[idx * PS];
    f32x4 o;
    float sc = 1.f;
    if constexpr (PF16) {
      typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
      const f16x4 v =
          *reinterpret_cast<const f16x4*>(static_cast<const _Float16*>(a.po) + idx * D + pos);
      o = f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
      sc = a.plse[idx * PS + 1];                // undoes the partial's power-of-two scaling
    } else {
      o = *reinterpret_cast<const f32x4*>(static_cast<const float*>(a.po) + idx * D + pos);
    }
    if (lam > M) {                               // the same for the row's lanes
      const float r = __builtin_amdgcn_exp2f(M - lam);
      W *= r;
      acc *= r;
      M = lam;
    }
    const float wl = __builtin_amdgcn_exp2f(lam - M);
    acc += o * (wl * sc);
    W += wl;
  }
  const f32x4 r = acc * (1.f / W);
  if constexpr (BF16) {
    unsigned short u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) u[i] = __builtin_bit_cast(unsigned short, (__bf16)r[i]);
    uint2 pk = make_uint2(u[0] | ((unsigned)u[1] << 16), u[2] | ((unsigned)u[3] << 16));
    *reinterpret_cast<uint2*>(static_cast<unsigned short*>(a.out) + row * D + 4 * sub) = pk;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + row * D + 4 * sub) = r;
  }
  if (sub == 0) a.lse[row] = (M + __builtin_amdgcn_logf(W)) * 0.69314718055994531f;
}

template <int D, bool BF16, bool PF16>
hipError_t launch_t(const MergeArgs& a, hipStream_t stream) {
  constexpr int RPB = 256 / (D / 4);
  const int64_t rows = (int64_t)a.B * a.Hq;
  const int grid = (int)((rows + RPB - 1) / RPB);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((k_merge<D, BF16, PF16>), dim3(grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <bool BF16, bool PF16>
hipError_t launch_d(const MergeArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 64) return launch_t<64, BF16, PF16>(a, stream);
  if (head_dim == 128) return launch_t<128, BF16, PF16>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int head_dim, bool bf16, bool part_f16,
                        hipStream_t stream) {
  if (bf16) return part_f16 ? launch_d<true, true>(a, head_dim, stream)
                            : launch_d<true, false>(a, head_dim, stream);
  return part_f16 ? launch_d<false, true>(a, head_dim, stream)
                  : launch_d<false, false>(a, head_dim, stream);
}

}  // namespace ga
