// Page-pool writes: storing new tokens' K and V in page slots (append) and moving tokens between
// page slots (copy).
//
// A decode step extends every active branch's newest segment by the token it produced, and a
// state's continuation is split into step segments (Alg. S.1, Stage 1).  Since every segment
// starts at slot 0 of a page of its own, forking a state into children needs no copy (each child
// opens new pages); moving the tokens after a cut inside a page to fresh pages does.
//
// A slot word w names page w / 16, slot w % 16.  One thread moves 16 bytes: token j's data is
// Hkv x 2 x ROW bytes (ROW = D x element size), and piece p of it is kv-head p / (2 PR), K or V
// (p / PR) % 2, 16-byte chunk p % PR of the token row (PR = ROW / 16), so consecutive threads
// read and write contiguous runs of a row.  Words outside [0, num_pages x 16) skip the token:
// nothing outside the pool is ever written.
#include "ga_internal.hpp"

namespace ga {
namespace {

__device__ __forceinline__ int64_t slot_offset(int32_t w, int h, int kv, int Hkv, int row_bytes) {
  return ((((int64_t)(w >> 4) * Hkv + h) * 2 + kv) * kPageTokens + (w & 15)) * row_bytes;
}

__global__ __launch_bounds__(256) void k_kv_write(KvWriteArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int pr = a.row_bytes / 16;
  const int ppt = a.Hkv * 2 * pr;
  const int64_t j = gid / ppt;
  if (j >= a.n) return;
  const int p = (int)(gid - j * ppt);
  const int h = p / (2 * pr), kv = (p / pr) & 1, c = p % pr;
  const int32_t dw = a.dst_words[j];
  if (dw < 0 || (int64_t)dw >= a.num_slots) return;
  const uint4* src;
  if (a.src_words) {
    const int32_t sw = a.src_words[j];
    if (sw < 0 || (int64_t)sw >= a.num_slots) return;
    src = reinterpret_cast<const uint4*>(a.pool + slot_offset(sw, h, kv, a.Hkv, a.row_bytes) +
                                         16 * c);
  } else {
    const unsigned char* base = kv ? a.v_new : a.k_new;
    src = reinterpret_cast<const uint4*>(base + (j * a.Hkv + h) * a.row_bytes + 16 * c);
  }
  *reinterpret_cast<uint4*>(a.pool + slot_offset(dw, h, kv, a.Hkv, a.row_bytes) + 16 * c) = *src;
}

}  // namespace

hipError_t launch_kv_write(const KvWriteArgs& a, hipStream_t stream) {
  const int64_t threads = (int64_t)a.n * a.Hkv * 2 * (a.row_bytes / 16);
  const int64_t grid = (threads + 255) / 256;
  if (grid == 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_kv_write, dim3((unsigned)grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ga
