// Device-side checks of the preconditions the fast path assumes but cannot
// see from the host, run before any other launch of a call when checking is
// on: every bf16 input finite, chunk positions strictly increasing, and the
// chunk's first position after the last cached one of each listed layer
// (stream positions only grow; the smoothing join and the recency term
// Sec. 3.1 / Sec. 3.2 rely on sorted positions).
#include "hermes_internal.h"

namespace hermes {
namespace {

constexpr int NT = 256;

// bit 0: a non-finite input; bit 1: positions not strictly increasing;
// bit 2: a chunk not after the cache.
__global__ __launch_bounds__(NT) void check_inputs(CheckArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * NT;
  unsigned bad = 0u;
  const int64_t n8 = (a.nq > a.nkv ? a.nq : a.nkv) / 8;   // 16-byte pieces
  for (int64_t e = gid; e < n8; e += stride) {
    const uint4 *src[3] = {reinterpret_cast<const uint4 *>(a.q), reinterpret_cast<const uint4 *>(a.k),
                           reinterpret_cast<const uint4 *>(a.v)};
    const int64_t lim[3] = {a.nq / 8, a.nkv / 8, a.nkv / 8};
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      if (e >= lim[t]) continue;
      const uint4 x = src[t][e];
      const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        // bf16 halves with an all-ones exponent are Inf or NaN
        if ((w[h] & 0x7f80u) == 0x7f80u || (w[h] & 0x7f800000u) == 0x7f800000u) bad |= 1u;
      }
    }
  }
  if (a.pos != nullptr) {
    for (int64_t i = gid; i + 1 < a.n_new; i += stride)
      if (a.pos[i] >= a.pos[i + 1]) bad |= 2u;
    if (gid < a.n_list) {
      const int l = a.layer_id[gid];
      const int len = a.len[gid];
      if (len > 0 && a.pos[0] <= a.tab[l].pos[a.cur[gid]][len - 1]) bad |= 4u;
    }
  }
  if (bad != 0u) atomicOr(a.flag, bad);
}

}  // namespace

hipError_t launch_check(const CheckArgs &a, hipStream_t s) {
  const int64_t n8 = (a.nq > a.nkv ? a.nq : a.nkv) / 8;
  int64_t blocks = (n8 + NT - 1) / NT;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(check_inputs, dim3((unsigned)blocks), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace hermes
