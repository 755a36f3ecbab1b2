// Data movement kernels for gfx950: the append copy of a chunk's K/V rows
// into the cache tail, and the order-preserving gather of kept rows
// (Sec. 3.2: K_l = K_l[I_l], V_l = V_l[I_l]) into the other buffer of each
// layer's ping-pong pair.  Rows are token-major (Hkv * d bf16 per row), moved
// in 16-byte pieces so every wave issues fully coalesced 1 KiB transactions.
#include "hermes_internal.h"

namespace hermes {
namespace {

constexpr int NT = 256;

__global__ __launch_bounds__(NT) void append_rows(AppendArgs a) {
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const int T0 = a.T0[jj];
  const int pieces = a.row_elems / 8;
  const int total = a.C * pieces;
  const uint16_t *kn = a.kn + a.slot[jj] * a.kv_lstride;
  const uint16_t *vn = a.vn + a.slot[jj] * a.kv_lstride;
  uint16_t *kd = L.k[cur] + (int64_t)T0 * a.row_elems;
  uint16_t *vd = L.v[cur] + (int64_t)T0 * a.row_elems;
  for (int e = blockIdx.x * NT + threadIdx.x; e < total; e += gridDim.x * NT) {
    const int64_t off = (int64_t)e * 8;
    *reinterpret_cast<uint4 *>(kd + off) = *reinterpret_cast<const uint4 *>(kn + off);
    *reinterpret_cast<uint4 *>(vd + off) = *reinterpret_cast<const uint4 *>(vn + off);
  }
  for (int e = blockIdx.x * NT + threadIdx.x; e < a.C; e += gridDim.x * NT) {
    L.pos[cur][T0 + e] = a.pos[e];
    if (L.rpos[cur] != nullptr) L.rpos[cur][T0 + e] = a.rope_pos != nullptr ? a.rope_pos[e] : a.pos[e];
    if (L.rpos_h[cur] != nullptr) {   // M-RoPE: h and w beside t
      L.rpos_h[cur][T0 + e] = a.rope_h[e];
      L.rpos_w[cur][T0 + e] = a.rope_w[e];
    }
  }
}

__global__ __launch_bounds__(NT) void gather_rows(GatherArgs a) {
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const int rows = a.row_start[jj + 1] - a.row_start[jj];
  const int pieces = a.row_elems / 8;
  const int total = rows * pieces;
  const int32_t *kept = a.kept + l * a.kept_lstride;
  const uint16_t *ks = L.k[cur];
  const uint16_t *vs = L.v[cur];
  uint16_t *kd = L.k[cur ^ 1];
  uint16_t *vd = L.v[cur ^ 1];
  for (int e = blockIdx.x * NT + threadIdx.x; e < total; e += gridDim.x * NT) {
    const int row = e / pieces;
    const int c = e - row * pieces;
    const int src = min(max(kept[row], 0), L.cap - 1);   // indices are < T <= cap
    const int64_t so = (int64_t)src * a.row_elems + 8 * c;
    const int64_t dof = (int64_t)row * a.row_elems + 8 * c;
    const uint4 kx = *reinterpret_cast<const uint4 *>(ks + so);
    const uint4 vx = *reinterpret_cast<const uint4 *>(vs + so);
    *reinterpret_cast<uint4 *>(kd + dof) = kx;
    *reinterpret_cast<uint4 *>(vd + dof) = vx;
    if (c == 0) {
      L.pos[cur ^ 1][row] = L.pos[cur][src];
      if (L.rpos[cur] != nullptr) L.rpos[cur ^ 1][row] = L.rpos[cur][src];
      if (L.rpos_h[cur] != nullptr) {
        L.rpos_h[cur ^ 1][row] = L.rpos_h[cur][src];
        L.rpos_w[cur ^ 1][row] = L.rpos_w[cur][src];
      }
    }
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs &a, hipStream_t s) {
  const int pieces = a.row_elems / 8;
  const int blocks = (a.C * pieces + NT - 1) / NT;
  hipLaunchKernelGGL(append_rows, dim3(blocks, a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, hipStream_t s) {
  const int pieces = a.row_elems / 8;
  int max_rows = 0;
  for (int j = 0; j < a.n_list; ++j) max_rows = max(max_rows, a.row_start[j + 1] - a.row_start[j]);
  const int blocks = (max_rows * pieces + NT - 1) / NT;
  hipLaunchKernelGGL(gather_rows, dim3(blocks, a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace hermes
