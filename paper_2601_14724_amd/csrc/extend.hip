// Kernels of the parts adjacent to the streaming step, for gfx950:
//
// summary_partial / summary_finalize
//     the summary token of every evicting deep layer (Sec. 3.2 last
//     paragraph; appendix algorithm "Summary Token Aggregation"): V is the
//     mean of the evicted rows, K the mean of the evicted keys after each is
//     rotated from its RoPE position to t, the RoPE position of the newest
//     evicted token.  Sums run in fp64 in a fixed order (per block of
//     kSummaryRows candidates, then over blocks), so the result does not
//     depend on scheduling.
// reindex_decide
//     the lazy re-indexing trigger (Sec. 3.3): the largest RoPE position any
//     layer retains after this compression, against the limit.
// gather_rope
//     the order-preserving gather with the summary row inserted at its sorted
//     place and, when re-indexing applies, every key rotated by the change of
//     its RoPE position (appendix, 1D re-indexing: p_new = offset + rank,
//     k_new = k_old * e^{i (p_new - p_old) theta}); layers that did not evict
//     are re-indexed in place.
//
// RoPE layout: rotate-half, channel j pairs with j + d/2 inside each head,
// theta_j = base^(-2j/d).  Angles, sines, cosines and rotations are fp64; a
// stored key is rounded fp64 -> fp32 -> bf16.  With d/2 dividing 64, lane l of
// a wave always handles frequency l % (d/2), so each lane evaluates one
// sine/cosine per row and reuses it for every KV head.
#include <climits>

#include "hermes_internal.h"

namespace hermes {
namespace {

constexpr int NT = 256;
constexpr int kMaxPairSlots = 8;   // Hkv * d / 2 <= 64 * 8 rotate pairs per row

__device__ __forceinline__ double bf16_to_f64(uint16_t b) {
  return (double)__builtin_bit_cast(float, (uint32_t)b << 16);
}

__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>((float)x));
}

// theta_j = base^(-2j/d), as (-2j)/d in double.
__device__ __forceinline__ double inv_freq(int j, int d, double base) {
  return pow(base, (-2.0 * (double)j) / (double)d);
}

// Index f of the first kept entry of the "tight" suffix kept[j] = T - M + j
// (the newest candidates all kept); the newest evicted candidate is
// T - M + f - 1 and exactly f kept entries precede it.  Tightness is closed
// upwards, so a binary search finds f.  Requires T > M.
__device__ int first_tight(const int32_t *kept, int T, int M) {
  int lo = 0, hi = M;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (kept[mid] == T - M + mid) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

__device__ int lower_bound(const int32_t *a, int n, int x) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// summary token: per-block fp64 sums of the evicted rows
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(NT) void summary_partial(SummaryArgs a) {
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const int T = a.len[jj], M = a.budget[jj];
  const int r0 = blockIdx.x * kSummaryRows;
  if (r0 >= T) return;
  const int r1 = min(T, r0 + kSummaryRows);
  const int32_t *kept = a.kept + l * a.kept_lstride;
  const int32_t *rpos = L.rpos[cur];
  const uint16_t *K = L.k[cur];
  const uint16_t *V = L.v[cur];
  const int RE = a.row_elems, d = a.head_dim, hd = d / 2;
  const int npairs = RE / 2;

  __shared__ int s_t, s_k0, s_k1;
  __shared__ uint8_t is_kept[kSummaryRows];
  __shared__ double red[4][2 * 64 * kMaxPairSlots * 2];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid == 0) {
    const int f = first_tight(kept, T, M);
    s_t = rpos[T - M + f - 1];
    s_k0 = lower_bound(kept, M, r0);
    s_k1 = lower_bound(kept, M, r1);
  }
  for (int i = tid; i < kSummaryRows; i += NT) is_kept[i] = 0;
  __syncthreads();
  for (int i = s_k0 + tid; i < s_k1; i += NT) is_kept[kept[i] - r0] = 1;
  __syncthreads();
  const int t = s_t;

  const double invf = inv_freq(lane % hd, d, a.theta);
  double ak[kMaxPairSlots][2], av[kMaxPairSlots][2];
#pragma unroll
  for (int q = 0; q < kMaxPairSlots; ++q) ak[q][0] = ak[q][1] = av[q][0] = av[q][1] = 0.0;
  for (int i = r0 + wave; i < r1; i += 4) {
    if (is_kept[i - r0]) continue;
    const double ang = (double)(t - rpos[i]) * invf;
    double sn, cs;
    sincos(ang, &sn, &cs);
    const uint16_t *kr = K + (int64_t)i * RE;
    const uint16_t *vr = V + (int64_t)i * RE;
#pragma unroll
    for (int q = 0; q < kMaxPairSlots; ++q) {
      const int p = lane + 64 * q;
      if (p >= npairs) break;
      const int e1 = (p / hd) * d + (p % hd), e2 = e1 + hd;
      const double x1 = bf16_to_f64(kr[e1]), x2 = bf16_to_f64(kr[e2]);
      ak[q][0] += x1 * cs - x2 * sn;
      ak[q][1] += x2 * cs + x1 * sn;
      av[q][0] += bf16_to_f64(vr[e1]);
      av[q][1] += bf16_to_f64(vr[e2]);
    }
  }
  // waves combine in a fixed order: element e of K at [e], of V at [RE + e]
#pragma unroll
  for (int q = 0; q < kMaxPairSlots; ++q) {
    const int p = lane + 64 * q;
    if (p >= npairs) break;
    const int e1 = (p / hd) * d + (p % hd), e2 = e1 + hd;
    red[wave][e1] = ak[q][0];
    red[wave][e2] = ak[q][1];
    red[wave][RE + e1] = av[q][0];
    red[wave][RE + e2] = av[q][1];
  }
  __syncthreads();
  double *out = a.part + l * a.part_lstride + (int64_t)blockIdx.x * 2 * RE;
  for (int e = tid; e < 2 * RE; e += NT) out[e] = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
}

// Mean over the blocks in block order, rounded to bf16, plus the summary's
// insert index, stream position and RoPE position.
__global__ __launch_bounds__(NT) void summary_finalize(SummaryArgs a) {
  const int jj = blockIdx.x;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const int T = a.len[jj], M = a.budget[jj];
  const int RE = a.row_elems;
  const int nb = (T + kSummaryRows - 1) / kSummaryRows;
  const double inv_e = 1.0 / (double)(T - M);
  const double *part = a.part + l * a.part_lstride;
  for (int e = threadIdx.x; e < 2 * RE; e += NT) {
    double s = 0.0;
    for (int b = 0; b < nb; ++b) s += part[(int64_t)b * 2 * RE + e];
    const uint16_t x = f64_to_bf16(s * inv_e);
    if (e < RE) a.sum_k[(int64_t)l * RE + e] = x;
    else a.sum_v[(int64_t)l * RE + e - RE] = x;
  }
  if (threadIdx.x == 0) {
    const int32_t *kept = a.kept + l * a.kept_lstride;
    const int f = first_tight(kept, T, M);
    const int newest = T - M + f - 1;
    int32_t *meta = a.sum_meta + 4 * l;
    meta[0] = f;                       // kept entries before it
    meta[1] = L.pos[cur][newest];
    meta[2] = L.rpos[cur][newest];
    meta[3] = T - M;                   // tokens folded in
  }
}

// ---------------------------------------------------------------------------
// lazy re-indexing decision
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(64) void reindex_decide(DecideArgs a) {
  const int l = threadIdx.x;
  long long r = LLONG_MIN;
  if (l < a.n_layers) {
    const LayerTable &L = a.tab[l];
    const int32_t *rp = L.rpos[a.cur[l]];
    if (a.evicts[l]) {
      r = rp[a.kept[l * a.kept_lstride + a.budget[l] - 1]];
      if (a.has_sum[l] && (long long)a.sum_meta[4 * l + 2] > r) r = a.sum_meta[4 * l + 2];
    } else if (a.len[l] > 0) {
      r = rp[a.len[l] - 1];
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const long long x = __shfl_xor(r, o);
    r = x > r ? x : r;
  }
  if (l == 0) a.flag[0] = (r != LLONG_MIN && r + (long long)a.headroom >= (long long)a.limit) ? 1 : 0;
}

// ---------------------------------------------------------------------------
// gather with summary insertion and re-indexing: one wave per output row
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(NT) void gather_rope(GatherArgs a) {
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const bool inplace = a.mode[jj] != 0;
  const int dst_buf = inplace ? cur : cur ^ 1;
  const int rows = a.row_start[jj + 1] - a.row_start[jj];
  const int RE = a.row_elems, d = a.head_dim, hd = d / 2;
  const int npairs = RE / 2, pieces = RE / 8;
  const bool rot = a.reindex == 1 || (a.reindex == 2 && a.flag[0] != 0);
  if (inplace && !rot) return;
  const bool has_sum = a.has_sum[jj] != 0;
  const int ins = has_sum ? a.sum_meta[4 * l] : -1;
  const int32_t *kept = a.kept + l * a.kept_lstride;
  const uint16_t *Ks = L.k[cur], *Vs = L.v[cur];
  uint16_t *Kd = L.k[dst_buf], *Vd = L.v[dst_buf];
  const int32_t *Ps = L.pos[cur], *Rs = L.rpos[cur];
  int32_t *Pd = L.pos[dst_buf], *Rd = L.rpos[dst_buf];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const double invf = inv_freq(lane % hd, d, a.theta);

  for (int j = blockIdx.x * 4 + wave; j < rows; j += gridDim.x * 4) {
    // source of output row j
    const bool is_sum = has_sum && j == ins;
    const uint16_t *kr, *vr;
    int p_src, r_src;
    if (inplace) {
      kr = Ks + (int64_t)j * RE;
      vr = nullptr;
      p_src = Ps[j];
      r_src = Rs[j];
    } else if (is_sum) {
      kr = a.sum_k + (int64_t)l * RE;
      vr = a.sum_v + (int64_t)l * RE;
      p_src = a.sum_meta[4 * l + 1];
      r_src = a.sum_meta[4 * l + 2];
    } else {
      const int src = min(max(kept[j - (has_sum && j > ins ? 1 : 0)], 0), L.cap - 1);
      kr = Ks + (int64_t)src * RE;
      vr = Vs + (int64_t)src * RE;
      p_src = Ps[src];
      r_src = Rs[src];
    }
    const int r_new = rot ? a.rope_offset + j : r_src;
    const int delta = r_new - r_src;
    uint16_t *kd = Kd + (int64_t)j * RE;
    if (delta != 0) {
      double sn, cs;
      sincos((double)delta * invf, &sn, &cs);
#pragma unroll
      for (int q = 0; q < kMaxPairSlots; ++q) {
        const int p = lane + 64 * q;
        if (p >= npairs) break;
        const int e1 = (p / hd) * d + (p % hd), e2 = e1 + hd;
        const double x1 = bf16_to_f64(kr[e1]), x2 = bf16_to_f64(kr[e2]);
        const uint16_t y1 = f64_to_bf16(x1 * cs - x2 * sn);
        const uint16_t y2 = f64_to_bf16(x2 * cs + x1 * sn);
        kd[e1] = y1;
        kd[e2] = y2;
      }
    } else if (!inplace) {
      for (int c = lane; c < pieces; c += 64)
        *reinterpret_cast<uint4 *>(kd + 8 * c) = *reinterpret_cast<const uint4 *>(kr + 8 * c);
    }
    if (!inplace) {
      uint16_t *vd = Vd + (int64_t)j * RE;
      for (int c = lane; c < pieces; c += 64)
        *reinterpret_cast<uint4 *>(vd + 8 * c) = *reinterpret_cast<const uint4 *>(vr + 8 * c);
      if (lane == 0) Pd[j] = p_src;
    }
    if (lane == 0) Rd[j] = r_new;
  }
}

}  // namespace

hipError_t launch_summary(const SummaryArgs &a, int max_T, hipStream_t s) {
  const int nb = (max_T + kSummaryRows - 1) / kSummaryRows;
  hipLaunchKernelGGL(summary_partial, dim3(nb, a.n_list), dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(summary_finalize, dim3(a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_decide(const DecideArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(reindex_decide, dim3(1), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_rope(const GatherArgs &a, hipStream_t s) {
  int max_rows = 0;
  for (int j = 0; j < a.n_list; ++j) max_rows = max(max_rows, a.row_start[j + 1] - a.row_start[j]);
  const int blocks = min((max_rows + 3) / 4, 2048);
  hipLaunchKernelGGL(gather_rope, dim3(max(blocks, 1), a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace hermes
