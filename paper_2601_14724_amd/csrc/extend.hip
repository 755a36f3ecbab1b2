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
// reindex_decide3 / mrope_rank
//     the same trigger over the t, h and w coordinates, and the per-axis
//     ranks of 3D M-RoPE re-indexing (appendix, Qwen2.5-VL): on each axis a
//     retained coordinate becomes offset + the number of distinct retained
//     coordinates below it (one workgroup per layer and axis, an LDS bitmap
//     of the coordinates and a prefix of its word popcounts);
// gather_rope
//     the order-preserving gather with the summary row inserted at its sorted
//     place and, when re-indexing applies, every key rotated by the change of
//     its RoPE position (appendix, 1D re-indexing: p_new = offset + rank,
//     k_new = k_old * e^{i (p_new - p_old) theta}); layers that did not evict
//     are re-indexed in place.  With M-RoPE the frequency pairs of a key are
//     split into t, h and w sections, and the pairs of each section turn by
//     the change of that section's coordinate.
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
// Rows of the summary and re-indexing kernels hold at most 1024 elements
// (Hkv * d <= 1024, checked by the host): at most two 16-byte pieces per lane.

__device__ __forceinline__ double bf16_to_f64(uint16_t b) {
  return (double)__builtin_bit_cast(float, (uint32_t)b << 16);
}

// fp64 -> fp32 (round to nearest even), then fp32 -> bf16 (round to nearest
// even) on the bits.  Written as two conversions, the compiler folds them
// into one rounding straight from fp64 (fp32 rounded to odd, then to bf16),
// which differs wherever the fp32 value lands on a bf16 midpoint.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, (float)x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// bf16 element i of a 16-byte piece
__device__ __forceinline__ uint16_t half16(const uint4 &v, int i) {
  const uint32_t w = (i >> 1) == 0 ? v.x : (i >> 1) == 1 ? v.y : (i >> 1) == 2 ? v.z : v.w;
  return (uint16_t)((i & 1) ? (w >> 16) : (w & 0xFFFFu));
}

__device__ __forceinline__ uint4 shfl_xor4(uint4 v, int m) {
  return uint4{(uint32_t)__shfl_xor((int)v.x, m), (uint32_t)__shfl_xor((int)v.y, m),
               (uint32_t)__shfl_xor((int)v.z, m), (uint32_t)__shfl_xor((int)v.w, m)};
}

// The first index in [0, n) where the monotone predicate (false, then true)
// holds, or n; searched by one whole wave.  Each round the 64 lanes probe 64
// evenly spaced points of the open interval and a ballot picks the segment,
// so n entries take about log64(n) dependent loads instead of log2(n).
// Invariant: the answer lies in [lo, hi], and hi is n or a known true index
// (probes at or beyond hi count as true).
template <class Pred>
__device__ int wave_search(int n, Pred pred) {
  const int lane = threadIdx.x & 63;
  int lo = 0, hi = n;
  while (lo < hi) {
    const int step = (hi - lo + 63) / 64;
    const int p = lo + (lane + 1) * step - 1;
    const unsigned long long m = __ballot(p >= hi || pred(p));
    if (m == 0ull) {
      lo = hi;
    } else {
      const int k = __builtin_ctzll(m);
      const int pk = lo + (k + 1) * step - 1;
      lo += k * step;
      hi = min(hi, pk);
    }
  }
  return lo;
}

// ---------------------------------------------------------------------------
// summary token: per-block fp64 sums of the evicted rows
// ---------------------------------------------------------------------------

// PG: 16-byte pieces per lane (the row has at most 64 * PG pieces).
template <int PG>
__global__ __launch_bounds__(NT) void summary_partial(SummaryArgs a) {
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const int T = a.len[jj], M = a.budget[jj];
  const int r0 = blockIdx.x * kSummaryRows;
  if (r0 >= T || a.row_elems / 8 > 64 * PG) return;
  const int r1 = min(T, r0 + kSummaryRows);
  const int32_t *kept = a.kept + l * a.kept_lstride;
  const int32_t *rpos = L.rpos[cur];
  const uint16_t *K = L.k[cur];
  const uint16_t *V = L.v[cur];
  const int RE = a.row_elems, d = a.head_dim, hd = d / 2;

  __shared__ int s_t, s_h, s_w, s_k0, s_k1;
  __shared__ uint8_t is_kept[kSummaryRows];
  __shared__ double red[4][2 * 64 * 8 * PG];
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  // Three wave-parallel searches of the kept list, one per wave.  The tight
  // suffix kept[j] = T - M + j (the newest candidates, all kept) starts at f,
  // so the newest evicted candidate is T - M + f - 1; tightness holds from f
  // on (kept is strictly increasing and kept[j] <= T - M + j), which makes it
  // a monotone predicate.
  if (wave == 0) {
    const int f = wave_search(M, [&](int j) { return kept[j] == T - M + j; });
    if (lane == 0) {
      const int newest = T - M + f - 1;
      s_t = rpos[newest];
      s_h = a.axes == 3 ? L.rpos_h[cur][newest] : 0;
      s_w = a.axes == 3 ? L.rpos_w[cur][newest] : 0;
    }
  } else if (wave == 1) {
    const int k0 = wave_search(M, [&](int j) { return kept[j] >= r0; });
    if (lane == 0) s_k0 = k0;
  } else if (wave == 2) {
    const int k1 = wave_search(M, [&](int j) { return kept[j] >= r1; });
    if (lane == 0) s_k1 = k1;
  }
  for (int i = tid; i < kSummaryRows; i += NT) is_kept[i] = 0;
  __syncthreads();
  for (int i = s_k0 + tid; i < s_k1; i += NT) is_kept[kept[i] - r0] = 1;
  __syncthreads();
  const int t = s_t, th = s_h, tw = s_w;

  // Lane c sums the 16-byte pieces c and c + 64 of the evicted rows' K
  // (turned to t; with M-RoPE each frequency pair by the change of its
  // section's coordinate, to the target's (t, h, w)) and V, in row order; the turn uses the pair partner from
  // the lane whose piece index differs in bit d/16 and one fp64 sine/cosine
  // per lane and row (lane f evaluates frequency f % (d/2)), shared through
  // LDS.  Four rows are loaded before the first is summed.
  constexpr int RW = 4;
  const int pieces = RE / 8;
  const int fj = lane % hd;
  const double invf = a.inv_freq[fj];
  const int pm = d / 16;
  const int f0 = 8 * (lane % pm);
  const bool second = (lane & pm) != 0;
  const bool three = a.axes == 3;
  const int my_axis = !three ? 0 : fj < a.section[0] ? 0 : fj < a.section[0] + a.section[1] ? 1 : 2;
  const int32_t *rph = three ? L.rpos_h[cur] : nullptr, *rpw = three ? L.rpos_w[cur] : nullptr;
  __shared__ double2 trig[NT / 64][64];
  double ak[PG][8], av[PG][8];
#pragma unroll
  for (int g = 0; g < PG; ++g)
#pragma unroll
    for (int i = 0; i < 8; ++i) ak[g][i] = av[g][i] = 0.0;
  for (int i0 = r0 + wave; i0 < r1; i0 += 4 * RW) {
    uint4 kx[RW][PG], vx[RW][PG];
    bool ev[RW];
#pragma unroll
    for (int u = 0; u < RW; ++u) {
      const int i = i0 + 4 * u;
      ev[u] = i < r1 && !is_kept[i - r0];
#pragma unroll
      for (int g = 0; g < PG; ++g) {
        const int c = lane + 64 * g;
        kx[u][g] = vx[u][g] = uint4{0u, 0u, 0u, 0u};
        if (ev[u] && c < pieces) {
          kx[u][g] = *reinterpret_cast<const uint4 *>(K + (int64_t)i * RE + 8 * c);
          vx[u][g] = *reinterpret_cast<const uint4 *>(V + (int64_t)i * RE + 8 * c);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < RW; ++u) {
      if (!ev[u]) continue;   // uniform over the wave (one row)
      const int i = i0 + 4 * u;
      const int delta = my_axis == 0 ? t - rpos[i] : my_axis == 1 ? th - rph[i] : tw - rpw[i];
      double sn, cs;
      sincos((double)delta * invf, &sn, &cs);
      trig[wave][lane] = double2{cs, sn};
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
#pragma unroll
      for (int g = 0; g < PG; ++g) {
        const uint4 px = shfl_xor4(kx[u][g], pm);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const double2 tr = trig[wave][f0 + e];
          const double x = bf16_to_f64(half16(kx[u][g], e)), y = bf16_to_f64(half16(px, e));
          // first half of a pair: x cos - y sin; second half: x cos + y sin
          ak[g][e] += second ? x * tr.x + y * tr.y : x * tr.x - y * tr.y;
          av[g][e] += bf16_to_f64(half16(vx[u][g], e));
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
  }
  // waves combine in a fixed order: element e of K at [e], of V at [RE + e]
#pragma unroll
  for (int g = 0; g < PG; ++g) {
    const int c = lane + 64 * g;
    if (c < pieces) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        red[wave][8 * c + e] = ak[g][e];
        red[wave][RE + 8 * c + e] = av[g][e];
      }
    }
  }
  __syncthreads();
  double *out = a.part + l * a.part_lstride + (int64_t)blockIdx.x * 2 * RE;
  for (int e = tid; e < 2 * RE; e += NT) out[e] = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
}

// Mean over the blocks in block order, rounded to bf16, plus the summary's
// insert index, stream position and RoPE position.
__global__ __launch_bounds__(NT) void summary_finalize(SummaryArgs a) {
  // grid (element blocks, layers): thread e sums element e over the blocks
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const int T = a.len[jj], M = a.budget[jj];
  const int RE = a.row_elems;
  const int nb = (T + kSummaryRows - 1) / kSummaryRows;
  const double inv_e = 1.0 / (double)(T - M);
  const double *part = a.part + l * a.part_lstride;
  const int e = blockIdx.x * NT + threadIdx.x;
  if (e < 2 * RE) {
    // eight loads in flight, then their sums in block order
    double s = 0.0;
    for (int b0 = 0; b0 < nb; b0 += 8) {
      double x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = b0 + u < nb ? part[(int64_t)(b0 + u) * 2 * RE + e] : 0.0;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (b0 + u < nb) s += x[u];
    }
    const uint16_t x = f64_to_bf16(s * inv_e);
    if (e < RE) a.sum_k[(int64_t)l * RE + e] = x;
    else a.sum_v[(int64_t)l * RE + e - RE] = x;
  }
  if (blockIdx.x == 0 && threadIdx.x < 64) {
    const int32_t *kept = a.kept + l * a.kept_lstride;
    const int f = wave_search(M, [&](int j) { return kept[j] == T - M + j; });
    if (threadIdx.x == 0) {
      const int newest = T - M + f - 1;
      int32_t *meta = a.sum_meta + kSumMeta * l;
      meta[0] = f;                       // kept entries before it
      meta[1] = L.pos[cur][newest];
      meta[2] = L.rpos[cur][newest];
      meta[3] = T - M;                   // tokens folded in
      if (a.axes == 3) {
        meta[4] = L.rpos_h[cur][newest];
        meta[5] = L.rpos_w[cur][newest];
      }
    }
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
      if (a.has_sum[l] && (long long)a.sum_meta[kSumMeta * l + 2] > r) r = a.sum_meta[kSumMeta * l + 2];
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

// Lazy trigger with M-RoPE: the largest retained coordinate on any axis of
// any layer (h and w are not monotone along the cache, so every retained row
// is read).
constexpr int RT = 1024;
__global__ __launch_bounds__(RT) void reindex_decide3(DecideArgs a) {
  long long r = LLONG_MIN;
  for (int l = 0; l < a.n_layers; ++l) {
    const LayerTable &L = a.tab[l];
    const int c = a.cur[l];
    const int rows = a.evicts[l] ? a.budget[l] : a.len[l];
    const int32_t *kept = a.kept + l * a.kept_lstride;
    for (int i = threadIdx.x; i < rows; i += RT) {
      const int src = a.evicts[l] ? min(max(kept[i], 0), L.cap - 1) : i;
      const long long m = max(L.rpos[c][src], max(L.rpos_h[c][src], L.rpos_w[c][src]));
      r = m > r ? m : r;
    }
    if (a.evicts[l] && a.has_sum[l] && threadIdx.x == 0) {   // the summary's (t, h, w)
      const int32_t *meta = a.sum_meta + kSumMeta * l;
      const long long m = max(meta[2], max(meta[4], meta[5]));
      r = m > r ? m : r;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const long long x = __shfl_xor(r, o);
    r = x > r ? x : r;
  }
  __shared__ long long wm[RT / 64];
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = r;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 0; w < RT / 64; ++w) r = wm[w] > r ? wm[w] : r;
    a.flag[0] = (r != LLONG_MIN && r + (long long)a.headroom >= (long long)a.limit) ? 1 : 0;
  }
}

// Distinct-rank compaction of one axis of one layer's retained coordinates.
constexpr int kSpanWords = kMropeWindow / 32;
__global__ __launch_bounds__(RT) void mrope_rank(RankArgs a) {
  const int jj = blockIdx.x, axis = blockIdx.y;
  const bool rot = a.reindex == 1 || (a.reindex == 2 && a.flag[0] != 0);
  if (!rot) return;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const bool inplace = a.mode[jj] != 0;
  const int rows = a.row_start[jj + 1] - a.row_start[jj];
  if (rows <= 0) return;
  const int32_t *C = axis == 0 ? L.rpos[cur] : axis == 1 ? L.rpos_h[cur] : L.rpos_w[cur];
  const int32_t *kept = a.kept + l * a.kept_lstride;
  int32_t *out = a.newc + (int64_t)(l * 3 + axis) * a.newc_lstride;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // output row r of an evicting layer with a summary: kept rows before the
  // summary's insert index, the summary, then the rest of the kept rows
  const bool has_sum = !inplace && a.has_sum[jj] != 0;
  const int32_t *meta = a.sum_meta + kSumMeta * l;
  const int ins = has_sum ? meta[0] : -1;
  const int sum_c = has_sum ? meta[axis == 0 ? 2 : axis == 1 ? 4 : 5] : 0;
  auto coord = [&](int r) {
    if (inplace) return C[r];
    if (r == ins) return sum_c;
    return C[min(max(kept[r - (has_sum && r > ins ? 1 : 0)], 0), L.cap - 1)];
  };

  __shared__ uint32_t bits[kSpanWords];
  __shared__ uint32_t wpre[kSpanWords];
  __shared__ int red[2][RT / 64];
  __shared__ long long rnext[RT / 64];
  __shared__ uint32_t wsum[RT / 64];
  // min and max of the retained coordinates
  int mn = INT_MAX, mx = INT_MIN;
  for (int r = tid; r < rows; r += RT) {
    const int c = coord(r);
    mn = min(mn, c);
    mx = max(mx, c);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mn = min(mn, __shfl_xor(mn, o));
    mx = max(mx, __shfl_xor(mx, o));
  }
  if (lane == 0) {
    red[0][wv] = mn;
    red[1][wv] = mx;
  }
  __syncthreads();
  for (int w = 0; w < RT / 64; ++w) {
    mn = min(mn, red[0][w]);
    mx = max(mx, red[1][w]);
  }
  // The ranks are counted window by window: each pass marks the retained
  // coordinates in [lo, lo + span) in the LDS bitmap, ranks the rows whose
  // coordinate falls there after the `below` distinct coordinates of the
  // earlier windows, and moves lo to the smallest coordinate past the window
  // (so empty stretches of a wide axis cost nothing).  Axes narrower than the
  // bitmap take one pass.
  constexpr long long kSpan = kMropeWindow;
  long long lo = mn;
  uint32_t below = 0;
  for (;;) {
    const long long hi_ex = lo + kSpan;   // window [lo, hi_ex)
    const long long top = (long long)mx + 1 < hi_ex ? (long long)mx + 1 : hi_ex;
    const int nwords = (int)((top - lo + 31) / 32);
    for (int w = tid; w < nwords; w += RT) bits[w] = 0u;
    __syncthreads();
    for (int r = tid; r < rows; r += RT) {
      const long long c = (long long)coord(r) - lo;
      if (c >= 0 && c < top - lo) atomicOr(&bits[c >> 5], 1u << (c & 31));
    }
    __syncthreads();
    // exclusive prefix of the word popcounts: thread t owns words [8t, 8t + 8)
    constexpr int WPT = kSpanWords / RT;
    uint32_t own = 0;
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int w = tid * WPT + u;
      own += w < nwords ? (uint32_t)__popc(bits[w]) : 0u;
    }
    uint32_t inc = own;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t x = __shfl_up(inc, o);
      if (lane >= o) inc += x;
    }
    if (lane == 63) wsum[wv] = inc;
    __syncthreads();
    uint32_t base = inc - own, total = 0;
    for (int w = 0; w < RT / 64; ++w) {
      base += w < wv ? wsum[w] : 0u;
      total += wsum[w];
    }
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int w = tid * WPT + u;
      if (w < nwords) {
        wpre[w] = base;
        base += (uint32_t)__popc(bits[w]);
      }
    }
    __syncthreads();
    // ranks of this window's rows, and the first coordinate past it
    long long nxt = LLONG_MAX;
    for (int r = tid; r < rows; r += RT) {
      const int cr = coord(r);
      const long long c = (long long)cr - lo;
      if (c >= 0 && c < top - lo) {
        const int w = (int)(c >> 5), b = (int)(c & 31);
        out[r] = a.offset + (int)(below + wpre[w] + (uint32_t)__popc(bits[w] & ((1u << b) - 1u)));
      } else if (c >= top - lo) {
        nxt = min(nxt, (long long)cr);
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const long long x = __shfl_xor(nxt, o);
      nxt = x < nxt ? x : nxt;
    }
    if (lane == 0) rnext[wv] = nxt;
    __syncthreads();
    for (int w = 0; w < RT / 64; ++w) nxt = rnext[w] < nxt ? rnext[w] : nxt;
    below += total;
    if (nxt == LLONG_MAX) break;   // uniform: every thread read the same rnext
    lo = nxt;
    __syncthreads();   // rnext, bits and wpre are rewritten by the next pass
  }
}

// ---------------------------------------------------------------------------
// gather with summary insertion and re-indexing: one wave per output row
// ---------------------------------------------------------------------------

// 16-byte pieces of a row held by one lane: piece lane + 64 g for g < PG.
template <int PG>
__global__ __launch_bounds__(NT) void gather_rope(GatherArgs a) {
  constexpr int RW = 4;   // rows per wave whose loads are all issued before the first is computed
  const int jj = blockIdx.y;
  const int l = a.layer_id[jj];
  const LayerTable &L = a.tab[l];
  const int cur = a.cur[jj];
  const bool inplace = a.mode[jj] != 0;
  const int dst_buf = inplace ? cur : cur ^ 1;
  const int rows = a.row_start[jj + 1] - a.row_start[jj];
  const int RE = a.row_elems, d = a.head_dim, hd = d / 2;
  const int pieces = RE / 8;
  const bool rot = a.reindex == 1 || (a.reindex == 2 && a.flag[0] != 0);
  if ((inplace && !rot) || pieces > 64 * PG) return;
  const bool has_sum = a.has_sum[jj] != 0;
  const int ins = has_sum ? a.sum_meta[kSumMeta * l] : -1;
  const int32_t *kept = a.kept + l * a.kept_lstride;
  const uint16_t *Ks = L.k[cur], *Vs = L.v[cur];
  uint16_t *Kd = L.k[dst_buf], *Vd = L.v[dst_buf];
  const int32_t *Ps = L.pos[cur], *Rs = L.rpos[cur];
  int32_t *Pd = L.pos[dst_buf], *Rd = L.rpos[dst_buf];
  // wave-uniform values are moved to scalar registers (readfirstlane)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  // Lane f evaluates frequency f % (d/2); the lane holding piece c needs the
  // 8 frequencies from 8 (c % (d/16)) on, and the other half of each of its
  // pairs sits in piece c ^ (d/16), held by lane lane ^ (d/16).
  const int fj = lane % hd;
  const double invf = a.inv_freq[fj];
  const int pm = d / 16;
  const int f0 = 8 * (lane % pm);
  const bool second = (lane & pm) != 0;
  // M-RoPE: the section (0 = t, 1 = h, 2 = w) of this lane's frequency
  const bool three = a.axes == 3;
  const int my_axis = fj < a.section[0] ? 0 : fj < a.section[0] + a.section[1] ? 1 : 2;
  const int32_t *Hs = three ? L.rpos_h[cur] : nullptr, *Ws = three ? L.rpos_w[cur] : nullptr;
  int32_t *Hd = three ? L.rpos_h[dst_buf] : nullptr, *Wd = three ? L.rpos_w[dst_buf] : nullptr;
  const int32_t *nc = three ? a.newc + (int64_t)l * 3 * a.newc_lstride : nullptr;
  __shared__ double2 trig[NT / 64][64];   // (cos, sin) by frequency, one row per wave

  const int stride = gridDim.x * (NT / 64);
  for (int j0 = blockIdx.x * (NT / 64) + wave; j0 < rows; j0 += stride * RW) {
    // sources of this wave's rows j0 + u * stride (every value is wave-uniform)
    const uint16_t *kr[RW], *vr[RW];
    int src[RW], p_src[RW], r_src[RW];
    int h_old[RW], w_old[RW], c_new[RW][3];   // M-RoPE coordinates before / after
#pragma unroll
    for (int u = 0; u < RW; ++u) {
      const int j = min(j0 + u * stride, rows - 1);
      if (inplace) {
        kr[u] = Kd + (int64_t)j * RE;
        vr[u] = nullptr;
        src[u] = j;
        p_src[u] = 0;
        r_src[u] = __builtin_amdgcn_readfirstlane(Rs[j]);
      } else if (has_sum && j == ins) {
        kr[u] = a.sum_k + (int64_t)l * RE;
        vr[u] = a.sum_v + (int64_t)l * RE;
        src[u] = -1;
        p_src[u] = a.sum_meta[kSumMeta * l + 1];
        r_src[u] = a.sum_meta[kSumMeta * l + 2];
      } else {
        src[u] = __builtin_amdgcn_readfirstlane(
            min(max(kept[j - (has_sum && j > ins ? 1 : 0)], 0), L.cap - 1));
        kr[u] = Ks + (int64_t)src[u] * RE;
        vr[u] = Vs + (int64_t)src[u] * RE;
        p_src[u] = __builtin_amdgcn_readfirstlane(Ps[src[u]]);
        r_src[u] = __builtin_amdgcn_readfirstlane(Rs[src[u]]);
      }
      h_old[u] = w_old[u] = c_new[u][0] = c_new[u][1] = c_new[u][2] = 0;
      if (three) {   // the summary row carries the target's (t, h, w)
        h_old[u] = src[u] < 0 ? a.sum_meta[kSumMeta * l + 4] : __builtin_amdgcn_readfirstlane(Hs[src[u]]);
        w_old[u] = src[u] < 0 ? a.sum_meta[kSumMeta * l + 5] : __builtin_amdgcn_readfirstlane(Ws[src[u]]);
#pragma unroll
        for (int x = 0; x < 3; ++x)
          c_new[u][x] = __builtin_amdgcn_readfirstlane(nc[x * a.newc_lstride + j]);
      }
    }
    uint4 kx[RW][PG], vx[RW][PG];
#pragma unroll
    for (int u = 0; u < RW; ++u) {
#pragma unroll
      for (int g = 0; g < PG; ++g) {
        const int c = lane + 64 * g;
        kx[u][g] = vx[u][g] = uint4{0u, 0u, 0u, 0u};
        if (c < pieces) {
          kx[u][g] = *reinterpret_cast<const uint4 *>(kr[u] + 8 * c);
          if (!inplace) vx[u][g] = *reinterpret_cast<const uint4 *>(vr[u] + 8 * c);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < RW; ++u) {
      const int j = j0 + u * stride;
      if (j >= rows) break;
      int r_new = rot ? a.rope_offset + j : r_src[u];
      int delta = r_new - r_src[u];
      int h_new = 0, w_new = 0;
      if (three) {
        r_new = rot ? c_new[u][0] : r_src[u];
        h_new = rot ? c_new[u][1] : h_old[u];
        w_new = rot ? c_new[u][2] : w_old[u];
        delta = my_axis == 0 ? r_new - r_src[u] : my_axis == 1 ? h_new - h_old[u] : w_new - w_old[u];
      }
      uint4 out[PG];
#pragma unroll
      for (int g = 0; g < PG; ++g) out[g] = kx[u][g];
      if (__any(delta != 0)) {   // uniform over the wave (one row)
        double sn, cs;
        sincos((double)delta * invf, &sn, &cs);
        trig[wave][lane] = double2{cs, sn};
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
#pragma unroll
        for (int g = 0; g < PG; ++g) {
          const uint4 px = shfl_xor4(kx[u][g], pm);
          uint32_t w[4];
#pragma unroll
          for (int i = 0; i < 8; i += 2) {
            uint32_t h2 = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const double2 t = trig[wave][f0 + i + h];
              const double x = bf16_to_f64(half16(kx[u][g], i + h));
              const double y = bf16_to_f64(half16(px, i + h));
              // first half: x cos - y sin; second half: x cos + y sin
              // (y is the other half of the pair), products rounded apart
              const double xc = __dmul_rn(x, t.x), ys = __dmul_rn(y, t.y);
              h2 |= (uint32_t)f64_to_bf16(second ? __dadd_rn(xc, ys) : __dsub_rn(xc, ys)) << (16 * h);
            }
            w[i >> 1] = h2;
          }
          out[g] = uint4{w[0], w[1], w[2], w[3]};
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      }
      uint16_t *kd = Kd + (int64_t)j * RE;
      uint16_t *vd = Vd + (int64_t)j * RE;
#pragma unroll
      for (int g = 0; g < PG; ++g) {
        const int c = lane + 64 * g;
        if (c < pieces) {
          *reinterpret_cast<uint4 *>(kd + 8 * c) = out[g];
          if (!inplace) *reinterpret_cast<uint4 *>(vd + 8 * c) = vx[u][g];
        }
      }
      if (lane == 0) {
        if (!inplace) Pd[j] = p_src[u];
        Rd[j] = r_new;
        if (three) {
          Hd[j] = h_new;
          Wd[j] = w_new;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_summary(const SummaryArgs &a, int max_T, hipStream_t s) {
  const int nb = (max_T + kSummaryRows - 1) / kSummaryRows;
  if (a.row_elems / 8 <= 64)
    hipLaunchKernelGGL(summary_partial<1>, dim3(nb, a.n_list), dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL(summary_partial<2>, dim3(nb, a.n_list), dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(summary_finalize, dim3((2 * a.row_elems + NT - 1) / NT, a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_decide(const DecideArgs &a, hipStream_t s) {
  if (a.axes == 3) hipLaunchKernelGGL(reindex_decide3, dim3(1), dim3(RT), 0, s, a);
  else hipLaunchKernelGGL(reindex_decide, dim3(1), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mrope_rank(const RankArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(mrope_rank, dim3(a.n_list, 3), dim3(RT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_rope(const GatherArgs &a, hipStream_t s) {
  int max_rows = 0;
  for (int j = 0; j < a.n_list; ++j) max_rows = max(max_rows, a.row_start[j + 1] - a.row_start[j]);
  // four rows per wave, four waves per workgroup
  const int blocks = max(1, min((max_rows + 15) / 16, 1024));
  if (a.row_elems / 8 <= 64)
    hipLaunchKernelGGL(gather_rope<1>, dim3(blocks, a.n_list), dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL(gather_rope<2>, dim3(blocks, a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace hermes
