// Scoring, cross-layer smoothing and TopK selection for gfx950, in two
// launches over the layers over budget:
//   score_keys   importance S^l_i by class (Sec. 3.1): recency
//                R_i = e^{-k(T-1-i)}/Z (shallow), attention A_i = alpha_i W_i
//                normalised to sum 1 (deep), (1 - omega_l) A + omega_l R
//                (middle), in fp64, the normaliser of A summed from the fp64
//                partials the mass reduction wrote with W; one-hop smoothing
//                S~^l = (1 - lambda_l) S^l + lambda_l S^{l+1}_{j(i)}
//                (Sec. 3.2), the partner j(i) found on layer l+1's sorted
//                positions (or at the equal physical index); S~ rounded to
//                fp32, whose bit pattern is an order-preserving uint32 key
//                (several workgroups per layer);
//   select_kept  the budget-th largest key by an MSB-first radix select over
//                the bits below the prefix all keys share (LDS histograms,
//                keys in registers), ties at that key to the higher index,
//                the kept indices emitted in ascending order from one block
//                scan (one workgroup per layer).
#include "hermes_internal.h"
#include "score_terms.h"

namespace hermes {
namespace {

constexpr int NT = 1024;
constexpr int NW = NT / 64;

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int ln = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (ln >= o) v += u;
  }
  return v;
}

struct SelectShared {
  unsigned hist[2][256];      // double-buffered: the next pass's is cleared during this scan
  int digit[2], above[2];
  uint32_t kmin[NW], kmax[NW];
  unsigned long long wtot[NW];
};

// Block-wide min and max of the keys; on return sh.hist[0] is cleared and
// every thread holds both.  kmin / kmax come in as this thread's own.
__device__ __forceinline__ void block_minmax(uint32_t &kmin, uint32_t &kmax, SelectShared &sh) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o));
  }
  if (lane == 0) {
    sh.kmin[wv] = kmin;
    sh.kmax[wv] = kmax;
  }
  if (tid < 256) sh.hist[0][tid] = 0u;
  __syncthreads();
  for (int w = 0; w < NW; ++w) {
    kmin = min(kmin, sh.kmin[w]);
    kmax = max(kmax, sh.kmax[w]);
  }
}

// The M-th largest key (0 < M < number of keys) by an MSB-first radix
// select, 8 bits per pass and two barriers per pass, over the bits below
// the prefix every key shares (the leading digits of nearby fp32 scores are
// nearly all equal, and a histogram of equal digits serialises on one LDS
// address).  Needs block_minmax first.  hist(h, pmask, prefix, shift, dm)
// adds this thread's keys k with (k & pmask) == prefix to h[(k >> shift) &
// dm].  *want gets how many keys equal to the result are kept.
template <typename Hist>
__device__ __forceinline__ uint32_t radix_select(int M, uint32_t kmin, uint32_t kmax, SelectShared &sh,
                                                 int *want_out, Hist hist) {
  const int tid = threadIdx.x;
  int hi = kmin == kmax ? 0 : 32 - __clz(kmin ^ kmax);   // bits below the shared prefix
  uint32_t pmask = hi >= 32 ? 0u : 0xffffffffu << hi;
  uint32_t prefix = kmin & pmask;
  int want = M;
  for (int pass = 0; hi > 0; ++pass) {
    const int width = min(8, hi), shift = hi - width, hb = pass & 1;
    const uint32_t dm = (1u << width) - 1u;
    hist(sh.hist[hb], pmask, prefix, shift, dm);
    __syncthreads();
    if (tid < 64) {
      // lane owns digits 255-4t .. 252-4t, visited from high to low
      int cnt[4], loc = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cnt[e] = (int)sh.hist[hb][255 - 4 * tid - e];
        loc += cnt[e];
      }
      int acc = wave_incl_scan(loc) - loc;   // keys whose digit is above this lane's
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (acc < want && want <= acc + cnt[e]) {
          sh.digit[hb] = 255 - 4 * tid - e;
          sh.above[hb] = acc;
        }
        acc += cnt[e];
      }
    } else if (tid < 64 + 256) {
      sh.hist[hb ^ 1][tid - 64] = 0u;
    }
    __syncthreads();
    want -= sh.above[hb];
    prefix |= (uint32_t)sh.digit[hb] << shift;
    pmask |= dm << shift;
    hi = shift;
  }
  *want_out = want;
  return prefix;
}

// Radix select over keys[0..T) read from memory with unit stride.
template <typename KeyPtr>
__device__ __forceinline__ uint32_t radix_threshold(KeyPtr keys, int T, int M, uint32_t kmin, uint32_t kmax,
                                                    SelectShared &sh, int *want_out) {
  return radix_select(M, kmin, kmax, sh, want_out,
                      [&](unsigned *h, uint32_t pmask, uint32_t prefix, int shift, uint32_t dm) {
                        for (int i = threadIdx.x; i < T; i += NT) {
                          const uint32_t k = keys[i];
                          if ((k & pmask) == prefix) atomicAdd(&h[(k >> shift) & dm], 1u);
                        }
                      });
}

// Keys spread over the threads for the radix passes: lane l takes the
// segment [l*seg, (l+1)*seg) of an odd length seg, wave w its offsets w,
// w+NW, ...  A wave's 64 reads then fall in 64 different places of the key
// array (scores are correlated with their index, so neighbouring keys share
// digits) and in distinct LDS banks.  Needs seg <= SR * NW.
template <int SR>
__device__ __forceinline__ void load_spread(const uint32_t *keys, int T, uint32_t (&ks)[SR], uint32_t &valid) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int seg = ((T + 63) / 64) | 1;
  valid = 0u;
#pragma unroll
  for (int u = 0; u < SR; ++u) {
    const int c = wv + NW * u, i = lane * seg + c;
    const bool ok = c < seg && i < T;
    ks[u] = ok ? keys[i] : 0u;
    valid |= (ok ? 1u : 0u) << u;
  }
}

template <int SR>
__device__ __forceinline__ uint32_t radix_threshold_regs(const uint32_t (&ks)[SR], uint32_t valid, int M,
                                                         uint32_t kmin, uint32_t kmax, SelectShared &sh,
                                                         int *want_out) {
  return radix_select(M, kmin, kmax, sh, want_out,
                      [&](unsigned *h, uint32_t pmask, uint32_t prefix, int shift, uint32_t dm) {
#pragma unroll
                        for (int u = 0; u < SR; ++u)
                          if (((valid >> u) & 1u) && (ks[u] & pmask) == prefix)
                            atomicAdd(&h[(ks[u] >> shift) & dm], 1u);
                      });
}

// Output place of a contiguous run holding gt keys above the threshold and
// eq equal to it, when the `want` equal keys of highest index are kept: one
// block scan of the packed (gt, eq) pair.  *skip gets how many of the run's
// equal keys (its first ones) are dropped.
__device__ __forceinline__ int kept_offset(unsigned gt, unsigned eq, int want, SelectShared &sh, int *skip) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const unsigned long long mine = ((unsigned long long)gt << 32) | eq;
  unsigned long long inc = mine;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long x = __shfl_up(inc, o);
    if (lane >= o) inc += x;
  }
  if (lane == 63) sh.wtot[wv] = inc;
  __syncthreads();
  unsigned long long before = inc - mine, total = 0;
  for (int w = 0; w < NW; ++w) {
    const unsigned long long x = sh.wtot[w];
    before += w < wv ? x : 0ull;
    total += x;
  }
  const int eq_total = (int)(uint32_t)total;
  const int eq_before = (int)(uint32_t)before, gt_before = (int)(before >> 32);
  const int drop = eq_total - want;   // ties dropped: those of lowest index
  *skip = min((int)eq, max(0, drop - eq_before));
  return gt_before + max(0, eq_before - drop);
}

// Output of a contiguous run [a0, a1) whose keys are in kr: the indices of
// those above thr, and of its share of the `want` kept ties (the highest
// indices), ascending from the run's place in out (and out2 if non-null).
template <int FR>
__device__ __forceinline__ void emit_run(const uint32_t (&kr)[FR], int a0, int a1, uint32_t thr, int want,
                                         int M, int32_t *out, int32_t *out2, SelectShared &sh) {
  unsigned gt = 0, eq = 0;
#pragma unroll
  for (int u = 0; u < FR; ++u)
    if (a0 + u < a1) {
      gt += kr[u] > thr;
      eq += kr[u] == thr;
    }
  int skip;
  int off = kept_offset(gt, eq, want, sh, &skip);
#pragma unroll
  for (int u = 0; u < FR; ++u) {
    const int i = a0 + u;
    if (i >= a1) break;
    bool keep = kr[u] > thr;
    if (kr[u] == thr) {
      if (skip > 0) --skip;
      else keep = true;
    }
    if (keep && off < M) {   // off < M always holds; the guard keeps writes in bounds
      out[off] = i;
      if (out2 != nullptr) out2[off] = i;
      ++off;
    }
  }
}

// Keep the M largest of keys[0..T) (M < T), ties to the higher index; write
// the kept indices ascending to out (and out2 if non-null).  Thread t owns
// the contiguous run [a0, a1) for the output.
template <typename KeyPtr>
__device__ __forceinline__ void select_top(KeyPtr keys, int T, int M, int32_t *out, int32_t *out2,
                                           SelectShared &sh) {
  const int tid = threadIdx.x;
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  for (int i = tid; i < T; i += NT) {
    const uint32_t k = keys[i];
    kmin = min(kmin, k);
    kmax = max(kmax, k);
  }
  block_minmax(kmin, kmax, sh);
  int want;
  const uint32_t thr = radix_threshold(keys, T, M, kmin, kmax, sh, &want);
  const int per = (T + NT - 1) / NT;
  const int a0 = min(T, tid * per), a1 = min(T, a0 + per);
  unsigned gt = 0, eq = 0;
  for (int i = a0; i < a1; ++i) {
    const uint32_t k = keys[i];
    gt += k > thr;
    eq += k == thr;
  }
  int skip;
  int off = kept_offset(gt, eq, want, sh, &skip);
  for (int i = a0; i < a1; ++i) {
    const uint32_t k = keys[i];
    bool keep = k > thr;
    if (k == thr) {
      if (skip > 0) --skip;
      else keep = true;
    }
    if (keep && off < M) {   // off < M always holds; the guard keeps writes in bounds
      out[off] = i;
      if (out2 != nullptr) out2[off] = i;
      ++off;
    }
  }
}

// The same for T <= FR * NT keys staged in LDS, with the keys in registers:
// the spread set for the radix passes, the contiguous run for the output.
template <int FR>
__device__ __forceinline__ void select_top_regs(const uint32_t *keys, int T, int M, int32_t *out,
                                                int32_t *out2, SelectShared &sh) {
  constexpr int SR = FR + 1;   // seg = ceil(T/64)|1 <= 16*FR + 1 <= SR * NW
  const int tid = threadIdx.x;
  const int per = (T + NT - 1) / NT;
  const int a0 = min(T, tid * per), a1 = min(T, a0 + per);
  uint32_t kr[FR], ks[SR], valid;
  uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
  for (int u = 0; u < FR; ++u) {
    kr[u] = a0 + u < a1 ? keys[a0 + u] : 0u;
    if (a0 + u < a1) {
      kmin = min(kmin, kr[u]);
      kmax = max(kmax, kr[u]);
    }
  }
  load_spread(keys, T, ks, valid);
  block_minmax(kmin, kmax, sh);
  int want;
  const uint32_t thr = radix_threshold_regs(ks, valid, M, kmin, kmax, sh, &want);
  emit_run<FR>(kr, a0, a1, thr, want, M, out, out2, sh);
}

__device__ __forceinline__ double class_score(int cls, double om, double a, double r) {
  if (cls == HERMES_SHALLOW) return r;
  if (cls == HERMES_DEEP) return a;
  return (1.0 - om) * a + om * r;
}

// Keys of layers with at most this many candidates are staged in LDS for the
// select passes; longer layers read them from global memory (L2-resident).
constexpr int kLdsKeys = 38400;   // 150 KiB
// Layers of at most kRegKeys * NT candidates keep their keys in registers.
constexpr int kRegKeys = 10;
// Positions of the layer above with at most this many candidates are staged
// in LDS for the partner search.
constexpr int kLdsPos = 12288;    // 48 KiB

// dst[0..n) = src[0..n) for a 4-byte aligned src, by the NTHR threads of the
// block: the elements before the first 16-byte boundary one by one, then
// 16-byte loads, R per thread issued before any is stored so their latencies
// overlap, then the last < 4 elements.  The caller synchronises.
template <int NTHR, int R>
__device__ __forceinline__ void stage_u32(const uint32_t *src, int n, uint32_t *dst) {
  const int tid = threadIdx.x;
  const int head = min(n, (int)(((16u - (uint32_t)(reinterpret_cast<uintptr_t>(src) & 15u)) & 15u) >> 2));
  if (tid < head) dst[tid] = src[tid];
  const int nv = (n - head) >> 2;
  const uint4 *s4 = reinterpret_cast<const uint4 *>(src + head);
  for (int b = 0; b < nv; b += NTHR * R) {
    uint4 r[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int q = b + u * NTHR + tid;
      if (q < nv) r[u] = s4[q];
    }
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int q = b + u * NTHR + tid;
      if (q < nv) {
        uint32_t *d = dst + head + 4 * q;
        d[0] = r[u].x;
        d[1] = r[u].y;
        d[2] = r[u].z;
        d[3] = r[u].w;
      }
    }
  }
  const int t0 = head + 4 * nv;
  if (t0 + tid < n) dst[t0 + tid] = src[t0 + tid];
}

// Normaliser of the attention score (Sec. 3.1): the fixed-order sum of the
// layer's per-block partials of alpha_i W_i (written with W), over the n
// blocks covering its T candidates.  Every wave computes it alone (lane b
// sums partials b, b+64, ... in order, then a fixed butterfly), so every
// wave of every workgroup gets the same bits.
__device__ __forceinline__ double sum_partials(const double *p, int n) {
  const int lane = threadIdx.x & 63;
  double s = 0.0;
  for (int b = lane; b < n; b += 64) s += p[b];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  return s;
}

// The same in two steps, so that the loads of up to 128 partials are issued
// long before the sum is needed (more are summed by sum_partials itself, in
// the same order).
struct Partials {
  const double *p;
  int n;
  double x0, x1;
};

__device__ __forceinline__ Partials load_partials(const double *p, int n) {
  const int lane = threadIdx.x & 63;
  Partials q;
  q.p = p;
  q.n = n;
  q.x0 = (n <= 128 && lane < n) ? p[lane] : 0.0;
  q.x1 = (n <= 128 && lane + 64 < n) ? p[lane + 64] : 0.0;
  return q;
}

__device__ __forceinline__ double reduce_partials(Partials q) {
  if (q.n > 128) return sum_partials(q.p, q.n);
  double s = q.x0 + q.x1;   // the order of sum_partials: b, then b + 64
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  return s;
}

// First index in [lo, n) of the sorted p with p[idx] >= x: a few linear
// steps (partners of consecutive candidates are usually adjacent), then a
// binary search.
template <typename Ptr>
__device__ __forceinline__ int lower_bound_from(Ptr p, int lo, int n, int x) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (lo >= n || p[lo] >= x) return lo;
    ++lo;
  }
  int hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (p[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Partners j(i) in the layer above of KU consecutive candidates with
// positions pv (ascending): one search for the first, a forward walk after.
template <int KU, typename Ptr>
__device__ __forceinline__ void partners(Ptr p1, int T1, const int *pv, int i0, int T, int *jx) {
  int lb = 0;
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    if (i0 + u >= T) {
      jx[u] = -1;
      continue;
    }
    if (u == 0 && i0 < T1 && p1[i0] == pv[0]) lb = i0;   // same physical index
    else lb = lower_bound_from(p1, lb, T1, pv[u]);
    jx[u] = (lb < T1 && p1[lb] == pv[u]) ? lb : -1;
  }
}

// A thread's share of one array copied to LDS by the whole block in one
// batch: the elements before src's first 16-byte boundary one by one, up to
// R 16-byte pieces, and the last < 4 elements.  stage_issue only loads, so
// several arrays' loads can be in flight before any is stored.
template <int R>
struct Staged {
  uint4 r[R];
  uint32_t h, t;
};

__device__ __forceinline__ int stage_head(const uint32_t *src, int n) {
  return min(n, (int)(((16u - (uint32_t)(reinterpret_cast<uintptr_t>(src) & 15u)) & 15u) >> 2));
}

template <int R>
__device__ __forceinline__ void stage_issue(const uint32_t *src, int n, Staged<R> &s) {
  const int tid = threadIdx.x;
  const int head = stage_head(src, n);
  const int nv = (n - head) >> 2;   // <= NT * R: one batch
  const uint4 *s4 = reinterpret_cast<const uint4 *>(src + head);
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const int q = u * NT + tid;
    if (q < nv) s.r[u] = s4[q];
  }
  if (tid < head) s.h = src[tid];
  const int t0 = head + 4 * nv;
  if (t0 + tid < n) s.t = src[t0 + tid];
}

template <int R>
__device__ __forceinline__ void stage_commit(const uint32_t *src, int n, const Staged<R> &s, uint32_t *dst) {
  const int tid = threadIdx.x;
  const int head = stage_head(src, n);
  const int nv = (n - head) >> 2;
  if (head == 0) {   // dst is 16-byte aligned
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int q = u * NT + tid;
      if (q < nv) reinterpret_cast<uint4 *>(dst)[q] = s.r[u];
    }
  } else {
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int q = u * NT + tid;
      if (q < nv) {
        uint32_t *d = dst + head + 4 * q;
        d[0] = s.r[u].x;
        d[1] = s.r[u].y;
        d[2] = s.r[u].z;
        d[3] = s.r[u].w;
      }
    }
  }
  if (tid < head) dst[tid] = s.h;
  const int t0 = head + 4 * nv;
  if (t0 + tid < n) dst[t0 + tid] = s.t;
}

// e^{-k (Tm1 - j)} for increasing j: from the previous value by factors of
// e^{k} when the gap is short (a few fp64 ulps from the direct form), else
// directly.
__device__ __forceinline__ double recency_next(double &val, int &jprev, int j, double k, double ek, int Tm1) {
  const int gap = j - jprev;
  if (jprev >= 0 && gap <= 4) {
    for (int g = 0; g < gap; ++g) val *= ek;
  } else {
    val = exp(-k * (double)(Tm1 - j));
  }
  jprev = j;
  return val;
}

// alpha_i W_i with the cached rows' 1/C as a product (a division only for
// the chunk's own rows).
__device__ __forceinline__ double mass_scaled(float w, int i, int T0, int C, int mode, double inv_c) {
  if (mode != 0) return (double)w;
  if (i < T0) return (double)w * inv_c;
  return (double)w / (double)(C - (i - T0));
}

// 1. Smoothed keys S~ of every candidate of the listed layers (Sec. 3.1
//    scores, Sec. 3.2 smoothing): workgroup (b, j) scores candidates
//    [b*MCH, (b+1)*MCH) of layer layer_id[j], MU consecutive ones per thread
//    (the second partner found by a forward search from the first), with
//    the positions and W of the layer above staged in LDS when they fit,
//    and writes the keys to global memory.
constexpr int MU = 2;
constexpr int MCH = NT * MU;

__global__ __launch_bounds__(NT) void score_keys(SelectArgs a) {
  __shared__ __align__(16) uint32_t s_buf[kLdsPos];   // positions of layer l+1
  __shared__ __align__(16) uint32_t s_w1[kLdsPos];    // W of layer l+1 as bits
  const int tid = threadIdx.x;
  const int l = a.layer_id[blockIdx.y];
  const int T = a.len[l];
  if ((int)blockIdx.x * MCH >= T) return;   // whole block past the layer's end (uniform)
  const LayerTable &L0 = a.tab[l];
  const int C = a.C;
  const int T0 = T - C;
  const int32_t *pos = L0.pos[a.cur[l]];
  const int cls = L0.cls;
  const double om = L0.omega, lam = L0.lambda, k = a.forget_rate;
  const bool has_next = (l + 1 < a.n_layers) && lam != 0.0;
  int T1 = 0, T01 = 0, cls1 = HERMES_SHALLOW;
  const int32_t *pos1 = nullptr;
  const float *w1 = nullptr;
  double om1 = 0.0;
  if (has_next) {
    const LayerTable &L1 = a.tab[l + 1];
    T1 = a.len[l + 1];
    T01 = T1 - C;
    pos1 = L1.pos[a.cur[l + 1]];
    w1 = L1.w;
    cls1 = L1.cls;
    om1 = L1.omega;
  }
  const int am0 = a.guide_rows[l] > 0 ? 1 : a.alpha_mode;
  const int am1 = (has_next && a.guide_rows[l + 1] > 0) ? 1 : a.alpha_mode;
  const bool needA0 = cls != HERMES_SHALLOW, needR0 = cls != HERMES_DEEP;
  const bool needA1 = has_next && cls1 != HERMES_SHALLOW;
  const bool needR1 = has_next && cls1 != HERMES_DEEP;
  const bool by_pos = has_next && a.align_mode == 0;
  const bool pos_lds = by_pos && T1 <= kLdsPos;

  // loads: normaliser partials, this thread's candidates, the staged positions
  const int nb0 = (T + kNormBlock - 1) / kNormBlock, nb1 = (T1 + kNormBlock - 1) / kNormBlock;
  Partials q0 = {nullptr, 0, 0.0, 0.0}, q1 = {nullptr, 0, 0.0, 0.0};
  if (needA0) q0 = load_partials(a.normpart + l * a.normpart_lstride, nb0);
  if (needA1) q1 = load_partials(a.normpart + (l + 1) * a.normpart_lstride, nb1);
  const int i0 = blockIdx.x * MCH + tid * MU;
  float wv[MU];
  int pv[MU];
#pragma unroll
  for (int u = 0; u < MU; ++u) {
    const bool ok = i0 + u < T;
    wv[u] = (ok && needA0) ? L0.w[i0 + u] : 0.f;
    pv[u] = (ok && by_pos) ? pos[i0 + u] : 0;
  }
  const bool w1_lds = needA1 && T1 <= kLdsPos;
  {
    Staged<3> g, h;
    if (pos_lds) stage_issue(reinterpret_cast<const uint32_t *>(pos1), T1, g);
    if (w1_lds) stage_issue(reinterpret_cast<const uint32_t *>(w1), T1, h);
    if (pos_lds) stage_commit(reinterpret_cast<const uint32_t *>(pos1), T1, g, s_buf);
    if (w1_lds) stage_commit(reinterpret_cast<const uint32_t *>(w1), T1, h, s_w1);
  }
  const double sa0 = needA0 ? reduce_partials(q0) : 0.0;
  const double sa1 = needA1 ? reduce_partials(q1) : 0.0;
  __syncthreads();

  // partners in layer l+1 and their W
  int jx[MU];
  if (pos_lds) partners<MU>(reinterpret_cast<const int32_t *>(s_buf), T1, pv, i0, T, jx);
  else if (by_pos) partners<MU>(pos1, T1, pv, i0, T, jx);
  else {
#pragma unroll
    for (int u = 0; u < MU; ++u) jx[u] = (has_next && i0 + u < T && i0 + u < T1) ? i0 + u : -1;
  }
  float w1v[MU];
#pragma unroll
  for (int u = 0; u < MU; ++u)
    w1v[u] = (jx[u] >= 0 && needA1)
                 ? (w1_lds ? __builtin_bit_cast(float, s_w1[jx[u]]) : w1[jx[u]])
                 : 0.f;

  // keys
  const double inv_sa0 = sa0 > 0.0 ? 1.0 / sa0 : 0.0, inv_sa1 = sa1 > 0.0 ? 1.0 / sa1 : 0.0;
  const double inv_z0 = a.inv_z[l], inv_z1 = has_next ? a.inv_z[l + 1] : 0.0;
  const double ek = a.ek, inv_c = a.inv_c;
  uint32_t *keys = a.keys + l * a.keys_lstride;
  int jp0 = -1, jp1 = -1;
  double rv0 = 0.0, rv1 = 0.0;
#pragma unroll
  for (int u = 0; u < MU; ++u) {
    const int i = i0 + u;
    if (i >= T) break;
    const double a_i = needA0 ? mass_scaled(wv[u], i, T0, C, am0, inv_c) * inv_sa0 : 0.0;
    const double r_i = needR0 ? recency_next(rv0, jp0, i, k, ek, T - 1) * inv_z0 : 0.0;
    double st = class_score(cls, om, a_i, r_i);
    if (has_next) {
      double sj = 0.0;
      const int j = jx[u];
      if (j >= 0) {
        const double a_j = needA1 ? mass_scaled(w1v[u], j, T01, C, am1, inv_c) * inv_sa1 : 0.0;
        const double r_j = needR1 ? recency_next(rv1, jp1, j, k, ek, T1 - 1) * inv_z1 : 0.0;
        sj = class_score(cls1, om1, a_j, r_j);
      }
      st = (1.0 - lam) * st + lam * sj;
    }
    const float f = (float)st;
    keys[i] = __builtin_bit_cast(uint32_t, f);
    if (L0.s_dbg != nullptr) L0.s_dbg[i] = f;
  }

}

// TopK of keys[0..T) (M < T) into out (and out2 if non-null): staged in LDS
// when they fit, held in registers for the radix passes when T <= kRegKeys
// * NT, read from global memory (L2-resident) otherwise.  Shared by the
// compression and the stand-alone entry point.
__device__ __forceinline__ void select_keys(const uint32_t *keys, int T, int M, int32_t *out, int32_t *out2,
                                            SelectShared &sh, uint32_t *big) {
  if (T <= kLdsKeys) {
    stage_u32<NT, 10>(keys, T, big);
    __syncthreads();
    if (T <= kRegKeys * NT) {
      // keys in registers: big is free once the radix passes are done and
      // takes the kept list, written out coalesced
      select_top_regs<kRegKeys>(big, T, M, reinterpret_cast<int32_t *>(big), nullptr, sh);
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kRegKeys; ++u) {
        const int i = u * NT + threadIdx.x;
        if (i < M) {   // M < T <= kRegKeys * NT
          const int32_t x = static_cast<int32_t>(big[i]);
          out[i] = x;
          if (out2 != nullptr) out2[i] = x;
        }
      }
    } else {
      select_top(static_cast<const uint32_t *>(big), T, M, out, out2, sh);
    }
  } else {
    select_top(keys, T, M, out, out2, sh);
  }
}

// 2. TopK of each listed layer from its keys.
__global__ __launch_bounds__(NT) void select_kept(SelectArgs a) {
  __shared__ SelectShared sh;
  __shared__ uint32_t big[kLdsKeys];
  const int l = a.layer_id[blockIdx.x];
  const LayerTable &L0 = a.tab[l];
  const int T = a.len[l];
  if (T <= L0.budget) return;
  select_keys(a.keys + l * a.keys_lstride, T, L0.budget, a.kept + l * a.kept_lstride, L0.kept_dbg, sh,
              big);
}

__global__ __launch_bounds__(NT) void topk_keys(const uint32_t *keys, int n, int k, int32_t *out) {
  __shared__ SelectShared sh;
  __shared__ uint32_t big[kLdsKeys];
  if (k >= n) {
    for (int i = threadIdx.x; i < n; i += NT) out[i] = i;
    return;
  }
  select_keys(keys, n, k, out, nullptr, sh, big);
}

}  // namespace

hipError_t launch_select(const SelectArgs &a, hipStream_t s) {
  int max_T = 0;
  for (int j = 0; j < a.n_list; ++j) max_T = max(max_T, a.len[a.layer_id[j]]);
  hipLaunchKernelGGL(score_keys, dim3((max_T + MCH - 1) / MCH, a.n_list), dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_kept, dim3(a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_topk(const float *keys, int n, int k, int32_t *out, hipStream_t s) {
  hipLaunchKernelGGL(topk_keys, dim3(1), dim3(NT), 0, s,
                     reinterpret_cast<const uint32_t *>(keys), n, k, out);
  return hipGetLastError();
}

}  // namespace hermes
