// Scoring, cross-layer smoothing and TopK selection for gfx950.
//
// One 1024-thread workgroup per layer over budget:
//   1. importance S^l_i by class (Sec. 3.1): recency R_i = e^{-k(T-1-i)}/Z
//      (shallow), attention A_i = alpha_i W_i normalised to sum 1 (deep), and
//      (1 - omega_l) A + omega_l R (middle), all in fp64;
//   2. one-hop smoothing S~^l = (1 - lambda_l) S^l + lambda_l S^{l+1}_{j(i)}
//      (Sec. 3.2), the partner j(i) found by binary search on layer l+1's
//      positions (or equal physical index);
//   3. S~ rounded to fp32; its bit pattern is an order-preserving uint32 key;
//   4. MSB-first radix select (4 passes of 8 bits, LDS histograms) finds the
//      budget-th largest key; ties at that key go to the higher index;
//   5. the kept indices are emitted in ascending order by two block scans.
#include "hermes_internal.h"

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

struct ScanShared {
  int wsum[NW];
  int woff[NW];
  int total;
};

// Exclusive prefix sum over the block in thread order; *total gets the sum.
__device__ int block_excl_scan(int v, ScanShared &sh, int *total) {
  const int w = threadIdx.x >> 6, ln = threadIdx.x & 63;
  const int inc = wave_incl_scan(v);
  if (ln == 63) sh.wsum[w] = inc;
  __syncthreads();
  if (w == 0) {
    const int x = ln < NW ? sh.wsum[ln] : 0;
    const int xi = wave_incl_scan(x);
    if (ln < NW) sh.woff[ln] = xi - x;
    if (ln == NW - 1) sh.total = xi;
  }
  __syncthreads();
  const int res = inc - v + sh.woff[w];
  *total = sh.total;
  __syncthreads();
  return res;
}

__device__ double block_sum_f64(double v, double *sh) {
  const int w = threadIdx.x >> 6, ln = threadIdx.x & 63;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (ln == 0) sh[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < NW; ++i) t += sh[i];   // fixed order: deterministic
  __syncthreads();
  return t;
}

// hist[d] += 1 for every active lane with d >= 0.  Lanes holding the same
// digit are merged with a ballot first (the leading digits of fp32 keys are
// shared by most candidates, so plain LDS atomics would serialise).
__device__ __forceinline__ void hist_add(unsigned *hist, int d) {
  const int lane = threadIdx.x & 63;
  unsigned long long active = __ballot(d >= 0);
  for (int it = 0; it < 3 && active != 0ull; ++it) {
    const int leader = __ffsll(active) - 1;
    const int dl = __shfl(d, leader);
    const unsigned long long m = __ballot(d == dl);
    if (lane == leader) atomicAdd(&hist[dl], (unsigned)__popcll(m));
    active &= ~m;
  }
  if ((active >> lane) & 1ull) atomicAdd(&hist[d], 1u);
}

struct SelectShared {
  unsigned hist[256];
  int digit, above;
  ScanShared scan;
  double red[NW];
};

// Keep the M largest of keys[0..T) (M < T), ties to the higher index; write
// the kept indices ascending to out (and out2 if non-null).
template <typename KeyPtr>
__device__ __forceinline__ void select_top(KeyPtr keys, int T, int M, int32_t *out, int32_t *out2,
                                           SelectShared &sh) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, pmask = 0u;
  int want = M;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < 256; i += NT) sh.hist[i] = 0u;
    if (tid == 0) {
      sh.digit = 0;
      sh.above = 0;
    }
    __syncthreads();
    for (int i = tid; i < T; i += NT) {
      const uint32_t k = keys[i];
      hist_add(sh.hist, (k & pmask) == prefix ? (int)((k >> shift) & 255u) : -1);
    }
    __syncthreads();
    if (tid < 64) {
      // lane ln owns digits 255-4ln .. 252-4ln, visited from high to low
      int cnt[4], loc = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cnt[e] = (int)sh.hist[255 - 4 * tid - e];
        loc += cnt[e];
      }
      const int incl = wave_incl_scan(loc);
      int acc = incl - loc;   // keys whose digit is above this lane's digits
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (acc < want && want <= acc + cnt[e]) {
          sh.digit = 255 - 4 * tid - e;
          sh.above = acc;
        }
        acc += cnt[e];
      }
    }
    __syncthreads();
    want -= sh.above;
    prefix |= (uint32_t)sh.digit << shift;
    pmask |= 255u << shift;
    __syncthreads();
  }
  const uint32_t thr = prefix;   // the M-th largest key; `want` ties of it are kept

  const int per = (T + NT - 1) / NT;
  const int a0 = min(T, tid * per), a1 = min(T, a0 + per);
  int gt = 0, eq = 0;
  for (int i = a0; i < a1; ++i) {
    const uint32_t k = keys[i];
    gt += k > thr;
    eq += k == thr;
  }
  int eq_total;
  const int eq_before = block_excl_scan(eq, sh.scan, &eq_total);
  const int eq_above = eq_total - eq_before - eq;        // ties at higher indices
  const int keep_eq = max(0, min(eq, want - eq_above));  // my highest keep_eq ties stay
  int kept_total;
  int off = block_excl_scan(gt + keep_eq, sh.scan, &kept_total);
  int skip = eq - keep_eq;
  for (int i = a0; i < a1; ++i) {
    const uint32_t k = keys[i];
    bool keep = k > thr;
    if (k == thr) {
      if (skip > 0) {
        --skip;
      } else {
        keep = true;
      }
    }
    if (keep && off < M) {   // off < M always holds; the guard keeps writes in bounds
      out[off] = i;
      if (out2 != nullptr) out2[off] = i;
      ++off;
    }
  }
}

__device__ __forceinline__ double mass_over_observers(float w, int i, int T0, int C, int mode) {
  if (mode != 0) return (double)w;
  const int n = i < T0 ? C : C - (i - T0);
  return (double)w / (double)n;
}

__device__ __forceinline__ double class_score(int cls, double om, double a, double r) {
  if (cls == HERMES_SHALLOW) return r;
  if (cls == HERMES_DEEP) return a;
  return (1.0 - om) * a + om * r;
}

// Candidates whose positions / keys fit in LDS take the LDS path; longer
// layers fall back to global memory (L2-resident) with the same arithmetic.
constexpr int kLdsKeys = 38400;   // 150 KiB

// Index of `target` in the sorted array p[0..n), or -1.
template <typename Ptr>
__device__ __forceinline__ int find_sorted(Ptr p, int n, int target, int hint) {
  if (hint < n && p[hint] == target) return hint;   // same physical index
  int lo = 0, hi = n - 1;
  while (lo <= hi) {
    const int mid = (lo + hi) >> 1;
    const int v = p[mid];
    if (v == target) return mid;
    if (v < target) lo = mid + 1; else hi = mid - 1;
  }
  return -1;
}

__global__ __launch_bounds__(NT) void score_select(SelectArgs a) {
  __shared__ SelectShared sh;
  __shared__ uint32_t big[kLdsKeys];
  const int tid = threadIdx.x;
  const int l = a.layer_id[blockIdx.x];
  const LayerTable &L0 = a.tab[l];
  const int C = a.C;
  const int T = a.len[l];
  const int T0 = T - C;
  const int32_t *pos = L0.pos[a.cur[l]];
  const float *w = L0.w;
  const int cls = L0.cls;
  const double om = L0.omega;
  const double lam = L0.lambda;
  const double k = a.forget_rate;
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
  // W from a guidance prompt: every candidate has the same observers, so the
  // normalised mass is W / sum W whatever alpha_mode says.
  const int am0 = a.guide_rows[l] > 0 ? 1 : a.alpha_mode;
  const int am1 = (has_next && a.guide_rows[l + 1] > 0) ? 1 : a.alpha_mode;
  const bool needA0 = cls != HERMES_SHALLOW, needR0 = cls != HERMES_DEEP;
  const bool needA1 = has_next && cls1 != HERMES_SHALLOW;
  const bool needR1 = has_next && cls1 != HERMES_DEEP;
  const bool lds = T <= kLdsKeys && T1 <= kLdsKeys;
  const bool by_pos = has_next && a.align_mode == 0;

  // Normalisers: the alpha-weighted mass summed in a fixed order, and the
  // recency curve's closed-form sum Z = (1 - e^{-kT}) / (1 - e^{-k}).
  double sa0 = 0.0, sa1 = 0.0;
  if (needA0)
    for (int i = tid; i < T; i += NT) sa0 += mass_over_observers(w[i], i, T0, C, am0);
  if (needA1)
    for (int i = tid; i < T1; i += NT) sa1 += mass_over_observers(w1[i], i, T01, C, am1);
  if (lds && by_pos)
    for (int i = tid; i < T1; i += NT) big[i] = (uint32_t)pos1[i];
  sa0 = block_sum_f64(sa0, sh.red);
  sa1 = block_sum_f64(sa1, sh.red);
  const double z0 = expm1(-k * (double)T) / expm1(-k);
  const double z1 = expm1(-k * (double)T1) / expm1(-k);

  uint32_t *keys = a.keys + l * a.keys_lstride;
  const double inv_sa0 = sa0 > 0.0 ? 1.0 / sa0 : 0.0, inv_sa1 = sa1 > 0.0 ? 1.0 / sa1 : 0.0;
  const double inv_z0 = 1.0 / z0, inv_z1 = T1 > 0 ? 1.0 / z1 : 0.0;
  constexpr int U = 4;   // candidates per thread per pass: their loads are in flight together
  for (int i0 = tid; i0 < T; i0 += U * NT) {
    int ii[U], pv[U], jx[U];
    float wv[U], w1v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      ii[u] = i0 + u * NT;
      const bool ok = ii[u] < T;
      wv[u] = (ok && needA0) ? w[ii[u]] : 0.f;
      pv[u] = (ok && by_pos) ? pos[ii[u]] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      jx[u] = -1;
      if (ii[u] < T && has_next) {
        if (by_pos) {
          jx[u] = lds ? find_sorted(reinterpret_cast<const int32_t *>(big), T1, pv[u], ii[u])
                      : find_sorted(pos1, T1, pv[u], ii[u]);
        } else {
          jx[u] = ii[u] < T1 ? ii[u] : -1;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) w1v[u] = (jx[u] >= 0 && needA1) ? w1[jx[u]] : 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = ii[u];
      if (i >= T) continue;
      const double a_i = needA0 ? mass_over_observers(wv[u], i, T0, C, am0) * inv_sa0 : 0.0;
      const double r_i = needR0 ? exp(-k * (double)(T - 1 - i)) * inv_z0 : 0.0;
      double st = class_score(cls, om, a_i, r_i);
      if (has_next) {
        double s1 = 0.0;
        const int j = jx[u];
        if (j >= 0) {
          const double a_j = needA1 ? mass_over_observers(w1v[u], j, T01, C, am1) * inv_sa1 : 0.0;
          const double r_j = needR1 ? exp(-k * (double)(T1 - 1 - j)) * inv_z1 : 0.0;
          s1 = class_score(cls1, om1, a_j, r_j);
        }
        st = (1.0 - lam) * st + lam * s1;
      }
      const float f = (float)st;
      keys[i] = __builtin_bit_cast(uint32_t, f);
      if (L0.s_dbg != nullptr) L0.s_dbg[i] = f;
    }
  }
  __syncthreads();
  if (T <= L0.budget) return;
  int32_t *kept = a.kept + l * a.kept_lstride;
  if (lds) {
    for (int i = tid; i < T; i += NT) big[i] = keys[i];
    __syncthreads();
    select_top(big, T, L0.budget, kept, L0.kept_dbg, sh);
  } else {
    select_top(keys, T, L0.budget, kept, L0.kept_dbg, sh);
  }
}

__global__ __launch_bounds__(NT) void topk_keys(const uint32_t *keys, int n, int k, int32_t *out) {
  __shared__ SelectShared sh;
  if (k >= n) {
    for (int i = threadIdx.x; i < n; i += NT) out[i] = i;
    return;
  }
  select_top(keys, n, k, out, nullptr, sh);
}

}  // namespace

hipError_t launch_select(const SelectArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(score_select, dim3(a.n_list), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_topk(const float *keys, int n, int k, int32_t *out, hipStream_t s) {
  hipLaunchKernelGGL(topk_keys, dim3(1), dim3(NT), 0, s,
                     reinterpret_cast<const uint32_t *>(keys), n, k, out);
  return hipGetLastError();
}

}  // namespace hermes
