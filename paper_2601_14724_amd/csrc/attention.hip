// Chunk attention for gfx950 (MFMA bf16, 64-wide waves).
//
// attn_fwd     causal GQA attention of the chunk (or query) rows over
//              [cache; new rows]: O and the per-row log-sum-exp.
// attn_colsum  attention mass W_i = sum over heads and rows of the softmax
//              probability on candidate i (Sec. 3.1, deep-layer score),
//              recomputed key-major from the row LSE so that every W_i is
//              summed by exactly one wave, in a fixed order, with no partials.
//
// Query rows are packed per KV head: packed row p = r * G + g holds chunk row
// r of query head kv * G + g, so the G heads that share a KV head share every
// K/V tile, and all rows of a tile share nearly the same causal boundary.
//
// MFMA layout (v_mfma_f32_32x32x16_bf16): lane l supplies A[m = l%32][k = 8(l/32)
// .. +7] and B[k = 8(l/32) .. +7][n = l%32]; result register j of lane l holds
// D[m = 8(j/4) + 4(l/32) + j%4][n = l%32].
#include "hermes_internal.h"

namespace hermes {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = kAttnRowsPerBlock;    // packed rows per workgroup (4 waves x 32)
constexpr int BN = 64;                   // keys per tile
constexpr int BK = kColsumKeysPerBlock;  // candidates per sweep workgroup (4 waves x 32)
constexpr int BQ = 64;                   // packed rows per sweep tile
constexpr int KPAD = 8;                  // u16 padding of K / Q rows in LDS
constexpr int VPAD = 4;                  // u16 padding of transposed V rows in LDS

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint16_t f2bf(float x) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int D>
__global__ __launch_bounds__(256) void attn_fwd(AttnArgs a) {
  const int j = blockIdx.z;
  const int kv = blockIdx.y;
  const int layer = a.layer_id[j];
  const LayerTable &lt = a.tab[layer];
  const int cur = a.cur[j];
  const int T0 = a.T0[j];
  const int C = a.C, Hq = a.Hq, Hkv = a.Hkv;
  const int G = Hq / Hkv;
  const int P = C * G;
  const int T = T0 + C;
  const int p0 = blockIdx.x * BM;
  if (p0 >= P) return;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int half = lane >> 5, l32 = lane & 31;

  const int slot = a.slot[j];
  const uint16_t *q = a.q + slot * a.q_lstride;
  const uint16_t *kn = a.kn + slot * a.kv_lstride;
  const uint16_t *vn = a.vn + slot * a.kv_lstride;
  uint16_t *out = a.out + slot * a.q_lstride;
  const uint16_t *kc = lt.k[cur];
  const uint16_t *vc = lt.v[cur];

  // This lane's query row (column n of the S^T tile).
  const int prow = p0 + wave * 32 + l32;
  const bool row_ok = prow < P;
  const int r = row_ok ? prow / G : 0;
  const int h = kv * G + (row_ok ? prow - r * G : 0);
  const int vis = row_ok ? T0 + r : -1;   // last candidate this row sees

  bf16x8 qf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    if (row_ok) {
      qf[kk] = *reinterpret_cast<const bf16x8 *>(q + ((int64_t)r * Hq + h) * D + 16 * kk + 8 * half);
    } else {
      qf[kk] = bf16x8{};
    }
  }

  const int pmax = min(p0 + BM, P) - 1;
  const int nkeys = T0 + pmax / G + 1;
  const int ntiles = (nkeys + BN - 1) / BN;

  __shared__ __attribute__((aligned(16))) uint16_t Ks[BN][D + KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D][BN + VPAD];

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) o[db] = f32x16{};
  float m_run = -1e30f, l_run = 0.f;
  const float c = a.scale_log2;

  for (int t = 0; t < ntiles; ++t) {
    const int k0 = t * BN;
    __syncthreads();
    constexpr int CH = D / 8;
    for (int e = tid; e < BN * CH; e += 256) {
      const int kr = e / CH, ch = e - (e / CH) * CH;
      const int i = k0 + kr;
      uint4 k4 = {0u, 0u, 0u, 0u}, v4 = {0u, 0u, 0u, 0u};
      if (i < T) {
        const uint16_t *ks, *vs;
        if (i < T0) {
          ks = kc + ((int64_t)i * Hkv + kv) * D;
          vs = vc + ((int64_t)i * Hkv + kv) * D;
        } else {
          ks = kn + ((int64_t)(i - T0) * Hkv + kv) * D;
          vs = vn + ((int64_t)(i - T0) * Hkv + kv) * D;
        }
        k4 = *reinterpret_cast<const uint4 *>(ks + ch * 8);
        v4 = *reinterpret_cast<const uint4 *>(vs + ch * 8);
      }
      *reinterpret_cast<uint4 *>(&Ks[kr][ch * 8]) = k4;
      const uint32_t vw[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        Vt[ch * 8 + 2 * e2][kr] = (uint16_t)(vw[e2] & 0xFFFFu);
        Vt[ch * 8 + 2 * e2 + 1][kr] = (uint16_t)(vw[e2] >> 16);
      }
    }
    __syncthreads();

    // S^T = K Q^T for two 32-key sub-tiles: lane = query row, register = key.
    f32x16 s[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      s[sub] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(&Ks[sub * 32 + l32][16 * kk + 8 * half]);
        s[sub] = mfma32(kf, qf[kk], s[sub]);
      }
    }
    float mt = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) {
        const int key = k0 + sub * 32 + 8 * (jj >> 2) + 4 * half + (jj & 3);
        const float x = key <= vis ? s[sub][jj] * c : -INFINITY;
        s[sub][jj] = x;
        mt = fmaxf(mt, x);
      }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] *= alpha;

    bf16x8 pf[4];
    float ls = 0.f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) {
        const float p = fast_exp2(s[sub][jj] - m_new);
        ls += p;
        pf[2 * sub + (jj >> 3)][jj & 7] = static_cast<__bf16>(p);
      }
    }
    l_run += ls;

    // O^T += V^T P^T: B element t of lane half hf in key group qq is key
    // 16 qq + 8 (t/4) + 4 hf + t%4, so A reads V^T at the same keys.
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const uint16_t *vrow = &Vt[32 * db + l32][0];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const uint2 lo = *reinterpret_cast<const uint2 *>(vrow + 16 * qq + 4 * half);
        const uint2 hi = *reinterpret_cast<const uint2 *>(vrow + 16 * qq + 8 + 4 * half);
        const uint4 packed = {lo.x, lo.y, hi.x, hi.y};
        const bf16x8 vf = __builtin_bit_cast(bf16x8, packed);
        o[db] = mfma32(vf, pf[qq], o[db]);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.f / l_tot;
  if (row_ok) {
    uint16_t *orow = out + ((int64_t)r * Hq + h) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int d0 = 32 * db + 8 * grp + 4 * half;
        const uint32_t w0 = (uint32_t)f2bf(o[db][4 * grp + 0] * inv) |
                            ((uint32_t)f2bf(o[db][4 * grp + 1] * inv) << 16);
        const uint32_t w1 = (uint32_t)f2bf(o[db][4 * grp + 2] * inv) |
                            ((uint32_t)f2bf(o[db][4 * grp + 3] * inv) << 16);
        *reinterpret_cast<uint2 *>(orow + d0) = uint2{w0, w1};
      }
    }
    if (a.lse != nullptr && half == 0) {
      a.lse[layer * a.lse_lstride + (int64_t)kv * P + prow] = m_run + log2f(l_tot);
    }
  }
}

template <int D>
__global__ __launch_bounds__(256) void attn_colsum(ColsumArgs a) {
  const int j = blockIdx.z;
  const int layer = a.layer_id[j];
  const LayerTable &lt = a.tab[layer];
  const int cur = a.cur[j];
  const int T0 = a.T0[j];
  const int C = a.C, Hq = a.Hq, Hkv = a.Hkv;
  const int G = Hq / Hkv;
  const int P = C * G;
  const int T = T0 + C;
  const int k0 = blockIdx.x * BK;
  if (k0 >= T) return;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int half = lane >> 5, l32 = lane & 31;
  const int key = k0 + wave * 32 + l32;          // column n of this lane
  const bool key_ok = key < T;
  const int pmin_key = key < T0 ? 0 : (key - T0) * G;
  const int p_begin = (k0 < T0 ? 0 : (k0 - T0) * G) & ~(BQ - 1);

  const int slot = a.slot[j];
  const uint16_t *q = a.q + slot * a.q_lstride;
  const uint16_t *kn = a.kn + slot * a.kv_lstride;
  const uint16_t *kc = lt.k[cur];
  const float c = a.scale_log2;

  __shared__ __attribute__((aligned(16))) uint16_t Qs[BQ][D + KPAD];
  __shared__ __attribute__((aligned(16))) float Ls[BQ];

  double wacc = 0.0;
  for (int kv = 0; kv < Hkv; ++kv) {
    bf16x8 kf[D / 16];
    const uint16_t *krow = key < T0 ? kc + ((int64_t)key * Hkv + kv) * D
                                    : kn + ((int64_t)(key - T0) * Hkv + kv) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      kf[kk] = key_ok ? *reinterpret_cast<const bf16x8 *>(krow + 16 * kk + 8 * half) : bf16x8{};
    }
    const float *lse = a.lse + layer * a.lse_lstride + (int64_t)kv * P;

    for (int pt = p_begin; pt < P; pt += BQ) {
      __syncthreads();
      constexpr int CH = D / 8;
      for (int e = tid; e < BQ * CH; e += 256) {
        const int rr = e / CH, ch = e - (e / CH) * CH;
        const int p = pt + rr;
        uint4 v = {0u, 0u, 0u, 0u};
        if (p < P) {
          const int r = p / G, g = p - (p / G) * G;
          v = *reinterpret_cast<const uint4 *>(q + ((int64_t)r * Hq + kv * G + g) * D + ch * 8);
        }
        *reinterpret_cast<uint4 *>(&Qs[rr][ch * 8]) = v;
      }
      if (tid < BQ) Ls[tid] = (pt + tid < P) ? lse[pt + tid] : INFINITY;
      __syncthreads();

#pragma unroll
      for (int rb = 0; rb < BQ / 32; ++rb) {
        // S = Q K^T: lane = candidate, register = query row.
        f32x16 s = f32x16{};
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          const bf16x8 qv = *reinterpret_cast<const bf16x8 *>(&Qs[rb * 32 + l32][16 * kk + 8 * half]);
          s = mfma32(qv, kf[kk], s);
        }
        float ts = 0.f;
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int rloc = rb * 32 + 8 * grp + 4 * half;
          const float4 l4 = *reinterpret_cast<const float4 *>(&Ls[rloc]);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float x = fmaf(s[4 * grp + e], c, -lv[e]);
            const float p = fast_exp2(x);
            ts += (pt + rloc + e >= pmin_key) ? p : 0.f;
          }
        }
        wacc += (double)ts;
      }
    }
  }
  wacc += __shfl_xor(wacc, 32);
  if (key_ok && half == 0) lt.w[key] = (float)wacc;
}

}  // namespace

hipError_t launch_attention(const AttnArgs &a, int n_list, int head_dim, hipStream_t s) {
  const int P = a.C * (a.Hq / a.Hkv);
  dim3 grid((P + BM - 1) / BM, a.Hkv, n_list);
  if (head_dim == 64) {
    hipLaunchKernelGGL(attn_fwd<64>, grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(attn_fwd<128>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_colsum(const ColsumArgs &a, int n_list, int max_T, int head_dim,
                         hipStream_t s) {
  dim3 grid((max_T + BK - 1) / BK, 1, n_list);
  if (head_dim == 64) {
    hipLaunchKernelGGL(attn_colsum<64>, grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(attn_colsum<128>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace hermes
