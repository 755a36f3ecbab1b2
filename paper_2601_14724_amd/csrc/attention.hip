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
#include <type_traits>

#include "hermes_internal.h"
#include "score_terms.h"

namespace hermes {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s4 __attribute__((ext_vector_type(4)));

constexpr int AT = 512;                  // attention workgroup: 8 waves, two per SIMD
constexpr int BM = kAttnRowsPerBlock;    // packed rows per workgroup (8 waves x 32)
constexpr int BN = 64;                   // keys per tile
constexpr int BK = kColsumKeysPerBlock;  // candidates per sweep workgroup (4 waves x 64)
constexpr int BQS = 32;                  // packed rows per sweep tile
constexpr int KPAD = 8;                  // u16 padding of K / Q rows in LDS
constexpr int VPAD = 32;                 // u16 padding of V rows in LDS
constexpr int kAheadK = 4;               // K fragment reads issued ahead of their MFMA
// fourth word of a raw buffer descriptor on gfx9-family chips (32-bit data,
// no swizzle; the range check uses the byte count in the third word)
constexpr int kBufferWord3 = 0x00020000;
constexpr int kAheadV = 4;               // V^T fragment pairs issued ahead of their MFMA

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint16_t f2bf(float x) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }


// 16-byte load through the global (not flat) address space, so outstanding
// prefetches are tracked by vmcnt only and never delay LDS waits.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 gload16(const uint16_t *p) {
  typedef const __attribute__((address_space(1))) u32x4 *gptr;
  const u32x4 v = *(gptr)(p);
  return uint4{v.x, v.y, v.z, v.w};
}

// ds_read_b64_tr_b16: inside each group of 16 lanes, lane j receives element
// j%4 of the 8-byte rows addressed by lanes j/4, 4 + j/4, 8 + j/4, 12 + j/4.
__device__ __forceinline__ s4 lds_tr16(const uint16_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)p);
}

// Workgroups are dispatched to the 8 XCDs round-robin by linear id; this
// maps linear ids so that consecutive logical tiles (the q-tiles of one
// layer and KV head, which stream the same K/V) run on the same XCD and
// share its L2.
__device__ __forceinline__ int xcd_remap(int i, int n) {
  const int q = n / 8, r = n % 8, x = i % 8, k = i / 8;
  return x < r ? x * (q + 1) + k : r * (q + 1) + (x - r) * q + k;
}

// STREAM: balanced short passes (query, guidance prompt).  The key tiles of
// every (entry, KV head) pair, concatenated in pair order (pair k = j Hkv +
// kv, st_tiles[j] tiles each, entry j's pairs from tile st_off[j]), are cut
// into st_units equal ranges; unit u is nqt workgroups with consecutive ids
// (one per query tile, sharing the K/V tiles in their XCD's L2) over tiles
// [u N / U, (u + 1) N / U).  The workgroup walks its range in one tile loop;
// where the range leaves a pair it writes the pair's unnormalised partial
// state (bf16 O, fp32 running maximum and row sum) to partial block (u + k)
// of its query tile (distinct for every (u, k): a later unit only covers
// later pairs) and switches to the next pair.  attn_combine merges a pair's
// blocks.  Otherwise: one workgroup per (entry, KV head, query tile) over its
// whole sequence, writing O (WRITE_O) and the row LSE.
template <int D, bool STREAM, bool WRITE_O>
__global__ __launch_bounds__(AT, 1) void attn_fwd(AttnArgs a, int nqt) {
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int qtile = lin % nqt;
  const int C = a.C, Hq = a.Hq, Hkv = a.Hkv;
  const int G = Hq / Hkv;
  const int P = C * G;
  const int p0 = qtile * BM;
  if (p0 >= P) return;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int half = lane >> 5, l32 = lane & 31;

  // This lane's query row (column n of the S^T tile).
  const int prow = p0 + wave * 32 + l32;
  const bool row_ok = prow < P;
  // A wave whose 32 rows all lie past P (in the last query tile of a head
  // group) still loads and stores its share of every tile and meets every
  // barrier, but issues no MFMAs.
  const bool wave_rows = __builtin_amdgcn_readfirstlane(p0 + wave * 32 < P ? 1 : 0) != 0;
  const int r = row_ok ? prow / G : 0;
  const int g = row_ok ? prow - r * G : 0;
  const int pmax = min(p0 + BM, P) - 1;

  // Pair state: entry j, KV head kv, its cache and new rows.
  int j = 0, kv = 0, T0 = 0, T = 0, vis = -1, vis_min = 0, ntiles = 0, n_pure = 0, first = 0;
  const uint16_t *q = nullptr, *kn = nullptr, *vn = nullptr, *kc = nullptr, *vc = nullptr;
  const int64_t row_stride = (int64_t)Hkv * D;
  constexpr int CH = D / 8;                 // 16-byte chunks per key row and head
  constexpr int NLD = BN * CH / AT;         // chunks per thread per tensor
  uint32_t cofs[NLD];
  bf16x8 qf[D / 16];
  // STREAM: this unit's tile range over the concatenated pairs
  int x_lo = 0, x_hi = 0, u = 0;
  if constexpr (STREAM) {
    u = lin / nqt;
    x_lo = (int)((int64_t)u * a.st_total / a.st_units);
    x_hi = (int)((int64_t)(u + 1) * a.st_total / a.st_units);
    if (x_lo >= x_hi) return;
  }
  auto enter = [&](int jj, int kvv) {
    j = jj;
    kv = kvv;
    const LayerTable &lt = a.tab[a.layer_id[j]];
    const int cur = a.cur[j];
    T0 = a.T0[j];
    T = T0 + C;
    vis = row_ok ? T0 + r : -1;             // last candidate this row sees
    vis_min = T0 + p0 / G;                  // every row of the block sees keys <= vis_min
    const int nkeys = T0 + pmax / G + 1;
    ntiles = (nkeys + BN - 1) / BN;
    // tiles [0, n_pure) lie wholly in the cache and below every row's causal
    // limit: they load with plain pointer strides and need no mask
    n_pure = min(ntiles, T0 / BN);
    const int slot = a.slot[j];
    q = a.q + slot * a.q_lstride;
    kn = a.kn + slot * a.kv_lstride;
    vn = a.vn + slot * a.kv_lstride;
    kc = lt.k[cur];
    vc = lt.v[cur];
    const int h = kv * G + g;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      qf[kk] = row_ok ? *reinterpret_cast<const bf16x8 *>(q + ((int64_t)r * Hq + h) * D + 16 * kk + 8 * half)
                      : bf16x8{};
    }
    // byte offset of this thread's chunk u inside a key tile of the cache; a
    // pure tile's loads are then a uniform base plus this 32-bit offset
#pragma unroll
    for (int uu = 0; uu < NLD; ++uu) {
      const int e = tid + uu * AT;
      cofs[uu] = (uint32_t)(((e / CH) * row_stride + kv * D + (e % CH) * 8) * sizeof(uint16_t));
    }
  };
  // the pair holding concatenated tile x (STREAM), its first tile in `first`
  auto locate = [&](int x, int &jj, int &kvv, int &f) {
    int e = 0;
    while (e + 1 < a.st_entries && x >= a.st_off[e + 1]) ++e;
    jj = e;
    kvv = (x - a.st_off[e]) / a.st_tiles[e];
    f = a.st_off[e] + kvv * a.st_tiles[e];
  };
  if constexpr (STREAM) {
    int jj, kvv;
    locate(x_lo, jj, kvv, first);
    enter(jj, kvv);
  } else {
    enter(lin / (nqt * Hkv), (lin / nqt) % Hkv);
  }

  // Double-buffered K and V tiles, both row-major [key][d]; V is read
  // transposed by ds_read_b64_tr_b16.  Row pads keep the K reads (16 B per
  // lane) and the transposed V reads (4 rows x 32 B per 16 lanes) spread
  // over the LDS banks.
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][BN][D + KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][BN][D + VPAD];
  uint4 kreg[NLD], vreg[NLD];
  // pure tiles load through buffer descriptors whose base is the tile's first
  // row (scalar arithmetic): each load is the descriptor plus the lane's
  // 32-bit offset, with no per-lane 64-bit address addition
  auto load_pure = [&](int k0) {
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(kc + (int64_t)k0 * row_stride), 0, 0x7FFFFFFF, kBufferWord3);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(vc + (int64_t)k0 * row_stride), 0, 0x7FFFFFFF, kBufferWord3);
#pragma unroll
    for (int uu = 0; uu < NLD; ++uu) {
      const auto kx = __builtin_amdgcn_raw_buffer_load_b128(kr, (int)cofs[uu], 0, 0);
      const auto vx = __builtin_amdgcn_raw_buffer_load_b128(vr, (int)cofs[uu], 0, 0);
      kreg[uu] = uint4{kx[0], kx[1], kx[2], kx[3]};
      vreg[uu] = uint4{vx[0], vx[1], vx[2], vx[3]};
    }
  };
  // a tile of any pair (its cache, new rows, lengths and KV head given)
  auto load_from = [&](int k0, const uint16_t *kcx, const uint16_t *vcx, const uint16_t *knx,
                       const uint16_t *vnx, int T0x, int Tx, int kvx) {
#pragma unroll
    for (int uu = 0; uu < NLD; ++uu) {
      const int e = tid + uu * AT;
      const int kr = e / CH, ch = e % CH;
      const int i = k0 + kr;
      uint4 k4 = {0u, 0u, 0u, 0u}, v4 = {0u, 0u, 0u, 0u};
      if (i < Tx) {
        const int64_t off = (i < T0x ? (int64_t)i : (int64_t)(i - T0x)) * row_stride + kvx * D + ch * 8;
        k4 = gload16((i < T0x ? kcx : knx) + off);
        v4 = gload16((i < T0x ? vcx : vnx) + off);
      }
      kreg[uu] = k4;
      vreg[uu] = v4;
    }
  };
  auto load_any = [&](int k0) { load_from(k0, kc, vc, kn, vn, T0, T, kv); };
  auto store_tile = [&](int b) {
#pragma unroll
    for (int uu = 0; uu < NLD; ++uu) {
      const int e = tid + uu * AT;
      const int kr = e / CH, ch = e % CH;
      *reinterpret_cast<uint4 *>(&Ks[b][kr][ch * 8]) = kreg[uu];
      *reinterpret_cast<uint4 *>(&Vs[b][kr][ch * 8]) = vreg[uu];
    }
  };

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) o[db] = f32x16{};
  float m_run = -1e30f, l_run = 0.f;
  const float c = a.scale_log2, inv_c = 1.f / c;
  float m_lim = (m_run + 8.f) * inv_c;

  // transposed-read coordinates of this lane inside its 16-lane group
  const int g16 = lane >> 4, s16 = lane & 15;
  const int tr_row = 4 * (g16 >> 1) + (s16 >> 2);
  const int tr_col = 16 * (g16 & 1) + 4 * (s16 & 3);

  // key tile t (keys from k0 = t * BN) of the current pair, in LDS buffer b.
  // `masked` is a std::integral_constant in the plain kernel's loops (the
  // mask code folds away per call site) and a uniform bool in stream mode,
  // whose single instance of this body fits the register budget (two
  // instances in one loop spill).
  auto compute = [&](int b, int t, auto masked) {
    const int k0 = t * BN;
    // S^T = K Q^T for two 32-key sub-tiles: lane = query row, register = key.
    f32x16 s[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      s[sub] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(&Ks[b][sub * 32 + l32][16 * kk + 8 * half]);
        s[sub] = mfma32(kf, qf[kk], s[sub]);
      }
    }
    // Schedule: kAheadK fragment reads, then one MFMA per read, so each MFMA's
    // operand was requested kAheadK MFMAs earlier (3% faster on the 7B
    // workload than all reads first).
#pragma unroll
    for (int i = 0; i < kAheadK; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
    for (int i = 0; i < 2 * (D / 16) - kAheadK; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < kAheadK; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (masked) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) {
          const int key = k0 + sub * 32 + 8 * (jj >> 2) + 4 * half + (jj & 3);
          if (key > vis) s[sub][jj] = -INFINITY;
        }
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) mx = fmaxf(mx, s[sub][jj]);
    }
    {
      // the other lane half's maximum (rows are split over the halves by key):
      // v_permlane32_swap exchanges the halves of a register pair, so the max
      // of its two results holds both halves' maxima in every lane
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      const float m0 = __uint_as_float(r[0]), m1 = __uint_as_float(r[1]);
      mx = m0 > m1 ? m0 : m1;   // (a compare and a select: fmaxf would first canonicalise both)
    }
    // Lazy rescaling: the running maximum only moves when a row's tile
    // maximum exceeds it by more than 2^8 (in the log2 domain), so
    // probabilities stay <= 256; the test compares the raw maximum with the
    // precomputed threshold (m_run + 8) / c.
    if (__any(mx > m_lim)) {
      const float m_new = fmaxf(m_run, mx * c);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      m_lim = (m_run + 8.f) * inv_c;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) o[db] *= alpha;
    }

    bf16x8 pf[4];
    float ls = 0.f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) {
        const float p = fast_exp2(fmaf(s[sub][jj], c, -m_run));
        ls += p;
        pf[2 * sub + (jj >> 3)][jj & 7] = static_cast<__bf16>(p);
      }
    }
    l_run += ls;

    // O^T += V^T P^T.  B element t of lane half hf in key group qq is key
    // 16 qq + 8 (t/4) + 4 hf + t%4; two transposed reads give the matching
    // V^T fragment (keys 16 qq + 4 hf + 0..3 and 16 qq + 8 + 4 hf + 0..3).
    // The wave streams these MFMAs at raised issue priority, so that the
    // other wave on the SIMD fills the issue cycles they leave free with its
    // softmax rather than competing with them (3% on the 7B workload).
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const uint16_t *vp = &Vs[b][16 * qq + tr_row][32 * db + tr_col];
        const s4 lo = lds_tr16(vp);
        const s4 hi = lds_tr16(vp + 8 * (D + VPAD));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        o[db] = mfma32(vf, pf[qq], o[db]);
      }
    }
    // the same for O^T += V^T P^T: two transposed reads per MFMA, kAheadV
    // MFMAs ahead
    constexpr int kPV = (D / 32) * 4;
#pragma unroll
    for (int i = 0; i < 2 * kAheadV; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
#pragma unroll
    for (int i = 0; i < kPV - kAheadV; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
    }
#pragma unroll
    for (int i = 0; i < kAheadV; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
    __builtin_amdgcn_s_setprio(0);
  };

  using NoMask = std::integral_constant<bool, false>;
  using Mask = std::integral_constant<bool, true>;
  // unnormalised partial state of the current pair into partial block blk:
  // bf16 O (half the bytes the combine reads back), fp32 running maximum and
  // row sum (they fix the LSE)
  auto flush = [&](int64_t blk) {
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (row_ok) {
      const int64_t row = blk * a.part_rows + prow;
      uint16_t *op = a.opart + row * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int d0 = 32 * db + 8 * grp + 4 * half;
          const uint32_t w0 = (uint32_t)f2bf(o[db][4 * grp + 0]) | ((uint32_t)f2bf(o[db][4 * grp + 1]) << 16);
          const uint32_t w1 = (uint32_t)f2bf(o[db][4 * grp + 2]) | ((uint32_t)f2bf(o[db][4 * grp + 3]) << 16);
          *reinterpret_cast<uint2 *>(op + d0) = uint2{w0, w1};
        }
      if (half == 0) *reinterpret_cast<float2 *>(a.mlpart + 2 * row) = float2{m_run, l_tot};
    }
  };
  if constexpr (STREAM) {
    // One tile loop over the range; leaving a pair (rare) flushes it, moves
    // to the next pair and loads that pair's first tile without prefetch.
    int t = x_lo - first;
    int pair_n = a.st_tiles[j];
    int k = j * Hkv + kv;
    if (t < n_pure) load_pure(t * BN); else load_any(t * BN);
    int b = 0;
    for (int x = x_lo; x < x_hi; ++x) {
      store_tile(b);
      __syncthreads();
      const bool pair_end = t + 1 == pair_n;
      if (!pair_end && x + 1 < x_hi) {
        if (t + 1 < n_pure) load_pure((t + 1) * BN); else load_any((t + 1) * BN);
      }
      // tiles past this query tile's own causal limit hold no visible key
      if (wave_rows && t < ntiles) compute(b, t, (t + 1) * BN - 1 > vis_min);
      if (pair_end && x + 1 < x_hi) {
        flush(u + k);
        if (kv + 1 < Hkv) enter(j, kv + 1); else enter(j + 1, 0);
        pair_n = a.st_tiles[j];
        ++k;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) o[db] = f32x16{};
        m_run = -1e30f;
        m_lim = (m_run + 8.f) * inv_c;
        l_run = 0.f;
        t = 0;
        if (n_pure > 0) load_pure(0); else load_any(0);
      } else {
        ++t;
      }
      b ^= 1;
    }
    flush(u + k);
    return;
  } else {
    // Steady state: the tile and the next one are pure (no branch in the
    // body); the last pure tile joins the general loop, where it is unmasked.
    if (n_pure > 0) load_pure(0); else load_any(0);
    int t = 0;
    // two tiles per trip, so that the LDS buffer of each is a constant and
    // its addresses fold into the instructions' offsets
    for (; t + 2 < n_pure; t += 2) {
      store_tile(0);
      __syncthreads();
      load_pure((t + 1) * BN);
      if (wave_rows) compute(0, t, NoMask{});
      store_tile(1);
      __syncthreads();
      load_pure((t + 2) * BN);
      if (wave_rows) compute(1, t + 1, NoMask{});
    }
    for (; t + 1 < n_pure; ++t) {
      store_tile(t & 1);
      __syncthreads();
      load_pure((t + 1) * BN);
      if (wave_rows) compute(t & 1, t, NoMask{});
    }
    for (; t < ntiles; ++t) {
      store_tile(t & 1);
      __syncthreads();
      if (t + 1 < ntiles) load_any((t + 1) * BN);
      if (!wave_rows) {
      } else if ((t + 1) * BN - 1 > vis_min) {
        compute(t & 1, t, Mask{});
      } else {
        compute(t & 1, t, NoMask{});
      }
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (row_ok) {
      if constexpr (WRITE_O) {
        uint16_t *orow = a.out + a.slot[j] * a.q_lstride + ((int64_t)r * Hq + kv * G + g) * D;
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
      }
      if (a.lse != nullptr && half == 0) {
        a.lse[a.layer_id[j] * a.lse_lstride + (int64_t)kv * P + prow] = m_run + log2f(l_tot);
      }
    }
  }
}


// Merge of a pair's partial blocks: m = max_s m_s, w_s = 2^(m_s - m),
// O = sum_s w_s O_s / sum_s w_s l_s, LSE = m + log2(sum_s w_s l_s).  Pair
// k = j Hkv + kv covers concatenated tiles [f, f + n); units u0 (holding
// tile f) to u1 (holding tile f + n - 1) wrote its blocks u0 + k .. u1 + k.
// One thread per (packed row, 8 channels), blocks summed in order.
template <int D>
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a) {
  const int j = blockIdx.z, kv = blockIdx.y;
  const int layer = a.layer_id[j];
  const int G = a.Hq / a.Hkv, P = a.C * G;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= P * (D / 8)) return;
  const int p = e / (D / 8), c8 = e % (D / 8);
  // the unit whose range [u N / U, (u + 1) N / U) holds tile x
  auto unit_of = [&](int64_t x) {
    return (int)(((x + 1) * a.st_units + a.st_total - 1) / a.st_total - 1);
  };
  const int64_t f = a.st_off[j] + (int64_t)kv * a.st_tiles[j];
  const int u0 = unit_of(f);
  const int nsp = unit_of(f + a.st_tiles[j] - 1) - u0 + 1;
  const int64_t row0 = ((int64_t)u0 + j * a.Hkv + kv) * a.part_rows + p;
  float m = -INFINITY;
  for (int s = 0; s < nsp; ++s) m = fmaxf(m, a.mlpart[2 * (row0 + (int64_t)s * a.part_rows)]);
  float lsum = 0.f, acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < nsp; ++s) {
    const int64_t row = row0 + (int64_t)s * a.part_rows;
    const float w = exp2f(a.mlpart[2 * row] - m);
    lsum += w * a.mlpart[2 * row + 1];
    const uint4 x = *reinterpret_cast<const uint4 *>(a.opart + row * D + 8 * c8);
    const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += w * __uint_as_float(xw[i] << 16);
      acc[2 * i + 1] += w * __uint_as_float(xw[i] & 0xffff0000u);
    }
  }
  const int r = p / G, h = kv * G + (p - r * G);
  if (a.out != nullptr) {
    const float inv = 1.f / lsum;
    uint16_t *orow = a.out + a.slot[j] * a.q_lstride + ((int64_t)r * a.Hq + h) * D + 8 * c8;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)f2bf(acc[2 * i] * inv) | ((uint32_t)f2bf(acc[2 * i + 1] * inv) << 16);
    *reinterpret_cast<uint4 *>(orow) = uint4{w[0], w[1], w[2], w[3]};
  }
  if (a.lse != nullptr && c8 == 0)
    a.lse[layer * a.lse_lstride + (int64_t)kv * P + p] = m + log2f(lsum);
}

template <int D>
__global__ __launch_bounds__(256, 3) void attn_colsum(ColsumArgs a, int nkb) {
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int kblk = lin % nkb;
  const int kv_blk = (lin / nkb) % a.Hkv;
  const int j = lin / (nkb * a.Hkv);
  const int layer = a.layer_id[j];
  const LayerTable &lt = a.tab[layer];
  const int cur = a.cur[j];
  const int T0 = a.T0[j];
  const int C = a.C, Hq = a.Hq, Hkv = a.Hkv;
  const int G = Hq / Hkv;
  const int P = C * G;
  const int T = a.ncand[j];        // candidates: T0 + C, or T0 for a prompt
  const int k0 = kblk * BK;
  if (k0 >= T) return;

  // wave index made scalar: the loop bounds below derive from it and stay uniform
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int half = lane >> 5, l32 = lane & 31;
  // Each wave owns 64 candidates (two MFMA column blocks of 32).
  const int kw0 = k0 + wave * 64;
  int key[2], pmin[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    key[kb] = kw0 + 32 * kb + l32;
    pmin[kb] = key[kb] < T0 ? 0 : (key[kb] - T0) * G;   // first packed row that sees it
  }
  // rows below pmask_end may be invisible to some candidate of this wave
  const int pmask_end = kw0 + 63 < T0 ? 0 : (kw0 + 63 - T0) * G + 1;
  const int p_begin = (k0 < T0 ? 0 : (k0 - T0) * G) & ~(BQS - 1);
  const int ntq = (P - p_begin + BQS - 1) / BQS;
  const int nit = ntq;

  const int slot = a.slot[j];
  const uint16_t *q = a.q + slot * a.q_lstride;
  const uint16_t *kn = a.kn + slot * a.kv_lstride;
  const uint16_t *kc = lt.k[cur];
  const float *lse_l = a.lse + layer * a.lse_lstride;
  const float c = a.scale_log2;

  // Ring of 32-row query tiles (four slots, so the slot index is a mask):
  // tile it is read by the MFMAs while tile it+2 is stored and tile it+3
  // loaded.
  __shared__ __attribute__((aligned(16))) uint16_t Qs[4][BQS][D + KPAD];
  __shared__ __attribute__((aligned(16))) float Ls[4][BQS];

  constexpr int CH = D / 8;
  constexpr int NLD = BQS * CH / 256;
  uint4 qreg[NLD];
  float lreg = INFINITY;
  auto tile_p = [&](int it) { return p_begin + it * BQS; };
  // Each thread loads NLD 16-byte pieces of one packed row of a tile (pieces
  // c and c + CH / NLD, ...), so one offset per thread serves all of them.
  // Tiles are loaded in order, so the thread's packed row p = (r, g) steps
  // by BQS per tile: r by BQS / G and g by BQS % G, plus one row when g wraps
  // past G; its byte offset moves by the matching fixed amounts.  The loads
  // go through a buffer descriptor over this slot's C chunk rows, so the
  // offset is a 32-bit register and rows past P (r >= C) lie outside the
  // descriptor's range, where the load returns zeros.
  constexpr int PPR = CH / NLD;             // pieces per thread-row group
  const int ld_row = tid / PPR, ld_c = tid % PPR;
  const __amdgpu_buffer_rsrc_t qrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)q, 0, C * Hq * D * (int)sizeof(uint16_t), kBufferWord3);
  const int step_r = BQS / G, step_g = BQS - (BQS / G) * G;
  const uint32_t ostep = (uint32_t)((step_r * Hq + step_g) * D * sizeof(uint16_t));
  const uint32_t owrap = (uint32_t)((Hq - G) * D * sizeof(uint16_t));
  int ld_g;
  uint32_t ld_o;
  {
    const int p = p_begin + ld_row;
    const int r0 = p / G;
    ld_g = p - r0 * G;
    ld_o = (uint32_t)((((int64_t)r0 * Hq + kv_blk * G + ld_g) * D + ld_c * 8) * sizeof(uint16_t));
  }
  // FULL: every row of the tile is < P (no bounds test on the LSE load)
  auto load_tile = [&](int it, auto full) {
    const int pt = tile_p(it);
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const auto x = __builtin_amdgcn_raw_buffer_load_b128(qrs, (int)(ld_o + u * PPR * 16), 0, 0);
      qreg[u] = uint4{x[0], x[1], x[2], x[3]};
    }
    ld_g += step_g;
    const bool wrap = ld_g >= G;
    ld_g -= wrap ? G : 0;
    ld_o += ostep + (wrap ? owrap : 0u);
    if (tid < BQS)
      lreg = (decltype(full)::value || pt + tid < P) ? lse_l[(int64_t)kv_blk * P + pt + tid] : INFINITY;
  };
  auto store_tile = [&](int b) {
#pragma unroll
    for (int u = 0; u < NLD; ++u)
      *reinterpret_cast<uint4 *>(&Qs[b][ld_row][(ld_c + u * PPR) * 8]) = qreg[u];
    if (tid < BQS) Ls[b][tid] = lreg;
  };

  bf16x8 kf[2][D / 16];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const bool ok = key[kb] < T;
    const uint16_t *krow = key[kb] < T0 ? kc + ((int64_t)key[kb] * Hkv + kv_blk) * D
                                        : kn + ((int64_t)(key[kb] - T0) * Hkv + kv_blk) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      kf[kb][kk] = ok ? __builtin_bit_cast(bf16x8, gload16(krow + 16 * kk + 8 * half)) : bf16x8{};
  }
  // S = Q K^T for one 32-row tile: lane = candidate, register = query row.
  auto scores = [&](int b, f32x16 *s) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const bf16x8 qv = *reinterpret_cast<const bf16x8 *>(&Qs[b][l32][16 * kk + 8 * half]);
      s[0] = mfma32(qv, kf[0][kk], s[0]);
      s[1] = mfma32(qv, kf[1][kk], s[1]);
    }
  };
  double wacc[2] = {0.0, 0.0};
  auto read_lse = [&](int b, float *lv) {
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const float4 l4 = *reinterpret_cast<const float4 *>(&Ls[b][8 * grp + 4 * half]);
      lv[4 * grp + 0] = l4.x;
      lv[4 * grp + 1] = l4.y;
      lv[4 * grp + 2] = l4.z;
      lv[4 * grp + 3] = l4.w;
    }
  };
  auto acc_masked = [&](int it, const f32x16 *s, const float *lv) {
    const int pt = tile_p(it);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float ts = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int prow = pt + 8 * (e >> 2) + 4 * half + (e & 3);
        const float p = fast_exp2(fmaf(s[kb][e], c, -lv[e]));
        ts += prow >= pmin[kb] ? p : 0.f;
      }
      wacc[kb] += (double)ts;
    }
  };
  auto acc_plain = [&](const f32x16 *s, const float *lv) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float t0 = fast_exp2(fmaf(s[kb][0], c, -lv[0]));
      float t1 = fast_exp2(fmaf(s[kb][1], c, -lv[1]));
#pragma unroll
      for (int e = 2; e < 16; e += 2) {
        t0 += fast_exp2(fmaf(s[kb][e], c, -lv[e]));
        t1 += fast_exp2(fmaf(s[kb][e + 1], c, -lv[e + 1]));
      }
      wacc[kb] += (double)(t0 + t1);
    }
  };
  // tiles [0, n_mask) touch the causal edge of this wave's candidates
  const int n_mask = min(nit, max(0, (pmask_end - p_begin + BQS - 1) / BQS));

  using Full = std::integral_constant<bool, true>;
  using Edge = std::integral_constant<bool, false>;
  // tiles [0, nfull) lie wholly below P
  const int nfull = (P - p_begin) / BQS;
  load_tile(0, Edge{});
  store_tile(0);
  if (nit > 1) {
    load_tile(1, Edge{});
    store_tile(1);
  }
  if (nit > 2) load_tile(2, Edge{});
  __syncthreads();
  // One tile per trip, scores then probabilities: without a second score
  // buffer the kernel fits three waves per SIMD, which hide the MFMA and LDS
  // latency better than overlapping two tiles inside one wave did.
  f32x16 s_cur[2];
  auto step = [&](int it, auto masked) {
    float lv[16];
    scores(it & 3, s_cur);
    read_lse(it & 3, lv);
    if constexpr (decltype(masked)::value) acc_masked(it, s_cur, lv); else acc_plain(s_cur, lv);
    if (it + 2 < nit) {
      store_tile((it + 2) & 3);
      if (it + 3 < nit) load_tile(it + 3, Edge{});
    }
    __syncthreads();
  };
  int it = 0;
  for (; it < n_mask; ++it) step(it, std::integral_constant<bool, true>{});
  // steady state: no branches inside the body
  for (; it + 3 < nfull; ++it) {
    float lv[16];
    scores(it & 3, s_cur);
    read_lse(it & 3, lv);
    acc_plain(s_cur, lv);
    store_tile((it + 2) & 3);
    load_tile(it + 3, Full{});
    __syncthreads();
  }
  for (; it < nit; ++it) step(it, std::integral_constant<bool, false>{});
  double *part = a.wpart + layer * a.wpart_lstride + (int64_t)kv_blk * a.wpart_hstride;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const double wsum = wacc[kb] + __shfl_xor(wacc[kb], 32);
    if (key[kb] < T && half == 0) part[key[kb]] = wsum;
  }
}

// W_i = sum over KV heads of the per-head partial masses, in head order.
// W_i = the head-order sum of the per-head fp64 partials, rounded to fp32;
// with it, per block of kNormBlock candidates, the fp64 partial of the
// attention-score normaliser sum_i alpha_i W_i over the rounded W (thread
// order within each wave by a fixed butterfly, then the waves in order).
__global__ __launch_bounds__(kNormBlock) void mass_reduce(ColsumArgs a) {
  const int j = blockIdx.y;
  const int layer = a.layer_id[j];
  const int T = a.ncand[j];
  if ((int)blockIdx.x * kNormBlock >= T) return;   // whole block past this layer's end
  const int i = blockIdx.x * kNormBlock + threadIdx.x;
  double m = 0.0;
  if (i < T) {
    const double *part = a.wpart + layer * a.wpart_lstride + i;
    double w = 0.0;
    for (int kv = 0; kv < a.Hkv; ++kv) w += part[(int64_t)kv * a.wpart_hstride];
    const float wf = (float)w;
    a.tab[layer].w[i] = wf;
    m = mass_over_observers(wf, i, a.T0[j], a.C, a.alpha_mode[j]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m += __shfl_xor(m, o);
  __shared__ double red[kNormBlock / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < kNormBlock / 64; ++w) s += red[w];
    a.normpart[layer * a.normpart_lstride + blockIdx.x] = s;
  }
}

}  // namespace

hipError_t launch_attention(const AttnArgs &a, int n_list, int head_dim, hipStream_t s) {
  const int P = a.C * (a.Hq / a.Hkv);
  const int nqt = (P + BM - 1) / BM;
  dim3 grid(nqt * a.Hkv * n_list);
  const bool wo = a.out != nullptr;
  if (head_dim == 64) {
    if (wo) hipLaunchKernelGGL((attn_fwd<64, false, true>), grid, dim3(AT), 0, s, a, nqt);
    else hipLaunchKernelGGL((attn_fwd<64, false, false>), grid, dim3(AT), 0, s, a, nqt);
  } else {
    if (wo) hipLaunchKernelGGL((attn_fwd<128, false, true>), grid, dim3(AT), 0, s, a, nqt);
    else hipLaunchKernelGGL((attn_fwd<128, false, false>), grid, dim3(AT), 0, s, a, nqt);
  }
  return hipGetLastError();
}

hipError_t launch_attention_stream(const AttnArgs &a, int n_list, int head_dim, hipStream_t s) {
  const int P = a.C * (a.Hq / a.Hkv);
  const int nqt = (P + BM - 1) / BM;
  dim3 grid(a.st_units * nqt);
  dim3 cgrid((P * (head_dim / 8) + 255) / 256, a.Hkv, n_list);
  if (head_dim == 64) {
    hipLaunchKernelGGL((attn_fwd<64, true, true>), grid, dim3(AT), 0, s, a, nqt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_combine<64>, cgrid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((attn_fwd<128, true, true>), grid, dim3(AT), 0, s, a, nqt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_combine<128>, cgrid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_colsum(const ColsumArgs &a, int n_list, int max_T, int head_dim,
                         hipStream_t s) {
  const int nkb = (max_T + BK - 1) / BK;
  dim3 grid(nkb * a.Hkv * n_list);
  if (head_dim == 64) {
    hipLaunchKernelGGL(attn_colsum<64>, grid, dim3(256), 0, s, a, nkb);
  } else {
    hipLaunchKernelGGL(attn_colsum<128>, grid, dim3(256), 0, s, a, nkb);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mass_reduce, dim3((max_T + kNormBlock - 1) / kNormBlock, n_list), dim3(kNormBlock), 0, s, a);
  return hipGetLastError();
}

}  // namespace hermes
