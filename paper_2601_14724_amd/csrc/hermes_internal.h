// Internal declarations shared by the host entry points (hermes_api.cpp) and
// the gfx950 kernels (*.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hermes.h"

namespace hermes {

constexpr int kMaxLayers = HERMES_MAX_LAYERS;
constexpr int kMaxHalfDim = 64;   // frequency pairs of the largest head size (128)
// Summary metadata per layer: insert index, stream position, RoPE position
// (t with M-RoPE), evicted count, then h and w with M-RoPE.
constexpr int kSumMeta = 8;
// 3D re-indexing ranks an axis's coordinates through an LDS bitmap over a
// window of this many consecutive values, one window after another.
constexpr int kMropeWindow = 262144;

// Static per-layer description, uploaded once into the workspace.
struct LayerTable {
  uint16_t *k[2];
  uint16_t *v[2];
  int32_t *pos[2];
  int32_t *rpos[2];         // RoPE positions of the stored keys (null when not kept); t with M-RoPE
  int32_t *rpos_h[2];       // M-RoPE h and w coordinates (null unless three axes)
  int32_t *rpos_w[2];
  float *w;
  float *s_dbg;
  int32_t *kept_dbg;
  int32_t cap;
  int32_t budget;
  int32_t cls;
  int32_t pad_;
  double lambda;
  double omega;
};

// Chunk (or query) attention: launch entry j covers layer layer_id[j], reads
// cached rows [0, T0[j]) of buffer cur[j] and new rows from the stacked inputs
// at slot j (stride *_lstride elements), writes out (if non-null) and lse (if
// non-null).
struct AttnArgs {
  const LayerTable *tab;
  const uint16_t *q, *kn, *vn;
  uint16_t *out;
  float *lse;               // [n_layers][Hkv][C*G] log2-domain row LSE, or null
  int64_t q_lstride, kv_lstride, lse_lstride;
  int32_t Hq, Hkv, C;
  float scale_log2;         // sm_scale * log2(e)
  int32_t T0[kMaxLayers];
  int8_t layer_id[kMaxLayers];
  int8_t slot[kMaxLayers];      // index of the layer's inputs in the stacked tensors
  int8_t cur[kMaxLayers];
  // Stream mode (short passes): the key tiles of every (entry, KV head) pair,
  // concatenated in pair order (entry j's Hkv pairs of st_tiles[j] tiles each
  // start at tile st_off[j]; st_total tiles in all), are cut into st_units
  // equal ranges of nqt workgroups each.  Unit u writes the unnormalised O
  // (bf16), running maximum and row sum (fp32) of each pair k it touches to
  // opart / mlpart block u + k ([block][part_rows]); a combine kernel merges
  // each pair's blocks.  st_units = 0: the plain kernel, one workgroup per
  // (entry, KV head, query tile).
  int32_t st_units, st_total, st_entries, part_rows;
  int32_t st_off[kMaxLayers + 1];
  int32_t st_tiles[kMaxLayers];
  uint16_t *opart;          // [..][part_rows][d] bf16 (unnormalised; its scale is in mlpart)
  float *mlpart;            // [..][part_rows][2] fp32 (max, sum)
};

// Attention-mass sweep: W_i for the candidates i < ncand[j] of layer
// layer_id[j] (ncand = T0 + C for the chunk's own mass, T0 for a guidance
// prompt, whose rows are not candidates).  Each KV head's share goes to
// wpart[layer][kv][i] (fp64), then is summed into the layer's w buffer in
// head order.
struct ColsumArgs {
  const LayerTable *tab;
  const uint16_t *q, *kn, *vn;
  const float *lse;
  double *wpart;
  double *normpart;         // [n_layers][normpart_lstride] fp64 partials of sum_i alpha_i W_i
  int64_t q_lstride, kv_lstride, lse_lstride, wpart_lstride, wpart_hstride, normpart_lstride;
  int32_t Hq, Hkv, C;
  float scale_log2;
  int32_t T0[kMaxLayers];
  int32_t ncand[kMaxLayers];
  int8_t layer_id[kMaxLayers];
  int8_t slot[kMaxLayers];
  int8_t cur[kMaxLayers];
  int8_t alpha_mode[kMaxLayers];   // weighting of the normaliser partials (0 per observer, 1 plain)
};

// Scoring, smoothing and selection; one workgroup per listed layer.  len and
// cur are indexed by LAYER (the smoothing reads layer l+1).
struct SelectArgs {
  const LayerTable *tab;
  uint32_t *keys;           // [n_layers][max_cap]
  int32_t *kept;            // [n_layers][max_budget]
  const double *normpart;   // normaliser partials written with W (kNormBlock candidates each)
  int64_t keys_lstride, kept_lstride, normpart_lstride;
  double forget_rate;
  int32_t n_layers, C, alpha_mode, align_mode;
  int32_t n_list;           // layers over budget, in layer_id
  int32_t len[kMaxLayers];
  int32_t guide_rows[kMaxLayers];   // by layer: > 0 = W came from that many prompt rows
  double inv_z[kMaxLayers];   // by layer: 1 / Z, Z = sum_{i<len} e^{-k i} = (1 - e^{-k len}) / (1 - e^{-k})
  double ek;                  // e^{k}
  double inv_c;               // 1 / C
  int8_t cur[kMaxLayers];
  int8_t layer_id[kMaxLayers];
};

// Order-preserving gather of kept rows into the other buffer of each pair,
// optionally with a summary row inserted and with RoPE re-indexing.
// mode[j] 0: rows [0, row_start[j+1] - row_start[j]) of the other buffer
// from the kept list (and the summary row when has_sum[j]); mode 1: the
// layer did not evict, re-index its current buffer in place.
struct GatherArgs {
  const LayerTable *tab;
  const int32_t *kept;
  int64_t kept_lstride;
  int32_t row_elems;        // Hkv * d
  int32_t head_dim;
  int32_t n_list;
  int32_t reindex;          // 0 never, 1 always, 2 when *flag != 0
  int32_t rope_offset;
  double inv_freq[kMaxHalfDim];   // RoPE frequencies theta_j = base^(-2j/d), host-computed
  const int32_t *flag;      // lazy re-indexing decision (device)
  const uint16_t *sum_k, *sum_v;   // [n_layers][row_elems] staged summary rows
  const int32_t *sum_meta;  // [n_layers][kSumMeta]
  int32_t axes;             // 1, or 3 for M-RoPE (t, h, w)
  int32_t section[3];       // M-RoPE: frequency pairs of the t, h, w sections
  const int32_t *newc;      // M-RoPE: [n_layers][3][newc_lstride] re-indexed coordinates by output row
  int64_t newc_lstride;
  int32_t row_start[kMaxLayers + 1];   // prefix of output rows over the list
  int8_t layer_id[kMaxLayers];
  int8_t cur[kMaxLayers];
  int8_t mode[kMaxLayers];
  int8_t has_sum[kMaxLayers];
};

// Summary token of every listed (deep, evicting) layer: fp64 partial sums of
// the evicted rows per block of kSummaryRows candidates, then the mean.
struct SummaryArgs {
  const LayerTable *tab;
  const int32_t *kept;
  int64_t kept_lstride;
  double *part;             // [n_layers][blocks][2 * row_elems]
  int64_t part_lstride;
  uint16_t *sum_k, *sum_v;  // [n_layers][row_elems]
  int32_t *sum_meta;        // [n_layers][kSumMeta]
  int32_t row_elems, head_dim, n_list;
  int32_t axes;             // 3: keys aligned to the target's (t, h, w) section by section
  int32_t section[3];
  double inv_freq[kMaxHalfDim];   // RoPE frequencies theta_j = base^(-2j/d), host-computed
  int32_t len[kMaxLayers];      // by entry: candidates T
  int32_t budget[kMaxLayers];   // by entry: kept M
  int8_t layer_id[kMaxLayers];
  int8_t cur[kMaxLayers];
};

// Lazy re-indexing decision: the largest RoPE position each layer retains
// after this compression, against limit - headroom.
struct DecideArgs {
  const LayerTable *tab;
  const int32_t *kept;
  int64_t kept_lstride;
  const int32_t *sum_meta;
  int32_t *flag;
  int32_t n_layers, limit, headroom;
  int32_t axes;             // 3: the largest of the t, h and w coordinates
  int32_t len[kMaxLayers];      // by layer: T before compression
  int32_t budget[kMaxLayers];
  int8_t cur[kMaxLayers];
  int8_t evicts[kMaxLayers];
  int8_t has_sum[kMaxLayers];
};

// M-RoPE ranks (appendix, 3D re-indexing): for list entry j and axis a, the
// coordinate of every output row (mode 0: kept row kept[r] of the current
// buffer; mode 1: row r in place) becomes offset + the number of distinct
// retained coordinates below it, written to newc[layer][a][r].
struct RankArgs {
  const LayerTable *tab;
  const int32_t *kept;
  int64_t kept_lstride;
  const int32_t *sum_meta;  // summary rows (has_sum): insert index and (t, h, w)
  int32_t *newc;
  int64_t newc_lstride;
  const int32_t *flag;      // lazy decision (device)
  int32_t reindex;          // 0 never, 1 always, 2 when *flag != 0
  int32_t offset;
  int32_t n_list;
  int32_t row_start[kMaxLayers + 1];
  int8_t layer_id[kMaxLayers];
  int8_t cur[kMaxLayers];
  int8_t mode[kMaxLayers];
  int8_t has_sum[kMaxLayers];
};

// Append copy: new K/V rows and positions into rows [T0, T0 + C) of the
// current buffer of each listed layer.
struct AppendArgs {
  const LayerTable *tab;
  const uint16_t *kn, *vn;
  const int32_t *pos;
  const int32_t *rope_pos;  // RoPE positions of the new rows (null: = pos); t with M-RoPE
  const int32_t *rope_h, *rope_w;   // M-RoPE h and w of the new rows (null unless three axes)
  int64_t kv_lstride;
  int32_t row_elems, C, n_list;
  int32_t T0[kMaxLayers];
  int8_t layer_id[kMaxLayers];
  int8_t slot[kMaxLayers];
  int8_t cur[kMaxLayers];
};

// Device scratch of the no-allocation context entry point (scratch.hip):
// kStaticWorkspaceBytes per GPU.  acquire looks up the array's address on the
// current device (once per device) and marks it owned: HERMES_ESTATE while
// another context owns it, HERMES_ENOTSUP beyond kMaxDevices GPUs.
constexpr size_t kStaticWorkspaceBytes = (size_t)HERMES_STATIC_WORKSPACE_BYTES;
constexpr int kMaxDevices = 64;
int static_workspace_acquire(void **ptr, int *device);
void static_workspace_release(int device);

// Launchers (return the hipError_t of the launch).
hipError_t launch_attention(const AttnArgs &a, int n_list, int head_dim, hipStream_t s);
hipError_t launch_attention_stream(const AttnArgs &a, int n_list, int head_dim, hipStream_t s);
hipError_t launch_colsum(const ColsumArgs &a, int n_list, int max_T, int head_dim,
                         hipStream_t s);
hipError_t launch_select(const SelectArgs &a, hipStream_t s);
// Precondition checks (device side): q, k, v bf16 with nq / nkv elements
// (multiples of 8, 16-byte aligned), the chunk positions pos[0..n_new) (or
// null) against the last cached position of each listed layer; violations
// are ORed into *flag.
struct CheckArgs {
  const LayerTable *tab;
  const uint16_t *q, *k, *v;
  int64_t nq, nkv;
  const int32_t *pos;
  int32_t n_new;
  int32_t n_list;
  int32_t len[kMaxLayers];
  int8_t layer_id[kMaxLayers];
  int8_t cur[kMaxLayers];
  int32_t *flag;
};

hipError_t launch_check(const CheckArgs &a, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);
hipError_t launch_append(const AppendArgs &a, hipStream_t s);
hipError_t launch_topk(const float *keys, int n, int k, int32_t *out, hipStream_t s);
hipError_t launch_summary(const SummaryArgs &a, int max_T, hipStream_t s);
hipError_t launch_decide(const DecideArgs &a, hipStream_t s);
hipError_t launch_gather_rope(const GatherArgs &a, hipStream_t s);
hipError_t launch_mrope_rank(const RankArgs &a, hipStream_t s);

// Geometry shared by host sizing and kernels.
constexpr int kAttnRowsPerBlock = 256;   // packed (row, head) pairs per attention workgroup
constexpr int kColsumKeysPerBlock = 256; // candidates per workgroup of the sweep
constexpr int kSummaryRows = 128;        // candidates per workgroup of the summary sums
constexpr int kSplitMaxTokens = 64;      // passes of at most this many rows use stream mode
constexpr int kStreamSlots = 256;        // resident attention workgroups (one per CU)
constexpr int kNormBlock = 256;         // candidates per fp64 partial of the score normaliser

}  // namespace hermes
