// Host side of libhermes.so: argument and state validation, per-layer
// bookkeeping, and the launches of the gfx950 kernels on the caller's stream.
// Every check runs before the first launch of a call, so a rejected call
// leaves device data and host lengths untouched.
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>
#include <utility>
#include <vector>

#include "hermes_internal.h"

using namespace hermes;

namespace {

constexpr double kLog2e = 1.4426950408889634;
constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Layout {
  size_t tab, lse, keys, kept, normpart, newc, wpart, spart, sumk, sumv, smeta, flag, opart, mlpart, total;
  int64_t lse_lstride, keys_lstride, kept_lstride, wpart_lstride, spart_lstride, normpart_lstride,
      newc_lstride;
  int32_t part_rows;
  int64_t part_blocks;      // stream-mode partial blocks of part_rows rows the workspace holds
};

int max_budget(const hermes_config *c) {
  int m = 1;
  for (int l = 0; l < c->n_layers; ++l) m = c->budget[l] > m ? c->budget[l] : m;
  return m;
}

int check_config(const hermes_config *c) {
  if (c == nullptr) return HERMES_EINVAL;
  if (c->n_layers < 1 || c->n_layers > HERMES_MAX_LAYERS) return HERMES_EINVAL;
  if (c->n_kv_heads < 1 || c->n_q_heads < c->n_kv_heads) return HERMES_EINVAL;
  if (c->n_q_heads % c->n_kv_heads != 0) return HERMES_EINVAL;
  if (c->head_dim != 64 && c->head_dim != 128) return HERMES_ENOTSUP;
  if (c->max_chunk < 1 || c->max_cap < 1) return HERMES_EINVAL;
  const int64_t packed = (int64_t)c->max_chunk * (c->n_q_heads / c->n_kv_heads);
  if (packed > (int64_t)1 << 30) return HERMES_EINVAL;
  if (c->budget == nullptr) return HERMES_EINVAL;
  for (int l = 0; l < c->n_layers; ++l) {
    if (c->budget[l] < 1) return HERMES_EINVAL;
    if (c->layer_class != nullptr && (c->layer_class[l] < HERMES_SHALLOW ||
                                      c->layer_class[l] > HERMES_DEEP))
      return HERMES_EINVAL;
    if (c->lambda != nullptr &&
        !(std::isfinite(c->lambda[l]) && c->lambda[l] >= 0.f && c->lambda[l] <= 1.f))
      return HERMES_EINVAL;
  }
  if (c->alpha_mode != 0 && c->alpha_mode != 1) return HERMES_EINVAL;
  if (c->align_mode != 0 && c->align_mode != 1) return HERMES_EINVAL;
  if (!std::isfinite(c->omega0) || !std::isfinite(c->gamma)) return HERMES_EINVAL;
  if (!std::isfinite(c->forget_rate) || !std::isfinite(c->sm_scale)) return HERMES_EINVAL;
  if (c->summary_mode != 0 && c->summary_mode != 1) return HERMES_EINVAL;
  if (c->reindex_mode < HERMES_REINDEX_NONE || c->reindex_mode > HERMES_REINDEX_LAZY)
    return HERMES_EINVAL;
  if (c->scoring_mode != HERMES_SCORE_CHUNK && c->scoring_mode != HERMES_SCORE_GUIDANCE)
    return HERMES_EINVAL;
  if (c->rope_offset < 0 || c->rope_limit < 0 || c->rope_headroom < 0) return HERMES_EINVAL;
  if (!std::isfinite(c->rope_theta)) return HERMES_EINVAL;
  if (c->rope_axes != 0 && c->rope_axes != 1 && c->rope_axes != 3) return HERMES_EINVAL;
  if (c->rope_axes == 3) {
    const int *sec = c->mrope_section;
    if (sec[0] != 0 || sec[1] != 0 || sec[2] != 0) {
      if (sec[0] < 0 || sec[1] < 0 || sec[2] < 0) return HERMES_EINVAL;
      if (sec[0] + sec[1] + sec[2] != c->head_dim / 2) return HERMES_EINVAL;
    }
  }
  // The RoPE kernels give each lane one frequency and at most 8 rotate pairs.
  if ((c->summary_mode || c->reindex_mode || c->rope_axes == 3) && c->n_kv_heads * c->head_dim > 1024)
    return HERMES_ENOTSUP;
  return HERMES_OK;
}

// Workspace layout of `c`; part_blocks < 0 sizes the stream-mode partial
// state for the most blocks any short pass can write (one per unit plus one
// per (layer, KV head) pair), else for that many partial blocks.
Layout layout_of(const hermes_config *c, int64_t part_blocks = -1) {
  Layout s;
  s.lse_lstride = (int64_t)c->n_q_heads * c->max_chunk;
  s.keys_lstride = c->max_cap;
  s.kept_lstride = max_budget(c);
  size_t off = 0;
  s.tab = off;
  off = round_up(off + sizeof(LayerTable) * c->n_layers);
  s.lse = off;
  off = round_up(off + sizeof(float) * (size_t)s.lse_lstride * c->n_layers);
  s.keys = off;
  off = round_up(off + sizeof(uint32_t) * (size_t)s.keys_lstride * c->n_layers);
  s.kept = off;
  off = round_up(off + sizeof(int32_t) * (size_t)s.kept_lstride * c->n_layers);
  // fp64 partials of the attention-score normaliser, one per kNormBlock candidates
  s.normpart_lstride = (c->max_cap + kNormBlock - 1) / kNormBlock;
  s.normpart = off;
  off = round_up(off + sizeof(double) * (size_t)s.normpart_lstride * c->n_layers);
  // M-RoPE: re-indexed (t, h, w) of every output row
  s.newc_lstride = c->rope_axes == 3 ? c->max_cap : 0;
  s.newc = off;
  off = round_up(off + sizeof(int32_t) * 3 * (size_t)s.newc_lstride * c->n_layers);
  s.wpart_lstride = (int64_t)c->n_kv_heads * c->max_cap;
  s.wpart = off;
  off = round_up(off + sizeof(double) * (size_t)s.wpart_lstride * c->n_layers);
  // summary token: fp64 block sums, staged bf16 rows and their metadata
  const int64_t row = (int64_t)c->n_kv_heads * c->head_dim;
  const int64_t nblk = c->summary_mode ? (c->max_cap + kSummaryRows - 1) / kSummaryRows : 0;
  s.spart_lstride = nblk * 2 * row;
  s.spart = off;
  off = round_up(off + sizeof(double) * (size_t)s.spart_lstride * c->n_layers);
  s.sumk = off;
  off = round_up(off + (c->summary_mode ? sizeof(uint16_t) * (size_t)row * c->n_layers : 0));
  s.sumv = off;
  off = round_up(off + (c->summary_mode ? sizeof(uint16_t) * (size_t)row * c->n_layers : 0));
  s.smeta = off;
  off = round_up(off + sizeof(int32_t) * kSumMeta * (size_t)c->n_layers);
  s.flag = off;
  off = round_up(off + sizeof(int32_t) * 4);
  // stream-mode partial state of short passes (query, guidance prompt)
  s.part_rows = kSplitMaxTokens * (c->n_q_heads / c->n_kv_heads);
  s.part_blocks = part_blocks >= 0 ? part_blocks : (int64_t)c->n_layers * c->n_kv_heads + kStreamSlots;
  const size_t prow = (size_t)s.part_blocks * s.part_rows;
  s.opart = off;
  off = round_up(off + sizeof(uint16_t) * prow * c->head_dim);
  s.mlpart = off;
  off = round_up(off + sizeof(float) * prow * 2);
  s.total = off;
  return s;
}

// The layout of `c` in at most `limit` bytes: the default one if it fits,
// else the same with as many stream-mode partial blocks as the rest leaves
// (possibly none: short passes then run the plain kernel).  false if even
// that exceeds `limit`.
bool layout_within(const hermes_config *c, size_t limit, Layout *out) {
  const Layout full = layout_of(c);
  if (full.total <= limit) {
    *out = full;
    return true;
  }
  const Layout none = layout_of(c, 0);
  if (none.total > limit) return false;
  const size_t per_block = (size_t)none.part_rows * (sizeof(uint16_t) * c->head_dim + 2 * sizeof(float));
  int64_t blocks = (int64_t)((limit - none.total) / per_block);
  // the two regions are rounded up separately: back off until it fits
  while (blocks > 0 && layout_of(c, blocks).total > limit) --blocks;
  *out = layout_of(c, blocks);
  return true;
}

// Stream plan of a short pass (n_rows <= kSplitMaxTokens rows per entry over
// caches of at.T0[j] tokens).  The plain kernel runs one workgroup per
// (entry, KV head, query tile) over its whole cache, so the entry with the
// longest cache sets the time while the other CUs idle.  Stream mode cuts
// the concatenated key tiles of all pairs into U equal ranges, U units of
// nqt workgroups filling one round of kStreamSlots, so every CU gets the same
// number of tiles; it pays a partial write per (unit, pair) touched and the
// combine launch.  Costs in key-tile times: a round also pays about two
// tiles of fixed work (query load, epilogue), the combine about two, and the
// partial writes about one tile per 64 * 128 / D workgroup blocks.  Stream
// mode is used when it promises at least 10% over the plain kernel and the
// workspace holds its U + pairs - 1 partial blocks.  Fills the st_* fields
// (st_units = 0 for the plain kernel).
void stream_plan(AttnArgs &at, int n_rows, int G, int Hkv, int n_list, int D, int64_t max_blocks) {
  const int nqt = (n_rows * G + kAttnRowsPerBlock - 1) / kAttnRowsPerBlock;
  at.st_units = 0;
  at.st_entries = n_list;
  int64_t total = 0;
  int max_tiles = 1;
  for (int j = 0; j < n_list; ++j) {
    const int tiles = (at.T0[j] + n_rows + 63) / 64;
    at.st_tiles[j] = tiles;
    at.st_off[j] = (int32_t)total;
    total += (int64_t)Hkv * tiles;
    max_tiles = tiles > max_tiles ? tiles : max_tiles;
  }
  at.st_off[n_list] = (int32_t)total;
  at.st_total = (int32_t)total;
  if (n_rows > kSplitMaxTokens || total > INT32_MAX / 2) return;
  const int64_t pairs = (int64_t)n_list * Hkv;
  int64_t units = kStreamSlots / nqt;
  units = units < total ? units : total;
  units = units < max_blocks - pairs + 1 ? units : max_blocks - pairs + 1;
  if (units < 2) return;
  auto rounds = [](int64_t w) { return (double)((w + kStreamSlots - 1) / kStreamSlots); };
  const double plain = rounds((int64_t)nqt * pairs) * (max_tiles + 2.0);
  const double per_unit = (double)((total + units - 1) / units);
  const double stream = per_unit + 2.0 + 2.0 + (double)(units + pairs) * nqt * D / (64.0 * 128.0);
  if (stream < 0.9 * plain) at.st_units = (int32_t)units;
}

// RoPE frequencies theta_j = base^(-2j/d), j < d/2 (rotate-half pairs), in
// double on the host: the kernels read them instead of evaluating pow.
void rope_frequencies(double base, int d, double *out) {
  for (int j = 0; j < d / 2 && j < kMaxHalfDim; ++j) out[j] = std::pow(base, (-2.0 * (double)j) / (double)d);
}

// 10% shallow, 60% middle, 30% deep (Sec. 4.1), rounded to nearest layer.
std::vector<int8_t> default_classes(int L) {
  const int n_sh = (int)std::floor(0.1 * L + 0.5);
  const int n_dp = (int)std::floor(0.3 * L + 0.5);
  std::vector<int8_t> c(L, HERMES_MIDDLE);
  for (int l = 0; l < L; ++l) {
    if (l < n_sh) c[l] = HERMES_SHALLOW;
    else if (l >= L - n_dp) c[l] = HERMES_DEEP;
  }
  return c;
}

struct EventPair {
  hipEvent_t start, stop;
};

}  // namespace

struct hermes_ctx {
  int L, Hq, Hkv, D, max_chunk, max_cap;
  double forget_rate, sm_scale;
  int alpha_mode, align_mode, force_scores;
  int summary_mode, reindex_mode, scoring_mode;
  int rope_offset, rope_limit, rope_headroom;
  double rope_theta;
  int rope_axes = 1;
  int section[3] = {0, 0, 0};       // M-RoPE frequency pairs of t, h, w
  bool keep_rpos = false;
  std::vector<int32_t> guided;      // prompt rows of this step's guidance score (0 = none)
  std::vector<int32_t> budget;
  std::vector<int8_t> cls;
  std::vector<double> lambda, omega;
  std::vector<hermes_layer_buffers> bufs;
  std::vector<int32_t> len;
  std::vector<int8_t> cur, appended, buf0_dirty;
  std::vector<int32_t> init_len;
  int32_t step_n_new = 0;
  int n_appended = 0;
  bool poisoned = false;
  Layout lay;
  char *ws = nullptr;
  LayerTable *d_tab = nullptr;
  bool prof = false;
  bool check = false;   // device-side precondition checks before each call's launches
  int static_dev = -1;  // device whose static scratch is the workspace (-1: the caller's)
  std::vector<EventPair> used[HERMES_K_COUNT];
  std::vector<EventPair> pool;

  int prof_begin(int id, hipStream_t s, EventPair *ep) {
    if (!prof) return HERMES_OK;
    if (pool.empty()) {
      EventPair e;
      if (hipEventCreate(&e.start) != hipSuccess) return HERMES_EHIP;
      if (hipEventCreate(&e.stop) != hipSuccess) return HERMES_EHIP;
      pool.push_back(e);
    }
    *ep = pool.back();
    pool.pop_back();
    if (hipEventRecord(ep->start, s) != hipSuccess) return HERMES_EHIP;
    (void)id;
    return HERMES_OK;
  }
  int prof_end(int id, hipStream_t s, const EventPair &ep) {
    if (!prof) return HERMES_OK;
    if (hipEventRecord(ep.stop, s) != hipSuccess) return HERMES_EHIP;
    used[id].push_back(ep);
    return HERMES_OK;
  }
  // Launch wrapper: events around the launch when profiling, poison on error.
  template <typename F>
  int run(int id, hipStream_t s, F &&launch) {
    EventPair ep{};
    if (prof_begin(id, s, &ep) != HERMES_OK) {
      poisoned = true;
      return HERMES_EHIP;
    }
    if (launch() != hipSuccess) {
      poisoned = true;
      return HERMES_EHIP;
    }
    if (prof_end(id, s, ep) != HERMES_OK) {
      poisoned = true;
      return HERMES_EHIP;
    }
    return HERMES_OK;
  }
};

// Device-side precondition checks of one call (when enabled): q, k, v of
// nq / nkv bf16 elements finite, and, with pos, the chunk positions strictly
// increasing and after the last cached position of every listed layer.  Waits
// for the verdict, so a failing call has launched nothing else: EINVAL.
static int run_checks(hermes_ctx *ctx, const std::vector<int> &list, const void *q, const void *k,
                      const void *v, int64_t nq, int64_t nkv, const int32_t *pos, int n_new,
                      hipStream_t s) {
  if (!ctx->check) return HERMES_OK;
  CheckArgs ca;
  std::memset(&ca, 0, sizeof(ca));
  ca.tab = ctx->d_tab;
  ca.q = static_cast<const uint16_t *>(q);
  ca.k = static_cast<const uint16_t *>(k);
  ca.v = static_cast<const uint16_t *>(v);
  ca.nq = nq;
  ca.nkv = nkv;
  ca.pos = pos;
  ca.n_new = n_new;
  ca.n_list = pos != nullptr ? (int)list.size() : 0;
  for (size_t j = 0; j < list.size(); ++j) {
    ca.layer_id[j] = (int8_t)list[j];
    ca.cur[j] = ctx->cur[list[j]];
    ca.len[j] = ctx->len[list[j]];
  }
  ca.flag = reinterpret_cast<int32_t *>(ctx->ws + ctx->lay.flag) + 2;   // [0] is the re-indexing decision
  int32_t verdict = 0;
  if (hipMemsetAsync(ca.flag, 0, sizeof(int32_t), s) != hipSuccess || launch_check(ca, s) != hipSuccess ||
      hipMemcpyAsync(&verdict, ca.flag, sizeof(int32_t), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess) {
    ctx->poisoned = true;
    return HERMES_EHIP;
  }
  return verdict == 0 ? HERMES_OK : HERMES_EINVAL;
}

extern "C" {

const char *hermes_strerror(int code) {
  switch (code) {
    case HERMES_OK: return "ok";
    case HERMES_EINVAL: return "invalid argument";
    case HERMES_ECAPACITY: return "buffer capacity exceeded";
    case HERMES_ESTATE: return "call not allowed in the current state";
    case HERMES_EHIP: return "HIP runtime error";
    case HERMES_ENOTSUP: return "unsupported shape";
    default: return "unknown error";
  }
}

size_t hermes_workspace_bytes(const hermes_config *cfg) {
  if (check_config(cfg) != HERMES_OK) return 0;
  return layout_of(cfg).total;
}

}  // extern "C"

// Buffer checks and context creation over a workspace of layout `lay`.
static int init_context(const hermes_config *cfg, const hermes_layer_buffers *layers, void *workspace,
                        const Layout &lay, hermes_ctx **out) {
  if (layers == nullptr) return HERMES_EINVAL;
  const int L = cfg->n_layers;
  for (int l = 0; l < L; ++l) {
    const hermes_layer_buffers &b = layers[l];
    for (int p = 0; p < 2; ++p) {
      if (b.k[p] == nullptr || b.v[p] == nullptr || b.pos[p] == nullptr) return HERMES_EINVAL;
      if (!aligned(b.k[p], 16) || !aligned(b.v[p], 16) || !aligned(b.pos[p], 4))
        return HERMES_EINVAL;
    }
    if (b.w == nullptr || !aligned(b.w, 4)) return HERMES_EINVAL;
    if (b.cap < 1 || b.init_len < 0) return HERMES_EINVAL;
    if (b.cap > cfg->max_cap || b.init_len > b.cap || cfg->budget[l] > b.cap)
      return HERMES_ECAPACITY;
    if (cfg->summary_mode || cfg->reindex_mode || cfg->rope_axes == 3) {
      for (int p = 0; p < 2; ++p)
        if (b.rpos[p] == nullptr || !aligned(b.rpos[p], 4)) return HERMES_EINVAL;
    }
    if (cfg->rope_axes == 3) {
      for (int p = 0; p < 2; ++p)
        if (b.rpos_h[p] == nullptr || b.rpos_w[p] == nullptr || !aligned(b.rpos_h[p], 4) ||
            !aligned(b.rpos_w[p], 4))
          return HERMES_EINVAL;
    }
  }
  if (cfg->summary_mode) {
    // an evicting deep layer holds budget + 1 rows after compression
    const std::vector<int8_t> cls = cfg->layer_class
        ? std::vector<int8_t>(cfg->layer_class, cfg->layer_class + L) : default_classes(L);
    for (int l = 0; l < L; ++l)
      if (cls[l] == HERMES_DEEP && cfg->budget[l] + 1 > layers[l].cap) return HERMES_ECAPACITY;
  }

  hermes_ctx *c = new (std::nothrow) hermes_ctx();
  if (c == nullptr) return HERMES_EINVAL;
  c->L = L;
  c->Hq = cfg->n_q_heads;
  c->Hkv = cfg->n_kv_heads;
  c->D = cfg->head_dim;
  c->max_chunk = cfg->max_chunk;
  c->max_cap = cfg->max_cap;
  c->forget_rate = cfg->forget_rate > 0.0 ? cfg->forget_rate : std::ldexp(1.0, -10);
  c->sm_scale = cfg->sm_scale > 0.0 ? cfg->sm_scale : 1.0 / std::sqrt((double)cfg->head_dim);
  c->alpha_mode = cfg->alpha_mode;
  c->align_mode = cfg->align_mode;
  c->force_scores = cfg->force_scores != 0;
  c->summary_mode = cfg->summary_mode;
  c->reindex_mode = cfg->reindex_mode;
  c->scoring_mode = cfg->scoring_mode;
  c->rope_offset = cfg->rope_offset;
  c->rope_limit = cfg->rope_limit;
  c->rope_headroom = cfg->rope_headroom;
  c->rope_theta = cfg->rope_theta > 0.0 ? cfg->rope_theta : 1.0e6;
  c->rope_axes = cfg->rope_axes == 3 ? 3 : 1;
  if (c->rope_axes == 3) {
    const int half = cfg->head_dim / 2;
    const int *sec = cfg->mrope_section;
    if (sec[0] == 0 && sec[1] == 0 && sec[2] == 0) {
      c->section[0] = half / 4;
      c->section[1] = (half - half / 4) / 2;
      c->section[2] = half - c->section[0] - c->section[1];
    } else {
      for (int a = 0; a < 3; ++a) c->section[a] = sec[a];
    }
  }
  c->keep_rpos = cfg->summary_mode != 0 || cfg->reindex_mode != 0 || c->rope_axes == 3;
  c->guided.assign(L, 0);
  c->budget.assign(cfg->budget, cfg->budget + L);
  c->cls = cfg->layer_class ? std::vector<int8_t>(cfg->layer_class, cfg->layer_class + L)
                            : default_classes(L);
  c->lambda.resize(L);
  static const double kLambda[3] = {0.1, 0.3, 0.4};   // Appendix C
  for (int l = 0; l < L; ++l)
    c->lambda[l] = cfg->lambda ? (double)cfg->lambda[l] : kLambda[(int)c->cls[l]];
  // omega_l for middle layers (Sec. 3.1), l_short/l_long = first/last middle layer.
  int l_s = -1, l_l = -1;
  for (int l = 0; l < L; ++l)
    if (c->cls[l] == HERMES_MIDDLE) {
      if (l_s < 0) l_s = l;
      l_l = l;
    }
  c->omega.assign(L, 0.0);
  for (int l = 0; l < L; ++l) {
    if (c->cls[l] != HERMES_MIDDLE) continue;
    c->omega[l] = (l_l == l_s) ? cfg->omega0
                               : cfg->omega0 - cfg->gamma * (double)(l - l_s) / (double)(l_l - l_s);
  }
  c->bufs.assign(layers, layers + L);
  c->len.resize(L);
  for (int l = 0; l < L; ++l) c->len[l] = layers[l].init_len;
  c->init_len = c->len;
  c->cur.assign(L, 0);
  c->appended.assign(L, 0);
  c->buf0_dirty.assign(L, 0);
  c->lay = lay;
  c->ws = static_cast<char *>(workspace);
  c->d_tab = reinterpret_cast<LayerTable *>(c->ws + lay.tab);
  {
    const char *env = std::getenv("HERMES_CHECK");
    c->check = env != nullptr && env[0] == '1';
  }

  std::vector<LayerTable> tab(L);
  for (int l = 0; l < L; ++l) {
    LayerTable &t = tab[l];
    std::memset(&t, 0, sizeof(t));
    for (int p = 0; p < 2; ++p) {
      t.k[p] = static_cast<uint16_t *>(layers[l].k[p]);
      t.v[p] = static_cast<uint16_t *>(layers[l].v[p]);
      t.pos[p] = layers[l].pos[p];
      t.rpos[p] = c->keep_rpos ? layers[l].rpos[p] : nullptr;
      t.rpos_h[p] = c->rope_axes == 3 ? layers[l].rpos_h[p] : nullptr;
      t.rpos_w[p] = c->rope_axes == 3 ? layers[l].rpos_w[p] : nullptr;
    }
    t.w = layers[l].w;
    t.s_dbg = layers[l].s_dbg;
    t.kept_dbg = layers[l].kept_dbg;
    t.cap = layers[l].cap;
    t.budget = c->budget[l];
    t.cls = c->cls[l];
    t.lambda = c->lambda[l];
    t.omega = c->omega[l];
  }
  if (hipMemcpy(c->d_tab, tab.data(), sizeof(LayerTable) * L, hipMemcpyHostToDevice) !=
      hipSuccess) {
    delete c;
    return HERMES_EHIP;
  }
  *out = c;
  return HERMES_OK;
}

extern "C" {

int hermes_kv_init(const hermes_config *cfg, const hermes_layer_buffers *layers, void *workspace,
                   size_t ws_bytes, hermes_ctx **out) {
  if (out == nullptr) return HERMES_EINVAL;
  *out = nullptr;
  const int rc = check_config(cfg);
  if (rc != HERMES_OK) return rc;
  if (layers == nullptr || workspace == nullptr || !aligned(workspace, kAlign)) return HERMES_EINVAL;
  const Layout lay = layout_of(cfg);
  if (ws_bytes < lay.total) return HERMES_ECAPACITY;
  return init_context(cfg, layers, workspace, lay, out);
}

int hermes_kv_init_static(const hermes_config *cfg, const hermes_layer_buffers *layers,
                          hermes_ctx **out) {
  if (out == nullptr) return HERMES_EINVAL;
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc != HERMES_OK) return rc;
  if (layers == nullptr) return HERMES_EINVAL;
  Layout lay;
  if (!layout_within(cfg, kStaticWorkspaceBytes, &lay)) return HERMES_ECAPACITY;
  void *ws = nullptr;
  int dev = -1;
  rc = static_workspace_acquire(&ws, &dev);
  if (rc != HERMES_OK) return rc;
  rc = init_context(cfg, layers, ws, lay, out);
  if (rc != HERMES_OK) {
    static_workspace_release(dev);
    return rc;
  }
  (*out)->static_dev = dev;
  return HERMES_OK;
}

void hermes_kv_destroy(hermes_ctx *ctx) {
  if (ctx == nullptr) return;
  if (ctx->static_dev >= 0) static_workspace_release(ctx->static_dev);
  for (auto &v : ctx->used)
    for (auto &e : v) {
      (void)hipEventDestroy(e.start);
      (void)hipEventDestroy(e.stop);
    }
  for (auto &e : ctx->pool) {
    (void)hipEventDestroy(e.start);
    (void)hipEventDestroy(e.stop);
  }
  delete ctx;
}

int hermes_kv_rewind(hermes_ctx *ctx) {
  if (ctx == nullptr) return HERMES_EINVAL;
  if (ctx->poisoned) return HERMES_ESTATE;
  for (int l = 0; l < ctx->L; ++l)
    if (ctx->buf0_dirty[l]) return HERMES_ESTATE;
  for (int l = 0; l < ctx->L; ++l) {
    ctx->len[l] = ctx->init_len[l];
    ctx->cur[l] = 0;
    ctx->appended[l] = 0;
    ctx->guided[l] = 0;
  }
  ctx->n_appended = 0;
  ctx->step_n_new = 0;
  return HERMES_OK;
}

int hermes_kv_view(const hermes_ctx *ctx, int32_t layer, const void **k, const void **v,
                   const int32_t **pos, int32_t *len) {
  if (ctx == nullptr || layer < 0 || layer >= ctx->L) return HERMES_EINVAL;
  const int p = ctx->cur[layer];
  if (k) *k = ctx->bufs[layer].k[p];
  if (v) *v = ctx->bufs[layer].v[p];
  if (pos) *pos = ctx->bufs[layer].pos[p];
  if (len) *len = ctx->len[layer];
  return HERMES_OK;
}

int hermes_kv_view_rope(const hermes_ctx *ctx, int32_t layer, const int32_t **rpos) {
  if (ctx == nullptr || layer < 0 || layer >= ctx->L || rpos == nullptr) return HERMES_EINVAL;
  *rpos = ctx->keep_rpos ? ctx->bufs[layer].rpos[ctx->cur[layer]] : nullptr;
  return HERMES_OK;
}

int hermes_kv_view_mrope(const hermes_ctx *ctx, int32_t layer, const int32_t **t,
                         const int32_t **h, const int32_t **w) {
  if (ctx == nullptr || layer < 0 || layer >= ctx->L || t == nullptr || h == nullptr ||
      w == nullptr)
    return HERMES_EINVAL;
  const bool three = ctx->rope_axes == 3;
  const int p = ctx->cur[layer];
  *t = three ? ctx->bufs[layer].rpos[p] : nullptr;
  *h = three ? ctx->bufs[layer].rpos_h[p] : nullptr;
  *w = three ? ctx->bufs[layer].rpos_w[p] : nullptr;
  return HERMES_OK;
}

int hermes_budget_from_weights(const double *weights, int32_t n_layers, int64_t total,
                               int32_t *budget) {
  if (weights == nullptr || budget == nullptr || n_layers < 1 || total < n_layers)
    return HERMES_EINVAL;
  double sum = 0.0;
  for (int l = 0; l < n_layers; ++l) {
    if (!std::isfinite(weights[l]) || weights[l] < 0.0) return HERMES_EINVAL;
    sum += weights[l];
  }
  if (!(sum > 0.0)) return HERMES_EINVAL;
  std::vector<int64_t> m(n_layers);
  int64_t acc = 0;
  for (int l = 0; l < n_layers; ++l) {
    m[l] = (int64_t)std::floor((weights[l] / sum) * (double)total);
    acc += m[l];
  }
  m[n_layers - 1] += total - acc;
  for (int l = 0; l < n_layers; ++l)
    if (m[l] < 1 || m[l] > INT32_MAX) return HERMES_EINVAL;
  for (int l = 0; l < n_layers; ++l) budget[l] = (int32_t)m[l];
  return HERMES_OK;
}

static int append_impl(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                       const void *v, const int32_t *pos, const int32_t *rope_pos,
                       const int32_t *rope_thw, int32_t n_new, void *out, void *stream) {
  if (ctx == nullptr) return HERMES_EINVAL;
  if (ctx->poisoned) return HERMES_ESTATE;
  // M-RoPE contexts take their chunks with (t, h, w) coordinates only
  if ((ctx->rope_axes == 3) != (rope_thw != nullptr)) return HERMES_ESTATE;
  if (!aligned(rope_thw, 4)) return HERMES_EINVAL;
  const int L = ctx->L;
  if (layer != HERMES_ALL_LAYERS && (layer < 0 || layer >= L)) return HERMES_EINVAL;
  if (q == nullptr || k == nullptr || v == nullptr || pos == nullptr || out == nullptr)
    return HERMES_EINVAL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(pos, 4) || !aligned(rope_pos, 4))
    return HERMES_EINVAL;
  if (n_new < 1 || n_new > ctx->max_chunk) return HERMES_EINVAL;
  std::vector<int> list;
  if (layer == HERMES_ALL_LAYERS) {
    for (int l = 0; l < L; ++l) list.push_back(l);
  } else {
    list.push_back(layer);
  }
  for (int l : list)
    if (ctx->appended[l]) return HERMES_ESTATE;
  if (ctx->n_appended > 0 && n_new != ctx->step_n_new) return HERMES_ESTATE;
  for (int l : list)
    if ((int64_t)ctx->len[l] + n_new > ctx->bufs[l].cap) return HERMES_ECAPACITY;
  {
    const int64_t rows = (int64_t)list.size() * n_new;
    const int rc = run_checks(ctx, list, q, k, v, rows * ctx->Hq * ctx->D, rows * ctx->Hkv * ctx->D, pos,
                              n_new, static_cast<hipStream_t>(stream));
    if (rc != HERMES_OK) return rc;
  }

  // Which layers' scores the coming compression needs (Sec. 3.1/3.2): a
  // non-shallow layer that evicts, or whose shallower neighbour evicts and
  // smooths with it.
  auto base_len = [&](int l) { return ctx->appended[l] ? ctx->len[l] - ctx->step_n_new : ctx->len[l]; };
  auto evicts = [&](int l) { return base_len(l) + n_new > ctx->budget[l]; };
  auto need_w = [&](int l) {
    if (ctx->scoring_mode == HERMES_SCORE_GUIDANCE) return false;   // W comes from the prompt
    if (ctx->force_scores) return true;
    if (ctx->cls[l] == HERMES_SHALLOW) return false;
    return evicts(l) || (l > 0 && evicts(l - 1) && ctx->lambda[l - 1] != 0.0);
  };

  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t q_ls = (layer == HERMES_ALL_LAYERS) ? (int64_t)n_new * ctx->Hq * ctx->D : 0;
  const int64_t kv_ls = (layer == HERMES_ALL_LAYERS) ? (int64_t)n_new * ctx->Hkv * ctx->D : 0;
  const float scale_log2 = (float)(ctx->sm_scale * kLog2e);

  AppendArgs ap;
  std::memset(&ap, 0, sizeof(ap));
  ap.tab = ctx->d_tab;
  ap.kn = static_cast<const uint16_t *>(k);
  ap.vn = static_cast<const uint16_t *>(v);
  ap.pos = pos;
  ap.rope_pos = rope_thw != nullptr ? rope_thw : rope_pos;
  ap.rope_h = rope_thw != nullptr ? rope_thw + n_new : nullptr;
  ap.rope_w = rope_thw != nullptr ? rope_thw + 2 * n_new : nullptr;
  ap.kv_lstride = kv_ls;
  ap.row_elems = ctx->Hkv * ctx->D;
  ap.C = n_new;
  ap.n_list = (int)list.size();

  AttnArgs at;
  std::memset(&at, 0, sizeof(at));
  at.tab = ctx->d_tab;
  at.q = static_cast<const uint16_t *>(q);
  at.kn = ap.kn;
  at.vn = ap.vn;
  at.out = static_cast<uint16_t *>(out);
  at.lse = reinterpret_cast<float *>(ctx->ws + ctx->lay.lse);
  at.q_lstride = q_ls;
  at.kv_lstride = kv_ls;
  at.lse_lstride = ctx->lay.lse_lstride;
  at.Hq = ctx->Hq;
  at.Hkv = ctx->Hkv;
  at.C = n_new;
  at.scale_log2 = scale_log2;

  ColsumArgs cs;
  std::memset(&cs, 0, sizeof(cs));
  cs.tab = ctx->d_tab;
  cs.q = at.q;
  cs.kn = ap.kn;
  cs.vn = ap.vn;
  cs.lse = at.lse;
  cs.wpart = reinterpret_cast<double *>(ctx->ws + ctx->lay.wpart);
  cs.wpart_lstride = ctx->lay.wpart_lstride;
  cs.wpart_hstride = ctx->max_cap;
  cs.normpart = reinterpret_cast<double *>(ctx->ws + ctx->lay.normpart);
  cs.normpart_lstride = ctx->lay.normpart_lstride;
  cs.q_lstride = q_ls;
  cs.kv_lstride = kv_ls;
  cs.lse_lstride = at.lse_lstride;
  cs.Hq = ctx->Hq;
  cs.Hkv = ctx->Hkv;
  cs.C = n_new;
  cs.scale_log2 = scale_log2;
  int n_cs = 0, max_T = 0;

  for (size_t j = 0; j < list.size(); ++j) {
    const int l = list[j];
    const int8_t slot = (int8_t)(layer == HERMES_ALL_LAYERS ? l : 0);
    ap.T0[j] = at.T0[j] = ctx->len[l];
    ap.layer_id[j] = at.layer_id[j] = (int8_t)l;
    ap.slot[j] = at.slot[j] = slot;
    ap.cur[j] = at.cur[j] = ctx->cur[l];
    if (need_w(l)) {
      cs.T0[n_cs] = ctx->len[l];
      cs.ncand[n_cs] = ctx->len[l] + n_new;
      cs.layer_id[n_cs] = (int8_t)l;
      cs.slot[n_cs] = slot;
      cs.cur[n_cs] = ctx->cur[l];
      cs.alpha_mode[n_cs] = (int8_t)ctx->alpha_mode;
      max_T = ctx->len[l] + n_new > max_T ? ctx->len[l] + n_new : max_T;
      ++n_cs;
    }
  }

  int rc = ctx->run(HERMES_K_APPEND, s, [&] { return launch_append(ap, s); });
  if (rc != HERMES_OK) return rc;
  rc = ctx->run(HERMES_K_ATTN, s, [&] { return launch_attention(at, (int)list.size(), ctx->D, s); });
  if (rc != HERMES_OK) return rc;
  if (n_cs > 0) {
    rc = ctx->run(HERMES_K_COLSUM, s, [&] { return launch_colsum(cs, n_cs, max_T, ctx->D, s); });
    if (rc != HERMES_OK) return rc;
  }
  for (int l : list) {
    ctx->len[l] += n_new;
    ctx->appended[l] = 1;
  }
  ctx->n_appended += (int)list.size();
  ctx->step_n_new = n_new;
  return HERMES_OK;
}

int hermes_append_chunk(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                        const void *v, const int32_t *pos, int32_t n_new, void *out,
                        void *stream) {
  return append_impl(ctx, layer, q, k, v, pos, nullptr, nullptr, n_new, out, stream);
}

int hermes_append_chunk_at(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                           const void *v, const int32_t *pos, const int32_t *rope_pos,
                           int32_t n_new, void *out, void *stream) {
  return append_impl(ctx, layer, q, k, v, pos, rope_pos, nullptr, n_new, out, stream);
}

int hermes_append_chunk_mrope(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                              const void *v, const int32_t *pos, const int32_t *rope_thw,
                              int32_t n_new, void *out, void *stream) {
  if (ctx == nullptr) return HERMES_EINVAL;
  if (ctx->rope_axes != 3) return HERMES_ESTATE;
  if (rope_thw == nullptr) return HERMES_EINVAL;
  return append_impl(ctx, layer, q, k, v, pos, nullptr, rope_thw, n_new, out, stream);
}

int hermes_guidance_score(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                          const void *v, int32_t n_rows, void *stream) {
  if (ctx == nullptr) return HERMES_EINVAL;
  if (ctx->poisoned) return HERMES_ESTATE;
  const int L = ctx->L;
  if (layer != HERMES_ALL_LAYERS && (layer < 0 || layer >= L)) return HERMES_EINVAL;
  if (q == nullptr || k == nullptr || v == nullptr) return HERMES_EINVAL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16)) return HERMES_EINVAL;
  if (n_rows < 1 || n_rows > ctx->max_chunk) return HERMES_EINVAL;
  if (ctx->scoring_mode != HERMES_SCORE_GUIDANCE) return HERMES_ESTATE;
  std::vector<int> list;
  for (int l = 0; l < L; ++l)
    if (layer == HERMES_ALL_LAYERS || l == layer) list.push_back(l);
  for (int l : list)
    if (!ctx->appended[l]) return HERMES_ESTATE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    const int64_t rows = (int64_t)list.size() * n_rows;
    const int rc = run_checks(ctx, list, q, k, v, rows * ctx->Hq * ctx->D, rows * ctx->Hkv * ctx->D, nullptr,
                              n_rows, s);
    if (rc != HERMES_OK) return rc;
  }
  const int64_t q_ls = (layer == HERMES_ALL_LAYERS) ? (int64_t)n_rows * ctx->Hq * ctx->D : 0;
  const int64_t kv_ls = (layer == HERMES_ALL_LAYERS) ? (int64_t)n_rows * ctx->Hkv * ctx->D : 0;
  const float scale_log2 = (float)(ctx->sm_scale * kLog2e);

  // The prompt follows the cache: its rows attend [cache; prompt] causally
  // (row LSE only), then the mass of the cached candidates only.
  AttnArgs at;
  std::memset(&at, 0, sizeof(at));
  at.tab = ctx->d_tab;
  at.q = static_cast<const uint16_t *>(q);
  at.kn = static_cast<const uint16_t *>(k);
  at.vn = static_cast<const uint16_t *>(v);
  at.out = nullptr;
  at.lse = reinterpret_cast<float *>(ctx->ws + ctx->lay.lse);
  at.q_lstride = q_ls;
  at.kv_lstride = kv_ls;
  at.lse_lstride = ctx->lay.lse_lstride;
  at.Hq = ctx->Hq;
  at.Hkv = ctx->Hkv;
  at.C = n_rows;
  at.scale_log2 = scale_log2;
  ColsumArgs cs;
  std::memset(&cs, 0, sizeof(cs));
  cs.tab = ctx->d_tab;
  cs.q = at.q;
  cs.kn = at.kn;
  cs.vn = at.vn;
  cs.lse = at.lse;
  cs.wpart = reinterpret_cast<double *>(ctx->ws + ctx->lay.wpart);
  cs.wpart_lstride = ctx->lay.wpart_lstride;
  cs.wpart_hstride = ctx->max_cap;
  cs.normpart = reinterpret_cast<double *>(ctx->ws + ctx->lay.normpart);
  cs.normpart_lstride = ctx->lay.normpart_lstride;
  cs.q_lstride = q_ls;
  cs.kv_lstride = kv_ls;
  cs.lse_lstride = at.lse_lstride;
  cs.Hq = ctx->Hq;
  cs.Hkv = ctx->Hkv;
  cs.C = n_rows;
  cs.scale_log2 = scale_log2;
  int max_T = 0;
  for (size_t j = 0; j < list.size(); ++j) {
    const int l = list[j];
    const int8_t slot = (int8_t)(layer == HERMES_ALL_LAYERS ? l : 0);
    at.T0[j] = cs.T0[j] = ctx->len[l];
    cs.ncand[j] = ctx->len[l];
    at.layer_id[j] = cs.layer_id[j] = (int8_t)l;
    at.slot[j] = cs.slot[j] = slot;
    at.cur[j] = cs.cur[j] = ctx->cur[l];
    cs.alpha_mode[j] = 1;   // every prompt row sees every candidate: A = W / sum W
    max_T = ctx->len[l] > max_T ? ctx->len[l] : max_T;
  }
  const int n = (int)list.size();
  stream_plan(at, n_rows, ctx->Hq / ctx->Hkv, ctx->Hkv, n, ctx->D, ctx->lay.part_blocks);
  at.part_rows = ctx->lay.part_rows;
  at.opart = reinterpret_cast<uint16_t *>(ctx->ws + ctx->lay.opart);
  at.mlpart = reinterpret_cast<float *>(ctx->ws + ctx->lay.mlpart);
  const int rc = ctx->run(HERMES_K_GUIDE, s, [&] {
    hipError_t e = at.st_units > 0 ? launch_attention_stream(at, n, ctx->D, s)
                                   : launch_attention(at, n, ctx->D, s);
    if (e != hipSuccess) return e;
    return launch_colsum(cs, n, max_T, ctx->D, s);
  });
  if (rc != HERMES_OK) return rc;
  for (int l : list) ctx->guided[l] = n_rows;
  return HERMES_OK;
}

int hermes_compress(hermes_ctx *ctx, void *stream) {
  if (ctx == nullptr) return HERMES_EINVAL;
  if (ctx->poisoned) return HERMES_ESTATE;
  if (ctx->n_appended == 0) return HERMES_OK;
  if (ctx->n_appended != ctx->L) return HERMES_ESTATE;
  const int L = ctx->L;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto evicts = [&](int l) { return ctx->len[l] > ctx->budget[l]; };
  if (ctx->scoring_mode == HERMES_SCORE_GUIDANCE) {
    // every layer whose decision reads W must have its prompt mass
    for (int l = 0; l < L; ++l) {
      if (ctx->cls[l] == HERMES_SHALLOW) continue;
      const bool need = ctx->force_scores || evicts(l) ||
                        (l > 0 && evicts(l - 1) && ctx->lambda[l - 1] != 0.0);
      if (need && ctx->guided[l] == 0) return HERMES_ESTATE;
    }
  }

  SelectArgs sa;
  std::memset(&sa, 0, sizeof(sa));
  sa.tab = ctx->d_tab;
  sa.keys = reinterpret_cast<uint32_t *>(ctx->ws + ctx->lay.keys);
  sa.kept = reinterpret_cast<int32_t *>(ctx->ws + ctx->lay.kept);
  sa.normpart = reinterpret_cast<const double *>(ctx->ws + ctx->lay.normpart);
  sa.normpart_lstride = ctx->lay.normpart_lstride;
  sa.keys_lstride = ctx->lay.keys_lstride;
  sa.kept_lstride = ctx->lay.kept_lstride;
  sa.forget_rate = ctx->forget_rate;
  sa.n_layers = L;
  sa.C = ctx->step_n_new;
  sa.ek = std::exp(ctx->forget_rate);
  sa.inv_c = 1.0 / (double)(sa.C > 0 ? sa.C : 1);
  sa.alpha_mode = ctx->alpha_mode;
  sa.align_mode = ctx->align_mode;
  GatherArgs ga;
  std::memset(&ga, 0, sizeof(ga));
  ga.tab = ctx->d_tab;
  ga.kept = sa.kept;
  ga.kept_lstride = sa.kept_lstride;
  ga.row_elems = ctx->Hkv * ctx->D;
  ga.head_dim = ctx->D;
  SummaryArgs sm;
  std::memset(&sm, 0, sizeof(sm));
  std::vector<int8_t> has_sum(L, 0);
  int n = 0, n_sum = 0, max_T_sum = 0;
  for (int l = 0; l < L; ++l) {
    sa.len[l] = ctx->len[l];
    sa.cur[l] = ctx->cur[l];
    sa.guide_rows[l] = ctx->scoring_mode == HERMES_SCORE_GUIDANCE ? ctx->guided[l] : 0;
    sa.inv_z[l] = 1.0 / (std::expm1(-ctx->forget_rate * (double)ctx->len[l]) / std::expm1(-ctx->forget_rate));
    if (evicts(l)) {
      has_sum[l] = ctx->summary_mode && ctx->cls[l] == HERMES_DEEP;
      sa.layer_id[n] = (int8_t)l;
      ga.layer_id[n] = (int8_t)l;
      ga.cur[n] = ctx->cur[l];
      ga.mode[n] = 0;
      ga.has_sum[n] = has_sum[l];
      ga.row_start[n + 1] = ga.row_start[n] + ctx->budget[l] + has_sum[l];
      ++n;
      if (has_sum[l]) {
        sm.layer_id[n_sum] = (int8_t)l;
        sm.cur[n_sum] = ctx->cur[l];
        sm.len[n_sum] = ctx->len[l];
        sm.budget[n_sum] = ctx->budget[l];
        max_T_sum = ctx->len[l] > max_T_sum ? ctx->len[l] : max_T_sum;
        ++n_sum;
      }
    }
  }
  sa.n_list = n;
  const int n_evict = n;
  int rc = HERMES_OK;
  if (n_evict > 0) {
    rc = ctx->run(HERMES_K_SELECT, s, [&] { return launch_select(sa, s); });
    if (rc != HERMES_OK) return rc;
  }
  if (!ctx->keep_rpos) {
    ga.n_list = n_evict;
    if (n_evict > 0) {
      rc = ctx->run(HERMES_K_GATHER, s, [&] { return launch_gather(ga, s); });
      if (rc != HERMES_OK) return rc;
    }
  } else {
    int32_t *meta = reinterpret_cast<int32_t *>(ctx->ws + ctx->lay.smeta);
    int32_t *flag = reinterpret_cast<int32_t *>(ctx->ws + ctx->lay.flag);
    if (n_sum > 0) {
      sm.tab = ctx->d_tab;
      sm.kept = sa.kept;
      sm.kept_lstride = sa.kept_lstride;
      sm.part = reinterpret_cast<double *>(ctx->ws + ctx->lay.spart);
      sm.part_lstride = ctx->lay.spart_lstride;
      sm.sum_k = reinterpret_cast<uint16_t *>(ctx->ws + ctx->lay.sumk);
      sm.sum_v = reinterpret_cast<uint16_t *>(ctx->ws + ctx->lay.sumv);
      sm.sum_meta = meta;
      sm.row_elems = ga.row_elems;
      sm.head_dim = ctx->D;
      sm.n_list = n_sum;
      sm.axes = ctx->rope_axes;
      for (int a = 0; a < 3; ++a) sm.section[a] = ctx->section[a];
      rope_frequencies(ctx->rope_theta, ctx->D, sm.inv_freq);
      rc = ctx->run(HERMES_K_SUMMARY, s, [&] { return launch_summary(sm, max_T_sum, s); });
      if (rc != HERMES_OK) return rc;
    }
    // layers that kept everything are re-indexed in place
    if (ctx->reindex_mode != HERMES_REINDEX_NONE) {
      for (int l = 0; l < L; ++l) {
        if (evicts(l) || ctx->len[l] == 0) continue;
        ga.layer_id[n] = (int8_t)l;
        ga.cur[n] = ctx->cur[l];
        ga.mode[n] = 1;
        ga.has_sum[n] = 0;
        ga.row_start[n + 1] = ga.row_start[n] + ctx->len[l];
        ++n;
      }
    }
    ga.n_list = n;
    ga.reindex = ctx->reindex_mode == HERMES_REINDEX_EAGER ? 1
               : ctx->reindex_mode == HERMES_REINDEX_LAZY ? 2 : 0;
    ga.rope_offset = ctx->rope_offset;
    rope_frequencies(ctx->rope_theta, ctx->D, ga.inv_freq);
    ga.flag = flag;
    ga.sum_k = reinterpret_cast<const uint16_t *>(ctx->ws + ctx->lay.sumk);
    ga.sum_v = reinterpret_cast<const uint16_t *>(ctx->ws + ctx->lay.sumv);
    ga.sum_meta = meta;
    ga.axes = ctx->rope_axes;
    for (int a = 0; a < 3; ++a) ga.section[a] = ctx->section[a];
    ga.newc = reinterpret_cast<const int32_t *>(ctx->ws + ctx->lay.newc);
    ga.newc_lstride = ctx->lay.newc_lstride;
    if (ctx->reindex_mode == HERMES_REINDEX_LAZY) {
      DecideArgs da;
      std::memset(&da, 0, sizeof(da));
      da.tab = ctx->d_tab;
      da.kept = sa.kept;
      da.kept_lstride = sa.kept_lstride;
      da.sum_meta = meta;
      da.flag = flag;
      da.n_layers = L;
      da.limit = ctx->rope_limit;
      da.headroom = ctx->rope_headroom;
      da.axes = ctx->rope_axes;
      for (int l = 0; l < L; ++l) {
        da.len[l] = ctx->len[l];
        da.budget[l] = ctx->budget[l];
        da.cur[l] = ctx->cur[l];
        da.evicts[l] = evicts(l);
        da.has_sum[l] = has_sum[l];
      }
      rc = ctx->run(HERMES_K_GATHER, s, [&] { return launch_decide(da, s); });
      if (rc != HERMES_OK) return rc;
    }
    if (n > 0 && ctx->rope_axes == 3 && ctx->reindex_mode != HERMES_REINDEX_NONE) {
      RankArgs ra;
      std::memset(&ra, 0, sizeof(ra));
      ra.tab = ctx->d_tab;
      ra.kept = sa.kept;
      ra.kept_lstride = sa.kept_lstride;
      ra.newc = reinterpret_cast<int32_t *>(ctx->ws + ctx->lay.newc);
      ra.newc_lstride = ctx->lay.newc_lstride;
      ra.sum_meta = meta;
      ra.flag = flag;
      ra.reindex = ga.reindex;
      ra.offset = ctx->rope_offset;
      ra.n_list = n;
      for (int j = 0; j < n; ++j) {
        ra.layer_id[j] = ga.layer_id[j];
        ra.cur[j] = ga.cur[j];
        ra.mode[j] = ga.mode[j];
        ra.has_sum[j] = ga.has_sum[j];
        ra.row_start[j + 1] = ga.row_start[j + 1];
      }
      rc = ctx->run(HERMES_K_GATHER, s, [&] { return launch_mrope_rank(ra, s); });
      if (rc != HERMES_OK) return rc;
    }
    if (n > 0) {
      rc = ctx->run(HERMES_K_GATHER, s, [&] { return launch_gather_rope(ga, s); });
      if (rc != HERMES_OK) return rc;
    }
  }
  for (int l = 0; l < L; ++l) {
    if (evicts(l)) {
      if (ctx->cur[l] == 1) ctx->buf0_dirty[l] = 1;
      ctx->cur[l] ^= 1;
      ctx->len[l] = ctx->budget[l] + has_sum[l];
    }
    ctx->appended[l] = 0;
    ctx->guided[l] = 0;
  }
  ctx->n_appended = 0;
  return HERMES_OK;
}

int hermes_query_attend(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                        const void *v, int32_t n_q, void *out, void *stream) {
  if (ctx == nullptr) return HERMES_EINVAL;
  if (ctx->poisoned) return HERMES_ESTATE;
  const int L = ctx->L;
  if (layer != HERMES_ALL_LAYERS && (layer < 0 || layer >= L)) return HERMES_EINVAL;
  if (q == nullptr || k == nullptr || v == nullptr || out == nullptr) return HERMES_EINVAL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16))
    return HERMES_EINVAL;
  if (n_q < 1 || n_q > ctx->max_chunk) return HERMES_EINVAL;
  if (ctx->n_appended != 0) return HERMES_ESTATE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    const int64_t rows = (int64_t)(layer == HERMES_ALL_LAYERS ? L : 1) * n_q;
    const int rc = run_checks(ctx, std::vector<int>(), q, k, v, rows * ctx->Hq * ctx->D,
                              rows * ctx->Hkv * ctx->D, nullptr, n_q, s);
    if (rc != HERMES_OK) return rc;
  }
  AttnArgs at;
  std::memset(&at, 0, sizeof(at));
  at.tab = ctx->d_tab;
  at.q = static_cast<const uint16_t *>(q);
  at.kn = static_cast<const uint16_t *>(k);
  at.vn = static_cast<const uint16_t *>(v);
  at.out = static_cast<uint16_t *>(out);
  at.lse = nullptr;
  at.q_lstride = (layer == HERMES_ALL_LAYERS) ? (int64_t)n_q * ctx->Hq * ctx->D : 0;
  at.kv_lstride = (layer == HERMES_ALL_LAYERS) ? (int64_t)n_q * ctx->Hkv * ctx->D : 0;
  at.Hq = ctx->Hq;
  at.Hkv = ctx->Hkv;
  at.C = n_q;
  at.scale_log2 = (float)(ctx->sm_scale * kLog2e);
  int n = 0;
  for (int l = 0; l < L; ++l) {
    if (layer != HERMES_ALL_LAYERS && l != layer) continue;
    at.T0[n] = ctx->len[l];
    at.layer_id[n] = (int8_t)l;
    at.slot[n] = (int8_t)(layer == HERMES_ALL_LAYERS ? l : 0);
    at.cur[n] = ctx->cur[l];
    ++n;
  }
  stream_plan(at, n_q, ctx->Hq / ctx->Hkv, ctx->Hkv, n, ctx->D, ctx->lay.part_blocks);
  at.part_rows = ctx->lay.part_rows;
  at.opart = reinterpret_cast<uint16_t *>(ctx->ws + ctx->lay.opart);
  at.mlpart = reinterpret_cast<float *>(ctx->ws + ctx->lay.mlpart);
  return ctx->run(HERMES_K_QUERY, s, [&] {
    return at.st_units > 0 ? launch_attention_stream(at, n, ctx->D, s)
                           : launch_attention(at, n, ctx->D, s);
  });
}

int hermes_select_topk(const float *keys, int32_t n, int32_t k, int32_t *out_idx, void *stream) {
  if (keys == nullptr || out_idx == nullptr || n < 1 || k < 1) return HERMES_EINVAL;
  if (!aligned(keys, 4) || !aligned(out_idx, 4)) return HERMES_EINVAL;
  return launch_topk(keys, n, k, out_idx, static_cast<hipStream_t>(stream)) == hipSuccess
             ? HERMES_OK
             : HERMES_EHIP;
}

int hermes_check_enable(hermes_ctx *ctx, int on) {
  if (ctx == nullptr) return HERMES_EINVAL;
  ctx->check = on != 0;
  return HERMES_OK;
}

int hermes_profile_enable(hermes_ctx *ctx, int on) {
  if (ctx == nullptr) return HERMES_EINVAL;
  ctx->prof = on != 0;
  return HERMES_OK;
}

int hermes_profile_read(hermes_ctx *ctx, int kernel_id, double *ms_total, int64_t *count) {
  if (ctx == nullptr || kernel_id < 0 || kernel_id >= HERMES_K_COUNT) return HERMES_EINVAL;
  double total = 0.0;
  int64_t cnt = 0;
  for (auto &e : ctx->used[kernel_id]) {
    if (hipEventSynchronize(e.stop) != hipSuccess) return HERMES_EHIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e.start, e.stop) != hipSuccess) return HERMES_EHIP;
    total += ms;
    ++cnt;
    ctx->pool.push_back(e);
  }
  ctx->used[kernel_id].clear();
  if (ms_total) *ms_total = total;
  if (count) *count = cnt;
  return HERMES_OK;
}

}  // extern "C"
