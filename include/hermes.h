/*
 * hermes.h -- C ABI of libhermes.so, the MI355X (gfx950) streaming step of
 * HERMES (arXiv 2601.14724): per-layer chunk append with causal GQA
 * attention, the attention mass every cached token receives, hierarchical
 * importance scoring, cross-layer smoothing, TopK eviction to the per-layer
 * budget and order-preserving compaction; plus query-time attention over the
 * compacted cache.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All device work is asynchronous on the caller's HIP stream (`stream` is
 *    a hipStream_t; NULL means the null stream).  No call synchronises the
 *    device except hermes_kv_init (one upload of a per-layer table) and
 *    hermes_profile_read.
 *  - The library never allocates device memory.  Every device buffer (K/V
 *    caches, positions, score buffers, the workspace, inputs, outputs) is
 *    owned by the caller and must stay alive until hermes_kv_destroy.
 *  - bfloat16 tensors are raw 16-bit patterns, row-major:
 *      cache K or V    [cap][n_kv_heads][head_dim]   (token-major rows)
 *      chunk Q / out   [n_new][n_q_heads][head_dim]
 *      chunk K or V    [n_new][n_kv_heads][head_dim]
 *    With layer == HERMES_ALL_LAYERS the per-layer tensors are stacked on a
 *    leading [n_layers] axis; positions are shared by all layers.
 *  - Query head h reads KV head h / (n_q_heads / n_kv_heads).
 *  - Every function returns 0 or a negative HERMES_E* code.  All argument,
 *    capacity and state checks run on the host BEFORE any launch, so a
 *    failing call changes neither device data nor host lengths.  A failed
 *    HIP launch returns HERMES_EHIP and poisons the context: later calls
 *    return HERMES_ESTATE until it is destroyed and re-initialised.
 *  - One context is driven by one host thread at a time.
 */
#ifndef HERMES_H
#define HERMES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hermes_ctx hermes_ctx;

enum {
  HERMES_OK = 0,
  HERMES_EINVAL = -1,      /* bad argument (null pointer, size, range)          */
  HERMES_ECAPACITY = -2,   /* a buffer is too small for the requested rows      */
  HERMES_ESTATE = -3,      /* call not allowed in the context's current state   */
  HERMES_EHIP = -4,        /* a HIP runtime call or launch failed               */
  HERMES_ENOTSUP = -5      /* shape the kernels do not implement (head_dim)     */
};

/* Layer classes of the hierarchical memory (Sec. 2 findings, Sec. 3.1). */
enum { HERMES_SHALLOW = 0, HERMES_MIDDLE = 1, HERMES_DEEP = 2 };
enum { HERMES_ALL_LAYERS = -1 };
enum { HERMES_MAX_LAYERS = 64 };

/*
 * Model shape and method parameters.
 *
 *  budget[l]     per-layer token budget |M|_l (Sec. 3.2 TopK equation;
 *                Sec. 4.4 layer-dependent budgets).  Host array, each >= 1.
 *  layer_class   host [n_layers] of HERMES_SHALLOW/MIDDLE/DEEP, or NULL for
 *                the 10% / 60% / 30% partition of Sec. 4.1, rounded as
 *                n_shallow = floor(0.1 L + 1/2), n_deep = floor(0.3 L + 1/2).
 *  lambda        host [n_layers] smoothing weights in [0,1], or NULL for
 *                0.1 / 0.3 / 0.4 by class (Appendix C).
 *  omega0, gamma middle-layer interpolation (Sec. 3.1): omega_l = omega0 -
 *                gamma (l - l_short)/(l_long - l_short), l_short / l_long the
 *                first / last middle layer.  Paper values 0.75 and 0.6.
 *  forget_rate   k of the recency curve e^{-k (T-1-i)} (Sec. 3.1; the paper
 *                gives no value).  <= 0 selects 2^-10 per token.
 *  sm_scale      softmax scale; <= 0 selects 1/sqrt(head_dim).
 *  alpha_mode    normalisation alpha of the attention score (Sec. 3.1):
 *                0 = divide each token's mass by the number of chunk rows
 *                    that can see it, then normalise to sum 1;
 *                1 = normalise the plain mass to sum 1.
 *  align_mode    partner of token i in layer l+1 for smoothing (Sec. 3.2):
 *                0 = same stream position, 1 = same physical index.
 *  force_scores  1 = compute the attention mass on every append and the
 *                smoothed keys for every layer over budget, even where the
 *                eviction decision does not need them (parity tests).
 *  max_chunk     largest n_new of an append or n_q of a query.
 *  max_cap       largest per-layer buffer capacity (sizes the workspace).
 */
typedef struct {
  int32_t n_layers;        /* 1 .. HERMES_MAX_LAYERS                            */
  int32_t n_q_heads;       /* multiple of n_kv_heads                            */
  int32_t n_kv_heads;
  int32_t head_dim;        /* 64 or 128                                         */
  int32_t max_chunk;
  int32_t max_cap;
  const int32_t *budget;
  const int8_t *layer_class;
  const float *lambda;
  double omega0, gamma;
  double forget_rate;
  double sm_scale;
  int32_t alpha_mode;
  int32_t align_mode;
  int32_t force_scores;
  /* Adjacent parts of the method; all zero = the core streaming step.  */
  int32_t summary_mode;    /* 1: every deep layer that evicts appends one summary
                              token (see hermes_compress); needs rpos buffers     */
  int32_t reindex_mode;    /* HERMES_REINDEX_*: position re-indexing at compress;
                              needs rpos buffers                                  */
  int32_t rope_offset;     /* length of the fixed system prefix: re-indexed
                              entries take positions offset, offset + 1, ...      */
  int32_t rope_limit;      /* lazy re-indexing: the model's position limit        */
  int32_t rope_headroom;   /* lazy re-indexing fires when the largest retained
                              RoPE position of any layer + headroom >= limit      */
  double rope_theta;       /* RoPE base; <= 0 selects 1e6                          */
  int32_t scoring_mode;    /* HERMES_SCORE_*: source of the attention mass W      */
  int32_t rope_axes;       /* 1 (0 reads as 1): one RoPE position per token (rpos);
                              3: M-RoPE (t, h, w) coordinates, t in rpos and h, w
                              in rpos_h / rpos_w, chunks appended through
                              hermes_append_chunk_mrope (appendix, 3D M-RoPE
                              re-indexing); with summary_mode 1 the summary
                              takes the newest evicted token's (t, h, w)        */
  int32_t mrope_section[3];/* rope_axes 3: frequency pairs j = 0 .. head_dim/2 - 1
                              of the t, h and w sections, in that order (sum
                              head_dim/2); all 0 selects head_dim/8 pairs for t
                              and the rest halved between h and w (16, 24, 24 at
                              head_dim 128)                                        */
} hermes_config;

/* Position re-indexing (Sec. 3.3; appendix, 1D RoPE re-indexing). */
enum { HERMES_REINDEX_NONE = 0, HERMES_REINDEX_EAGER = 1, HERMES_REINDEX_LAZY = 2 };
/* Source of W: the chunk's own queries (default) or a guidance prompt used as
 * a pseudo-query (Sec. 3.1 deep-layer paragraph; appendix guidance prompts). */
enum { HERMES_SCORE_CHUNK = 0, HERMES_SCORE_GUIDANCE = 1 };

/*
 * Caller-owned device memory for ONE layer.
 *  k[2], v[2]   ping-pong pair of bf16 caches [cap][n_kv_heads][head_dim];
 *               buffer 0 holds the initial `init_len` tokens.  Compaction
 *               writes the kept rows into the other buffer of the pair.
 *  pos[2]       int32 stream positions [cap] for each buffer, strictly
 *               increasing along the cache.
 *  w            fp32 [cap]: attention mass of every candidate, written by
 *               append where the layer's score needs it.
 *  s_dbg        fp32 [cap] or NULL: smoothed selection keys S~ (parity).
 *  kept_dbg     int32 [budget] or NULL: kept indices of the last compaction.
 *  cap          rows per buffer; must be >= max(init_len, budget) + the
 *               largest chunk ever appended (budget + 1 in deep layers when
 *               summary_mode is on).
 *  rpos[2]      int32 [cap] RoPE positions the stored keys were rotated with,
 *               one per buffer, strictly increasing along the cache; buffer 0
 *               holds the initial `init_len` values.  Required (non-NULL) when
 *               summary_mode or reindex_mode is on, or rope_axes is 3, else
 *               ignored (may be NULL).  With rope_axes 3: the t coordinates.
 *  rpos_h[2], rpos_w[2]
 *               rope_axes 3: int32 [cap] h and w coordinates, laid out like
 *               rpos (buffer 0 holds the initial values); else ignored.
 */
typedef struct {
  void *k[2];
  void *v[2];
  int32_t *pos[2];
  float *w;
  float *s_dbg;
  int32_t *kept_dbg;
  int32_t cap;
  int32_t init_len;
  int32_t *rpos[2];
  int32_t *rpos_h[2];
  int32_t *rpos_w[2];
} hermes_layer_buffers;

/* Bytes of device workspace hermes_kv_init needs for `cfg` (0 on a bad cfg). */
size_t hermes_workspace_bytes(const hermes_config *cfg);

/*
 * Create a context over caller-owned buffers.  `layers` is a host array of
 * n_layers descriptors; `workspace` is device memory of at least
 * hermes_workspace_bytes(cfg) bytes, 256-byte aligned.  The per-layer
 * pointer table is uploaded into the workspace (one synchronous copy).
 * Errors: EINVAL (null/invalid fields), ECAPACITY (cap or workspace too
 * small), ENOTSUP (head_dim), EHIP.
 */
int hermes_kv_init(const hermes_config *cfg, const hermes_layer_buffers *layers,
                   void *workspace, size_t ws_bytes, hermes_ctx **out);

/*
 * hermes_kv_init for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the workspace is the library's own device scratch, a file-scope array of
 * HERMES_STATIC_WORKSPACE_BYTES that every GPU the library runs on holds
 * until the process ends.  Nothing is allocated (no hipMalloc, no library
 * routine that allocates); the scratch of the current device is looked up
 * once per device and is owned by the returned context until
 * hermes_kv_destroy.  The caller still owns the layer buffers, inputs and
 * outputs.  One such context per device at a time: a second call on the same
 * device returns HERMES_ESTATE while the first is alive, since both would
 * share (and race on) the one array; nothing in it needs to start at zero
 * (every word is written before it is read).  When the configuration's
 * workspace (hermes_workspace_bytes) exceeds the scratch, the stream-mode
 * partial state of queries and guidance prompts is cut to what fits (those
 * passes then use fewer stream units, or one workgroup per layer, KV head and
 * query tile: same results up to rounding order);
 * HERMES_ECAPACITY when even the rest exceeds it.  Errors otherwise as
 * hermes_kv_init (ENOTSUP also beyond 64 devices).
 */
enum { HERMES_STATIC_WORKSPACE_BYTES = 64 << 20 };
int hermes_kv_init_static(const hermes_config *cfg, const hermes_layer_buffers *layers,
                          hermes_ctx **out);

/*
 * Chunk-wise prefill of one layer or of all layers (Sec. 2 setup, Sec. 4.1):
 * append n_new tokens (q, k, v device bf16; pos device int32 [n_new]) to the
 * cache, and write the attention output `out` (device bf16) of the chunk's
 * queries over [cache; chunk], causally.  Where the coming compression needs
 * it, the same call writes the layer's attention mass w[i] (sum over heads
 * and rows of the softmax probability on candidate i, Sec. 3.1 deep-layer
 * score).  A layer may be appended once per step; every layer must be
 * appended with the same n_new before hermes_compress.
 * Errors: EINVAL (null pointer, layer out of range, n_new > max_chunk),
 * ECAPACITY (len + n_new > cap), ESTATE (layer already appended this step,
 * different n_new than other layers, poisoned context), EHIP.
 */
int hermes_append_chunk(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                        const void *v, const int32_t *pos, int32_t n_new, void *out,
                        void *stream);

/*
 * hermes_append_chunk for callers that rotate the chunk's Q/K at RoPE
 * positions other than its stream positions (after re-indexing, Sec. 3.3):
 * rope_pos is device int32 [n_new], the positions the chunk's keys carry,
 * stored in rpos; NULL means rope_pos = pos.  They must exceed every RoPE
 * position already in the layer.  Same errors as hermes_append_chunk.
 */
int hermes_append_chunk_at(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                           const void *v, const int32_t *pos, const int32_t *rope_pos,
                           int32_t n_new, void *out, void *stream);

/*
 * hermes_append_chunk for M-RoPE coordinates (rope_axes 3; appendix, 3D
 * M-RoPE re-indexing): rope_thw is device int32 [3][n_new], the t, then the
 * h, then the w coordinate of every new row (the same for every layer with
 * HERMES_ALL_LAYERS), stored in rpos / rpos_h / rpos_w; the chunk's keys
 * carry these coordinates.  The plain appends are refused (ESTATE) when
 * rope_axes is 3, and this one when it is not.  Errors otherwise as
 * hermes_append_chunk (EINVAL also for a null or misaligned rope_thw).
 */
int hermes_append_chunk_mrope(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                              const void *v, const int32_t *pos, const int32_t *rope_thw,
                              int32_t n_new, void *out, void *stream);

/*
 * Guidance-prompt scoring (scoring_mode HERMES_SCORE_GUIDANCE; Sec. 3.1
 * deep-layer paragraph and the appendix guidance prompts): n_rows prompt
 * tokens (q, k, v: device bf16, layout as hermes_append_chunk; stacked over
 * layers for HERMES_ALL_LAYERS) are placed after every cached token of the
 * layer; their causal attention over [cache; prompt] gives w[i] for the
 * cached candidates i < len.  The prompt is not stored.  Call it after the
 * step's append and before hermes_compress, for every layer whose score
 * needs W (non-shallow layers; middle layers take the hybrid local + global
 * prompt, deep layers the global one).  Every candidate is seen by all
 * prompt rows, so A = W / sum W.
 * Errors: EINVAL (null pointer, layer, n_rows < 1 or > max_chunk), ESTATE
 * (scoring_mode is not guidance, layer not appended this step, poisoned), EHIP.
 */
int hermes_guidance_score(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                          const void *v, int32_t n_rows, void *stream);

/*
 * Close the step: for every layer whose length T exceeds its budget, score
 * the candidates (Sec. 3.1), smooth with layer l+1 (Sec. 3.2), keep the
 * budget largest keys (ties to the newer token) and compact K, V and
 * positions in stream order into the other buffer (Sec. 3.2 TopK/gather).
 * Layers within budget are untouched.  Lengths become min(T, budget) on the
 * host, without a device read-back.  Requires every layer to have been
 * appended this step (or none, which makes the call a no-op).
 *
 * summary_mode 1 (Sec. 3.2 last paragraph; appendix summary-token
 * algorithm): each evicting deep layer folds its evicted tokens into one
 * token, V = mean of the evicted values, K = mean of the evicted keys each
 * rotated from its RoPE position to t, the RoPE position of the newest
 * evicted token (with rope_axes 3: each frequency pair turned by the change
 * of its section's coordinate to the newest evicted token's (t, h, w)).
 * The summary takes that token's stream and RoPE position (coordinates) and
 * its sorted place among the kept rows, in addition to the budget (length
 * budget + 1).  K and V are accumulated in fp64, stored as bf16.
 *
 * reindex_mode (Sec. 3.3; appendix 1D re-indexing): EAGER re-indexes every
 * layer at every call, LAZY only when the largest retained RoPE position of
 * any layer + rope_headroom >= rope_limit (decided on the device).  Entry j
 * of a re-indexed layer gets RoPE position rope_offset + j and its key is
 * rotated by the position change (rotate-half pairs, angles and rotation in
 * fp64, stored as bf16); V is unchanged.
 *
 * With rope_axes 3 (appendix, 3D M-RoPE re-indexing) each axis is compacted
 * on its own: a retained entry's t (h, w) coordinate becomes rope_offset +
 * the number of distinct t (h, w) coordinates the layer retains below it,
 * so entries that shared a coordinate still share it, and frequency pair j
 * of its key turns by the change of the coordinate of the section j falls
 * in (mrope_section).  LAZY fires when the largest retained coordinate on
 * any axis of any layer + rope_headroom >= rope_limit.
 *
 * scoring_mode GUIDANCE: W must have been written by hermes_guidance_score
 * this step for every layer whose decision needs it, else ESTATE.
 * Errors: ESTATE, EHIP.
 */
int hermes_compress(hermes_ctx *ctx, void *stream);

/*
 * Query-time attention (Sec. 3: the query is answered directly from the
 * compact cache): n_q query tokens attend the layer's current cache plus
 * their own earlier tokens, causally; the cache is not modified.
 * Layout as hermes_append_chunk.  Not allowed between an append and its
 * compress.  Errors: EINVAL, ESTATE, EHIP.
 */
int hermes_query_attend(hermes_ctx *ctx, int32_t layer, const void *q, const void *k,
                        const void *v, int32_t n_q, void *out, void *stream);

/*
 * Return every layer to its state right after hermes_kv_init (initial length,
 * buffer 0 current), dropping any step in progress.  Host-only.  Allowed only
 * while no compaction has written into buffer 0 since init (each layer
 * compacted at most once), so the initial rows are still intact; otherwise
 * HERMES_ESTATE.  Used to replay one step on the same initial cache.
 */
int hermes_kv_rewind(hermes_ctx *ctx);

/* Current buffer pointers and host-tracked length of one layer. */
int hermes_kv_view(const hermes_ctx *ctx, int32_t layer, const void **k, const void **v,
                   const int32_t **pos, int32_t *len);

/* Current RoPE-position buffer of one layer (NULL when the context keeps
 * none); it has the length hermes_kv_view reports. */
int hermes_kv_view_rope(const hermes_ctx *ctx, int32_t layer, const int32_t **rpos);

/* Current t, h and w coordinate buffers of one layer (rope_axes 3; all NULL
 * otherwise); they have the length hermes_kv_view reports. */
int hermes_kv_view_mrope(const hermes_ctx *ctx, int32_t layer, const int32_t **t,
                         const int32_t **h, const int32_t **w);

/*
 * Layer-dependent budgets from layer weights (Sec. 4 ablation "Layer-
 * dependent Memory Budget"): budget[i] = floor((w[i] / sum_j w[j]) * total),
 * evaluated in double with the sum taken in layer order, and the rounding
 * residue added to the last layer so the budgets sum to `total`.  Host only.
 * Errors: EINVAL (null pointer, n_layers < 1, a weight not finite or < 0,
 * all weights 0, total < n_layers, a resulting budget < 1).
 */
int hermes_budget_from_weights(const double *weights, int32_t n_layers, int64_t total,
                               int32_t *budget);

/* Free the host context (device buffers stay with the caller). */
void hermes_kv_destroy(hermes_ctx *ctx);

/* Static message for a return code. */
const char *hermes_strerror(int code);

/*
 * Stand-alone TopK (Sec. 3.2 TopK equation) over caller keys, through the
 * selection routine the compression runs per layer (keys held in registers
 * up to 10240 of them, staged in LDS up to 38400, read from memory beyond):
 * keys is device fp32 [n] of non-negative finite values, out_idx device
 * int32 [k]; writes the k largest keys' indices in ascending order, ties to
 * the higher index.  k >= n writes 0..n-1.  One workgroup, no scratch memory.
 * Errors: EINVAL (null pointer, n < 1, k < 1), EHIP.
 */
int hermes_select_topk(const float *keys, int32_t n, int32_t k, int32_t *out_idx,
                       void *stream);

/*
 * Precondition checks on the device, for callers that want the inputs the
 * fast path trusts verified: while enabled, hermes_append_chunk (all forms)
 * first checks that q, k and v hold only finite bf16 values, that pos is
 * strictly increasing and that pos[0] is greater than the last cached
 * position of every appended layer (stream positions only grow: the
 * cross-layer smoothing join and the recency term of Sec. 3.1 / 3.2 rely on
 * sorted positions); hermes_query_attend and hermes_guidance_score check
 * that q, k and v are finite.  The check runs on the call's stream and the
 * call waits for it (one stream synchronisation), so a violation returns
 * HERMES_EINVAL before anything else is launched: device data and host
 * lengths are untouched.  Off by default; the environment variable
 * HERMES_CHECK=1 at hermes_kv_init turns it on for that context.  Uses a
 * word of the context's workspace; not for use under graph capture.
 * Errors: EINVAL (null context), EHIP from the check's own launches (the
 * context is then poisoned).
 */
int hermes_check_enable(hermes_ctx *ctx, int on);

/*
 * Kernel timing with HIP events recorded on the launch stream around every
 * launch of one kernel class while enabled.  Kernel ids: 0 append copy,
 * 1 chunk attention, 2 attention-mass sweep, 3 score+select, 4 gather (and
 * re-indexing), 5 query attention, 6 summary reduction, 7 guidance scoring.  hermes_profile_read waits for the recorded events and
 * returns the summed milliseconds and the launch count since the last read.
 */
enum { HERMES_K_APPEND = 0, HERMES_K_ATTN = 1, HERMES_K_COLSUM = 2, HERMES_K_SELECT = 3,
       HERMES_K_GATHER = 4, HERMES_K_QUERY = 5, HERMES_K_SUMMARY = 6, HERMES_K_GUIDE = 7,
       HERMES_K_COUNT = 8 };
int hermes_profile_enable(hermes_ctx *ctx, int on);
int hermes_profile_read(hermes_ctx *ctx, int kernel_id, double *ms_total, int64_t *count);

#ifdef __cplusplus
}
#endif
#endif /* HERMES_H */
