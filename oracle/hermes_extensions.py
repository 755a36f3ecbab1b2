"""Plain fp64 CPU oracle for the parts adjacent to the HERMES streaming step.

TEST INFRASTRUCTURE ONLY, like oracle/hermes_oracle.py: nothing in the product
path may import, call or execute this module.  It imports numpy and the step
oracle only and shares no code with the HIP library.

What it computes (arXiv 2601.14724):

  * summary token (Sec. 3.2 last paragraph, Algorithm "Summary Token
    Aggregation" in the appendix): in every deep layer that evicts, the
    evicted tokens are folded into one token; V is the plain mean of the
    evicted values, K the mean of the evicted keys after each key is rotated
    from its own RoPE position to the target position t;
  * position re-indexing with a fixed system prefix (Sec. 3.3, appendix
    "Re-indexing for LLaVA-OV (1D RoPE)", the three equations there):
    retained tokens get p_new = offset + rank(p_old) and their cached keys are
    rotated by the relative phase e^{i (p_new - p_old) theta}; eager mode does
    it at every compression, lazy mode only when positions approach the
    model's limit;
  * guidance-prompt pseudo-query scoring (Sec. 3.1 deep-layer paragraph,
    appendix "Guidance Prompt"): the attention mass W comes from the prompt's
    query rows placed after every cached token, instead of from the chunk;
  * layer-weighted budget allocation (Sec. 4 ablation "Layer-dependent Memory
    Budget"): m_i = floor(w_i / sum_j w_j * |M|), residue to the last layer;
  * 3D M-RoPE re-indexing (appendix "Re-indexing for Qwen2.5-VL (3D
    M-RoPE)", its three equations): every axis d in {t, h, w} is left-
    compacted on its own, p_new^(d) = offset + rank of p_old^(d) among the
    layer's retained coordinates on that axis, and every cached key is
    rotated section by section by e^{i (p_new^(d) - p_old^(d)) theta^(d)}.

Readings where the paper is silent (each listed in the design notes):
  * RoPE uses the rotate-half channel layout (pairs (j, j + d/2)) with
    inv_freq_j = theta^(-2j/d), theta = 1e6 by default (the backbone's);
  * the summary target t is the RoPE position of the newest evicted token,
    the summary takes that token's stream position and is inserted at its
    sorted place, so stream order, RoPE order and physical order coincide;
  * the summary does not count against the budget (the algorithm
    concatenates it to the |M| kept tokens), so an evicting deep layer holds
    |M| + 1 entries; an earlier summary is an ordinary candidate later on
    (it can be kept, or evicted and folded into the next summary);
  * stored K/V are bfloat16: the summary's K and V and every re-indexed key
    are rounded from the exact fp64 value to float32 and then to bfloat16
    (round to nearest even both times);
  * re-indexing ranks every retained entry of a layer (summaries included) in
    physical order, p_new = offset + j; eager mode re-indexes every layer at
    every compression, lazy mode re-indexes every layer when the largest
    retained position of any layer plus a headroom reaches the limit;
  * 3D M-RoPE: the d/2 frequency pairs (frequencies theta^(-2j/d) as in
    1D) are split into three contiguous sections, t first, then h, then w,
    with the section sizes an input (by default a quarter of the pairs for t
    and the rest halved between h and w: 16/24/24 at d = 128, the backbone's
    split); the rank on an axis counts DISTINCT retained coordinates, so
    tokens that shared a coordinate still share it; the same offset applies
    to every axis;
  * summary tokens with 3D coordinates: the target is the newest evicted
    token's (t, h, w), each evicted key is aligned to it section by section
    (pair j turns by the change of the coordinate of its section), and the
    summary takes that token's stream position and coordinates, inserted at
    its sorted place as in 1D;
  * guidance rows attend every token of the cache and their own earlier rows
    (the prompt follows the video); only the cached tokens are candidates and
    every one of them is seen by all prompt rows, so alpha_mode 0 divides by
    the prompt's row count for every token.
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction
from typing import List, Optional, Sequence

import numpy as np

from oracle import hermes_oracle as ho

DEFAULT_ROPE_THETA = 1.0e6
REINDEX_NONE, REINDEX_EAGER, REINDEX_LAZY = 0, 1, 2
SCORE_CHUNK, SCORE_GUIDANCE = 0, 1


# --------------------------------------------------------------------------
# bfloat16 storage rounding (independent of the input generator)
# --------------------------------------------------------------------------

def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp64 -> float32 -> bfloat16, both round-to-nearest-even; returned as
    the exact fp64 value of the bfloat16."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    up = (bits + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    out = (up << np.uint64(16)).astype(np.uint32).view(np.float32)
    return out.astype(np.float64)


# --------------------------------------------------------------------------
# RotaryDelta (appendix, 1D re-indexing: third equation)
# --------------------------------------------------------------------------

def inv_freq(head_dim: int, theta: float = DEFAULT_ROPE_THETA) -> np.ndarray:
    """theta_j = theta^(-2j/d), j < d/2: the RoPE frequency vector."""
    return theta ** (-np.arange(head_dim // 2, dtype=np.float64) * 2.0 / head_dim)


def rotary_delta(k: np.ndarray, delta: np.ndarray, theta: float = DEFAULT_ROPE_THETA) -> np.ndarray:
    """k [n][H][d] times e^{i delta_n theta} on the complex pairs
    (k_j, k_{j + d/2}): each key is moved delta_n positions along RoPE."""
    d = k.shape[-1]
    half = d // 2
    ang = np.asarray(delta, dtype=np.float64)[:, None] * inv_freq(d, theta)[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    re, im = k[..., :half], k[..., half:]
    return np.concatenate([re * c - im * s, im * c + re * s], axis=-1)


# --------------------------------------------------------------------------
# summary token (appendix algorithm "Summary Token Aggregation")
# --------------------------------------------------------------------------

def summary_token(k_ev: np.ndarray, v_ev: np.ndarray, rpos_ev: np.ndarray,
                  theta: float = DEFAULT_ROPE_THETA):
    """Step 1: v_sum = Mean(V_p).  Step 2: every pruned key is aligned to the
    target phase t by RotaryDelta(P_p -> t), then k_sum = Mean(K_aligned).
    Returns (k_sum [H][d], v_sum [H][d], t) in fp64, before storage rounding."""
    t = int(np.max(rpos_ev))
    v_sum = v_ev.mean(axis=0)
    aligned = rotary_delta(k_ev, t - np.asarray(rpos_ev, dtype=np.int64), theta)
    return aligned.mean(axis=0), v_sum, t


# --------------------------------------------------------------------------
# re-indexing (appendix, 1D re-indexing: first two equations)
# --------------------------------------------------------------------------

def reindex_positions(rpos: np.ndarray, offset: int) -> np.ndarray:
    """p_new = offset + rank_P(p_old): the retained positions, left-compacted
    behind the fixed prefix of length `offset`."""
    ranks = np.argsort(np.argsort(np.asarray(rpos), kind="stable"), kind="stable")
    return offset + ranks.astype(np.int64)


def reindex_keys(k: np.ndarray, rpos: np.ndarray, offset: int,
                 theta: float = DEFAULT_ROPE_THETA):
    """k_new = k_old * RotaryDelta(p_old, p_new), stored as bfloat16."""
    new = reindex_positions(rpos, offset)
    return round_to_bf16(rotary_delta(k, new - np.asarray(rpos, dtype=np.int64), theta)), new


# --------------------------------------------------------------------------
# 3D M-RoPE re-indexing (appendix, Qwen2.5-VL: its three equations)
# --------------------------------------------------------------------------

def default_mrope_section(head_dim: int):
    """Frequency pairs per axis (t, h, w): a quarter of the d/2 pairs for t,
    the rest halved between h and w (16/24/24 at d = 128)."""
    half = head_dim // 2
    t = half // 4
    h = (half - t) // 2
    return (t, h, half - t - h)


def mrope_pair_axis(head_dim: int, section) -> np.ndarray:
    """Axis (0 = t, 1 = h, 2 = w) of each of the d/2 frequency pairs."""
    s = [int(x) for x in section]
    assert len(s) == 3 and min(s) >= 0 and sum(s) == head_dim // 2, section
    return np.repeat(np.arange(3), s)


def rotary_delta3(k: np.ndarray, delta3: np.ndarray, section,
                  theta: float = DEFAULT_ROPE_THETA) -> np.ndarray:
    """k [n][H][d] times the concatenation over the sections of
    e^{i delta^(d) theta^(d)}: pair j turns by delta[axis(j)] * theta_j."""
    d = k.shape[-1]
    half = d // 2
    axis = mrope_pair_axis(d, section)
    ang = np.asarray(delta3, dtype=np.float64)[:, axis] * inv_freq(d, theta)[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    re, im = k[..., :half], k[..., half:]
    return np.concatenate([re * c - im * s, im * c + re * s], axis=-1)


def summary_token3(k_ev: np.ndarray, v_ev: np.ndarray, coords_ev: np.ndarray, section,
                   theta: float = DEFAULT_ROPE_THETA):
    """The summary-token algorithm with 3D coordinates: v_sum = Mean(V_p);
    every pruned key is aligned to the target (t, h, w) of the newest pruned
    token (the last in stream order) by the sectioned RotaryDelta, then
    k_sum = Mean(K_aligned).  Returns (k_sum [H][d], v_sum [H][d], target
    [3]) in fp64, before storage rounding."""
    coords_ev = np.asarray(coords_ev, dtype=np.int64)
    target = coords_ev[-1].copy()
    v_sum = v_ev.mean(axis=0)
    aligned = rotary_delta3(k_ev, target[None, :] - coords_ev, section, theta)
    return aligned.mean(axis=0), v_sum, target


def reindex_coords3(coords: np.ndarray, offset: int) -> np.ndarray:
    """p_new^(d) = offset + rank of p_old^(d) in the sorted set of the
    retained coordinates on axis d, for d = t, h, w independently."""
    coords = np.asarray(coords, dtype=np.int64)
    out = np.empty_like(coords)
    for a in range(3):
        values = np.unique(coords[:, a])          # the sorted set P^(d)
        out[:, a] = offset + np.searchsorted(values, coords[:, a])
    return out


def reindex_keys3(k: np.ndarray, coords: np.ndarray, offset: int, section,
                  theta: float = DEFAULT_ROPE_THETA):
    """k_new = k_old * RotaryDelta(p_old, p_new) section by section, stored
    as bfloat16; returns (keys, new coordinates)."""
    new = reindex_coords3(coords, offset)
    return round_to_bf16(rotary_delta3(k, new - np.asarray(coords, dtype=np.int64), section, theta)), new


# --------------------------------------------------------------------------
# guidance-prompt pseudo-query (Sec. 3.1 deep layers, appendix prompts)
# --------------------------------------------------------------------------

def guidance_mass(q_g: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                  k_g: np.ndarray, v_g: np.ndarray, sm_scale: Optional[float] = None) -> np.ndarray:
    """W_i over the cached tokens from the prompt rows: the prompt follows the
    video, so row r sees every cached token and prompt rows 0..r."""
    _, w = ho.chunk_attention(q_g, k_cache, v_cache, k_g, v_g, sm_scale)
    return w[:k_cache.shape[0]]


def guidance_importance(w_cache: np.ndarray, n_rows: int, alpha_mode: int = 0) -> np.ndarray:
    """A_i = alpha_i W_i normalised to sum 1; every cached token has the same
    n_rows observers."""
    a_hat = w_cache / float(n_rows) if alpha_mode == 0 else w_cache.astype(np.float64)
    return a_hat / a_hat.sum()


# --------------------------------------------------------------------------
# layer-weighted budgets (Sec. 4 ablation)
# --------------------------------------------------------------------------

def budget_allocation(weights: Sequence[float], total: int) -> List[int]:
    """m_i = floor(w_i / sum_j w_j * |M|); the rounding residue goes to the
    last layer so that sum_i m_i = |M|.  Evaluated in fp64 as
    floor((w_i / sum) * total), the sum taken in layer order."""
    s = 0.0
    for w in weights:
        s += float(w)
    m = [int(np.floor((float(w) / s) * float(total))) for w in weights]
    m[-1] += int(total) - sum(m)
    return m


def budget_allocation_exact(weights: Sequence[str], total: int) -> List[int]:
    """The same rule in exact rational arithmetic (weights as decimal strings),
    used to pin the fp64 evaluation away from rounding boundaries."""
    ws = [Fraction(w) for w in weights]
    s = sum(ws)
    m = [int((w / s) * total) for w in ws]   # floor for non-negative rationals
    m[-1] += total - sum(m)
    return m


# --------------------------------------------------------------------------
# the extended streaming step
# --------------------------------------------------------------------------

@dataclasses.dataclass
class ExtConfig:
    summary: bool = False              # summary token in evicting deep layers
    reindex_mode: int = REINDEX_NONE   # none / eager / lazy
    rope_theta: float = DEFAULT_ROPE_THETA
    rope_offset: int = 0               # length of the fixed system prefix
    rope_limit: int = 1 << 30          # lazy mode: the model's position limit
    rope_headroom: int = 0             # lazy mode: positions kept free below it
    scoring_mode: int = SCORE_CHUNK    # W from the chunk or from a guidance prompt
    rope_axes: int = 1                 # 1: one RoPE position; 3: M-RoPE (t, h, w)
    mrope_section: tuple = ()          # pairs per axis; () = default_mrope_section(d)


@dataclasses.dataclass
class ExtLayerCache:
    k: np.ndarray      # [T][Hkv][d] float64 (exact bfloat16 values)
    v: np.ndarray
    pos: np.ndarray    # [T] stream positions (token identity), strictly increasing
    rpos: np.ndarray   # [T] RoPE positions the stored keys carry, strictly increasing
                       # (3D: the t coordinates, non-decreasing)
    rpos3: Optional[np.ndarray] = None   # [T][3] (t, h, w) coordinates in 3D mode


def stream_step_ext(caches: List[ExtLayerCache], chunks: List[dict], cfg: ho.OracleConfig,
                    ext: ExtConfig, prompts: Optional[List[dict]] = None,
                    compute_attention: bool = True) -> dict:
    """One chunk append + compression with the extensions above.

    chunks[l]: q, k, v (float64), pos and optionally rope_pos (default pos).
    prompts[l] (guidance scoring): q, k, v of the prompt rows of layer l (the
    hybrid local+global prompt for middle layers, the global one for deep
    layers); shallow layers need none."""
    L = len(caches)
    cfg = cfg.resolved(L)
    outs, ws, t0s, cats = [], [], [], []
    for l in range(L):
        c, ch = caches[l], chunks[l]
        T0, C = c.k.shape[0], ch["q"].shape[0]
        want_w = ext.scoring_mode == SCORE_CHUNK
        if compute_attention:
            o, w = ho.chunk_attention(ch["q"], c.k, c.v, ch["k"], ch["v"], cfg.sm_scale, want_w=want_w)
        else:
            o, w = None, None
        outs.append(o)
        if ext.rope_axes == 3:
            thw = np.asarray(ch["rope_thw"], dtype=np.int64).T          # [C][3]
            r3 = np.concatenate([c.rpos3, thw]).astype(np.int64)
            cats.append(ExtLayerCache(np.concatenate([c.k, ch["k"]]), np.concatenate([c.v, ch["v"]]),
                                      np.concatenate([c.pos, ch["pos"]]).astype(np.int64),
                                      r3[:, 0].copy(), r3))
        else:
            rp = np.asarray(ch.get("rope_pos", ch["pos"]), dtype=np.int64)
            cats.append(ExtLayerCache(np.concatenate([c.k, ch["k"]]), np.concatenate([c.v, ch["v"]]),
                                      np.concatenate([c.pos, ch["pos"]]).astype(np.int64),
                                      np.concatenate([c.rpos, rp]).astype(np.int64)))
        if ext.scoring_mode == SCORE_GUIDANCE and cfg.classes[l] != ho.SHALLOW and compute_attention:
            p = prompts[l]
            w = guidance_mass(p["q"], cats[l].k, cats[l].v, p["k"], p["v"], cfg.sm_scale)
        ws.append(w)
        t0s.append(T0)
    scores = []
    for l in range(L):
        T = cats[l].k.shape[0]
        C = T - t0s[l]
        r = ho.recency_importance(T, cfg.forget_rate)
        a = None
        if cfg.classes[l] != ho.SHALLOW:
            if ext.scoring_mode == SCORE_GUIDANCE:
                a = guidance_importance(ws[l], prompts[l]["q"].shape[0], cfg.alpha_mode)
            else:
                a = ho.attention_importance(ws[l], t0s[l], C, cfg.alpha_mode)
        om = ho.omega(l, cfg.classes, cfg.omega0, cfg.gamma) if cfg.classes[l] == ho.MIDDLE else 0.0
        scores.append(ho.raw_importance(cfg.classes[l], om, a, r))
    smoothed, kept, compact, summaries = [], [], [], []
    for l in range(L):
        nxt = l + 1 < L
        st = ho.smooth(scores[l], scores[l + 1] if nxt else None, cats[l].pos,
                       cats[l + 1].pos if nxt else None, cfg.lambdas[l], cfg.align_mode)
        smoothed.append(st)
        idx = ho.topk_indices(st, cfg.budgets[l])
        kept.append(idx)
        c, summ = compact_layer(cats[l], idx, cfg.classes[l] == ho.DEEP, ext)
        summaries.append(summ)
        compact.append(c)
    compact, reindexed = reindex_layers(compact, ext)
    return {"out": outs, "w": ws, "scores": scores, "smoothed": smoothed, "kept": kept,
            "caches": compact, "appended": cats, "summaries": summaries, "reindexed": reindexed}


def compact_layer(cat: ExtLayerCache, idx: np.ndarray, deep: bool, ext: ExtConfig):
    """Gather the kept rows of one appended layer (Sec. 3.2) and, for an
    evicting deep layer with summaries on, insert the summary token of the
    evicted rows at the sorted place of the newest evicted token."""
    T = cat.k.shape[0]
    k, v, pos, rpos = cat.k[idx], cat.v[idx], cat.pos[idx], cat.rpos[idx]
    three = ext.rope_axes == 3
    rpos3 = cat.rpos3[idx] if three else None
    summ = None
    if ext.summary and deep and len(idx) < T:
        mask = np.ones(T, dtype=bool)
        mask[idx] = False
        ev = np.nonzero(mask)[0]
        if three:
            section = ext.mrope_section or default_mrope_section(cat.k.shape[-1])
            ks, vs, tgt = summary_token3(cat.k[ev], cat.v[ev], cat.rpos3[ev], section, ext.rope_theta)
            t = int(tgt[0])
        else:
            ks, vs, t = summary_token(cat.k[ev], cat.v[ev], cat.rpos[ev], ext.rope_theta)
        newest = int(ev[-1])
        ins = int(np.searchsorted(idx, newest))
        k = np.insert(k, ins, round_to_bf16(ks), axis=0)
        v = np.insert(v, ins, round_to_bf16(vs), axis=0)
        pos = np.insert(pos, ins, cat.pos[newest])
        rpos = np.insert(rpos, ins, t)
        if three:
            rpos3 = np.insert(rpos3, ins, tgt, axis=0)
        summ = {"index": ins, "source": newest, "t": t, "evicted": ev,
                "k": round_to_bf16(ks), "v": round_to_bf16(vs)}
        if three:
            summ["target"] = tgt
    return ExtLayerCache(k, v, pos, rpos, rpos3), summ


def reindex_layers(compact: List[ExtLayerCache], ext: ExtConfig):
    """Eager: re-index every layer.  Lazy: re-index every layer when the
    largest retained RoPE position of any layer + headroom reaches the limit."""
    reindexed = False
    if ext.reindex_mode == REINDEX_EAGER:
        reindexed = True
    elif ext.reindex_mode == REINDEX_LAZY:
        if ext.rope_axes == 3:
            top = max(int(c.rpos3.max()) for c in compact if len(c.rpos))
        else:
            top = max(int(c.rpos[-1]) for c in compact if len(c.rpos))
        reindexed = top + ext.rope_headroom >= ext.rope_limit
    if not reindexed:
        return compact, False
    out = []
    if ext.rope_axes == 3:
        for c in compact:
            section = ext.mrope_section or default_mrope_section(c.k.shape[-1])
            k_new, r_new = reindex_keys3(c.k, c.rpos3, ext.rope_offset, section, ext.rope_theta)
            out.append(ExtLayerCache(k_new, c.v, c.pos, r_new[:, 0].copy(), r_new))
        return out, True
    for c in compact:
        k_new, r_new = reindex_keys(c.k, c.rpos, ext.rope_offset, ext.rope_theta)
        out.append(ExtLayerCache(k_new, c.v, c.pos, r_new))
    return out, True
