"""Plain, slow fp64 CPU oracle for the HERMES streaming step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module; only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library: it imports
numpy only, and receives its inputs as arrays.

What it computes, in the paper's order and notation (arXiv 2601.14724):

  1. chunk-wise prefill: the chunk's queries attend the layer's cached tokens
     plus the chunk's own earlier tokens (Sec. 2 setup, Sec. 4.1); the same
     pass yields W_i, the attention mass every candidate token receives;
  2. per-layer importance S_i^l (Sec. 3.1): recency for shallow layers (first
     equation of Sec. 3.1), attention for deep layers (second equation), the
     omega-weighted mix for middle layers (third and fourth equations), with
     the 10/60/30 layer partition of Sec. 4.1;
  3. cross-layer smoothing S~^l = (1 - lambda_l) S^l + lambda_l S^{l+1}
     (Sec. 3.2, first equation), lambda by layer class (Appendix C);
  4. TopK to the per-layer budget and gather of K/V (Sec. 3.2, second
     equation);
  5. query-time attention over the compact cache (Sec. 3 overview: the
     query is answered from the cache with no retrieval).

Readings where the paper is silent or ambiguous (each is a parameter here):
  * alpha (the normalisation factor of the first two equations of Sec. 3.1):
    alpha_mode 0 divides each token's attention mass by the number of chunk
    rows that can see it (causal mask) and then normalises to sum 1;
    alpha_mode 1 only normalises to sum 1.  The recency term is normalised to
    sum 1.
  * forget rate k: not given; default 2^-10 per token.
  * T and i in Delta t = T - 1 - i: T = cached + chunk tokens, i = physical
    index in the order-preserving cache.
  * W comes from the chunk's own queries (all heads, all rows), not from the
    guidance-prompt pseudo-query.
  * candidates: every cached token and every chunk token.
  * eviction: a layer evicts iff T > |M|_l, down to exactly |M|_l.
  * partition rounding: n_shallow = floor(0.1 L + 1/2), n_deep = floor(0.3 L
    + 1/2), the rest middle.
  * l_short / l_long: the first and last middle layer.
  * smoothing is one hop with the RAW S^{l+1}; the last layer keeps S.
    align_mode 0 pairs a token with the token of the same stream position in
    layer l+1 (absent -> contributes 0); align_mode 1 pairs equal physical
    indices.
  * TopK ties: keys are S~ rounded to float32; order is (key descending,
    index descending); the kept index list is emitted ascending.
  * attention scale 1/sqrt(d); row r sees the whole cache plus chunk rows
    0..r.

Parity pins live in tests/test_oracle_pins.py.  The paper prints no worked
example with scores or kept sets, so no expected value here comes from it;
every function and each reading above is pinned through closed forms,
invariants, library routines (torch SDPA and softmax) and brute force.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

SHALLOW, MIDDLE, DEEP = 0, 1, 2

DEFAULT_OMEGA0 = 0.75       # Sec. 3.1, middle-layer interpolation
DEFAULT_GAMMA = 0.6         # Sec. 3.1, middle-layer interpolation
DEFAULT_FORGET_RATE = 2.0 ** -10
LAMBDA_BY_CLASS = {SHALLOW: 0.1, MIDDLE: 0.3, DEEP: 0.4}   # Appendix C


# --------------------------------------------------------------------------
# configuration (Sec. 4.1 partition, Appendix C lambda, Sec. 3.1 omega)
# --------------------------------------------------------------------------

def layer_partition(n_layers: int) -> List[int]:
    """10% shallow, 60% middle, 30% deep, in layer order (Sec. 4.1)."""
    n_sh = int(math.floor(0.1 * n_layers + 0.5))
    n_dp = int(math.floor(0.3 * n_layers + 0.5))
    n_mid = n_layers - n_sh - n_dp
    return [SHALLOW] * n_sh + [MIDDLE] * n_mid + [DEEP] * n_dp


def smoothing_lambdas(classes: Sequence[int]) -> List[float]:
    """lambda_l by the class of layer l (Appendix C)."""
    return [LAMBDA_BY_CLASS[c] for c in classes]


def omega(layer: int, classes: Sequence[int], omega0: float = DEFAULT_OMEGA0,
          gamma: float = DEFAULT_GAMMA) -> float:
    """omega^l = omega0 - gamma (l - l_short) / (l_long - l_short) (Sec. 3.1)."""
    middle = [l for l, c in enumerate(classes) if c == MIDDLE]
    l_short, l_long = middle[0], middle[-1]
    if l_long == l_short:
        return omega0
    return omega0 - gamma * (layer - l_short) / (l_long - l_short)


@dataclasses.dataclass
class OracleConfig:
    budgets: Sequence[int]
    classes: Optional[Sequence[int]] = None
    lambdas: Optional[Sequence[float]] = None
    omega0: float = DEFAULT_OMEGA0
    gamma: float = DEFAULT_GAMMA
    forget_rate: float = DEFAULT_FORGET_RATE
    sm_scale: Optional[float] = None
    alpha_mode: int = 0
    align_mode: int = 0

    def resolved(self, n_layers: int) -> "OracleConfig":
        classes = list(self.classes) if self.classes is not None else layer_partition(n_layers)
        lambdas = list(self.lambdas) if self.lambdas is not None else smoothing_lambdas(classes)
        return dataclasses.replace(self, classes=classes, lambdas=lambdas)


# --------------------------------------------------------------------------
# step 1: chunk attention and the attention mass W (Sec. 3.1, deep layers)
# --------------------------------------------------------------------------

def chunk_attention(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                    k_new: np.ndarray, v_new: np.ndarray, sm_scale: Optional[float] = None,
                    want_w: bool = True, row_block: int = 64):
    """Causal GQA attention of the chunk over [cache; chunk], in float64.

    q [C][Hq][d]; k_cache, v_cache [T0][Hkv][d]; k_new, v_new [C][Hkv][d].
    Query head h reads KV head h // (Hq/Hkv).  Row r sees candidates
    0 .. T0 + r.  Returns O [C][Hq][d] and W [T0 + C], where W_i is the sum
    over heads and rows of the softmax probability given to candidate i.
    """
    C, Hq, d = q.shape
    T0 = k_cache.shape[0]
    Hkv = k_cache.shape[1] if T0 else k_new.shape[1]
    G = Hq // Hkv
    T = T0 + C
    scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    k_all = np.concatenate([k_cache.reshape(T0, Hkv, d), k_new], axis=0)
    v_all = np.concatenate([v_cache.reshape(T0, Hkv, d), v_new], axis=0)
    out = np.zeros((C, Hq, d))
    w = np.zeros(T)
    for h in range(Hq):
        kv = h // G
        kh = k_all[:, kv, :]
        vh = v_all[:, kv, :]
        for r0 in range(0, C, row_block):
            r1 = min(C, r0 + row_block)
            s = scale * (q[r0:r1, h, :] @ kh.T)                 # [rows][T]
            rows = np.arange(r0, r1)[:, None]
            visible = np.arange(T)[None, :] <= T0 + rows
            s = np.where(visible, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p = p / p.sum(axis=1, keepdims=True)
            out[r0:r1, h, :] = p @ vh
            if want_w:
                w += p.sum(axis=0)
    return out, (w if want_w else None)


# --------------------------------------------------------------------------
# step 2: per-layer importance (Sec. 3.1)
# --------------------------------------------------------------------------

def observer_counts(T0: int, C: int) -> np.ndarray:
    """How many chunk rows (per head) can see each candidate under the causal
    mask: every row sees a cached token, rows j..C-1 see chunk token j."""
    return np.concatenate([np.full(T0, float(C)), C - np.arange(C, dtype=np.float64)])


def attention_importance(w: np.ndarray, T0: int, C: int, alpha_mode: int = 0) -> np.ndarray:
    """A_i = alpha_i W_i, normalised to sum 1 (Sec. 3.1, deep-layer equation)."""
    if alpha_mode == 0:
        a_hat = w / observer_counts(T0, C)
    else:
        a_hat = w.astype(np.float64)
    return a_hat / a_hat.sum()


def recency_importance(T: int, forget_rate: float) -> np.ndarray:
    """R_i = alpha e^{-k Delta t_i}, Delta t_i = T - 1 - i, normalised to sum 1
    (Sec. 3.1, shallow-layer equation)."""
    dt = (T - 1) - np.arange(T, dtype=np.float64)
    r = np.exp(-forget_rate * dt)
    return r / r.sum()


def raw_importance(cls: int, om: float, a: Optional[np.ndarray], r: np.ndarray) -> np.ndarray:
    """S^l by layer class: R (shallow), A (deep), (1-omega)A + omega R (middle)."""
    if cls == SHALLOW:
        return r
    if cls == DEEP:
        return a
    return (1.0 - om) * a + om * r


# --------------------------------------------------------------------------
# step 3: cross-layer smoothing (Sec. 3.2)
# --------------------------------------------------------------------------

def smooth(s_l: np.ndarray, s_next: Optional[np.ndarray], pos_l: np.ndarray,
           pos_next: Optional[np.ndarray], lam: float, align_mode: int = 0) -> np.ndarray:
    """S~^l_i = (1 - lambda) S^l_i + lambda S^{l+1}_{j(i)}; j(i) is the token of
    layer l+1 at the same stream position (align_mode 0) or the same physical
    index (align_mode 1); a token with no partner gets 0 from layer l+1.
    s_next None marks the last layer, which keeps S."""
    if s_next is None:
        return s_l.copy()
    partner = np.zeros_like(s_l)
    if align_mode == 0:
        where = {int(p): j for j, p in enumerate(pos_next)}
        for i, p in enumerate(pos_l):
            j = where.get(int(p))
            if j is not None:
                partner[i] = s_next[j]
    else:
        n = min(len(s_l), len(s_next))
        partner[:n] = s_next[:n]
    return (1.0 - lam) * s_l + lam * partner


# --------------------------------------------------------------------------
# step 4: TopK and gather (Sec. 3.2, second equation)
# --------------------------------------------------------------------------

def selection_keys(s_tilde: np.ndarray) -> np.ndarray:
    """The selection compares S~ rounded to float32."""
    return s_tilde.astype(np.float32)


def topk_indices(s_tilde: np.ndarray, budget: int) -> np.ndarray:
    """I_l = TopK(S~_l, |M|): the budget largest keys, ties to the higher index,
    emitted in ascending index order (the cache keeps stream order)."""
    T = len(s_tilde)
    if T <= budget:
        return np.arange(T, dtype=np.int64)
    keys = selection_keys(s_tilde).astype(np.float64)
    order = np.lexsort((-np.arange(T), -keys))
    return np.sort(order[:budget])


def gather(k: np.ndarray, v: np.ndarray, pos: np.ndarray, idx: np.ndarray):
    """K_l = K_l[I_l], V_l = V_l[I_l], positions alike."""
    return k[idx], v[idx], pos[idx]


# --------------------------------------------------------------------------
# the whole streaming step over all layers
# --------------------------------------------------------------------------

@dataclasses.dataclass
class LayerCache:
    k: np.ndarray      # [T][Hkv][d] float64 (exact bfloat16 values)
    v: np.ndarray
    pos: np.ndarray    # [T] int


def stream_step(caches: List[LayerCache], chunks: List[dict], cfg: OracleConfig,
                compute_attention: bool = True) -> dict:
    """One chunk append + compression over every layer.

    chunks[l] holds q [C][Hq][d], k, v [C][Hkv][d] (float64) and pos [C].
    Returns per-layer O, W, S, S~, kept indices and the new caches."""
    L = len(caches)
    cfg = cfg.resolved(L)
    outs, ws, t0s, cats = [], [], [], []
    for l in range(L):
        c, ch = caches[l], chunks[l]
        T0, C = c.k.shape[0], ch["q"].shape[0]
        o, w = (chunk_attention(ch["q"], c.k, c.v, ch["k"], ch["v"], cfg.sm_scale)
                if compute_attention else (None, None))
        outs.append(o)
        ws.append(w)
        t0s.append(T0)
        cats.append(LayerCache(np.concatenate([c.k, ch["k"]]), np.concatenate([c.v, ch["v"]]),
                               np.concatenate([c.pos, ch["pos"]])))
    scores = []
    for l in range(L):
        T = cats[l].k.shape[0]
        C = T - t0s[l]
        r = recency_importance(T, cfg.forget_rate)
        a = (attention_importance(ws[l], t0s[l], C, cfg.alpha_mode)
             if cfg.classes[l] != SHALLOW else None)
        om = omega(l, cfg.classes, cfg.omega0, cfg.gamma) if cfg.classes[l] == MIDDLE else 0.0
        scores.append(raw_importance(cfg.classes[l], om, a, r))
    smoothed, kept, new_caches = [], [], []
    for l in range(L):
        nxt = l + 1 < L
        st = smooth(scores[l], scores[l + 1] if nxt else None, cats[l].pos,
                    cats[l + 1].pos if nxt else None, cfg.lambdas[l], cfg.align_mode)
        smoothed.append(st)
        idx = topk_indices(st, cfg.budgets[l])
        kept.append(idx)
        new_caches.append(LayerCache(*gather(cats[l].k, cats[l].v, cats[l].pos, idx)))
    return {"out": outs, "w": ws, "scores": scores, "smoothed": smoothed, "kept": kept,
            "caches": new_caches, "appended": cats}


def query_attention(cache: LayerCache, q: np.ndarray, k: np.ndarray, v: np.ndarray,
                    sm_scale: Optional[float] = None) -> np.ndarray:
    """Query tokens attend the compact cache plus their own earlier tokens;
    the cache is not modified."""
    o, _ = chunk_attention(q, cache.k, cache.v, k, v, sm_scale, want_w=False)
    return o
