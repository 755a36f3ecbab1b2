"""Seeded synthetic inputs shaped like the paper's streaming workloads.

This module produces DATA only: the per-layer K/V caches, each chunk's Q/K/V
and the token positions, exactly as a video LLM backbone would hand them to
the cache manager.  It holds none of the cache manager's arithmetic (no
attention, scoring, smoothing, selection or compaction), so both the HIP path
and the CPU oracle can consume the same arrays without sharing method code.

Shapes follow the paper's setting: every video frame becomes 196 tokens
(Sec. 2, investigation setup), chunks carry 4, 8 or 16 frames (Sec. 2 and
Sec. 4.1 implementation details), and the 0.5B / 7B backbones (Qwen2-based
LLaVA-OV) use 14q/2kv heads with d=64 and 28q/4kv heads with d=128.  The
datasets the paper streams are not available; Gaussian Q/K/V stand in for
them (the recipe is stated per workload below).

Generation recipe (per tensor):
  * rng = numpy default_rng(SeedSequence([workload_id, step, layer, tensor_id]))
    tensor ids: chunk Q=0, chunk K=1, chunk V=2, cache K=3, cache V=4,
    low-rank basis U=5, chunk low-rank coefficients=6, cache coefficients=7,
    query Q=8, query K=9, query V=10, guidance-prompt Q=11, K=12, V=13 (step
    id 1000 for the global prompt, 1001 for the hybrid local + global one),
    anchor direction=14, anchor strengths=15, anchor value signs=16;
  * draw float64 N(0,1), scale by 0.5 (standard deviation 0.5);
  * the low-rank key workload adds 1.0 * (z @ U), U in R^{8 x d} with entries
    N(0, 1/8) per (layer, kv head) and z ~ N(0, I_8) per token, before scaling
    the noise term by 0.5;
  * rotary position embedding (rotate-half convention, theta = 1e6,
    inv_freq_j = theta^(-2j/d)) applied in float64 to Q and K at the token's
    stream position;  V gets none;
  * cast to float32, then to bfloat16 by round-to-nearest-even.

Sharp-attention variant (anchor_period > 0), for checks whose attention
outputs must be far above the rounding noise: every token whose stream
position is a multiple of anchor_period is an anchor.  Per (layer, kv head) a
unit direction u lives on the four lowest-frequency rotary pairs (RoPE turns
it by at most a few hundredths of a radian over the workloads' spans), drawn
once from tensor id 14 at step 0.  An anchor key gets + a_p * u with a_p =
d^(1/4) * U(1, 5) (tensor id 15, drawn per anchor from its own position), an
anchor value gets + 0.5 * (a random sign per element, tensor id 16); every
query row (chunk, text query, guidance prompt) of query head h gets
+ 3 d^(1/4) * u of its kv head.  Scores of anchors then stand 3..15 above the
rest (in units of the softmax exponent), so a few anchors spread over the
cache dominate each row and |O| is of order 0.5.  Added before RoPE.

bfloat16 tensors are returned as numpy uint16 bit patterns so that the two
consumers can view them without a conversion step of their own.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

ROPE_THETA = 1.0e6
TOKENS_PER_FRAME = 196

T_CHUNK_Q, T_CHUNK_K, T_CHUNK_V = 0, 1, 2
T_CACHE_K, T_CACHE_V = 3, 4
T_LOWRANK_U, T_CHUNK_Z, T_CACHE_Z = 5, 6, 7
T_QUERY_Q, T_QUERY_K, T_QUERY_V = 8, 9, 10
T_PROMPT_Q, T_PROMPT_K, T_PROMPT_V = 11, 12, 13
T_ANCHOR_U, T_ANCHOR_A, T_ANCHOR_V = 14, 15, 16
PROMPT_GLOBAL, PROMPT_HYBRID = 0, 1


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic streaming workload (shapes, budgets, input recipe)."""

    name: str
    workload_id: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    init_len: int            # tokens already cached in every layer
    chunk: int               # tokens appended per step
    n_steps: int             # chunks streamed in sequence
    budgets: tuple           # per-layer token budget |M|_l
    query_len: int = 0       # text-query tokens attending the compact cache
    low_rank_keys: bool = False
    scale: float = 0.5
    anchor_period: int = 0   # > 0: sharp-attention variant (planted anchor tokens)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def row_elems(self) -> int:
        return self.n_kv_heads * self.head_dim

    def cap(self) -> int:
        """Rows a per-layer buffer needs: the larger of the initial cache and
        the budget, plus one chunk (and room for the chunk at every step)."""
        top = max(self.init_len, max(self.budgets))
        return top + max(self.chunk, self.query_len)

    def chunk_positions(self, step: int) -> np.ndarray:
        start = self.init_len + step * self.chunk
        return np.arange(start, start + self.chunk, dtype=np.int32)

    def query_positions(self) -> np.ndarray:
        start = self.init_len + self.n_steps * self.chunk
        return np.arange(start, start + self.query_len, dtype=np.int32)


def _ramp(lo: int, hi: int, n: int) -> tuple:
    return tuple(lo + ((hi - lo) * l) // (n - 1) for l in range(n))


WORKLOADS = {
    # single layer, 0.5B-like shape, one frame appended to a 1024-token cache
    "c1_0p5b_1layer": Workload("c1_0p5b_1layer", 1, 1, 14, 2, 64, 1024, 196, 1, (512,)),
    # 24 layers, 0.5B-like shape, 4 frames appended to a 4096-token cache
    "c2_0p5b_24layer": Workload("c2_0p5b_24layer", 2, 24, 14, 2, 64, 4096, 784, 1,
                                (2048,) * 24),
    # 28 layers, 7B-like shape, 4 frames onto an 8192-token cache, budgets
    # ramping 2048 -> 6144, low-rank keys so attention mass is skewed
    "c3_7b_28layer": Workload("c3_7b_28layer", 3, 28, 28, 4, 128, 8192, 784, 1,
                              _ramp(2048, 6144, 28), low_rank_keys=True),
    # 28 layers, 7B shape, 64 successive 4-frame chunks from an empty cache
    "c4_7b_stream64": Workload("c4_7b_stream64", 4, 28, 28, 4, 128, 0, 784, 64,
                               (6144,) * 28),
    # 28 layers, 7B shape, 16 frames onto a 32768-token cache, then a
    # 64-token text query over the compacted cache
    "c5_7b_long": Workload("c5_7b_long", 5, 28, 28, 4, 128, 32768, 3136, 1,
                           _ramp(4096, 16384, 28), query_len=64),
}


def _rng(wl: Workload, step: int, layer: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([wl.workload_id, step, layer, tensor_id]))


def rope_f64(x: np.ndarray, positions: np.ndarray, theta: float = ROPE_THETA) -> np.ndarray:
    """Rotary embedding (rotate-half layout) of x [n][heads][d] at positions [n]."""
    d = x.shape[-1]
    half = d // 2
    inv_freq = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = positions.astype(np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float64."""
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _gauss(rng: np.random.Generator, shape, scale: float) -> np.ndarray:
    return rng.standard_normal(shape) * scale


def _anchor_dir(wl: Workload, layer: int) -> np.ndarray:
    """[Hkv][d] unit directions on the four lowest-frequency rotary pairs."""
    d, half = wl.head_dim, wl.head_dim // 2
    cols = np.concatenate([np.arange(half - 4, half), np.arange(d - 4, d)])
    u = np.zeros((wl.n_kv_heads, d))
    u[:, cols] = _rng(wl, 0, layer, T_ANCHOR_U).standard_normal((wl.n_kv_heads, cols.size))
    return u / np.linalg.norm(u, axis=1, keepdims=True)


def _is_anchor(wl: Workload, positions: np.ndarray) -> np.ndarray:
    return (positions % wl.anchor_period) == 0


def _anchor_keys(wl: Workload, layer: int, positions: np.ndarray, k: np.ndarray) -> np.ndarray:
    if wl.anchor_period <= 0:
        return k
    u = _anchor_dir(wl, layer)
    q4 = wl.head_dim ** 0.25
    k = k.copy()
    for i in np.nonzero(_is_anchor(wl, positions))[0]:
        a = q4 * _rng(wl, int(positions[i]), layer, T_ANCHOR_A).uniform(1.0, 5.0, wl.n_kv_heads)
        k[i] += a[:, None] * u
    return k


def _anchor_values(wl: Workload, layer: int, positions: np.ndarray, v: np.ndarray) -> np.ndarray:
    if wl.anchor_period <= 0:
        return v
    v = v.copy()
    for i in np.nonzero(_is_anchor(wl, positions))[0]:
        sgn = _rng(wl, int(positions[i]), layer, T_ANCHOR_V).integers(0, 2, v.shape[1:]) * 2 - 1
        v[i] += 0.5 * sgn
    return v


def _anchor_queries(wl: Workload, layer: int, q: np.ndarray) -> np.ndarray:
    if wl.anchor_period <= 0:
        return q
    u = _anchor_dir(wl, layer)
    return q + 3.0 * wl.head_dim ** 0.25 * np.repeat(u, wl.group, axis=0)[None]


def _keys(wl: Workload, step: int, layer: int, n: int, noise_id: int, coef_id: int,
          positions: np.ndarray) -> np.ndarray:
    shape = (n, wl.n_kv_heads, wl.head_dim)
    k = _gauss(_rng(wl, step, layer, noise_id), shape, wl.scale)
    if wl.low_rank_keys:
        basis = _rng(wl, 0, layer, T_LOWRANK_U).standard_normal(
            (wl.n_kv_heads, 8, wl.head_dim)) * np.sqrt(1.0 / 8.0)
        z = _rng(wl, step, layer, coef_id).standard_normal((n, wl.n_kv_heads, 8))
        k = k + 1.0 * np.einsum("nhr,hrd->nhd", z, basis)
    return rope_f64(_anchor_keys(wl, layer, positions, k), positions)


def _to_bits(x: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(x.astype(np.float32))


def gen_cache(wl: Workload, layer: int) -> dict:
    """The tokens already cached in `layer` before the first step."""
    n = wl.init_len
    pos = np.arange(n, dtype=np.int32)
    k = _keys(wl, 0, layer, n, T_CACHE_K, T_CACHE_Z, pos)
    v = _gauss(_rng(wl, 0, layer, T_CACHE_V), (n, wl.n_kv_heads, wl.head_dim), wl.scale)
    v = _anchor_values(wl, layer, pos, v)
    return {"k": _to_bits(k), "v": _to_bits(v), "pos": pos}


def gen_chunk(wl: Workload, step: int, layer: int) -> dict:
    """The chunk appended to `layer` at `step`: Q, K, V and positions."""
    n = wl.chunk
    pos = wl.chunk_positions(step)
    q = rope_f64(_anchor_queries(wl, layer, _gauss(_rng(wl, step, layer, T_CHUNK_Q),
                                                   (n, wl.n_q_heads, wl.head_dim), wl.scale)), pos)
    k = _keys(wl, step, layer, n, T_CHUNK_K, T_CHUNK_Z, pos)
    v = _gauss(_rng(wl, step, layer, T_CHUNK_V), (n, wl.n_kv_heads, wl.head_dim), wl.scale)
    v = _anchor_values(wl, layer, pos, v)
    return {"q": _to_bits(q), "k": _to_bits(k), "v": _to_bits(v), "pos": pos}


def gen_query(wl: Workload, layer: int) -> dict:
    """The text query's Q/K/V for `layer`, placed after the whole stream."""
    n = wl.query_len
    pos = wl.query_positions()
    q = rope_f64(_anchor_queries(wl, layer, _gauss(_rng(wl, 0, layer, T_QUERY_Q),
                                                   (n, wl.n_q_heads, wl.head_dim), wl.scale)), pos)
    k = rope_f64(_gauss(_rng(wl, 0, layer, T_QUERY_K), (n, wl.n_kv_heads, wl.head_dim),
                        wl.scale), pos)
    v = _gauss(_rng(wl, 0, layer, T_QUERY_V), (n, wl.n_kv_heads, wl.head_dim), wl.scale)
    return {"q": _to_bits(q), "k": _to_bits(k), "v": _to_bits(v), "pos": pos}


def gen_prompt(wl: Workload, layer: int, n_rows: int, kind: int = PROMPT_GLOBAL,
               start: Optional[int] = None) -> dict:
    """Guidance-prompt Q/K/V of `layer` (the tokenised prompt is not
    available; Gaussian rows of the prompt's length stand in), placed after the
    stream at positions start.. (default: right after the first chunk)."""
    if start is None:
        start = wl.init_len + wl.chunk
    pos = np.arange(start, start + n_rows, dtype=np.int32)
    step = 1000 + kind
    q = rope_f64(_anchor_queries(wl, layer, _gauss(_rng(wl, step, layer, T_PROMPT_Q),
                                                   (n_rows, wl.n_q_heads, wl.head_dim), wl.scale)), pos)
    k = rope_f64(_gauss(_rng(wl, step, layer, T_PROMPT_K), (n_rows, wl.n_kv_heads, wl.head_dim),
                        wl.scale), pos)
    v = _gauss(_rng(wl, step, layer, T_PROMPT_V), (n_rows, wl.n_kv_heads, wl.head_dim), wl.scale)
    return {"q": _to_bits(q), "k": _to_bits(k), "v": _to_bits(v), "pos": pos}


def scaled(wl: Workload, **changes) -> Workload:
    """A copy of `wl` with some fields replaced (smaller parity-test variants)."""
    return dataclasses.replace(wl, **changes)


def custom(name: str, workload_id: int, n_layers: int, n_q_heads: int, n_kv_heads: int,
           head_dim: int, init_len: int, chunk: int, budgets: Sequence[int], n_steps: int = 1,
           query_len: int = 0, low_rank_keys: bool = False,
           scale: float = 0.5, anchor_period: int = 0) -> Workload:
    return Workload(name, workload_id, n_layers, n_q_heads, n_kv_heads, head_dim, init_len,
                    chunk, n_steps, tuple(int(b) for b in budgets), query_len, low_rank_keys,
                    scale, anchor_period)


def stack_chunks(wl: Workload, step: int, layers: Optional[Sequence[int]] = None,
                 threads: int = 8) -> dict:
    """All layers' chunk inputs stacked on a leading layer axis."""
    import concurrent.futures as cf
    layers = list(range(wl.n_layers) if layers is None else layers)
    with cf.ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        parts = list(ex.map(lambda l: gen_chunk(wl, step, l), layers))
    return {key: np.stack([p[key] for p in parts]) for key in ("q", "k", "v")} | {
        "pos": parts[0]["pos"]}
