"""Thin ctypes binding of libhermes.so (argument marshalling only).

Every step of the streaming path runs in the library's HIP kernels; this
module only allocates device buffers with torch, passes raw pointers and the
current HIP stream, and turns negative return codes into exceptions.  If the
library has not been built it raises at import time: there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhermes.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2601_14724_amd.build`"
                      " (or __graft_entry__.build()) before using the HIP path")
lib = ctypes.CDLL(_LIB_PATH)

OK, EINVAL, ECAPACITY, ESTATE, EHIP, ENOTSUP = 0, -1, -2, -3, -4, -5
SHALLOW, MIDDLE, DEEP = 0, 1, 2
ALL_LAYERS = -1
MAX_LAYERS = 64
K_APPEND, K_ATTN, K_COLSUM, K_SELECT, K_GATHER, K_QUERY, K_SUMMARY, K_GUIDE = range(8)
KERNEL_NAMES = ("append", "attention", "colsum", "select", "gather", "query", "summary", "guide")
REINDEX_NONE, REINDEX_EAGER, REINDEX_LAZY = 0, 1, 2
SCORE_CHUNK, SCORE_GUIDANCE = 0, 1

EXPORTED = ("hermes_workspace_bytes", "hermes_kv_init", "hermes_append_chunk",
            "hermes_append_chunk_at", "hermes_guidance_score", "hermes_compress",
            "hermes_append_chunk_mrope", "hermes_query_attend", "hermes_kv_rewind",
            "hermes_kv_view", "hermes_kv_view_rope", "hermes_kv_view_mrope",
            "hermes_budget_from_weights", "hermes_kv_destroy", "hermes_strerror",
            "hermes_select_topk", "hermes_profile_enable", "hermes_profile_read",
            "hermes_check_enable", "hermes_kv_init_static")
STATIC_WORKSPACE_BYTES = 64 << 20


class HermesConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_chunk", ctypes.c_int32), ("max_cap", ctypes.c_int32),
                ("budget", ctypes.POINTER(ctypes.c_int32)),
                ("layer_class", ctypes.POINTER(ctypes.c_int8)),
                ("lambda_", ctypes.POINTER(ctypes.c_float)),
                ("omega0", ctypes.c_double), ("gamma", ctypes.c_double),
                ("forget_rate", ctypes.c_double), ("sm_scale", ctypes.c_double),
                ("alpha_mode", ctypes.c_int32), ("align_mode", ctypes.c_int32),
                ("force_scores", ctypes.c_int32),
                ("summary_mode", ctypes.c_int32), ("reindex_mode", ctypes.c_int32),
                ("rope_offset", ctypes.c_int32), ("rope_limit", ctypes.c_int32),
                ("rope_headroom", ctypes.c_int32), ("rope_theta", ctypes.c_double),
                ("scoring_mode", ctypes.c_int32), ("rope_axes", ctypes.c_int32),
                ("mrope_section", ctypes.c_int32 * 3)]


class LayerBuffers(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p * 2), ("v", ctypes.c_void_p * 2),
                ("pos", ctypes.c_void_p * 2), ("w", ctypes.c_void_p),
                ("s_dbg", ctypes.c_void_p), ("kept_dbg", ctypes.c_void_p),
                ("cap", ctypes.c_int32), ("init_len", ctypes.c_int32),
                ("rpos", ctypes.c_void_p * 2), ("rpos_h", ctypes.c_void_p * 2),
                ("rpos_w", ctypes.c_void_p * 2)]


_vp, _i32, _i64, _dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
lib.hermes_workspace_bytes.restype = ctypes.c_size_t
lib.hermes_workspace_bytes.argtypes = [ctypes.POINTER(HermesConfig)]
lib.hermes_kv_init.restype = ctypes.c_int
lib.hermes_kv_init.argtypes = [ctypes.POINTER(HermesConfig), ctypes.POINTER(LayerBuffers), _vp,
                               ctypes.c_size_t, ctypes.POINTER(_vp)]
lib.hermes_kv_init_static.restype = ctypes.c_int
lib.hermes_kv_init_static.argtypes = [ctypes.POINTER(HermesConfig), ctypes.POINTER(LayerBuffers),
                                      ctypes.POINTER(_vp)]
lib.hermes_append_chunk.restype = ctypes.c_int
lib.hermes_append_chunk.argtypes = [_vp, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp]
lib.hermes_append_chunk_at.restype = ctypes.c_int
lib.hermes_append_chunk_at.argtypes = [_vp, _i32, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp]
lib.hermes_append_chunk_mrope.restype = ctypes.c_int
lib.hermes_append_chunk_mrope.argtypes = [_vp, _i32, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp]
lib.hermes_kv_view_mrope.restype = ctypes.c_int
lib.hermes_kv_view_mrope.argtypes = [_vp, _i32, ctypes.POINTER(_vp), ctypes.POINTER(_vp),
                                     ctypes.POINTER(_vp)]
lib.hermes_guidance_score.restype = ctypes.c_int
lib.hermes_guidance_score.argtypes = [_vp, _i32, _vp, _vp, _vp, _i32, _vp]
lib.hermes_kv_view_rope.restype = ctypes.c_int
lib.hermes_kv_view_rope.argtypes = [_vp, _i32, ctypes.POINTER(_vp)]
lib.hermes_budget_from_weights.restype = ctypes.c_int
lib.hermes_budget_from_weights.argtypes = [ctypes.POINTER(_dbl), _i32, _i64, ctypes.POINTER(_i32)]
lib.hermes_compress.restype = ctypes.c_int
lib.hermes_compress.argtypes = [_vp, _vp]
lib.hermes_query_attend.restype = ctypes.c_int
lib.hermes_query_attend.argtypes = [_vp, _i32, _vp, _vp, _vp, _i32, _vp, _vp]
lib.hermes_kv_rewind.restype = ctypes.c_int
lib.hermes_kv_rewind.argtypes = [_vp]
lib.hermes_kv_view.restype = ctypes.c_int
lib.hermes_kv_view.argtypes = [_vp, _i32, ctypes.POINTER(_vp), ctypes.POINTER(_vp),
                               ctypes.POINTER(_vp), ctypes.POINTER(_i32)]
lib.hermes_kv_destroy.restype = None
lib.hermes_kv_destroy.argtypes = [_vp]
lib.hermes_strerror.restype = ctypes.c_char_p
lib.hermes_strerror.argtypes = [ctypes.c_int]
lib.hermes_select_topk.restype = ctypes.c_int
lib.hermes_select_topk.argtypes = [_vp, _i32, _i32, _vp, _vp]
lib.hermes_check_enable.restype = ctypes.c_int
lib.hermes_check_enable.argtypes = [_vp, ctypes.c_int]
lib.hermes_profile_enable.restype = ctypes.c_int
lib.hermes_profile_enable.argtypes = [_vp, ctypes.c_int]
lib.hermes_profile_read.restype = ctypes.c_int
lib.hermes_profile_read.argtypes = [_vp, ctypes.c_int, ctypes.POINTER(_dbl), ctypes.POINTER(_i64)]


class HermesError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {lib.hermes_strerror(code).decode()} ({code})")
        self.code = code


def check(code: int, what: str) -> None:
    if code != OK:
        raise HermesError(code, what)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _need(t: torch.Tensor, dtype: torch.dtype, shape: tuple, name: str) -> None:
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or tuple(t.shape) != shape:
        raise ValueError(f"{name}: expected {dtype} {shape}, got "
                         f"{getattr(t, 'dtype', None)} {tuple(getattr(t, 'shape', ()))}")
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name}: must be a contiguous device tensor")


def budget_from_weights(weights: Sequence[float], total: int) -> list:
    """Per-layer budgets floor(w_i / sum w * total), residue to the last layer
    (the library's host helper)."""
    n = len(weights)
    w = (ctypes.c_double * n)(*[float(x) for x in weights])
    out = (ctypes.c_int32 * n)()
    check(lib.hermes_budget_from_weights(w, n, int(total), out), "hermes_budget_from_weights")
    return list(out)


def select_topk(keys: torch.Tensor, k: int) -> torch.Tensor:
    """Indices (ascending) of the k largest non-negative fp32 keys, ties to the
    higher index, computed by the library's TopK kernel."""
    _need(keys, torch.float32, (keys.numel(),), "keys")
    out = torch.empty(min(k, keys.numel()), dtype=torch.int32, device=keys.device)
    check(lib.hermes_select_topk(keys.data_ptr(), keys.numel(), k, out.data_ptr(), _stream()),
          "hermes_select_topk")
    return out


class HermesKV:
    """Per-layer KV caches managed by libhermes.

    Device memory (two ping-pong buffers per layer, positions, the attention
    mass, optional debug outputs and the workspace) is allocated here with
    torch; the library only receives pointers.  `init` optionally gives each
    layer's initial (k, v, pos) as device tensors of shapes [n][Hkv][d] bf16,
    [n][Hkv][d] bf16 and [n] int32, then optionally its RoPE positions [n]
    (rope_axes 1) or its (t, h, w) coordinates [3][n] int32 (rope_axes 3).
    """

    def __init__(self, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 budgets: Sequence[int], max_chunk: int, cap: Optional[int] = None,
                 init: Optional[Sequence[tuple]] = None,
                 layer_class: Optional[Sequence[int]] = None,
                 lambdas: Optional[Sequence[float]] = None, omega0: float = 0.75,
                 gamma: float = 0.6, forget_rate: float = 2.0 ** -10,
                 sm_scale: Optional[float] = None, alpha_mode: int = 0, align_mode: int = 0,
                 force_scores: bool = False, debug: bool = False, device: str = "cuda",
                 summary_mode: int = 0, reindex_mode: int = REINDEX_NONE, rope_offset: int = 0,
                 rope_limit: int = 0, rope_headroom: int = 0, rope_theta: float = 1.0e6,
                 scoring_mode: int = SCORE_CHUNK, rope_axes: int = 1,
                 mrope_section: Sequence[int] = (0, 0, 0), static_workspace: bool = False):
        self.L, self.Hq, self.Hkv, self.d = n_layers, n_q_heads, n_kv_heads, head_dim
        self.budgets = [int(b) for b in budgets]
        self.max_chunk = int(max_chunk)
        init_lens = [0] * n_layers if init is None else [int(t[0].shape[0]) for t in init]
        if cap is None:
            cap = max(max(init_lens), max(self.budgets) + int(bool(summary_mode))) + self.max_chunk
        self.rope_axes = 3 if rope_axes == 3 else 1
        self.keep_rpos = bool(summary_mode) or reindex_mode != REINDEX_NONE or self.rope_axes == 3
        self.cap = int(cap)
        self.device = torch.device(device)
        dev = self.device
        shp = (self.cap, n_kv_heads, head_dim)
        self.k = [[torch.zeros(shp, dtype=torch.bfloat16, device=dev) for _ in range(2)]
                  for _ in range(n_layers)]
        self.v = [[torch.zeros(shp, dtype=torch.bfloat16, device=dev) for _ in range(2)]
                  for _ in range(n_layers)]
        self.pos = [[torch.zeros(self.cap, dtype=torch.int32, device=dev) for _ in range(2)]
                    for _ in range(n_layers)]
        self.rpos = ([[torch.zeros(self.cap, dtype=torch.int32, device=dev) for _ in range(2)]
                      for _ in range(n_layers)] if self.keep_rpos else None)
        three = self.rope_axes == 3
        self.rpos_h = ([[torch.zeros(self.cap, dtype=torch.int32, device=dev) for _ in range(2)]
                        for _ in range(n_layers)] if three else None)
        self.rpos_w = ([[torch.zeros(self.cap, dtype=torch.int32, device=dev) for _ in range(2)]
                        for _ in range(n_layers)] if three else None)
        self.w = [torch.zeros(self.cap, dtype=torch.float32, device=dev) for _ in range(n_layers)]
        self.s_dbg = ([torch.zeros(self.cap, dtype=torch.float32, device=dev)
                       for _ in range(n_layers)] if debug else None)
        self.kept_dbg = ([torch.zeros(b, dtype=torch.int32, device=dev) for b in self.budgets]
                         if debug else None)
        if init is not None:
            for l, t in enumerate(init):
                k0, v0, p0 = t[:3]
                n = k0.shape[0]
                self.k[l][0][:n].copy_(k0)
                self.v[l][0][:n].copy_(v0)
                self.pos[l][0][:n].copy_(p0)
                if three and n > 0:   # (t, h, w) coordinates [3][n] (4th element)
                    if len(t) < 4:
                        raise ValueError("rope_axes 3: init needs (k, v, pos, thw)")
                    self.rpos[l][0][:n].copy_(t[3][0])
                    self.rpos_h[l][0][:n].copy_(t[3][1])
                    self.rpos_w[l][0][:n].copy_(t[3][2])
                elif self.keep_rpos and not three:   # RoPE positions (4th element), default the stream ones
                    self.rpos[l][0][:n].copy_(t[3] if len(t) > 3 else p0)
        self._budget_arr = (ctypes.c_int32 * n_layers)(*self.budgets)
        self._class_arr = ((ctypes.c_int8 * n_layers)(*layer_class)
                           if layer_class is not None else None)
        self._lambda_arr = ((ctypes.c_float * n_layers)(*lambdas) if lambdas is not None else None)
        cfg = HermesConfig()
        cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim = (n_layers, n_q_heads,
                                                                     n_kv_heads, head_dim)
        cfg.max_chunk, cfg.max_cap = self.max_chunk, self.cap
        cfg.budget = self._budget_arr
        cfg.layer_class = (ctypes.cast(self._class_arr, ctypes.POINTER(ctypes.c_int8))
                           if self._class_arr is not None else None)
        cfg.lambda_ = (ctypes.cast(self._lambda_arr, ctypes.POINTER(ctypes.c_float))
                       if self._lambda_arr is not None else None)
        cfg.omega0, cfg.gamma, cfg.forget_rate = omega0, gamma, forget_rate
        cfg.sm_scale = sm_scale if sm_scale is not None else 0.0
        cfg.alpha_mode, cfg.align_mode, cfg.force_scores = alpha_mode, align_mode, int(force_scores)
        cfg.summary_mode, cfg.reindex_mode, cfg.scoring_mode = int(summary_mode), reindex_mode, scoring_mode
        cfg.rope_offset, cfg.rope_limit, cfg.rope_headroom = rope_offset, rope_limit, rope_headroom
        cfg.rope_theta = rope_theta
        cfg.rope_axes = int(rope_axes)
        for a in range(3):
            cfg.mrope_section[a] = int(mrope_section[a])
        self._cfg = cfg
        nbytes = lib.hermes_workspace_bytes(ctypes.byref(cfg))
        if nbytes == 0:
            raise HermesError(EINVAL, "hermes_workspace_bytes")
        # static_workspace: the library's own device scratch (hermes_kv_init_static)
        self.workspace = (None if static_workspace
                          else torch.empty(nbytes, dtype=torch.uint8, device=dev))
        bufs = (LayerBuffers * n_layers)()
        for l in range(n_layers):
            b = bufs[l]
            for p in range(2):
                b.k[p] = self.k[l][p].data_ptr()
                b.v[p] = self.v[l][p].data_ptr()
                b.pos[p] = self.pos[l][p].data_ptr()
            b.w = self.w[l].data_ptr()
            b.s_dbg = _ptr(self.s_dbg[l]) if debug else None
            b.kept_dbg = _ptr(self.kept_dbg[l]) if debug else None
            b.cap = self.cap
            b.init_len = init_lens[l]
            if self.keep_rpos:
                for p in range(2):
                    b.rpos[p] = self.rpos[l][p].data_ptr()
            if three:
                for p in range(2):
                    b.rpos_h[p] = self.rpos_h[l][p].data_ptr()
                    b.rpos_w[p] = self.rpos_w[l][p].data_ptr()
        self._bufs = bufs
        ctx = ctypes.c_void_p()
        if static_workspace:
            with torch.cuda.device(dev):
                check(lib.hermes_kv_init_static(ctypes.byref(cfg), bufs, ctypes.byref(ctx)),
                      "hermes_kv_init_static")
        else:
            check(lib.hermes_kv_init(ctypes.byref(cfg), bufs, self.workspace.data_ptr(), nbytes,
                                     ctypes.byref(ctx)), "hermes_kv_init")
        self.ctx = ctx

    # ------------------------------------------------------------------ calls
    def _check_inputs(self, q, k, v, n, layer):
        lead = () if layer != ALL_LAYERS else (self.L,)
        _need(q, torch.bfloat16, lead + (n, self.Hq, self.d), "q")
        _need(k, torch.bfloat16, lead + (n, self.Hkv, self.d), "k")
        _need(v, torch.bfloat16, lead + (n, self.Hkv, self.d), "v")

    def append(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, pos: torch.Tensor,
               layer: int = ALL_LAYERS, out: Optional[torch.Tensor] = None,
               rope_pos: Optional[torch.Tensor] = None,
               rope_thw: Optional[torch.Tensor] = None) -> torch.Tensor:
        n = q.shape[-3]
        self._check_inputs(q, k, v, n, layer)
        _need(pos, torch.int32, (n,), "pos")
        if out is None:
            out = torch.empty_like(q)
        if rope_thw is not None:
            _need(rope_thw, torch.int32, (3, n), "rope_thw")
            check(lib.hermes_append_chunk_mrope(self.ctx, layer, q.data_ptr(), k.data_ptr(),
                                                v.data_ptr(), pos.data_ptr(), rope_thw.data_ptr(),
                                                n, out.data_ptr(), _stream()),
                  "hermes_append_chunk_mrope")
        elif rope_pos is None:
            check(lib.hermes_append_chunk(self.ctx, layer, q.data_ptr(), k.data_ptr(),
                                          v.data_ptr(), pos.data_ptr(), n, out.data_ptr(),
                                          _stream()), "hermes_append_chunk")
        else:
            _need(rope_pos, torch.int32, (n,), "rope_pos")
            check(lib.hermes_append_chunk_at(self.ctx, layer, q.data_ptr(), k.data_ptr(),
                                             v.data_ptr(), pos.data_ptr(), rope_pos.data_ptr(), n,
                                             out.data_ptr(), _stream()), "hermes_append_chunk_at")
        return out

    def guidance(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                 layer: int = ALL_LAYERS) -> None:
        """Attention mass of the cached tokens from guidance-prompt rows."""
        n = q.shape[-3]
        self._check_inputs(q, k, v, n, layer)
        check(lib.hermes_guidance_score(self.ctx, layer, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                        n, _stream()), "hermes_guidance_score")

    def compress(self) -> None:
        check(lib.hermes_compress(self.ctx, _stream()), "hermes_compress")

    def query(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
              layer: int = ALL_LAYERS, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        n = q.shape[-3]
        self._check_inputs(q, k, v, n, layer)
        if out is None:
            out = torch.empty_like(q)
        check(lib.hermes_query_attend(self.ctx, layer, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                      n, out.data_ptr(), _stream()), "hermes_query_attend")
        return out

    def rewind(self) -> None:
        check(lib.hermes_kv_rewind(self.ctx), "hermes_kv_rewind")

    def length(self, layer: int) -> int:
        ln = ctypes.c_int32()
        check(lib.hermes_kv_view(self.ctx, layer, None, None, None, ctypes.byref(ln)),
              "hermes_kv_view")
        return ln.value

    def view(self, layer: int):
        """(k, v, pos) tensors of the layer's current buffer, first `len` rows."""
        kp, vp, pp, ln = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_int32()
        check(lib.hermes_kv_view(self.ctx, layer, ctypes.byref(kp), ctypes.byref(vp),
                                 ctypes.byref(pp), ctypes.byref(ln)), "hermes_kv_view")
        p = 0 if kp.value == self.k[layer][0].data_ptr() else 1
        n = ln.value
        return self.k[layer][p][:n], self.v[layer][p][:n], self.pos[layer][p][:n]

    def view_rope(self, layer: int) -> torch.Tensor:
        """RoPE positions of the layer's current buffer, first `len` rows."""
        rp = ctypes.c_void_p()
        check(lib.hermes_kv_view_rope(self.ctx, layer, ctypes.byref(rp)), "hermes_kv_view_rope")
        if not rp.value:
            raise ValueError("this cache keeps no RoPE positions")
        p = 0 if rp.value == self.rpos[layer][0].data_ptr() else 1
        return self.rpos[layer][p][:self.length(layer)]

    def view_mrope(self, layer: int) -> torch.Tensor:
        """(t, h, w) coordinates [3][len] of the layer's current buffer."""
        t, h, w = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p()
        check(lib.hermes_kv_view_mrope(self.ctx, layer, ctypes.byref(t), ctypes.byref(h),
                                       ctypes.byref(w)), "hermes_kv_view_mrope")
        if not t.value:
            raise ValueError("this cache keeps no M-RoPE coordinates")
        p = 0 if t.value == self.rpos[layer][0].data_ptr() else 1
        n = self.length(layer)
        return torch.stack([self.rpos[layer][p][:n], self.rpos_h[layer][p][:n],
                            self.rpos_w[layer][p][:n]])

    # -------------------------------------------------------------- profiling
    def check_preconditions(self, on: bool = True) -> None:
        """Device-side checks of positions and finiteness before each call."""
        check(lib.hermes_check_enable(self.ctx, int(on)), "hermes_check_enable")

    def profile(self, on: bool = True) -> None:
        check(lib.hermes_profile_enable(self.ctx, int(on)), "hermes_profile_enable")

    def profile_read(self, kernel_id: int):
        ms, cnt = ctypes.c_double(), ctypes.c_int64()
        check(lib.hermes_profile_read(self.ctx, kernel_id, ctypes.byref(ms), ctypes.byref(cnt)),
              "hermes_profile_read")
        return ms.value, cnt.value

    def close(self) -> None:
        if getattr(self, "ctx", None) is not None and self.ctx.value:
            lib.hermes_kv_destroy(self.ctx)
            self.ctx = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def default_sm_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
