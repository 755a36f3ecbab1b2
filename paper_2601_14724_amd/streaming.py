"""Device-side set-up of a synthetic streaming workload (marshalling only).

Uploads the seeded inputs of :mod:`paper_2601_14724_amd.workloads` into torch
device tensors and builds the :class:`~paper_2601_14724_amd.hermes.HermesKV`
that the library operates on.  No step of the streaming path runs here.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import workloads as wk
from .hermes import HermesKV


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def make_cache(wl: wk.Workload, device="cuda", max_chunk: Optional[int] = None,
               cap: Optional[int] = None, caches: Optional[Sequence[dict]] = None,
               **kw) -> HermesKV:
    """A HermesKV holding every layer's initial cache of `wl`."""
    if caches is None:
        caches = [wk.gen_cache(wl, l) for l in range(wl.n_layers)]
    init = []
    for c in caches:
        t = (bf16_tensor(c["k"], device), bf16_tensor(c["v"], device),
             torch.from_numpy(c["pos"]).to(device))
        if "thw" in c:        # M-RoPE (t, h, w) coordinates [3][n]
            t = t + (torch.from_numpy(np.ascontiguousarray(c["thw"], dtype=np.int32)).to(device),)
        init.append(t)
    mc = max_chunk if max_chunk is not None else max(wl.chunk, wl.query_len)
    return HermesKV(wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.budgets, mc,
                    cap=cap if cap is not None else wl.cap(), init=init, device=device, **kw)


def chunk_tensors(chunks: dict, device="cuda") -> dict:
    """Stacked chunk inputs (numpy bit patterns) as device tensors."""
    return {"q": bf16_tensor(chunks["q"], device), "k": bf16_tensor(chunks["k"], device),
            "v": bf16_tensor(chunks["v"], device),
            "pos": torch.from_numpy(np.ascontiguousarray(chunks["pos"])).to(device)}
