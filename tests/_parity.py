"""Shared helpers of the GPU parity tests: run one streaming step through the
C ABI and through the fp64 oracle on the same seeded inputs, and compare to
the tolerances of the streaming-step contract:

  * attention outputs within max-abs 2e-2 (bf16 inputs, fp32 accumulation),
    and, so that the bar can fail where the outputs themselves are small
    (long caches spread the softmax thin), within 2e-2 of max|O_ref| and
    within 1e-2 relative in the L2 norm;
  * attention mass W and smoothed keys S~ within 1e-3 relative;
  * kept index sets bit-exact, except tokens whose oracle S~ lies within 1e-6
    relative of the budget-th largest;
  * compacted K/V rows and positions bit-exact copies of the kept inputs.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import hermes_oracle as orc
from paper_2601_14724_amd import streaming, workloads as wk

O_ATOL = 2e-2
O_RREL = 2e-2    # max |O - O_ref| / max |O_ref|
O_L2REL = 1e-2   # ||O - O_ref||_2 / ||O_ref||_2
W_RTOL = 1e-3
S_RTOL = 1e-3
BAND = 1e-6

f64 = wk.bf16_bits_to_f64


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check_o(got, want, what):
    """Attention output against the oracle: max-abs 2e-2 (the contract), plus
    the two signal-relative bars, which an all-zero or a mis-normalised output
    fails however small the outputs are.  Returns and prints the errors."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    diff = np.abs(got - want)
    err = float(diff.max())
    scale = float(np.abs(want).max())
    rel = err / scale if scale > 0 else err
    l2 = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))
    say(f"{what}: O max-abs {err:.3e} (max|O_ref| {scale:.3e}, rel {rel:.3e}), L2 rel {l2:.3e}")
    assert err <= O_ATOL, f"{what}: attention max-abs {err}"
    assert rel <= O_RREL, f"{what}: attention error {rel} of max|O_ref|"
    assert l2 <= O_L2REL, f"{what}: attention L2 relative error {l2}"
    return {"o_maxabs": err, "o_rel": rel, "o_l2rel": l2}


def gen(wl, step=0, layers=None):
    layers = range(wl.n_layers) if layers is None else layers
    caches = [wk.gen_cache(wl, l) for l in layers]
    chunks = [wk.gen_chunk(wl, step, l) for l in layers]
    return caches, chunks


def stacked(chunks):
    return {k: np.stack([c[k] for c in chunks]) for k in ("q", "k", "v")} | {"pos": chunks[0]["pos"]}


def oracle_caches(caches):
    return [orc.LayerCache(f64(c["k"]), f64(c["v"]), c["pos"].astype(np.int64)) for c in caches]


def oracle_chunks(chunks):
    return [{"q": f64(c["q"]), "k": f64(c["k"]), "v": f64(c["v"]), "pos": c["pos"]} for c in chunks]


def oracle_config(wl, **kw):
    return orc.OracleConfig(budgets=list(wl.budgets), **kw)


def run_gpu_step(wl, caches, chunks, device="cuda", **kw):
    kv = streaming.make_cache(wl, device=device, caches=caches, debug=True, **kw)
    t = streaming.chunk_tensors(stacked(chunks), device)
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    torch.cuda.synchronize()
    w = [kv.w[l].cpu().numpy().copy() for l in range(wl.n_layers)]
    kv.compress()
    torch.cuda.synchronize()
    return kv, out.float().cpu().numpy(), w


def band_of(st, budget):
    kth = np.sort(st)[::-1][budget - 1]
    return np.abs(st - kth) <= BAND * kth


def check_layer(l, kv, out_gpu, w_gpu, ref, budget, chunk, check_w=True, check_s=True,
                report=None):
    """Compare one layer of a GPU step with the oracle; returns error stats."""
    stats = check_o(out_gpu[l], ref["out"][l], f"layer {l}")
    T = ref["appended"][l].k.shape[0]
    if check_w:
        wr = ref["w"][l]
        rel = float((np.abs(w_gpu[l][:T] - wr) / wr).max())
        stats["w_rel"] = rel
        assert rel <= W_RTOL, f"layer {l}: attention mass rel error {rel}"
    st = ref["smoothed"][l]
    if T > budget:
        if check_s:
            sg = kv.s_dbg[l][:T].cpu().numpy().astype(np.float64)
            rel = float((np.abs(sg - st) / st).max())
            stats["s_rel"] = rel
            assert rel <= S_RTOL, f"layer {l}: smoothed key rel error {rel}"
        idx_gpu = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
        assert len(idx_gpu) == budget and np.all(np.diff(idx_gpu) > 0), f"layer {l}: bad index list"
        idx_ref = ref["kept"][l]
        diff = np.setxor1d(idx_gpu, idx_ref)
        band = band_of(st, budget)
        outside = [int(i) for i in diff if not band[i]]
        assert not outside, f"layer {l}: kept sets differ outside the 1e-6 band at {outside[:10]}"
        stats["kept_diff"] = len(diff)
    else:
        idx_gpu = np.arange(T)
    k_g, v_g, p_g = kv.view(l)
    n = len(idx_gpu)
    assert k_g.shape[0] == n
    app = ref["appended"][l]
    kb = torch.from_numpy(np.concatenate([report["cache_k"][l], report["chunk_k"][l]]).view(np.int16))
    vb = torch.from_numpy(np.concatenate([report["cache_v"][l], report["chunk_v"][l]]).view(np.int16))
    idx_t = torch.from_numpy(idx_gpu)
    assert torch.equal(k_g.view(torch.int16).cpu(), kb[idx_t]), f"layer {l}: compacted K differs"
    assert torch.equal(v_g.view(torch.int16).cpu(), vb[idx_t]), f"layer {l}: compacted V differs"
    assert np.array_equal(p_g.cpu().numpy(), app.pos[idx_gpu]), f"layer {l}: positions differ"
    return stats


def raw_bits(caches, chunks):
    return {"cache_k": [c["k"] for c in caches], "cache_v": [c["v"] for c in caches],
            "chunk_k": [c["k"] for c in chunks], "chunk_v": [c["v"] for c in chunks]}


# ---------------------------------------------------------------------------
# per-layer oracle composition for full-size workloads (sampled layers)
# ---------------------------------------------------------------------------

def oracle_layer_attention(cache, chunk):
    """Oracle O and W of one layer (cache/chunk as generated bit patterns)."""
    return orc.chunk_attention(f64(chunk["q"]), f64(cache["k"]), f64(cache["v"]),
                               f64(chunk["k"]), f64(chunk["v"]))


def oracle_layer_score(l, classes, w, T0, C, forget_rate=orc.DEFAULT_FORGET_RATE, alpha_mode=0):
    """Raw importance S^l from the oracle's scoring functions (Sec. 3.1)."""
    T = T0 + C
    r = orc.recency_importance(T, forget_rate)
    a = orc.attention_importance(w, T0, C, alpha_mode) if classes[l] != orc.SHALLOW else None
    om = orc.omega(l, classes) if classes[l] == orc.MIDDLE else 0.0
    return orc.raw_importance(classes[l], om, a, r)


def check_kept(idx_gpu, st, budget, what):
    """Kept sets bit-exact except inside the 1e-6 band of the budget-th score."""
    idx_ref = orc.topk_indices(st, budget)
    assert len(idx_gpu) == budget and np.all(np.diff(idx_gpu) > 0), f"{what}: bad index list"
    diff = np.setxor1d(idx_gpu, idx_ref)
    band = band_of(st, budget)
    outside = [int(i) for i in diff if not band[i]]
    assert not outside, f"{what}: kept sets differ outside the 1e-6 band at {outside[:10]}"
    return len(diff)
