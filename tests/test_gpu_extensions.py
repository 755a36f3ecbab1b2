"""GPU parity of the adjacent rows through the C ABI: summary tokens,
eager / lazy RoPE re-indexing, guidance-prompt scoring and the budget helper,
against the extension oracle on the same seeded inputs.

Kept sets follow the core contract (bit-exact outside the 1e-6 band of the
budget-th key).  The compacted cache is then rebuilt by the oracle from the
GPU's own kept set, so near-tie swaps cannot leak into the comparison of the
summary rows and the rotated keys.  Those are computed in fp64 on both sides
and stored as bf16 through fp32 (two roundings to nearest even, also on the
device, where the compiler would otherwise fold them into one); the RoPE
frequencies come from the host's pow on both sides, so the two fp64 values
differ only where the device's sincos or summation order differs from the
host's at the 1e-16 level, which changes the stored bf16 only for a value
within about 1e-16 of a rounding boundary.  The bar: every element within
one bf16 ulp and at most 1e-6 of the elements off by one."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import hermes_extensions as he
from oracle import hermes_oracle as orc
from paper_2601_14724_amd import hermes as H
from paper_2601_14724_amd import streaming, workloads as wk

from _parity import check_kept, f64, say

pytestmark = pytest.mark.gpu

S, M, D = orc.SHALLOW, orc.MIDDLE, orc.DEEP


def _wl(name, wid, L, Hq, Hkv, d, T0, C, budgets, n_steps=1):
    return wk.custom(name, wid, L, Hq, Hkv, d, T0, C, budgets, n_steps=n_steps)


def _ext_caches(caches):
    return [he.ExtLayerCache(f64(c["k"]), f64(c["v"]), c["pos"].astype(np.int64),
                             c.get("rpos", c["pos"]).astype(np.int64)) for c in caches]


def _ext_chunks(chunks):
    return [{"q": f64(c["q"]), "k": f64(c["k"]), "v": f64(c["v"]), "pos": c["pos"]} for c in chunks]


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _cmp_layer(l, kv, exp: he.ExtLayerCache, what):
    k, v, p = kv.view(l)
    rp = kv.view_rope(l)
    n = len(exp.pos)
    assert k.shape[0] == n, f"{what} layer {l}: length {k.shape[0]} != {n}"
    assert np.array_equal(p.cpu().numpy(), exp.pos), f"{what} layer {l}: positions differ"
    assert np.array_equal(rp.cpu().numpy(), exp.rpos), f"{what} layer {l}: RoPE positions differ"
    kg = wk.bf16_bits_to_f64(_bits(k).reshape(exp.k.shape))
    vg = wk.bf16_bits_to_f64(_bits(v).reshape(exp.v.shape))
    for name, g, e in (("K", kg, exp.k), ("V", vg, exp.v)):
        diff = g != e
        if diff.any():
            ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(e), 1e-30))) - 7)
            worst = float(np.max(np.abs(g - e)[diff] / ulp[diff]))
            say(f"{what} layer {l} {name}: {int(diff.sum())} of {diff.size} differ, worst {worst} ulp")
            assert worst <= 1.0 and diff.mean() <= 1e-6, f"{what} layer {l}: {name} differs"


def _run(wl, classes, ext: he.ExtConfig, caches, chunks, prompts=None, prompts_stacked=False,
         **kw):
    kv = streaming.make_cache(wl, device="cuda", caches=caches, debug=True, layer_class=classes,
                              summary_mode=int(ext.summary), reindex_mode=ext.reindex_mode,
                              rope_offset=ext.rope_offset, rope_limit=ext.rope_limit,
                              rope_headroom=ext.rope_headroom, rope_theta=ext.rope_theta,
                              scoring_mode=ext.scoring_mode, **kw)
    t = streaming.chunk_tensors(_stack(chunks), "cuda")
    kv.append(t["q"], t["k"], t["v"], t["pos"])
    if prompts is not None and prompts_stacked:   # one pass over every layer
        pt = {k2: streaming.bf16_tensor(np.stack([p[k2] for p in prompts]), "cuda")
              for k2 in ("q", "k", "v")}
        kv.guidance(pt["q"], pt["k"], pt["v"])
    elif prompts is not None:
        for l, p in enumerate(prompts):
            if p is None:
                continue
            pt = {k2: streaming.bf16_tensor(p[k2], "cuda") for k2 in ("q", "k", "v")}
            kv.guidance(pt["q"], pt["k"], pt["v"], layer=l)
    torch.cuda.synchronize()
    w = [kv.w[l].cpu().numpy().copy() for l in range(wl.n_layers)]
    kv.compress()
    torch.cuda.synchronize()
    return kv, w


def _stack(chunks):
    return {k: np.stack([c[k] for c in chunks]) for k in ("q", "k", "v")} | {"pos": chunks[0]["pos"]}


def _check_step(wl, classes, ext, kv, ref, what):
    """Kept sets against the oracle, then the compacted caches rebuilt by the
    oracle from the GPU's kept sets."""
    compact = []
    for l in range(wl.n_layers):
        cat = ref["appended"][l]
        T = len(cat.pos)
        if T > wl.budgets[l]:
            idx = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
            check_kept(idx, ref["smoothed"][l], wl.budgets[l], f"{what} layer {l}")
        else:
            idx = np.arange(T)
        c, _ = he.compact_layer(cat, idx, classes[l] == D, ext)
        compact.append(c)
    compact, reidx = he.reindex_layers(compact, ext)
    for l in range(wl.n_layers):
        _cmp_layer(l, kv, compact[l], what)
    return compact, reidx


# (32, 8, 128): 1024-element rows, two 16-byte pieces per lane in the
# summary and re-indexing kernels
@pytest.mark.parametrize("shape", [(14, 2, 64), (28, 4, 128), (32, 8, 128)])
@pytest.mark.parametrize("reindex", [he.REINDEX_NONE, he.REINDEX_EAGER])
def test_summary_tokens(shape, reindex):
    Hq, Hkv, d = shape
    classes = [S, M, D, D]
    wl = _wl("ext_sum", 40 + d, 4, Hq, Hkv, d, 1024, 196, (512, 600, 512, 700))
    caches = [wk.gen_cache(wl, l) for l in range(4)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(4)]
    ext = he.ExtConfig(summary=True, reindex_mode=reindex, rope_offset=11)
    say(f"summary tokens {shape} reindex {reindex}")
    kv, _ = _run(wl, classes, ext, caches, chunks)
    cfg = orc.OracleConfig(budgets=list(wl.budgets), classes=classes)
    ref = he.stream_step_ext(_ext_caches(caches), _ext_chunks(chunks), cfg, ext)
    compact, reidx = _check_step(wl, classes, ext, kv, ref, "summary")
    assert reidx == (reindex == he.REINDEX_EAGER)
    for l in (2, 3):
        assert kv.length(l) == wl.budgets[l] + 1
    kv.close()


def test_eager_reindex_in_place_for_layers_within_budget():
    """Layers that keep everything are re-indexed in their current buffer."""
    classes = [S, M, D, D]
    wl = _wl("ext_inplace", 50, 4, 14, 2, 64, 700, 196, (2000, 512, 2000, 512))
    caches = [wk.gen_cache(wl, l) for l in range(4)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(4)]
    ext = he.ExtConfig(summary=True, reindex_mode=he.REINDEX_EAGER, rope_offset=3)
    say("eager re-index, two layers within budget")
    kv, _ = _run(wl, classes, ext, caches, chunks)
    cfg = orc.OracleConfig(budgets=list(wl.budgets), classes=classes)
    ref = he.stream_step_ext(_ext_caches(caches), _ext_chunks(chunks), cfg, ext)
    _check_step(wl, classes, ext, kv, ref, "in-place")
    assert kv.length(0) == 896 and kv.length(2) == 896 and kv.length(3) == 513
    kv.close()


@pytest.mark.parametrize("limit,fires", [(1220 + 100, False), (1219 + 100, True)])
def test_lazy_reindex_trigger(limit, fires):
    """The largest retained position is 1219 (the chunk's last token is kept
    by every recency-scored layer); lazy re-indexing fires when
    1219 + headroom >= limit."""
    classes = [S, M, D, D]
    wl = _wl("ext_lazy", 51, 4, 14, 2, 64, 1024, 196, (512, 512, 512, 512))
    caches = [wk.gen_cache(wl, l) for l in range(4)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(4)]
    ext = he.ExtConfig(summary=True, reindex_mode=he.REINDEX_LAZY, rope_offset=0,
                       rope_limit=limit, rope_headroom=100)
    say(f"lazy re-index limit {limit}")
    kv, _ = _run(wl, classes, ext, caches, chunks)
    cfg = orc.OracleConfig(budgets=list(wl.budgets), classes=classes)
    ref = he.stream_step_ext(_ext_caches(caches), _ext_chunks(chunks), cfg, ext)
    _, reidx = _check_step(wl, classes, ext, kv, ref, "lazy")
    assert reidx == fires
    kv.close()


def test_stream_with_summaries_and_eager_reindex():
    """Four successive chunks; after each step the oracle continues from the
    GPU's compacted state read back from the device, so an element one ulp off
    at one step cannot drift further at the next."""
    classes = [S, M, M, D, D]
    L, C = 5, 196
    wl = _wl("ext_stream", 52, L, 14, 2, 64, 600, C, (700, 650, 600, 640, 560), n_steps=4)
    caches = [wk.gen_cache(wl, l) for l in range(L)]
    ext = he.ExtConfig(summary=True, reindex_mode=he.REINDEX_EAGER, rope_offset=5)
    kv = streaming.make_cache(wl, device="cuda", caches=caches, debug=True, layer_class=classes,
                              summary_mode=1, reindex_mode=he.REINDEX_EAGER, rope_offset=5)
    cfg = orc.OracleConfig(budgets=list(wl.budgets), classes=classes)
    state = _ext_caches(caches)
    for step in range(4):
        chunks = [wk.gen_chunk(wl, step, l) for l in range(L)]
        # after re-indexing the next chunk's keys would be rotated at positions
        # following the re-indexed cache; the stream positions serve as both
        # here, which only needs them to exceed every retained RoPE position
        say(f"stream step {step}")
        t = streaming.chunk_tensors(_stack(chunks), "cuda")
        kv.append(t["q"], t["k"], t["v"], t["pos"])
        kv.compress()
        torch.cuda.synchronize()
        ref = he.stream_step_ext(state, _ext_chunks(chunks), cfg, ext)
        _check_step(wl, classes, ext, kv, ref, f"step {step}")
        state = _gpu_state(kv, L)     # continue from the GPU's exact state
    kv.close()


def _gpu_state(kv, L):
    out = []
    for l in range(L):
        k, v, p = kv.view(l)
        shp = (k.shape[0], k.shape[1], k.shape[2])
        out.append(he.ExtLayerCache(wk.bf16_bits_to_f64(_bits(k).reshape(shp)),
                                    wk.bf16_bits_to_f64(_bits(v).reshape(shp)),
                                    p.cpu().numpy().astype(np.int64),
                                    kv.view_rope(l).cpu().numpy().astype(np.int64)))
    return out


def test_guidance_prompt_scoring():
    """W from guidance rows (global prompt for deep layers, hybrid prompt for
    middle layers), then scoring, smoothing and selection."""
    classes = [S, M, M, D, D]
    L = 5
    wl = _wl("ext_guide", 53, L, 14, 2, 64, 1024, 196, (512, 600, 550, 512, 640))
    caches = [wk.gen_cache(wl, l) for l in range(L)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(L)]
    n_rows = {M: 40, D: 24}
    prompts = [None if classes[l] == S else
               wk.gen_prompt(wl, l, n_rows[classes[l]],
                             wk.PROMPT_HYBRID if classes[l] == M else wk.PROMPT_GLOBAL)
               for l in range(L)]
    ext = he.ExtConfig(scoring_mode=he.SCORE_GUIDANCE)
    say("guidance-prompt scoring")
    kv, w = _run(wl, classes, ext, caches, chunks, prompts=prompts)
    cfg = orc.OracleConfig(budgets=list(wl.budgets), classes=classes)
    pr = [None if p is None else {"q": f64(p["q"]), "k": f64(p["k"]), "v": f64(p["v"])}
          for p in prompts]
    ref = he.stream_step_ext(_ext_caches(caches), _ext_chunks(chunks), cfg, ext, prompts=pr)
    for l in range(L):
        T = len(ref["appended"][l].pos)
        if classes[l] != S:
            rel = float(np.max(np.abs(w[l][:T] - ref["w"][l]) / ref["w"][l]))
            say(f"layer {l}: W rel {rel:.2e}")
            assert rel <= 1e-3
            sg = kv.s_dbg[l][:T].cpu().numpy().astype(np.float64)
            srel = float(np.max(np.abs(sg - ref["smoothed"][l]) / ref["smoothed"][l]))
            assert srel <= 1e-3, f"layer {l}: smoothed key rel {srel}"
        idx = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
        check_kept(idx, ref["smoothed"][l], wl.budgets[l], f"guidance layer {l}")
    kv.close()


def test_guidance_prompt_all_layers_one_pass():
    """A 64-row prompt for all 28 layers of the 7B head shape in one call:
    the caches are equal in length and the row pass fills one round of
    workgroups, so it runs one workgroup per (layer, KV head, query tile)
    (the row-LSE-only attention kernel, not stream mode); W, smoothed keys
    and kept sets against the oracle."""
    L = 28
    classes = [S] * 3 + [M] * 17 + [D] * 8
    wl = _wl("ext_guide_all", 55, L, 28, 4, 128, 256, 64, tuple(200 + 3 * l for l in range(L)))
    caches = [wk.gen_cache(wl, l) for l in range(L)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(L)]
    prompts = [wk.gen_prompt(wl, l, 64, wk.PROMPT_HYBRID if classes[l] == M else wk.PROMPT_GLOBAL)
               for l in range(L)]
    ext = he.ExtConfig(scoring_mode=he.SCORE_GUIDANCE)
    say("guidance-prompt scoring, all layers in one pass")
    kv, w = _run(wl, classes, ext, caches, chunks, prompts=prompts, prompts_stacked=True)
    cfg = orc.OracleConfig(budgets=list(wl.budgets), classes=classes)
    pr = [None if classes[l] == S else {"q": f64(p["q"]), "k": f64(p["k"]), "v": f64(p["v"])}
          for l, p in enumerate(prompts)]
    ref = he.stream_step_ext(_ext_caches(caches), _ext_chunks(chunks), cfg, ext, prompts=pr)
    worst = 0.0
    for l in range(L):
        T = len(ref["appended"][l].pos)
        if classes[l] != S:
            rel = float(np.max(np.abs(w[l][:T] - ref["w"][l]) / ref["w"][l]))
            worst = max(worst, rel)
            assert rel <= 1e-3, f"layer {l}: W rel {rel}"
            sg = kv.s_dbg[l][:T].cpu().numpy().astype(np.float64)
            srel = float(np.max(np.abs(sg - ref["smoothed"][l]) / ref["smoothed"][l]))
            assert srel <= 1e-3, f"layer {l}: smoothed key rel {srel}"
        idx = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
        check_kept(idx, ref["smoothed"][l], wl.budgets[l], f"guidance layer {l}")
    say(f"worst W rel {worst:.2e}")
    kv.close()


def test_guidance_state_errors():
    classes = [S, M, D]
    wl = _wl("ext_guide_err", 54, 3, 14, 2, 64, 300, 64, (200, 200, 200))
    caches = [wk.gen_cache(wl, l) for l in range(3)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(3)]
    t = streaming.chunk_tensors(_stack(chunks), "cuda")
    p = wk.gen_prompt(wl, 2, 16)
    pt = {k2: streaming.bf16_tensor(p[k2], "cuda") for k2 in ("q", "k", "v")}
    # chunk scoring: the guidance entry point is refused
    kv = streaming.make_cache(wl, device="cuda", caches=caches, layer_class=classes)
    kv.append(t["q"], t["k"], t["v"], t["pos"])
    with pytest.raises(H.HermesError) as e:
        kv.guidance(pt["q"], pt["k"], pt["v"], layer=2)
    assert e.value.code == H.ESTATE
    kv.close()
    # guidance scoring: compress needs the prompt mass of layers 1 and 2
    kv = streaming.make_cache(wl, device="cuda", caches=caches, layer_class=classes,
                              scoring_mode=H.SCORE_GUIDANCE)
    with pytest.raises(H.HermesError) as e:       # not appended yet
        kv.guidance(pt["q"], pt["k"], pt["v"], layer=2)
    assert e.value.code == H.ESTATE
    kv.append(t["q"], t["k"], t["v"], t["pos"])
    kv.guidance(pt["q"], pt["k"], pt["v"], layer=2)
    with pytest.raises(H.HermesError) as e:       # layer 1 missing
        kv.compress()
    assert e.value.code == H.ESTATE
    p1 = wk.gen_prompt(wl, 1, 16)
    kv.guidance(*(streaming.bf16_tensor(p1[k2], "cuda") for k2 in ("q", "k", "v")), layer=1)
    kv.compress()
    torch.cuda.synchronize()
    assert [kv.length(l) for l in range(3)] == [200, 200, 200]
    kv.close()


def test_fullsize_7b_summary_and_eager_reindex():
    """28 layers at the 7B shape (8192 cached + 784 new, budgets 2048..6144)
    with summaries and eager re-indexing: every layer's compacted cache,
    rebuilt by the oracle from the GPU's kept set, matches bit for bit."""
    wl = wk.WORKLOADS["c3_7b_28layer"]
    classes = orc.layer_partition(wl.n_layers)
    say("c3 full size: generating inputs")
    caches = [wk.gen_cache(wl, l) for l in range(wl.n_layers)]
    st = wk.stack_chunks(wl, 0)
    ext = he.ExtConfig(summary=True, reindex_mode=he.REINDEX_EAGER, rope_offset=14)
    kv = streaming.make_cache(wl, device="cuda", caches=caches, debug=True, summary_mode=1,
                              reindex_mode=he.REINDEX_EAGER, rope_offset=14)
    t = streaming.chunk_tensors(st, "cuda")
    kv.append(t["q"], t["k"], t["v"], t["pos"])
    kv.compress()
    torch.cuda.synchronize()
    say("c3 full size: comparing")
    compact = []
    for l in range(wl.n_layers):
        cat = he.ExtLayerCache(np.concatenate([f64(caches[l]["k"]), f64(st["k"][l])]),
                               np.concatenate([f64(caches[l]["v"]), f64(st["v"][l])]),
                               np.concatenate([caches[l]["pos"], st["pos"]]).astype(np.int64),
                               np.concatenate([caches[l]["pos"], st["pos"]]).astype(np.int64))
        idx = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
        assert len(idx) == wl.budgets[l] and np.all(np.diff(idx) > 0)
        c, _ = he.compact_layer(cat, idx, classes[l] == D, ext)
        compact.append(c)
    compact, _ = he.reindex_layers(compact, ext)
    for l in range(wl.n_layers):
        _cmp_layer(l, kv, compact[l], "c3")
    kv.close()


# ------------------------------------------------------------- 3D M-RoPE

def _grid(n, H, W, offset, t_step):
    """(t, h, w) [n][3] of tokens laid out frame by frame, row by row."""
    s = np.arange(n)
    f, r = s // (H * W), s % (H * W)
    return np.stack([offset + f * t_step, offset + r // W, offset + r % W], 1).astype(np.int64)


def _mrope_case(shape, mode, section_gpu, section_oracle, t_step=2, frames=5, summary=False):
    """`frames` cached frames of 14 x 14 tokens (text prefix 3) + 1 new frame;
    the last layer keeps everything and is re-indexed in place; with
    summary, the evicting deep layer folds its evicted tokens into one."""
    Hq, Hkv, d = shape
    classes = [S, M, D, D]
    T0, C = frames * 196, 196
    wl = _wl("ext_mrope", (60 if t_step == 2 else 160) + d, 4, Hq, Hkv, d, T0, C,
             (500, 600, 700, T0 + C + 24))
    caches = [wk.gen_cache(wl, l) for l in range(4)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(4)]
    g = _grid(T0 + C, 14, 14, offset=3, t_step=t_step)
    for c in caches:
        c["thw"] = g[:T0].T.copy()
    # the largest coordinate retained anywhere is h = w = 3 + 13 = 16 (with
    # t step 2, t reaches 13)
    limit = {"eager": 0, "lazy_fires": 18, "lazy_waits": 19, "none": 0}[mode]
    rmode = {"eager": he.REINDEX_EAGER, "none": he.REINDEX_NONE}.get(mode, he.REINDEX_LAZY)
    ext = he.ExtConfig(summary=summary, reindex_mode=rmode, rope_offset=5, rope_limit=limit,
                       rope_headroom=2, rope_axes=3, mrope_section=section_oracle)
    say(f"mrope {shape} {mode} section {section_gpu} t step {t_step}")
    ext_caches = [he.ExtLayerCache(f64(c["k"]), f64(c["v"]), c["pos"].astype(np.int64),
                                   g[:T0, 0].copy(), g[:T0].copy()) for c in caches]
    ext_chunks = [dict(ch, rope_thw=g[T0:].T.copy()) for ch in _ext_chunks(chunks)]
    ref = he.stream_step_ext(ext_caches, ext_chunks, orc.OracleConfig(budgets=list(wl.budgets),
                                                                      classes=classes), ext)
    assert ref["reindexed"] == (mode not in ("lazy_waits", "none"))
    if summary:
        assert ref["summaries"][2] is not None
    kv = streaming.make_cache(wl, device="cuda", caches=caches, debug=True, layer_class=classes,
                              summary_mode=int(summary), reindex_mode=ext.reindex_mode, rope_offset=5,
                              rope_limit=limit, rope_headroom=2, rope_axes=3,
                              mrope_section=section_gpu)
    t = streaming.chunk_tensors(_stack(chunks), "cuda")
    thw = torch.from_numpy(np.ascontiguousarray(g[T0:].T, dtype=np.int32)).cuda()
    kv.append(t["q"], t["k"], t["v"], t["pos"], rope_thw=thw)
    kv.compress()
    torch.cuda.synchronize()
    compact, reidx = _check_step(wl, classes, ext, kv, ref, f"mrope {mode}")
    assert reidx == ref["reindexed"]
    for l in range(4):
        got = kv.view_mrope(l).cpu().numpy().T
        assert np.array_equal(got, compact[l].rpos3), f"layer {l}: coordinates differ"
    kv.close()


@pytest.mark.parametrize("shape", [(14, 2, 64), (28, 4, 128), (32, 8, 128)])
@pytest.mark.parametrize("mode", ["eager", "lazy_fires", "lazy_waits"])
def test_mrope_reindex(shape, mode):
    d = shape[2]
    section = (8, 12, 12) if d == 64 else (16, 24, 24)
    _mrope_case(shape, mode, section, section)


@pytest.mark.parametrize("shape", [(14, 2, 64), (28, 4, 128)])
def test_mrope_reindex_default_section(shape):
    """mrope_section (0, 0, 0) selects the library's default split, which
    must be the oracle's default (16/24/24 at d = 128, 8/12/12 at d = 64);
    the benchmark's 3D re-indexing leg runs with it."""
    _mrope_case(shape, "eager", (0, 0, 0), ())


@pytest.mark.parametrize("shape", [(14, 2, 64), (28, 4, 128), (32, 8, 128)])
@pytest.mark.parametrize("mode", ["none", "eager", "lazy_fires"])
def test_mrope_summary_tokens(shape, mode):
    """Summary tokens with 3D coordinates (appendix summary algorithm with the
    3D re-indexing's sectioned RotaryDelta): the evicting deep layer's
    evicted keys are turned to the newest evicted token's (t, h, w) and
    averaged; the summary row (K, V, stream position and coordinates) and,
    with re-indexing, the ranks that now include it, against the oracle."""
    d = shape[2]
    section = (8, 12, 12) if d == 64 else (16, 24, 24)
    _mrope_case(shape, mode, section, section, summary=True)


@pytest.mark.parametrize("t_step", [70001, 300007])
def test_mrope_reindex_wide_t_axis(t_step):
    """Temporal coordinates far apart (6 frames, t step 70001 or 300007: the
    retained t values span more than one rank window of 2^18 values, with
    empty stretches between frames): every axis is still ranked over all its
    distinct retained coordinates (the appendix's sorted sets have no bound)."""
    _mrope_case((28, 4, 128), "eager", (16, 24, 24), (16, 24, 24), t_step=t_step)


def test_mrope_append_entry_points_follow_the_context():
    wl = _wl("ext_mrope_state", 70, 2, 4, 2, 64, 0, 8, (64, 64))
    caches = [wk.gen_cache(wl, l) for l in range(2)]
    chunks = [wk.gen_chunk(wl, 0, l) for l in range(2)]
    t = streaming.chunk_tensors(_stack(chunks), "cuda")
    thw = torch.zeros((3, 8), dtype=torch.int32, device="cuda")
    three = streaming.make_cache(wl, device="cuda", caches=caches, rope_axes=3)
    with pytest.raises(H.HermesError) as e:
        three.append(t["q"], t["k"], t["v"], t["pos"])
    assert e.value.code == H.ESTATE
    three.close()
    one = streaming.make_cache(wl, device="cuda", caches=caches)
    with pytest.raises(H.HermesError) as e:
        one.append(t["q"], t["k"], t["v"], t["pos"], rope_thw=thw)
    assert e.value.code == H.ESTATE
    one.close()
