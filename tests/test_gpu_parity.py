"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Sizes span several tiles of every kernel plus ragged tails (packed query rows
not a multiple of 128, candidates not a multiple of 64/128, chunk lengths of
1 and of several hundred) and the edge cases: empty cache, single-token
chunk, a budget at least the candidate count (nothing evicted), every layer
class, G = 1 (no grouping) and G = 7.
"""
import numpy as np
import pytest
import torch

from oracle import hermes_oracle as orc
from paper_2601_14724_amd import workloads as wk

from _parity import (check_layer, check_o, gen, oracle_caches, oracle_chunks, oracle_config,
                     raw_bits, run_gpu_step, say)

pytestmark = pytest.mark.gpu


def _step_parity(wl, classes=None, lambdas=None, check_w=True, **kw):
    say(f"[parity] {wl.name}: L={wl.n_layers} Hq={wl.n_q_heads} Hkv={wl.n_kv_heads} "
        f"d={wl.head_dim} T0={wl.init_len} C={wl.chunk} budgets={wl.budgets[:4]}...")
    caches, chunks = gen(wl)
    kv, out, w = run_gpu_step(wl, caches, chunks, layer_class=classes, lambdas=lambdas,
                              force_scores=True, **kw)
    ref = orc.stream_step(oracle_caches(caches), oracle_chunks(chunks),
                          oracle_config(wl, classes=classes, lambdas=lambdas,
                                        alpha_mode=kw.get("alpha_mode", 0),
                                        align_mode=kw.get("align_mode", 0)))
    bits = raw_bits(caches, chunks)
    worst = {}
    for l in range(wl.n_layers):
        st = check_layer(l, kv, out, w, ref, wl.budgets[l], wl.chunk, check_w=check_w,
                         report=bits)
        for k, v in st.items():
            worst[k] = max(worst.get(k, 0), v)
    say(f"[parity] {wl.name} worst: {worst}")
    kv.close()
    return worst


ATTN_SHAPES = [
    # name, Hq, Hkv, d, T0, C, budget
    ("g7_d64", 14, 2, 64, 100, 50, 400),
    ("g7_d128", 28, 4, 128, 300, 77, 1000),
    ("g1_empty_cache", 4, 4, 64, 0, 33, 100),
    ("g7_one_cached", 7, 1, 128, 1, 129, 400),
    ("one_token_chunk", 8, 2, 64, 257, 1, 1000),
    ("g2_ragged", 6, 3, 128, 191, 65, 1000),
]


@pytest.mark.parametrize("name,Hq,Hkv,d,T0,C,budget", ATTN_SHAPES)
def test_attention_and_mass_parity_no_eviction(name, Hq, Hkv, d, T0, C, budget):
    wl = wk.custom(f"attn_{name}", 100 + len(name), 2, Hq, Hkv, d, T0, C, (budget, budget))
    _step_parity(wl, classes=[orc.DEEP, orc.DEEP])


@pytest.mark.parametrize("cls", [orc.SHALLOW, orc.MIDDLE, orc.DEEP])
def test_c1_single_layer_each_class(cls):
    """1 layer, 0.5B shape, 1024 cached + 196 new, budget 512."""
    wl = wk.WORKLOADS["c1_0p5b_1layer"]
    worst = _step_parity(wl, classes=[cls], lambdas=[0.0])
    assert worst["kept_diff"] <= 2


def test_small_multilayer_eviction_all_classes():
    wl = wk.custom("multi", 120, 10, 14, 2, 64, 300, 97, [150, 170, 200, 230, 260, 290, 320,
                                                         350, 380, 396])
    _step_parity(wl)


@pytest.mark.parametrize("alpha_mode,align_mode", [(1, 0), (0, 1)])
def test_alternate_readings(alpha_mode, align_mode):
    wl = wk.custom("readings", 121, 6, 8, 2, 128, 200, 64, [100, 120, 140, 160, 180, 200])
    _step_parity(wl, alpha_mode=alpha_mode, align_mode=align_mode)


def test_c2_full():
    """24 layers, 0.5B shape, 4096 cached + 784 new, budget 2048 per layer."""
    _step_parity(wk.WORKLOADS["c2_0p5b_24layer"])


def test_topk_kernel_matches_oracle_with_ties():
    from paper_2601_14724_amd import hermes as H
    rng = np.random.default_rng(5)
    # register-resident (n <= 10240), LDS-staged (n <= 38400) and global paths
    for n, k in [(1, 1), (7, 3), (1000, 999), (5000, 1234), (10240, 3), (10241, 10000),
                 (36000, 16000), (40000, 20000), (100, 200), (4096, 4096)]:
        keys = rng.random(n).astype(np.float32)
        keys[rng.integers(0, n, n // 5)] = keys[0]           # a block of exact ties
        say(f"[topk] n={n} k={k}")
        got = H.select_topk(torch.from_numpy(keys).cuda(), k).cpu().numpy()
        want = orc.topk_indices(keys.astype(np.float64), k)
        assert np.array_equal(got, want), (n, k)


@pytest.mark.parametrize("anchors", [0, 37])
def test_query_after_compress_matches_oracle(anchors):
    """Compress, then a 64-token query over the compacted caches; with
    anchors the outputs are of order 0.5, so the bars measure the PV path
    and the slice merge, not only the rounding of near-zero outputs."""
    wl = wk.custom("query", 122, 3, 28, 4, 128, 400, 100, (256, 300, 600), query_len=64,
                   anchor_period=anchors)
    say(f"[query] compress then 64-token query (anchor period {anchors})")
    caches, chunks = gen(wl)
    kv, out, w = run_gpu_step(wl, caches, chunks)
    ref = orc.stream_step(oracle_caches(caches), oracle_chunks(chunks), oracle_config(wl))
    from paper_2601_14724_amd import streaming
    for l in range(wl.n_layers):
        check_o(out[l], ref["out"][l], f"[query] chunk layer {l}")
    qry = [wk.gen_query(wl, l) for l in range(wl.n_layers)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    o = kv.query(qt["q"], qt["k"], qt["v"]).float().cpu().numpy()
    f64 = wk.bf16_bits_to_f64
    for l in range(wl.n_layers):
        # continue the oracle from the GPU's kept set (identical bf16 rows)
        k_g, v_g, p_g = kv.view(l)
        cache = orc.LayerCache(k_g.float().double().cpu().numpy(), v_g.float().double().cpu().numpy(),
                               p_g.cpu().numpy())
        want = orc.query_attention(cache, f64(qry[l]["q"]), f64(qry[l]["k"]), f64(qry[l]["v"]))
        check_o(o[l], want, f"[query] layer {l}")
    kv.close()


def test_max_layer_count_step_and_query():
    """HERMES_MAX_LAYERS (64) layers in one context: every per-layer table and
    launch-argument array at its limit.  Budgets ramp across the layers so
    that some evict and the last ones keep everything; the append + compress
    step of every layer against the oracle, then an 8-token query over the
    64 compacted caches of different lengths."""
    from paper_2601_14724_amd import hermes as H
    from paper_2601_14724_amd import streaming
    L = H.MAX_LAYERS
    budgets = [60 + (200 * l) // (L - 1) for l in range(L)]   # 60 .. 260 against T = 224
    wl = wk.custom("maxlayers", 125, L, 4, 2, 64, 200, 24, budgets, query_len=8, anchor_period=29)
    say(f"[maxlayers] {L} layers, budgets {budgets[0]}..{budgets[-1]}, T = 224")
    caches, chunks = gen(wl)
    kv, out, w = run_gpu_step(wl, caches, chunks, force_scores=True)
    ref = orc.stream_step(oracle_caches(caches), oracle_chunks(chunks), oracle_config(wl))
    bits = raw_bits(caches, chunks)
    for l in range(L):
        check_layer(l, kv, out, w, ref, wl.budgets[l], wl.chunk, report=bits)
    assert [kv.length(l) for l in range(L)] == [min(224, b) for b in budgets]
    qry = [wk.gen_query(wl, l) for l in range(L)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    o = kv.query(qt["q"], qt["k"], qt["v"]).float().cpu().numpy()
    f64 = wk.bf16_bits_to_f64
    for l in range(L):
        k_g, v_g, p_g = kv.view(l)
        cache = orc.LayerCache(k_g.float().double().cpu().numpy(), v_g.float().double().cpu().numpy(),
                               p_g.cpu().numpy())
        want = orc.query_attention(cache, f64(qry[l]["q"]), f64(qry[l]["k"]), f64(qry[l]["v"]))
        check_o(o[l], want, f"[maxlayers] query layer {l} ({kv.length(l)} cached)")
    kv.close()


def test_determinism_bitwise():
    wl = wk.WORKLOADS["c1_0p5b_1layer"]
    caches, chunks = gen(wl)
    res = []
    for _ in range(2):
        kv, out, w = run_gpu_step(wl, caches, chunks, force_scores=True)
        res.append((out, w[0], kv.s_dbg[0].cpu().numpy(), kv.kept_dbg[0].cpu().numpy(),
                    kv.view(0)[0].view(torch.int16).cpu().numpy()))
        kv.close()
    for a, b in zip(*res):
        assert np.array_equal(a, b)


def test_degenerate_budgets_keep_one_evict_one_keep_all():
    """Budgets 1 (keep one candidate), T - 1 (evict exactly one) and T (keep
    everything) on the same step."""
    wl = wk.custom("degenerate", 122, 3, 4, 2, 64, 200, 40, [1, 239, 240])
    _step_parity(wl, classes=[orc.MIDDLE, orc.DEEP, orc.DEEP])


def test_first_chunk_larger_than_the_budget():
    """An empty cache and a 150-token first chunk against budgets 40, 75 and
    149: every layer evicts among the chunk's own tokens, whose candidates
    are each seen by a different number of chunk rows (Eq.2 with T0 = 0)."""
    wl = wk.custom("first_chunk_evicts", 126, 3, 8, 2, 64, 0, 150, [40, 75, 149])
    _step_parity(wl)


def test_long_layers_past_the_lds_staging_limits():
    """40000 cached + 32 new candidates: the selection keys no longer fit in
    LDS (read from global memory), the partner positions of the layer above
    are searched in global memory, and the normaliser has more partials than
    one wave loads at once."""
    wl = wk.custom("long", 123, 2, 2, 1, 64, 40000, 32, [20000, 30000])
    _step_parity(wl, classes=[orc.MIDDLE, orc.DEEP])


@pytest.mark.parametrize("anchors,n_q", [(0, 9), (61, 9), (61, 1)])
def test_query_stream_mode_over_unequal_caches(anchors, n_q):
    """Layers of very different cache lengths (300, 2000 and 8000 tokens): the
    host runs the query in stream mode, the 326 key tiles of the six (layer,
    KV head) pairs cut into 256 unit ranges, so the longest layer's keys are
    spread over about 100 units whose partial states the combine merges; each
    layer's query output against the oracle's attention over that layer's
    cache.  With anchors every range holds tokens that dominate some rows, so
    a block merged with a wrong weight, or dropped, moves the output by far
    more than the bars."""
    from paper_2601_14724_amd import streaming
    wl = wk.custom("slices", 123, 3, 4, 2, 64, 8000, 9, (8000, 8000, 8000), query_len=n_q,
                   anchor_period=anchors)
    lens = (300, 2000, 8000)
    caches = []
    for l in range(wl.n_layers):
        c = wk.gen_cache(wl, l)
        caches.append({k: np.ascontiguousarray(c[k][:lens[l]]) for k in ("k", "v", "pos")})
    kv = streaming.make_cache(wl, caches=caches)
    assert [kv.length(l) for l in range(wl.n_layers)] == list(lens)
    qry = [wk.gen_query(wl, l) for l in range(wl.n_layers)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    o = kv.query(qt["q"], qt["k"], qt["v"]).float().cpu().numpy()
    f64 = wk.bf16_bits_to_f64
    for l in range(wl.n_layers):
        cache = orc.LayerCache(f64(caches[l]["k"]), f64(caches[l]["v"]),
                               caches[l]["pos"].astype(np.int64))
        want = orc.query_attention(cache, f64(qry[l]["q"]), f64(qry[l]["k"]), f64(qry[l]["v"]))
        check_o(o[l], want, f"[stream] layer {l} ({lens[l]} cached, anchors {anchors}, {n_q} tokens)")
    kv.close()


def test_exact_ties_through_compress_keep_the_newest():
    """Every selection key equal (Sec. 3.2 TopK with the tie reading: the
    newer token wins): a one-token chunk of all-zero queries gives every
    candidate the same score 0, so the softmax is uniform and every W_i is the
    same float; the single deep layer (no smoothing partner) then has
    identical keys, and the kept set must be the budget newest candidates.
    T = 8001 <= 10240 candidates, so the selection runs the register-resident
    radix path of the compression."""
    from paper_2601_14724_amd import streaming
    wl = wk.custom("ties", 124, 1, 4, 2, 64, 8000, 1, (3000,))
    caches, chunks = gen(wl)
    chunks[0]["q"][:] = 0
    kv, out, w = run_gpu_step(wl, caches, chunks, layer_class=[orc.DEEP], force_scores=True)
    T = wl.init_len + wl.chunk
    wt = w[0][:T]
    assert np.all(wt == wt[0]), "uniform attention must give bit-identical masses"
    assert abs(float(wt.sum()) - wl.n_q_heads) < 1e-4 * wl.n_q_heads
    keys = kv.s_dbg[0][:T].cpu().numpy()
    assert np.all(keys == keys[0])
    idx = kv.kept_dbg[0].cpu().numpy().astype(np.int64)
    assert np.array_equal(idx, np.arange(T - 3000, T)), "ties must keep the newest candidates"
    assert np.array_equal(kv.view(0)[2].cpu().numpy(), np.arange(T - 3000, T))
    # the oracle agrees: uniform W, identical keys, the newest budget kept
    ref = orc.stream_step(oracle_caches(caches), oracle_chunks(chunks),
                          oracle_config(wl, classes=[orc.DEEP], lambdas=[0.0]))
    assert np.array_equal(ref["kept"][0], idx)
    kv.close()
