"""Full-size GPU parity on the 28-layer 7B-shaped workloads, in the launch
configuration the benchmark times (all layers in one append + one compress).

The oracle cannot afford every layer at these sizes, so it checks sampled
layers completely (attention output, attention mass, smoothed keys, kept set,
compacted rows) and every layer through properties that hold at any size
(mass sums to C*Hq, kept sets are the budget-th largest of the smoothed keys,
lengths, ordered positions).  The long-stream test resynchronises the oracle
to the GPU's cache before each checked step (the kept rows are bit-identical
copies, so both sides then start from the same state)."""
import numpy as np
import pytest
import torch

from oracle import hermes_oracle as orc
from paper_2601_14724_amd import streaming, workloads as wk

from _parity import (S_RTOL, W_RTOL, check_kept, check_o, f64, oracle_layer_attention,
                     oracle_layer_score, say, stacked)

pytestmark = pytest.mark.gpu


def _gen_all(wl, step=0):
    import concurrent.futures as cf
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        caches = list(ex.map(lambda l: wk.gen_cache(wl, l), range(wl.n_layers)))
        chunks = list(ex.map(lambda l: wk.gen_chunk(wl, step, l), range(wl.n_layers)))
    return caches, chunks


def _oracle_mass_threaded(cache, chunk, wl, row_parts=4):
    """The oracle's attention mass W of one layer, computed per (KV-head
    group, block of chunk rows) on parallel threads and summed in a fixed
    order.  Query heads kv*G .. kv*G+G-1 with KV head kv is exactly the
    oracle's head mapping, and rows [r0, r1) of the chunk see the cache plus
    chunk rows before r0 as cached tokens and their own block causally, which
    is the oracle's mask; BLAS runs one thread per worker."""
    import concurrent.futures as cf

    from threadpoolctl import threadpool_limits
    G, C = wl.group, wl.chunk
    q, kc, vc = f64(chunk["q"]), f64(cache["k"]), f64(cache["v"])
    kn, vn = f64(chunk["k"]), f64(chunk["v"])
    T0 = kc.shape[0]
    cuts = [C * i // row_parts for i in range(row_parts + 1)]

    def one(job):
        kv, part = job
        r0, r1 = cuts[part], cuts[part + 1]
        sl = slice(kv * G, (kv + 1) * G)
        k_pre = np.concatenate([kc[:, kv:kv + 1], kn[:r0, kv:kv + 1]])
        v_pre = np.concatenate([vc[:, kv:kv + 1], vn[:r0, kv:kv + 1]])
        w = orc.chunk_attention(q[r0:r1, sl], k_pre, v_pre, kn[r0:r1, kv:kv + 1],
                                vn[r0:r1, kv:kv + 1])[1]
        return np.concatenate([w, np.zeros(T0 + C - len(w))])
    jobs = [(kv, p) for kv in range(wl.n_kv_heads) for p in range(row_parts)]
    with threadpool_limits(1), cf.ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        parts = list(ex.map(one, jobs))
    w = np.zeros(T0 + C)
    for p in parts:
        w += p
    return w


def test_c3_full_step_sampled_layers():
    """28 layers, 28q/4kv, d=128, 8192 cached + 784 new, budgets 2048..6144."""
    wl = wk.WORKLOADS["c3_7b_28layer"]
    say("[c3] generating inputs")
    caches, chunks = _gen_all(wl)
    kv = streaming.make_cache(wl, caches=caches, debug=True)
    t = streaming.chunk_tensors(stacked(chunks))
    say("[c3] append + compress on the GPU")
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    torch.cuda.synchronize()
    w_gpu = [kv.w[l].cpu().numpy().copy() for l in range(wl.n_layers)]
    out = out.float().cpu().numpy()
    kv.compress()
    torch.cuda.synchronize()
    classes = orc.layer_partition(wl.n_layers)
    lambdas = orc.smoothing_lambdas(classes)
    C, T0 = wl.chunk, wl.init_len
    T = T0 + C
    # every layer: lengths, ordered positions, mass of non-shallow layers
    for l in range(wl.n_layers):
        k_g, v_g, p_g = kv.view(l)
        assert k_g.shape[0] == wl.budgets[l]
        p = p_g.cpu().numpy()
        assert np.all(np.diff(p) > 0) and p[0] >= 0 and p[-1] < T
        if classes[l] != orc.SHALLOW:
            assert abs(w_gpu[l][:T].sum() - C * wl.n_q_heads) < 1e-4 * C * wl.n_q_heads
    sample = [2, 11, 19, 26, 27]
    needed = sorted(set(sample) | {l + 1 for l in sample if l + 1 < wl.n_layers})
    ref_o, ref_w = {}, {}
    for l in needed:
        say(f"[c3] oracle attention layer {l}")
        ref_o[l], ref_w[l] = oracle_layer_attention(caches[l], chunks[l])
    for l in sample:
        err = check_o(out[l], ref_o[l], f"[c3] layer {l}")["o_maxabs"]
        s_l = oracle_layer_score(l, classes, ref_w[l], T0, C)
        if classes[l] != orc.SHALLOW:
            rel = (np.abs(w_gpu[l][:T] - ref_w[l]) / ref_w[l]).max()
            assert rel <= W_RTOL, (l, rel)
        if l + 1 < wl.n_layers:
            s_n = oracle_layer_score(l + 1, classes, ref_w[l + 1], T0, C)
            pos = np.arange(T)
            st = orc.smooth(s_l, s_n, pos, pos, lambdas[l])
        else:
            st = s_l
        sg = kv.s_dbg[l][:T].cpu().numpy().astype(np.float64)
        srel = (np.abs(sg - st) / st).max()
        assert srel <= S_RTOL, (l, srel)
        idx = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
        nd = check_kept(idx, st, wl.budgets[l], f"c3 layer {l}")
        k_g, v_g, p_g = kv.view(l)
        kb = np.concatenate([caches[l]["k"], chunks[l]["k"]]).view(np.int16)
        assert np.array_equal(k_g.view(torch.int16).cpu().numpy(), kb[idx])
        assert np.array_equal(p_g.cpu().numpy(), np.arange(T)[idx])
        say(f"[c3] layer {l}: O err {err:.2e}, S~ rel {srel:.2e}, kept diff {nd}")
    kv.close()


def test_c4_stream_64_chunks_resync():
    """28 layers, 7B shape, 64 chunks of 784 from an empty cache, budget 6144:
    every step checks lengths and positions; steps 7 (first eviction), 8 and
    63 check two adjacent layers against the oracle resynchronised to the
    GPU's cache before the step."""
    wl = wk.WORKLOADS["c4_7b_stream64"]
    kv = streaming.make_cache(wl, debug=True, cap=6144 + 784)
    classes = orc.layer_partition(wl.n_layers)
    lambdas = orc.smoothing_lambdas(classes)
    check_steps = {7: [19, 20], 8: [2, 3], 63: [26, 27]}
    for s in range(wl.n_steps):
        chunks = None
        if s in check_steps:
            layers = check_steps[s]
            before = {}
            for l in layers:
                k_, v_, p_ = kv.view(l)
                before[l] = (k_.view(torch.int16).cpu().numpy().copy(),
                             v_.view(torch.int16).cpu().numpy().copy(), p_.cpu().numpy().copy())
        st_all = wk.stack_chunks(wl, s)
        t = streaming.chunk_tensors(st_all)
        out = kv.append(t["q"], t["k"], t["v"], t["pos"])
        if s in check_steps:
            torch.cuda.synchronize()
            w_gpu = {l: kv.w[l].cpu().numpy().copy() for l in layers}
            o_gpu = out.float().cpu().numpy()
        kv.compress()
        torch.cuda.synchronize()
        for l in range(wl.n_layers):
            assert kv.length(l) == min(784 * (s + 1), 6144)
        if s not in check_steps:
            continue
        say(f"[c4] step {s}: oracle on layers {layers}")
        l0, l1 = layers
        scores, cats = {}, {}
        for l in layers:
            k0, v0, p0 = before[l]
            ch = {"q": st_all["q"][l], "k": st_all["k"][l], "v": st_all["v"][l],
                  "pos": st_all["pos"]}
            cache = {"k": k0.view(np.uint16), "v": v0.view(np.uint16)}
            o, w = oracle_layer_attention(cache, ch)
            T0 = k0.shape[0]
            check_o(o_gpu[l], o, f"[c4] step {s} layer {l}")
            if classes[l] != orc.SHALLOW:
                assert (np.abs(w_gpu[l][:T0 + 784] - w) / w).max() <= W_RTOL
            scores[l] = oracle_layer_score(l, classes, w, T0, 784)
            cats[l] = (np.concatenate([p0, st_all["pos"]]), T0)
        st = orc.smooth(scores[l0], scores[l1], cats[l0][0], cats[l1][0], lambdas[l0])
        T = cats[l0][1] + 784
        if T > wl.budgets[l0]:
            sg = kv.s_dbg[l0][:T].cpu().numpy().astype(np.float64)
            assert (np.abs(sg - st) / st).max() <= S_RTOL
            idx = kv.kept_dbg[l0].cpu().numpy().astype(np.int64)
            nd = check_kept(idx, st, wl.budgets[l0], f"c4 step {s} layer {l0}")
            assert np.array_equal(kv.view(l0)[2].cpu().numpy(), cats[l0][0][idx])
            say(f"[c4] step {s} layer {l0}: kept diff {nd}")
    kv.close()


def test_c5_long_cache_and_query():
    """28 layers, 7B shape, 32768 cached + 3136 new, budgets 4096..16384, then
    a 64-token query.  Checked exactly: attention rows sampled across the
    chunk, the attention mass of the newest 8 candidates (seen only by the
    last 8 rows), the smoothed keys and kept sets of every layer recomputed
    from the GPU's own attention mass with the oracle's scoring, and the
    query attention over the compacted cache."""
    wl = wk.WORKLOADS["c5_7b_long"]
    say("[c5] generating inputs")
    caches, chunks = _gen_all(wl)
    kv = streaming.make_cache(wl, caches=caches, debug=True)
    t = streaming.chunk_tensors(stacked(chunks))
    say("[c5] append + compress on the GPU")
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    torch.cuda.synchronize()
    w_gpu = [kv.w[l].cpu().numpy().astype(np.float64) for l in range(wl.n_layers)]
    kv.compress()
    torch.cuda.synchronize()
    classes = orc.layer_partition(wl.n_layers)
    lambdas = orc.smoothing_lambdas(classes)
    C, T0 = wl.chunk, wl.init_len
    T = T0 + C
    G = wl.group
    rows = np.array([0, 1, 977, 2048, C - 9, C - 1])
    for l in (0, 13, 27):
        say(f"[c5] sampled rows of layer {l}")
        ch, ca = chunks[l], caches[l]
        k_all = np.concatenate([f64(ca["k"]), f64(ch["k"])])
        v_all = np.concatenate([f64(ca["v"]), f64(ch["v"])])
        q = f64(ch["q"])
        o_g = out[l].float().cpu().numpy()
        w_tail = np.zeros(8)
        o_want = {}
        for r in sorted(set(rows.tolist()) | set(range(C - 8, C))):
            o_r, w_r = orc.chunk_attention(q[r:r + 1], k_all[:T0 + r], v_all[:T0 + r],
                                           k_all[T0 + r:T0 + r + 1], v_all[T0 + r:T0 + r + 1])
            if r in rows:
                o_want[r] = o_r[0]
            if r >= C - 8:
                w_tail[:r - (C - 8) + 1] += w_r[T - 8:T0 + r + 1]
        check_o(o_g[rows], np.stack([o_want[r] for r in rows]), f"[c5] layer {l} sampled rows")
        if classes[l] != orc.SHALLOW:
            assert (np.abs(w_gpu[l][T - 8:T] - w_tail) / w_tail).max() <= W_RTOL, l
    # the whole attention mass of one middle and one deep layer (all 35,904
    # candidates; the oracle in head groups on the host's threads)
    for l in (14, 26):
        say(f"[c5] oracle attention mass of layer {l} over all {T} candidates")
        w_ref = _oracle_mass_threaded(caches[l], chunks[l], wl)
        rel = float((np.abs(w_gpu[l][:T] - w_ref) / w_ref).max())
        say(f"[c5] layer {l}: W rel error {rel:.3e} over {T} candidates")
        assert rel <= W_RTOL, (l, rel)
    # scoring, smoothing and selection of every layer from the GPU's mass
    s_raw = [oracle_layer_score(l, classes, w_gpu[l][:T], T0, C) for l in range(wl.n_layers)]
    pos = np.arange(T)
    for l in range(wl.n_layers):
        if classes[l] != orc.SHALLOW:
            assert abs(w_gpu[l][:T].sum() - C * wl.n_q_heads) < 1e-4 * C * wl.n_q_heads
        st = orc.smooth(s_raw[l], s_raw[l + 1] if l + 1 < wl.n_layers else None, pos,
                        pos if l + 1 < wl.n_layers else None, lambdas[l])
        sg = kv.s_dbg[l][:T].cpu().numpy().astype(np.float64)
        assert (np.abs(sg - st) / st).max() <= 1e-6, l
        idx = kv.kept_dbg[l].cpu().numpy().astype(np.int64)
        check_kept(idx, st, wl.budgets[l], f"c5 layer {l}")
        assert np.array_equal(kv.view(l)[2].cpu().numpy(), pos[idx])
    # the 64-token query over the compacted caches
    qry = [wk.gen_query(wl, l) for l in range(wl.n_layers)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    oq = kv.query(qt["q"], qt["k"], qt["v"]).float().cpu().numpy()
    for l in (0, 27):
        k_g, v_g, p_g = kv.view(l)
        cache = orc.LayerCache(k_g.float().double().cpu().numpy(), v_g.float().double().cpu().numpy(),
                               p_g.cpu().numpy())
        want = orc.query_attention(cache, f64(qry[l]["q"]), f64(qry[l]["k"]), f64(qry[l]["v"]))
        check_o(oq[l], want, f"[c5] query layer {l}")
    kv.close()


def _sharp(wl, period):
    return wk.scaled(wl, anchor_period=period, workload_id=wl.workload_id + 100)


def test_c3_sharp_attention_step_and_query():
    """The 28-layer 7B workload with planted anchor tokens (every 64th
    position; anchors dominate each row, so |O| is of order 0.5): one append +
    compress and the 64-token query, in the benchmark's launch configuration.
    The oracle checks the chunk attention and the attention mass of a middle
    and a deep layer, and the query output of the shortest and longest
    compacted layers (the query runs in stream mode, its partial states merged
    by the combine)."""
    wl = _sharp(wk.WORKLOADS["c3_7b_28layer"], 64)
    say("[c3 sharp] generating inputs")
    caches, chunks = _gen_all(wl)
    kv = streaming.make_cache(wl, caches=caches, debug=True, max_chunk=wl.chunk)
    t = streaming.chunk_tensors(stacked(chunks))
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    torch.cuda.synchronize()
    w_gpu = [kv.w[l].cpu().numpy().copy() for l in range(wl.n_layers)]
    out = out.float().cpu().numpy()
    kv.compress()
    torch.cuda.synchronize()
    T = wl.init_len + wl.chunk
    for l in (11, 26):
        say(f"[c3 sharp] oracle attention layer {l}")
        o_ref, w_ref = oracle_layer_attention(caches[l], chunks[l])
        check_o(out[l], o_ref, f"[c3 sharp] layer {l}")
        rel = float((np.abs(w_gpu[l][:T] - w_ref) / w_ref).max())
        say(f"[c3 sharp] layer {l}: W rel {rel:.3e}")
        assert rel <= W_RTOL, (l, rel)
    qw = wk.scaled(wl, query_len=64)
    qry = [wk.gen_query(qw, l) for l in range(wl.n_layers)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    oq = kv.query(qt["q"], qt["k"], qt["v"]).float().cpu().numpy()
    for l in (0, 27):
        k_g, v_g, p_g = kv.view(l)
        cache = orc.LayerCache(k_g.float().double().cpu().numpy(), v_g.float().double().cpu().numpy(),
                               p_g.cpu().numpy())
        want = orc.query_attention(cache, f64(qry[l]["q"]), f64(qry[l]["k"]), f64(qry[l]["v"]))
        check_o(oq[l], want, f"[c3 sharp] query layer {l} ({kv.length(l)} cached)")
    kv.close()


def test_c5_sharp_query_over_long_caches():
    """The long-cache workload (32768 + 3136 tokens, budgets 4096..16384) with
    planted anchors every 128th position: append + compress, then the 64-token
    query in stream mode (its longest layers spread over the most units); sampled
    chunk rows and the query output of the shortest and longest layer against
    the oracle."""
    wl = _sharp(wk.WORKLOADS["c5_7b_long"], 128)
    say("[c5 sharp] generating inputs")
    caches, chunks = _gen_all(wl)
    kv = streaming.make_cache(wl, caches=caches)
    t = streaming.chunk_tensors(stacked(chunks))
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    kv.compress()
    torch.cuda.synchronize()
    C, T0 = wl.chunk, wl.init_len
    rows = np.array([0, 977, C - 1])
    for l in (13, 27):
        ch, ca = chunks[l], caches[l]
        k_all = np.concatenate([f64(ca["k"]), f64(ch["k"])])
        v_all = np.concatenate([f64(ca["v"]), f64(ch["v"])])
        q = f64(ch["q"])
        want = np.stack([orc.chunk_attention(q[r:r + 1], k_all[:T0 + r], v_all[:T0 + r],
                                             k_all[T0 + r:T0 + r + 1], v_all[T0 + r:T0 + r + 1])[0][0]
                         for r in rows])
        check_o(out[l].float().cpu().numpy()[rows], want, f"[c5 sharp] layer {l} sampled rows")
    qry = [wk.gen_query(wl, l) for l in range(wl.n_layers)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    oq = kv.query(qt["q"], qt["k"], qt["v"]).float().cpu().numpy()
    for l in (0, 27):
        k_g, v_g, p_g = kv.view(l)
        cache = orc.LayerCache(k_g.float().double().cpu().numpy(), v_g.float().double().cpu().numpy(),
                               p_g.cpu().numpy())
        want = orc.query_attention(cache, f64(qry[l]["q"]), f64(qry[l]["k"]), f64(qry[l]["v"]))
        check_o(oq[l], want, f"[c5 sharp] query layer {l} ({kv.length(l)} cached)")
    kv.close()
