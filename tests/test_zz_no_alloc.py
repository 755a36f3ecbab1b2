"""The no-allocation context entry point, hermes_kv_init_static (the
workspace is the library's own device scratch), against hermes_kv_init with
a caller workspace: on the same seeded inputs every output of an append +
compress + query must be bit-identical (same kernels, same launch plan).
Two calls in a row, the second with a smaller input, so the second context
runs on the scratch exactly as the first left it."""
import numpy as np
import pytest
import torch

from paper_2601_14724_amd import hermes as H, streaming, workloads as wk

from _parity import gen, say, stacked

pytestmark = pytest.mark.gpu


def _run(wl, caches, chunks, static):
    kv = streaming.make_cache(wl, caches=caches, debug=True, force_scores=True,
                              static_workspace=static)
    t = streaming.chunk_tensors(stacked(chunks))
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    torch.cuda.synchronize()
    res = {"out": out.view(torch.int16).cpu().numpy(),
           "w": [kv.w[l].cpu().numpy().copy() for l in range(wl.n_layers)]}
    kv.compress()
    qry = [wk.gen_query(wl, l) for l in range(wl.n_layers)]
    qt = {k: streaming.bf16_tensor(np.stack([x[k] for x in qry]), "cuda") for k in ("q", "k", "v")}
    res["query"] = kv.query(qt["q"], qt["k"], qt["v"]).view(torch.int16).cpu().numpy()
    torch.cuda.synchronize()
    res["s"] = [kv.s_dbg[l].cpu().numpy() for l in range(wl.n_layers)]
    res["kept"] = [kv.kept_dbg[l].cpu().numpy() for l in range(wl.n_layers)]
    res["cache"] = []
    for l in range(wl.n_layers):
        k, v, p = kv.view(l)
        res["cache"].append((k.view(torch.int16).cpu().numpy(), v.view(torch.int16).cpu().numpy(),
                             p.cpu().numpy()))
    return kv, res


def _same(a, b, what):
    if isinstance(a, (list, tuple)):
        assert len(a) == len(b), what
        for i, (x, y) in enumerate(zip(a, b)):
            _same(x, y, f"{what}[{i}]")
    else:
        assert np.array_equal(a, b), f"{what} differs"


def test_static_workspace_matches_caller_workspace():
    cases = [wk.custom("noalloc_a", 130, 3, 14, 2, 64, 1024, 196, (512, 700, 1300), query_len=64),
             wk.custom("noalloc_b", 131, 2, 4, 2, 64, 300, 37, (100, 400), query_len=9)]
    for n, wl in enumerate(cases):
        say(f"[no-alloc] call {n}: {wl.name} L={wl.n_layers} T0={wl.init_len} C={wl.chunk}")
        caches, chunks = gen(wl)
        kv_s, got = _run(wl, caches, chunks, static=True)
        if n == 0:
            # the device's scratch has one owner at a time
            with pytest.raises(H.HermesError) as e:
                streaming.make_cache(wl, caches=caches, static_workspace=True)
            assert e.value.code == H.ESTATE
        kv_r, want = _run(wl, caches, chunks, static=False)
        for key in want:
            _same(got[key], want[key], f"call {n} {key}")
        kv_s.close()
        kv_r.close()
    # released by close: a new static context can be made again
    wl = cases[1]
    caches, _ = gen(wl)
    streaming.make_cache(wl, caches=caches, static_workspace=True).close()
