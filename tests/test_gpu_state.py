"""State machine of the C ABI on a real device: every rejected call returns
its code before any launch and leaves lengths untouched."""
import numpy as np
import pytest
import torch

from paper_2601_14724_amd import hermes as H
from paper_2601_14724_amd import streaming, workloads as wk

pytestmark = pytest.mark.gpu


def _setup():
    wl = wk.custom("state", 130, 3, 4, 2, 64, 20, 8, (16, 24, 40))
    kv = streaming.make_cache(wl, max_chunk=8, cap=40)
    t = streaming.chunk_tensors(wk.stack_chunks(wl, 0))
    return wl, kv, t


def test_append_compress_state_machine():
    wl, kv, t = _setup()
    one = {k: t[k][0].contiguous() for k in ("q", "k", "v")}
    kv.append(one["q"], one["k"], one["v"], t["pos"], layer=0)
    with pytest.raises(H.HermesError) as e:
        kv.append(one["q"], one["k"], one["v"], t["pos"], layer=0)       # twice in one step
    assert e.value.code == H.ESTATE
    with pytest.raises(H.HermesError) as e:
        kv.compress()                                                      # not all layers yet
    assert e.value.code == H.ESTATE
    with pytest.raises(H.HermesError) as e:
        kv.query(one["q"], one["k"], one["v"], layer=1)                    # mid-step query
    assert e.value.code == H.ESTATE
    short = {k: one[k][:4].contiguous() for k in one}
    with pytest.raises(H.HermesError) as e:                                # different n_new
        kv.append(short["q"], short["k"], short["v"], t["pos"][:4].contiguous(), layer=1)
    assert e.value.code == H.ESTATE
    assert kv.length(1) == 20
    for l in (1, 2):
        kv.append(one["q"], one["k"], one["v"], t["pos"], layer=l)
    kv.compress()
    torch.cuda.synchronize()
    assert [kv.length(l) for l in range(3)] == [16, 24, 28]
    kv.compress()                                                          # no-op
    kv.rewind()
    assert [kv.length(l) for l in range(3)] == [20, 20, 20]
    kv.close()


def test_capacity_and_argument_errors():
    wl, kv, t = _setup()
    ctx = kv.ctx
    one = {k: t[k][0].contiguous() for k in ("q", "k", "v")}
    assert H.lib.hermes_append_chunk(ctx, 5, one["q"].data_ptr(), one["k"].data_ptr(),
                                     one["v"].data_ptr(), t["pos"].data_ptr(), 8,
                                     one["q"].data_ptr(), None) == H.EINVAL  # layer out of range
    assert H.lib.hermes_append_chunk(ctx, 0, one["q"].data_ptr() + 2, one["k"].data_ptr(),
                                     one["v"].data_ptr(), t["pos"].data_ptr(), 8,
                                     one["q"].data_ptr(), None) == H.EINVAL  # misaligned input
    assert H.lib.hermes_append_chunk(ctx, H.ALL_LAYERS, t["q"].data_ptr(), t["k"].data_ptr(),
                                     t["v"].data_ptr(), t["pos"].data_ptr(), 9,
                                     t["q"].data_ptr(), None) == H.EINVAL   # > max_chunk
    assert H.lib.hermes_append_chunk(ctx, H.ALL_LAYERS, t["q"].data_ptr(), t["k"].data_ptr(),
                                     t["v"].data_ptr(), t["pos"].data_ptr(), 0,
                                     t["q"].data_ptr(), None) == H.EINVAL   # empty chunk
    # fill layer 2 (budget 40 = cap) up to capacity: 20 + 8 + 8 = 36, next append overflows
    for _ in range(2):
        kv.append(t["q"], t["k"], t["v"], t["pos"])
        kv.compress()
    torch.cuda.synchronize()
    assert kv.length(2) == 36
    with pytest.raises(H.HermesError) as e:
        kv.append(t["q"], t["k"], t["v"], t["pos"])
    assert e.value.code == H.ECAPACITY
    assert [kv.length(l) for l in range(3)] == [16, 24, 36]
    with pytest.raises(H.HermesError) as e:
        kv.rewind()                            # layers 0/1 compacted twice: buffer 0 overwritten
    assert e.value.code == H.ESTATE
    kv.close()


def test_profiling_counts_launches():
    wl, kv, t = _setup()
    kv.profile(True)
    kv.append(t["q"], t["k"], t["v"], t["pos"])
    kv.compress()
    ms, n = kv.profile_read(H.K_ATTN)
    assert n == 1 and ms > 0
    ms, n = kv.profile_read(H.K_GATHER)
    assert n == 1
    ms, n = kv.profile_read(H.K_ATTN)
    assert n == 0 and ms == 0
    kv.close()


def test_precondition_checks_reject_before_any_launch(monkeypatch):
    """With device-side checks on, a chunk whose positions are not strictly
    increasing or not after the cache, or whose inputs are not finite, is
    rejected with EINVAL and changes nothing; valid inputs give bitwise the
    same results as an unchecked context."""
    wl, kv, t = _setup()
    _, ref, _ = _setup()
    kv.check_preconditions(True)
    bad_order = t["pos"].clone()
    bad_order[3] = bad_order[2]
    early = t["pos"] - 1                       # first position equals the last cached one
    q_nan = t["q"].clone()
    q_nan.view(-1)[5] = float("nan")
    v_inf = t["v"].clone()
    v_inf.view(-1)[-1] = float("inf")
    for q, k, v, pos in ((t["q"], t["k"], t["v"], bad_order), (t["q"], t["k"], t["v"], early),
                         (q_nan, t["k"], t["v"], t["pos"]), (t["q"], t["k"], v_inf, t["pos"])):
        with pytest.raises(H.HermesError) as e:
            kv.append(q, k, v, pos)
        assert e.value.code == H.EINVAL
        assert [kv.length(l) for l in range(3)] == [20, 20, 20]
    one = {k: t[k][1].contiguous() for k in ("q", "k", "v")}
    bad_one = one["q"].clone()
    bad_one.view(-1)[0] = float("-inf")
    with pytest.raises(H.HermesError) as e:   # one layer; earlier ones stay appendable
        kv.append(bad_one, one["k"], one["v"], t["pos"], layer=1)
    assert e.value.code == H.EINVAL
    out = kv.append(t["q"], t["k"], t["v"], t["pos"])
    out_ref = ref.append(t["q"], t["k"], t["v"], t["pos"])
    kv.compress()
    ref.compress()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out_ref.view(torch.int16))
    for l in range(3):
        a, b = kv.view(l), ref.view(l)
        assert torch.equal(a[2], b[2])
        assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    with pytest.raises(H.HermesError) as e:   # query inputs are checked for finiteness too
        kv.query(q_nan, t["k"], t["v"])
    assert e.value.code == H.EINVAL
    qo = kv.query(t["q"], t["k"], t["v"])
    qo_ref = ref.query(t["q"], t["k"], t["v"])
    torch.cuda.synchronize()
    assert torch.equal(qo.view(torch.int16), qo_ref.view(torch.int16))
    kv.close()
    ref.close()
    # HERMES_CHECK=1 turns the checks on for contexts created while it is set
    monkeypatch.setenv("HERMES_CHECK", "1")
    _, envkv, _ = _setup()
    with pytest.raises(H.HermesError) as e:
        envkv.append(t["q"], t["k"], t["v"], bad_order)
    assert e.value.code == H.EINVAL
    envkv.check_preconditions(False)          # and the toggle turns them off again: a chunk
    envkv.append(t["q"], t["k"], t["v"], early)   # overlapping the cache's last position passes
    torch.cuda.synchronize()
    assert [envkv.length(l) for l in range(3)] == [28, 28, 28]
    envkv.close()


def test_checkpoint_resume_is_bitwise():
    """Checkpoint / resume: after three append + compress steps the per-layer
    state is read back through hermes_kv_view (K, V and positions of each
    layer's current buffer, its length), copied to host memory, and a fresh
    context is created from it (init_len = the lengths).  Three more steps on
    the original and on the resumed context then give bit-identical outputs,
    attention mass and compacted caches: the context holds no other state
    that the next steps read."""
    wl = wk.custom("resume", 131, 4, 8, 2, 64, 600, 48, (300, 400, 500, 600), n_steps=6)
    kv = streaming.make_cache(wl, max_chunk=wl.chunk)
    steps = [streaming.chunk_tensors(wk.stack_chunks(wl, s)) for s in range(6)]
    for s in range(3):
        t = steps[s]
        kv.append(t["q"], t["k"], t["v"], t["pos"])
        kv.compress()
    snap = [tuple(x.cpu().clone() for x in kv.view(l)) for l in range(wl.n_layers)]
    lens = [kv.length(l) for l in range(wl.n_layers)]
    assert lens == [min(b, wl.init_len + 3 * wl.chunk) for b in wl.budgets]
    init = [tuple(x.to("cuda") for x in snap[l]) for l in range(wl.n_layers)]
    kv2 = H.HermesKV(wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.budgets,
                     wl.chunk, cap=kv.cap, init=init)
    assert [kv2.length(l) for l in range(wl.n_layers)] == lens
    for s in range(3, 6):
        t = steps[s]
        o1 = kv.append(t["q"], t["k"], t["v"], t["pos"]).clone()
        o2 = kv2.append(t["q"], t["k"], t["v"], t["pos"]).clone()
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)), f"step {s}: O differs"
        for l in range(wl.n_layers):
            n = kv.length(l)
            assert torch.equal(kv.w[l][:n], kv2.w[l][:n]), f"step {s} layer {l}: W differs"
        kv.compress()
        kv2.compress()
        for l in range(wl.n_layers):
            a, b = kv.view(l), kv2.view(l)
            assert len(a[2]) == len(b[2])
            for x, y in zip(a, b):
                assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                                   y.view(torch.int16) if y.dtype == torch.bfloat16 else y), \
                    f"step {s} layer {l}: compacted state differs"
    kv.close()
    kv2.close()
