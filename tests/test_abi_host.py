"""Host-side checks of the C ABI: every symbol the header declares is
exported, and the argument checks that run before any device work reject bad
calls with the documented codes.  Nothing here launches a kernel or touches
device memory (every init call below fails validation before its upload)."""
import ctypes
import os
import re

import pytest

from paper_2601_14724_amd import hermes as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x100000   # aligned, never dereferenced: every call below fails validation first


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "hermes.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hermes_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(H.lib, n), f"{n} declared in hermes.h but not exported"
    assert set(names) == set(H.EXPORTED)


def test_strerror():
    for code in (H.OK, H.EINVAL, H.ECAPACITY, H.ESTATE, H.EHIP, H.ENOTSUP, -99):
        assert isinstance(H.lib.hermes_strerror(code), bytes)
    assert H.lib.hermes_strerror(H.EINVAL) == b"invalid argument"


def _cfg(**over):
    L = over.pop("n_layers", 3)
    budgets = over.pop("budgets", [8] * L)
    cfg = H.HermesConfig()
    cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim = L, 4, 2, 64
    cfg.max_chunk, cfg.max_cap = 16, 64
    arr = (ctypes.c_int32 * len(budgets))(*budgets)
    cfg.budget = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))
    cfg.omega0, cfg.gamma, cfg.forget_rate, cfg.sm_scale = 0.75, 0.6, 2.0 ** -10, 0.0
    for k, v in over.items():
        setattr(cfg, k, v)
    cfg._keep = arr
    return cfg


def _bufs(L, cap=64, init_len=0, **over):
    b = (H.LayerBuffers * L)()
    for l in range(L):
        for p in range(2):
            b[l].k[p] = FAKE
            b[l].v[p] = FAKE
            b[l].pos[p] = FAKE
        b[l].w = FAKE
        b[l].cap = cap
        b[l].init_len = init_len
    for k, v in over.items():
        setattr(b[0], k, v)
    return b


def _init(cfg, bufs, ws=FAKE, nbytes=None):
    if nbytes is None:
        nbytes = H.lib.hermes_workspace_bytes(ctypes.byref(cfg))
    ctx = ctypes.c_void_p()
    rc = H.lib.hermes_kv_init(ctypes.byref(cfg), bufs, ws, nbytes, ctypes.byref(ctx))
    return rc, ctx


def test_static_init_rejects_workspaces_beyond_the_scratch():
    """hermes_kv_init_static refuses a configuration whose workspace, even
    without the stream-mode partial state, exceeds the library's static device
    scratch; the size check runs before any device call."""
    cfg = _cfg(max_cap=1 << 22)
    need = H.lib.hermes_workspace_bytes(ctypes.byref(cfg))
    assert need > H.STATIC_WORKSPACE_BYTES
    bufs = (H.LayerBuffers * cfg.n_layers)()
    ctx = ctypes.c_void_p()
    assert H.lib.hermes_kv_init_static(ctypes.byref(cfg), bufs, ctypes.byref(ctx)) == H.ECAPACITY
    assert not ctx.value
    assert H.lib.hermes_kv_init_static(None, bufs, ctypes.byref(ctx)) == H.EINVAL


def test_workspace_bytes():
    good = H.lib.hermes_workspace_bytes(ctypes.byref(_cfg()))
    assert good > 0 and good % 256 == 0
    bigger = H.lib.hermes_workspace_bytes(ctypes.byref(_cfg(max_cap=4096)))
    assert bigger > good
    assert H.lib.hermes_workspace_bytes(None) == 0
    assert H.lib.hermes_workspace_bytes(ctypes.byref(_cfg(head_dim=96))) == 0


@pytest.mark.parametrize("over,code", [
    ({"n_layers": 0, "budgets": [8]}, H.EINVAL),
    ({"n_layers": 65, "budgets": [8] * 65}, H.EINVAL),
    ({"n_q_heads": 5}, H.EINVAL),
    ({"n_kv_heads": 0}, H.EINVAL),
    ({"head_dim": 96}, H.ENOTSUP),
    ({"max_chunk": 0}, H.EINVAL),
    ({"budgets": [8, 0, 8]}, H.EINVAL),
    ({"alpha_mode": 2}, H.EINVAL),
    ({"align_mode": -1}, H.EINVAL),
    ({"omega0": float("nan")}, H.EINVAL),
])
def test_init_rejects_bad_config(over, code):
    cfg = _cfg(**over)
    rc, ctx = _init(cfg, _bufs(max(1, min(cfg.n_layers, 64))), nbytes=1 << 30)
    assert rc == code and not ctx.value


def test_init_rejects_bad_class_and_lambda():
    cls = (ctypes.c_int8 * 3)(0, 1, 3)
    cfg = _cfg()
    cfg.layer_class = ctypes.cast(cls, ctypes.POINTER(ctypes.c_int8))
    assert _init(cfg, _bufs(3))[0] == H.EINVAL
    lam = (ctypes.c_float * 3)(0.1, 1.5, 0.3)
    cfg = _cfg()
    cfg.lambda_ = ctypes.cast(lam, ctypes.POINTER(ctypes.c_float))
    assert _init(cfg, _bufs(3))[0] == H.EINVAL


def test_init_rejects_bad_buffers_and_workspace():
    cfg = _cfg()
    assert _init(cfg, _bufs(3), ws=FAKE + 8)[0] == H.EINVAL            # misaligned workspace
    assert _init(cfg, _bufs(3), ws=None)[0] == H.EINVAL
    assert _init(cfg, _bufs(3), nbytes=1024)[0] == H.ECAPACITY          # workspace too small
    assert _init(cfg, _bufs(3, cap=4))[0] == H.ECAPACITY                # cap < budget
    assert _init(cfg, _bufs(3, cap=128))[0] == H.ECAPACITY              # cap > max_cap
    assert _init(cfg, _bufs(3, init_len=65))[0] == H.ECAPACITY          # init_len > cap
    assert _init(cfg, _bufs(3, init_len=-1))[0] == H.EINVAL
    b = _bufs(3)
    b[1].w = None
    assert _init(cfg, b)[0] == H.EINVAL
    b = _bufs(3)
    b[2].k[1] = FAKE + 2                                                # misaligned cache
    assert _init(cfg, b)[0] == H.EINVAL
    b = _bufs(3)
    b[0].pos[0] = None
    assert _init(cfg, b)[0] == H.EINVAL
    ctx = ctypes.c_void_p()
    assert H.lib.hermes_kv_init(ctypes.byref(cfg), None, FAKE, 1 << 30, ctypes.byref(ctx)) == H.EINVAL
    assert H.lib.hermes_kv_init(ctypes.byref(cfg), _bufs(3), FAKE, 1 << 30, None) == H.EINVAL


def test_null_context_calls():
    assert H.lib.hermes_append_chunk(None, 0, FAKE, FAKE, FAKE, FAKE, 4, FAKE, None) == H.EINVAL
    assert H.lib.hermes_compress(None, None) == H.EINVAL
    assert H.lib.hermes_query_attend(None, 0, FAKE, FAKE, FAKE, 4, FAKE, None) == H.EINVAL
    assert H.lib.hermes_kv_rewind(None) == H.EINVAL
    assert H.lib.hermes_kv_view(None, 0, None, None, None, None) == H.EINVAL
    assert H.lib.hermes_profile_enable(None, 1) == H.EINVAL
    assert H.lib.hermes_profile_read(None, 0, None, None) == H.EINVAL
    H.lib.hermes_kv_destroy(None)


def test_topk_argument_checks():
    assert H.lib.hermes_select_topk(None, 10, 3, FAKE, None) == H.EINVAL
    assert H.lib.hermes_select_topk(FAKE, 0, 3, FAKE, None) == H.EINVAL
    assert H.lib.hermes_select_topk(FAKE, 10, 0, FAKE, None) == H.EINVAL
    assert H.lib.hermes_select_topk(FAKE, 10, 3, None, None) == H.EINVAL
    assert H.lib.hermes_select_topk(FAKE + 1, 10, 3, FAKE, None) == H.EINVAL


@pytest.mark.parametrize("over,code", [
    ({"summary_mode": 2}, H.EINVAL),
    ({"reindex_mode": 3}, H.EINVAL),
    ({"scoring_mode": -1}, H.EINVAL),
    ({"rope_offset": -1}, H.EINVAL),
    ({"rope_headroom": -5}, H.EINVAL),
    ({"rope_theta": float("inf")}, H.EINVAL),
    ({"summary_mode": 1, "n_q_heads": 16, "n_kv_heads": 16, "head_dim": 128}, H.ENOTSUP),
])
def test_init_rejects_bad_extension_config(over, code):
    cfg = _cfg(**over)
    rc, ctx = _init(cfg, _bufs(3), nbytes=1 << 30)
    assert rc == code and not ctx.value


def test_extensions_need_rope_buffers_and_room_for_the_summary():
    # summary or re-indexing without RoPE-position buffers
    for over in ({"summary_mode": 1}, {"reindex_mode": H.REINDEX_EAGER}):
        assert _init(_cfg(**over), _bufs(3))[0] == H.EINVAL
    b = _bufs(3)
    for l in range(3):
        b[l].rpos[0] = FAKE
        b[l].rpos[1] = FAKE + 2            # misaligned
    assert _init(_cfg(reindex_mode=H.REINDEX_LAZY), b)[0] == H.EINVAL
    # a deep layer with summaries needs budget + 1 rows (default classes of 3
    # layers: shallow, middle, deep)
    b = _bufs(3, cap=8)
    for l in range(3):
        b[l].rpos[0] = b[l].rpos[1] = FAKE
    cfg = _cfg(summary_mode=1, max_cap=8)
    assert _init(cfg, b)[0] == H.ECAPACITY


def test_workspace_grows_with_summary_buffers():
    base = H.lib.hermes_workspace_bytes(ctypes.byref(_cfg(max_cap=4096)))
    summ = H.lib.hermes_workspace_bytes(ctypes.byref(_cfg(max_cap=4096, summary_mode=1)))
    # fp64 block sums: ceil(4096 / 512) blocks x 2 x Hkv*d doubles per layer
    assert summ - base >= 3 * 8 * 2 * 128 * 8


def test_budget_from_weights_matches_oracle():
    from oracle import hermes_extensions as he
    from oracle import hermes_oracle as ho
    cls = ho.layer_partition(28)
    for wts in ((1.0, 1.0, 1.0), (1.3, 1.0, 0.7), (0.7, 1.6, 0.7), (0.7, 1.0, 1.3)):
        w = [wts[c] for c in cls]
        assert H.budget_from_weights(w, 6000 * 28) == he.budget_allocation(w, 6000 * 28)
    rng = __import__("numpy").random.default_rng(7)
    for _ in range(20):
        w = list(rng.uniform(0.1, 3.0, size=24))
        total = int(rng.integers(24 * 10, 24 * 9000))
        assert H.budget_from_weights(w, total) == he.budget_allocation(w, total)


@pytest.mark.parametrize("weights,total", [
    ([1.0, float("nan")], 100), ([1.0, -1.0], 100), ([0.0, 0.0], 100), ([1.0, 1.0], 1),
    ([1e-9, 1.0], 100),           # the first layer would get 0 tokens
])
def test_budget_from_weights_rejects(weights, total):
    with pytest.raises(H.HermesError) as e:
        H.budget_from_weights(weights, total)
    assert e.value.code == H.EINVAL


def _sec(a, b, c):
    return (ctypes.c_int32 * 3)(a, b, c)


@pytest.mark.parametrize("over,code", [
    ({"rope_axes": 2}, H.EINVAL),
    ({"rope_axes": -1}, H.EINVAL),
    ({"rope_axes": 3, "mrope_section": _sec(8, 8, 8)}, H.EINVAL),      # sums to 24, not d/2 = 32
    ({"rope_axes": 3, "mrope_section": _sec(-1, 17, 16)}, H.EINVAL),
    ({"rope_axes": 3, "n_q_heads": 16, "n_kv_heads": 16, "head_dim": 128}, H.ENOTSUP),
])
def test_init_rejects_bad_mrope_config(over, code):
    rc, ctx = _init(_cfg(**over), _bufs(3), nbytes=1 << 30)
    assert rc == code and not ctx.value


def test_mrope_needs_all_three_coordinate_buffers():
    b = _bufs(3)
    for l in range(3):
        b[l].rpos[0] = b[l].rpos[1] = FAKE
    assert _init(_cfg(rope_axes=3), b)[0] == H.EINVAL          # no h / w buffers
    for l in range(3):
        b[l].rpos_h[0] = b[l].rpos_h[1] = FAKE
        b[l].rpos_w[0] = FAKE
        b[l].rpos_w[1] = FAKE + 2                                # misaligned
    assert _init(_cfg(rope_axes=3), b)[0] == H.EINVAL


def test_workspace_grows_with_mrope_coordinates():
    base = H.lib.hermes_workspace_bytes(ctypes.byref(_cfg(max_cap=4096)))
    three = H.lib.hermes_workspace_bytes(ctypes.byref(_cfg(max_cap=4096, rope_axes=3)))
    assert three - base >= 3 * 3 * 4096 * 4        # (t, h, w) of every row of 3 layers
