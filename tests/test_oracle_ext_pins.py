"""Pins of the extension oracle (summary token, re-indexing, guidance-prompt
scoring, layer-weighted budgets) against facts that do not come from the
oracle itself: the input generator's independent RoPE, closed forms, exact
integer arithmetic written out here, and invariants."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import hermes_extensions as he
from oracle import hermes_oracle as ho
from paper_2601_14724_amd import workloads as wk

RNG = np.random.default_rng(20260114)


def _raw(n, h=2, d=16):
    return RNG.standard_normal((n, h, d))


# ---------------------------------------------------------------- rounding

def test_round_to_bf16_matches_generator_rounding():
    x = RNG.standard_normal(4096).astype(np.float32).astype(np.float64) * 3.0
    ours = he.round_to_bf16(x)
    gen = wk.bf16_bits_to_f64(wk.f32_to_bf16_bits(x.astype(np.float32)))
    assert np.array_equal(ours, gen)


def test_round_to_bf16_ties_to_even():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7: ties go to the even 1.0;
    # 1 + 3 * 2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: goes to 1 + 2^-6
    assert he.round_to_bf16(np.array([1 + 2.0 ** -8]))[0] == 1.0
    assert he.round_to_bf16(np.array([1 + 3 * 2.0 ** -8]))[0] == 1 + 2.0 ** -6


# ---------------------------------------------------------------- RotaryDelta

def test_rotary_delta_zero_is_identity():
    k = _raw(5)
    assert np.array_equal(he.rotary_delta(k, np.zeros(5, dtype=np.int64)), k)


@pytest.mark.parametrize("d", [16, 64, 128])
def test_rotary_delta_moves_rope_positions(d):
    """Re-rotating a key made at p_old by p_new - p_old gives the key made at
    p_new (the generator's RoPE is an independent implementation)."""
    x = _raw(7, 3, d)
    p_old = np.array([0, 5, 17, 300, 9000, 20000, 35903])
    p_new = np.array([3, 4, 5, 6, 7, 8, 36000])
    k_old = wk.rope_f64(x, p_old)
    got = he.rotary_delta(k_old, p_new - p_old)
    want = wk.rope_f64(x, p_new)
    assert np.max(np.abs(got - want)) < 1e-9


def test_rotary_delta_composes_and_preserves_pair_norms():
    k = _raw(6, 2, 32)
    a = np.array([1, -4, 100, 7, 0, 12345])
    b = np.array([9, 4, -50, 1000, 3, -12345])
    assert np.max(np.abs(he.rotary_delta(he.rotary_delta(k, a), b) - he.rotary_delta(k, a + b))) < 1e-10
    r = he.rotary_delta(k, a)
    n0 = k[..., :16] ** 2 + k[..., 16:] ** 2
    n1 = r[..., :16] ** 2 + r[..., 16:] ** 2
    assert np.max(np.abs(n0 - n1)) < 1e-12


# ---------------------------------------------------------------- summary token

def test_summary_key_is_mean_raw_key_at_target():
    """Keys made at positions p_i and aligned to t average to the key made at
    t from the mean unrotated vector."""
    x = _raw(11, 2, 64)
    p = np.sort(RNG.choice(5000, size=11, replace=False))
    k = wk.rope_f64(x, p)
    v = _raw(11, 2, 64)
    ks, vs, t = he.summary_token(k, v, p)
    assert t == p.max()
    want = wk.rope_f64(x.mean(axis=0)[None], np.array([t]))[0]
    assert np.max(np.abs(ks - want)) < 1e-10
    # V: rows a_i * u average to mean(a) * u
    a = RNG.standard_normal(11)
    u = _raw(1, 2, 64)[0]
    _, vs2, _ = he.summary_token(k, a[:, None, None] * u[None], p)
    assert np.max(np.abs(vs2 - a.mean() * u)) < 1e-12


def test_summary_of_one_token_is_that_token():
    k, v = _raw(1, 2, 32), _raw(1, 2, 32)
    ks, vs, t = he.summary_token(k, v, np.array([77]))
    assert t == 77 and np.array_equal(ks, k[0]) and np.array_equal(vs, v[0])


# ---------------------------------------------------------------- re-indexing

def test_reindex_positions_left_compacts_behind_prefix():
    assert list(he.reindex_positions(np.array([5, 9, 100, 101]), 3)) == [3, 4, 5, 6]
    assert list(he.reindex_positions(np.array([0, 1, 2]), 0)) == [0, 1, 2]


def test_reindex_of_contiguous_positions_changes_nothing():
    k = he.round_to_bf16(_raw(4, 2, 32))
    rp = np.array([10, 11, 12, 13])
    k_new, p_new = he.reindex_keys(k, rp, 10)
    assert list(p_new) == [10, 11, 12, 13] and np.array_equal(k_new, k)


def test_reindexed_keys_are_keys_made_at_new_positions():
    x = _raw(5, 2, 64)
    p_old = np.array([100, 2000, 2001, 30000, 35000])
    k_new, p_new = he.reindex_keys(wk.rope_f64(x, p_old), p_old, 7)
    assert list(p_new) == [7, 8, 9, 10, 11]
    want = he.round_to_bf16(wk.rope_f64(x, p_new))
    # both sides round fp64 values that agree to ~1e-12: at most one bf16 ulp apart
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(want), 1e-30))) - 7)
    assert np.all(np.abs(k_new - want) <= ulp)


# ---------------------------------------------------------------- guidance scoring

def test_guidance_mass_uniform_closed_form():
    """Zero queries: prompt row r attends T + r + 1 keys uniformly, so each
    cached token receives Hq * sum_r 1 / (T + r + 1)."""
    T, n, Hq, Hkv, d = 37, 5, 4, 2, 16
    kc, vc = _raw(T, Hkv, d), _raw(T, Hkv, d)
    kg, vg = _raw(n, Hkv, d), _raw(n, Hkv, d)
    w = he.guidance_mass(np.zeros((n, Hq, d)), kc, vc, kg, vg)
    want = Hq * sum(1.0 / (T + r + 1) for r in range(n))
    assert w.shape == (T,) and np.max(np.abs(w - want)) < 1e-13


def test_guidance_mass_plus_self_mass_is_rows_times_heads():
    T, n, Hq, Hkv, d = 50, 6, 4, 2, 16
    q, kc, vc, kg, vg = _raw(n, Hq, d), _raw(T, Hkv, d), _raw(T, Hkv, d), _raw(n, Hkv, d), _raw(n, Hkv, d)
    _, w_all = ho.chunk_attention(q, kc, vc, kg, vg)
    w = he.guidance_mass(q, kc, vc, kg, vg)
    assert np.array_equal(w, w_all[:T])
    assert abs(w_all.sum() - n * Hq) < 1e-12
    a = he.guidance_importance(w, n)
    assert abs(a.sum() - 1.0) < 1e-14


# ---------------------------------------------------------------- budgets

def test_budget_allocation_paper_weights_by_hand():
    """Weights 0.7 / 1.0 / 1.3 (shallow / middle / deep) over the 3/17/8
    partition of 28 layers and |M| = 6000 * 28, in integer arithmetic:
    floor(7 * 168000 / 295) = 3986, floor(10 * 168000 / 295) = 5694,
    floor(13 * 168000 / 295) = 7403, residue 168000 - 167980 = 20."""
    cls = ho.layer_partition(28)
    w = [{ho.SHALLOW: 0.7, ho.MIDDLE: 1.0, ho.DEEP: 1.3}[c] for c in cls]
    m = he.budget_allocation(w, 6000 * 28)
    assert m[:3] == [3986] * 3 and m[3:20] == [5694] * 17 and m[20:27] == [7403] * 7
    assert m[27] == 7403 + 20 and sum(m) == 168000


@pytest.mark.parametrize("wts", [("1.0", "1.0", "1.0"), ("1.3", "1.0", "0.7"),
                                 ("0.7", "1.6", "0.7"), ("0.7", "1.0", "1.3")])
def test_budget_allocation_fp64_equals_exact(wts):
    cls = ho.layer_partition(28)
    ws = [wts[c] for c in cls]
    m = he.budget_allocation([float(x) for x in ws], 6000 * 28)
    assert m == he.budget_allocation_exact(ws, 6000 * 28)
    assert sum(m) == 6000 * 28


def test_budget_allocation_equal_weights():
    m = he.budget_allocation([1.0] * 5, 103)
    assert m == [20, 20, 20, 20, 23]


# ---------------------------------------------------------------- the extended step

def _tiny(L=4, T0=40, C=12, Hq=4, Hkv=2, d=16, budgets=(30, 30, 30, 30), seed=3):
    rng = np.random.default_rng(seed)
    r = lambda *s: he.round_to_bf16(rng.standard_normal(s) * 0.5)
    caches = [he.ExtLayerCache(r(T0, Hkv, d), r(T0, Hkv, d), np.arange(T0), np.arange(T0)) for _ in range(L)]
    chunks = [{"q": r(C, Hq, d), "k": r(C, Hkv, d), "v": r(C, Hkv, d), "pos": np.arange(T0, T0 + C)}
              for _ in range(L)]
    cfg = ho.OracleConfig(budgets=list(budgets), classes=[ho.SHALLOW, ho.MIDDLE, ho.DEEP, ho.DEEP])
    return caches, chunks, cfg


def test_ext_step_without_extensions_equals_step():
    caches, chunks, cfg = _tiny()
    a = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig())
    b = ho.stream_step([ho.LayerCache(c.k, c.v, c.pos) for c in caches], chunks, cfg)
    for l in range(4):
        assert np.array_equal(a["kept"][l], b["kept"][l])
        assert np.array_equal(a["caches"][l].k, b["caches"][l].k)
        assert np.array_equal(a["caches"][l].pos, b["caches"][l].pos)


def test_ext_step_summary_tokens():
    caches, chunks, cfg = _tiny()
    res = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(summary=True))
    for l in range(4):
        c, kept = res["caches"][l], res["kept"][l]
        s = res["summaries"][l]
        if cfg.classes[l] != ho.DEEP:
            assert s is None and len(c.pos) == 30
            continue
        assert len(c.pos) == 31                      # |M| kept + the summary
        ev = np.setdiff1d(np.arange(52), kept)
        assert np.array_equal(s["evicted"], ev) and s["source"] == ev[-1]
        assert c.pos[s["index"]] == res["appended"][l].pos[ev[-1]]
        assert np.all(np.diff(c.pos) > 0) and np.all(np.diff(c.rpos) > 0)
        assert np.array_equal(np.delete(c.pos, s["index"]), res["appended"][l].pos[kept])


def test_ext_step_eager_and_lazy_reindex():
    caches, chunks, cfg = _tiny()
    eager = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(summary=True, reindex_mode=he.REINDEX_EAGER,
                                                                 rope_offset=5))
    assert eager["reindexed"]
    for c in eager["caches"]:
        assert list(c.rpos) == list(range(5, 5 + len(c.rpos)))
    # largest retained position is 51; the lazy rule fires at 51 + 12 >= limit
    lazy_no = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(reindex_mode=he.REINDEX_LAZY,
                                                                   rope_limit=64, rope_headroom=12))
    lazy_yes = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(reindex_mode=he.REINDEX_LAZY,
                                                                    rope_limit=63, rope_headroom=12))
    assert not lazy_no["reindexed"] and lazy_yes["reindexed"]
    plain = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig())
    for l in range(4):
        assert np.array_equal(lazy_no["caches"][l].k, plain["caches"][l].k)
        assert list(lazy_yes["caches"][l].rpos) == list(range(len(lazy_yes["caches"][l].rpos)))


def test_ext_step_guidance_zero_queries_keep_newest_in_deep_layers():
    """A zero-query prompt spreads its mass evenly over the cache, so deep-layer
    scores tie and the tie rule keeps the newest |M| tokens (lambda = 0)."""
    caches, chunks, cfg = _tiny()
    cfg.lambdas = [0.0] * 4
    prompts = [{"q": np.zeros((3, 4, 16)), "k": np.zeros((3, 2, 16)), "v": np.zeros((3, 2, 16))}] * 4
    res = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(scoring_mode=he.SCORE_GUIDANCE), prompts)
    for l in (2, 3):
        assert np.allclose(res["w"][l], res["w"][l][0], rtol=1e-14)
        assert list(res["kept"][l]) == list(range(22, 52))


# ---------------------------------------------------------------- 3D M-RoPE

def _grid(frames, H, W, offset=0, t_step=1):
    """(t, h, w) of a video laid out frame by frame, row by row (the order
    tokens are appended in), written out here independently of the oracle."""
    out = []
    for f in range(frames):
        for y in range(H):
            for x in range(W):
                out.append((offset + f * t_step, offset + y, offset + x))
    return np.array(out, dtype=np.int64)


@pytest.mark.parametrize("d,want", [(128, (16, 24, 24)), (64, (8, 12, 12)), (256, (32, 48, 48))])
def test_default_mrope_section(d, want):
    """The default split of the d/2 frequency pairs over (t, h, w): the
    backbone's published M-RoPE section sizes, 16/24/24 pairs at head size
    128 (the paper only names "the channel section allocated for dimension
    d"), i.e. a quarter of the pairs for t and the rest halved, contiguous in
    the order t, h, w and covering every pair once."""
    assert he.default_mrope_section(d) == want
    axis = he.mrope_pair_axis(d, want)
    assert len(axis) == d // 2 and np.all(np.diff(axis) >= 0)
    assert [int((axis == a).sum()) for a in range(3)] == list(want)


def test_mrope_with_one_section_reduces_to_1d():
    """All pairs in the t section: the sectioned rotation is the 1D rotation
    by the t delta, and ranking strictly increasing t is the 1D rank."""
    k = _raw(9, 2, 16)
    d3 = np.stack([RNG.integers(-50, 50, 9), RNG.integers(-50, 50, 9), RNG.integers(-50, 50, 9)], 1)
    assert np.array_equal(he.rotary_delta3(k, d3, (8, 0, 0)), he.rotary_delta(k, d3[:, 0]))
    t = np.sort(RNG.choice(1000, 9, replace=False))
    c = np.stack([t, RNG.integers(0, 5, 9), RNG.integers(0, 5, 9)], 1)
    assert np.array_equal(he.reindex_coords3(c, 7)[:, 0], he.reindex_positions(t, 7))


def test_mrope_full_grid_is_unchanged():
    g = _grid(3, 4, 5, offset=11)
    assert np.array_equal(he.reindex_coords3(g, 11), g)
    k = he.round_to_bf16(_raw(len(g), 2, 32))
    kn, new = he.reindex_keys3(k, g, 11, (4, 6, 6))
    assert np.array_equal(kn, k) and np.array_equal(new, g)


def test_mrope_dropping_a_frame_and_a_column():
    """Frame 1 and column 2 evicted everywhere: later frames move one step
    down in t, later columns one step down in w, rows keep their h."""
    F, H, W, off = 4, 3, 5, 2
    g = _grid(F, H, W, offset=off)
    f = (g[:, 0] - off)
    x = (g[:, 2] - off)
    keep = (f != 1) & (x != 2)
    new = he.reindex_coords3(g[keep], off)
    exp_t = off + np.where(f[keep] > 1, f[keep] - 1, f[keep])
    exp_w = off + np.where(x[keep] > 2, x[keep] - 1, x[keep])
    assert np.array_equal(new[:, 0], exp_t)
    assert np.array_equal(new[:, 1], g[keep][:, 1])
    assert np.array_equal(new[:, 2], exp_w)


def test_mrope_ranks_are_dense_and_shared_coordinates_stay_shared():
    c = np.stack([RNG.integers(0, 40, 200) * 3, RNG.integers(0, 9, 200) + 100, RNG.integers(5, 30, 200)], 1)
    new = he.reindex_coords3(c, 4)
    for a in range(3):
        distinct = sorted(set(c[:, a].tolist()))
        assert sorted(set(new[:, a].tolist())) == list(range(4, 4 + len(distinct)))
        for i in range(0, 200, 7):
            for j in range(0, 200, 11):
                assert (c[i, a] < c[j, a]) == (new[i, a] < new[j, a])
                assert (c[i, a] == c[j, a]) == (new[i, a] == new[j, a])


def test_mrope_reindexed_keys_equal_keys_made_at_new_coordinates():
    """A raw key made at 3D coordinates p by multiplying each complex pair
    (x_j + i x_{j+d/2}) by e^{i p_axis(j) theta_j}, computed here with complex
    exponentials; the oracle's RotaryDelta from old to new coordinates turns
    the key made at the old coordinates into the one made at the new."""
    d, section = 32, (4, 6, 6)
    axis = np.array([0] * section[0] + [1] * section[1] + [2] * section[2])
    freq = 1.0e6 ** (-np.arange(d // 2) * 2.0 / d)

    def made_at(x, p):
        z = x[..., : d // 2] + 1j * x[..., d // 2:]
        z = z * np.exp(1j * p[:, axis][:, None, :] * freq[None, None, :])
        return np.concatenate([z.real, z.imag], axis=-1)

    g = _grid(3, 4, 4, offset=9)
    keep = RNG.random(len(g)) < 0.6
    old = g[keep]
    x = _raw(len(old), 2, d)
    new = he.reindex_coords3(old, 9)
    moved = he.rotary_delta3(made_at(x, old), new - old, section)
    assert np.abs(moved - made_at(x, new)).max() < 1e-12


def test_summary3_key_is_mean_raw_key_at_the_target_coordinates():
    """Summary token with 3D coordinates: keys made at (t, h, w)_i (complex
    exponentials per section, computed here) and aligned to the newest
    evicted token's coordinates average to the key made at those coordinates
    from the mean unrotated vector; V is the plain mean; the target is the
    last row's coordinates."""
    d, section = 32, (4, 6, 6)
    axis = np.array([0] * section[0] + [1] * section[1] + [2] * section[2])
    freq = 1.0e6 ** (-np.arange(d // 2) * 2.0 / d)

    def made_at(x, p):
        z = x[..., : d // 2] + 1j * x[..., d // 2:]
        z = z * np.exp(1j * p[:, axis][:, None, :] * freq[None, None, :])
        return np.concatenate([z.real, z.imag], axis=-1)

    g = _grid(3, 4, 4, offset=5)
    ev = np.sort(RNG.choice(len(g), size=13, replace=False))
    c = g[ev]
    x = _raw(13, 2, d)
    v = _raw(13, 2, d)
    ks, vs, tgt = he.summary_token3(made_at(x, c), v, c, section)
    assert np.array_equal(tgt, c[-1])
    assert np.abs(ks - made_at(x.mean(axis=0)[None], c[-1:])[0]).max() < 1e-12
    assert np.abs(vs - v.mean(axis=0)).max() < 1e-15


def test_summary3_with_one_section_is_the_1d_summary_on_t():
    """All frequency pairs in the t section: the 3D summary is the 1D summary
    over the t coordinates (h and w play no part)."""
    k, v = _raw(9, 2, 16), _raw(9, 2, 16)
    t = np.sort(RNG.choice(3000, 9, replace=False))
    c = np.stack([t, RNG.integers(0, 50, 9), RNG.integers(0, 50, 9)], 1)
    ks3, vs3, tgt = he.summary_token3(k, v, c, (8, 0, 0))
    ks1, vs1, t1 = he.summary_token(k, v, t)
    assert tgt[0] == t1 and np.array_equal(ks3, ks1) and np.array_equal(vs3, vs1)
    ks_one, vs_one, tgt_one = he.summary_token3(k[:1], v[:1], c[:1], (4, 2, 2))
    assert np.array_equal(ks_one, k[0]) and np.array_equal(vs_one, v[0]) and np.array_equal(tgt_one, c[0])


def _tiny_mrope(L=3, frames0=4, frames=1, H=3, W=4, Hq=4, Hkv=2, d=16, budgets=(30, 30, 30), seed=5):
    rng = np.random.default_rng(seed)
    r = lambda *s: he.round_to_bf16(rng.standard_normal(s) * 0.5)
    T0, C = frames0 * H * W, frames * H * W
    g = _grid(frames0 + frames, H, W, offset=3)
    caches = [he.ExtLayerCache(r(T0, Hkv, d), r(T0, Hkv, d), np.arange(T0), g[:T0, 0].copy(), g[:T0].copy())
              for _ in range(L)]
    chunks = [{"q": r(C, Hq, d), "k": r(C, Hkv, d), "v": r(C, Hkv, d), "pos": np.arange(T0, T0 + C),
               "rope_thw": g[T0:].T.copy()} for _ in range(L)]
    cfg = ho.OracleConfig(budgets=list(budgets), classes=[ho.SHALLOW, ho.MIDDLE, ho.DEEP])
    return caches, chunks, cfg, g


def test_ext_step_mrope_eager_and_lazy():
    caches, chunks, cfg, g = _tiny_mrope()
    ext = he.ExtConfig(reindex_mode=he.REINDEX_EAGER, rope_offset=3, rope_axes=3)
    res = he.stream_step_ext(caches, chunks, cfg, ext)
    assert res["reindexed"]
    plain = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(rope_axes=3))
    for l in range(3):
        c, p = res["caches"][l], plain["caches"][l]
        assert np.array_equal(c.pos, p.pos) and np.array_equal(c.v, p.v)
        assert np.array_equal(p.rpos3, g[res["kept"][l]])
        for a in range(3):
            n = len(set(p.rpos3[:, a].tolist()))
            assert sorted(set(c.rpos3[:, a].tolist())) == list(range(3, 3 + n))
    # largest retained coordinate is t = 3 + 4 = 7: the lazy rule fires at 7 + 2 >= limit
    no = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(reindex_mode=he.REINDEX_LAZY, rope_axes=3,
                                                              rope_limit=10, rope_headroom=2))
    yes = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(reindex_mode=he.REINDEX_LAZY, rope_axes=3,
                                                               rope_limit=9, rope_headroom=2, rope_offset=3))
    assert not no["reindexed"] and yes["reindexed"]
    for l in range(3):
        assert np.array_equal(yes["caches"][l].k, res["caches"][l].k)


def test_ext_step_mrope_with_summary_tokens():
    """3D coordinates with summary tokens: every evicting deep layer holds
    budget + 1 rows, the summary at the sorted place of the newest evicted
    token with that token's stream position and (t, h, w); eager re-indexing
    then ranks the summary's coordinates with the kept rows'."""
    caches, chunks, cfg, g = _tiny_mrope(budgets=(30, 30, 30))
    ext = he.ExtConfig(summary=True, rope_axes=3)
    res = he.stream_step_ext(caches, chunks, cfg, ext)
    cat = res["appended"][2]
    summ = res["summaries"][2]
    assert summ is not None and res["summaries"][0] is None and res["summaries"][1] is None
    c = res["caches"][2]
    assert len(c.pos) == 31
    newest = summ["source"]
    assert newest == summ["evicted"][-1]
    assert np.array_equal(c.rpos3[summ["index"]], cat.rpos3[newest])
    assert c.pos[summ["index"]] == cat.pos[newest] and np.all(np.diff(c.pos) > 0)
    assert np.array_equal(summ["target"], cat.rpos3[newest])
    eager = he.stream_step_ext(caches, chunks, cfg, he.ExtConfig(summary=True, rope_axes=3,
                                                                reindex_mode=he.REINDEX_EAGER,
                                                                rope_offset=3))
    e = eager["caches"][2]
    assert np.array_equal(e.rpos3, he.reindex_coords3(c.rpos3, 3))
