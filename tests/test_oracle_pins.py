"""Pins of the fp64 oracle against what the paper and mathematics fix.

None of these checks re-types the oracle's own formula: each one compares it
with a library routine (torch SDPA / softmax), a closed form, an invariant,
a hand-derived fixture under tests/golden/, or brute force on tiny inputs.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import hermes_oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _frac(pairs):
    return np.array([a / b for a, b in pairs])


def _rand_inputs(rng, T0, C, Hq, Hkv, d, scale=0.5):
    q = rng.standard_normal((C, Hq, d)) * scale
    kc = rng.standard_normal((T0, Hkv, d)) * scale
    vc = rng.standard_normal((T0, Hkv, d)) * scale
    kn = rng.standard_normal((C, Hkv, d)) * scale
    vn = rng.standard_normal((C, Hkv, d)) * scale
    return q, kc, vc, kn, vn


# ---------------------------------------------------------------- attention

@pytest.mark.parametrize("T0,C,Hq,Hkv,d", [(0, 5, 2, 1, 4), (7, 3, 4, 2, 8), (33, 17, 14, 2, 16),
                                           (64, 40, 28, 4, 8)])
def test_mass_invariant_rows_sum_to_one(T0, C, Hq, Hkv, d):
    """Every softmax row sums to 1, so sum_i W_i = C * Hq."""
    rng = np.random.default_rng(1)
    q, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
    _, w = orc.chunk_attention(q, kc, vc, kn, vn, row_block=4)
    assert w.shape == (T0 + C,)
    assert abs(w.sum() - C * Hq) <= 1e-12 * C * Hq
    assert np.all(w > 0)


@pytest.mark.parametrize("T0,C,Hq,Hkv,d", [(0, 6, 2, 2, 8), (9, 5, 4, 2, 8), (20, 11, 14, 2, 16),
                                           (31, 9, 28, 4, 32)])
def test_attention_matches_torch_sdpa(T0, C, Hq, Hkv, d):
    """Library special case: torch SDPA in float64 with the causal chunk mask and
    KV heads expanded by repeat_interleave (the HF repeat_kv convention)."""
    rng = np.random.default_rng(2)
    q, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
    o, _ = orc.chunk_attention(q, kc, vc, kn, vn, row_block=3)
    G = Hq // Hkv
    k_all = torch.from_numpy(np.concatenate([kc, kn])).permute(1, 0, 2)
    v_all = torch.from_numpy(np.concatenate([vc, vn])).permute(1, 0, 2)
    k_all = k_all.repeat_interleave(G, dim=0)
    v_all = v_all.repeat_interleave(G, dim=0)
    qt = torch.from_numpy(q).permute(1, 0, 2)
    T = T0 + C
    mask = torch.arange(T)[None, :] <= (T0 + torch.arange(C))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, k_all, v_all, attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-12)


def test_w_matches_torch_softmax_column_sums():
    """W_i = sum over heads and rows of torch.softmax of the masked logits."""
    rng = np.random.default_rng(3)
    T0, C, Hq, Hkv, d = 13, 7, 6, 3, 8
    q, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
    _, w = orc.chunk_attention(q, kc, vc, kn, vn, row_block=2)
    G = Hq // Hkv
    k_all = torch.from_numpy(np.concatenate([kc, kn]))
    T = T0 + C
    mask = torch.arange(T)[None, :] <= (T0 + torch.arange(C))[:, None]
    ref = torch.zeros(T, dtype=torch.float64)
    for h in range(Hq):
        logits = torch.from_numpy(q[:, h, :]) @ k_all[:, h // G, :].T / math.sqrt(d)
        logits = logits.masked_fill(~mask, float("-inf"))
        ref += torch.softmax(logits, dim=1).sum(dim=0)
    np.testing.assert_allclose(w, ref.numpy(), rtol=1e-13)


def test_uniform_attention_closed_form():
    """Zero queries give a uniform softmax over the visible candidates: row r
    puts 1/(T0+r+1) on each, so W_i = Hq * sum_{r >= max(0, i-T0)} 1/(T0+r+1)
    and O[r] is the mean of the visible values."""
    rng = np.random.default_rng(4)
    T0, C, Hq, Hkv, d = 11, 6, 4, 2, 8
    _, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
    q = np.zeros((C, Hq, d))
    o, w = orc.chunk_attention(q, kc, vc, kn, vn)
    expect = np.array([Hq * sum(1.0 / (T0 + r + 1) for r in range(max(0, i - T0), C))
                       for i in range(T0 + C)])
    np.testing.assert_allclose(w, expect, rtol=1e-14)
    v_all = np.concatenate([vc, vn])
    for r in range(C):
        for h in range(Hq):
            np.testing.assert_allclose(o[r, h], v_all[:T0 + r + 1, h // 2].mean(axis=0),
                                       rtol=1e-13, atol=1e-15)


def test_golden_uniform_attention_and_importance():
    """Hand-derived fixture: W, A (both alpha readings) and R at k = ln 2."""
    g = _golden("uniform_attention_T0_2_C_2.json")
    T0, C = g["T0"], g["C"]
    rng = np.random.default_rng(5)
    _, kc, vc, kn, vn = _rand_inputs(rng, T0, C, 1, 1, 4)
    _, w = orc.chunk_attention(np.zeros((C, 1, 4)), kc, vc, kn, vn)
    np.testing.assert_allclose(w, _frac(g["W"]), rtol=1e-15)
    np.testing.assert_allclose(orc.attention_importance(w, T0, C, 0), _frac(g["A_alpha0"]),
                               rtol=1e-14)
    np.testing.assert_allclose(orc.attention_importance(w, T0, C, 1), _frac(g["A_alpha1"]),
                               rtol=1e-14)
    np.testing.assert_allclose(orc.recency_importance(4, math.log(2.0)), _frac(g["R_k_ln2"]),
                               rtol=1e-14)


def test_observer_counts_closed_form():
    assert orc.observer_counts(3, 4).tolist() == [4, 4, 4, 4, 3, 2, 1]
    assert orc.observer_counts(0, 2).tolist() == [2, 1]


# ---------------------------------------------------------------- scores

def test_recency_normaliser_closed_form():
    """Z = sum_i e^{-k(T-1-i)} = (1 - e^{-kT}) / (1 - e^{-k}); the newest token
    gets 1/Z and R increases strictly with i."""
    k = 2.0 ** -10
    for T in (1, 2, 196, 8976, 35904):
        r = orc.recency_importance(T, k)
        z = (1.0 - math.exp(-k * T)) / (1.0 - math.exp(-k))
        assert abs(r[-1] - 1.0 / z) <= 1e-13 / z
        assert abs(r.sum() - 1.0) < 1e-12
        assert np.all(np.diff(r) > 0)
    z8976 = (1.0 - math.exp(-k * 8976)) / (1.0 - math.exp(-k))
    assert abs(z8976 - 1024.34) < 0.01


def test_partition_counts():
    """10/60/30 partition (Sec. 4.1) rounded to the nearest layer."""
    c28 = orc.layer_partition(28)
    assert (c28.count(0), c28.count(1), c28.count(2)) == (3, 17, 8)
    assert c28 == sorted(c28)
    c24 = orc.layer_partition(24)
    assert (c24.count(0), c24.count(1), c24.count(2)) == (2, 15, 7)
    assert orc.smoothing_lambdas([0, 1, 2]) == [0.1, 0.3, 0.4]


def test_omega_endpoints():
    """omega runs from omega0 = 0.75 at the first middle layer down by gamma =
    0.6 to 0.15 at the last, 0.45 half way (Sec. 3.1)."""
    c = orc.layer_partition(28)          # middle layers 3..19
    assert orc.omega(3, c) == pytest.approx(0.75, abs=1e-15)
    assert orc.omega(19, c) == pytest.approx(0.15, abs=1e-15)
    assert orc.omega(11, c) == pytest.approx(0.45, abs=1e-15)
    assert orc.omega(0, [orc.SHALLOW, orc.MIDDLE, orc.DEEP]) == 0.75


def test_middle_mix_and_smoothing_through_stream_step():
    """Three layers (middle, middle, deep) with zero queries: every layer has
    the golden A and R, S^0 = 0.25A + 0.75R, S^1 = 0.85A + 0.15R, S^2 = A, and
    S~^l = (1 - lambda_l) S^l + lambda_l S^{l+1} with lambda = 0.3, 0.3 and the
    last layer unsmoothed."""
    g = _golden("uniform_attention_T0_2_C_2.json")
    A, R = _frac(g["A_alpha0"]), _frac(g["R_k_ln2"])
    rng = np.random.default_rng(6)
    caches, chunks = [], []
    for _ in range(3):
        _, kc, vc, kn, vn = _rand_inputs(rng, 2, 2, 1, 1, 4)
        caches.append(orc.LayerCache(kc, vc, np.arange(2)))
        chunks.append({"q": np.zeros((2, 1, 4)), "k": kn, "v": vn, "pos": np.arange(2, 4)})
    cfg = orc.OracleConfig(budgets=[3, 3, 3], classes=[orc.MIDDLE, orc.MIDDLE, orc.DEEP],
                           forget_rate=math.log(2.0))
    res = orc.stream_step(caches, chunks, cfg)
    s0, s1, s2 = 0.25 * A + 0.75 * R, 0.85 * A + 0.15 * R, A
    for got, want in zip(res["scores"], (s0, s1, s2)):
        np.testing.assert_allclose(got, want, rtol=1e-13)
    np.testing.assert_allclose(res["smoothed"][0], 0.7 * s0 + 0.3 * s1, rtol=1e-13)
    np.testing.assert_allclose(res["smoothed"][1], 0.7 * s1 + 0.3 * s2, rtol=1e-13)
    np.testing.assert_allclose(res["smoothed"][2], s2, rtol=1e-13)
    # A = [7,7,7,6]/27 in the deep layer: the 6/27 token goes, ties keep the
    # higher indices among the 7/27 tokens (all three fit here)
    assert res["kept"][2].tolist() == [0, 1, 2]


def test_golden_smoothing_join():
    g = _golden("smoothing_join.json")
    args = (np.array(g["S_l"]), np.array(g["S_next"]), np.array(g["pos_l"]),
            np.array(g["pos_next"]), g["lambda"])
    np.testing.assert_allclose(orc.smooth(*args, align_mode=0), g["by_position"], rtol=1e-15)
    np.testing.assert_allclose(orc.smooth(*args, align_mode=1), g["by_index"], rtol=1e-15)
    np.testing.assert_allclose(orc.smooth(args[0], None, args[2], None, 0.4), g["S_l"])


# ---------------------------------------------------------------- selection

def test_topk_matches_bruteforce_subset_enumeration():
    """For distinct keys, the kept set maximises the sum of kept keys over all
    subsets of size M (exhaustive on T <= 10)."""
    rng = np.random.default_rng(7)
    for trial in range(60):
        T = int(rng.integers(1, 11))
        M = int(rng.integers(1, 6))
        s = rng.random(T)
        keys = s.astype(np.float32).astype(np.float64)
        if len(set(keys.tolist())) < T:
            continue
        got = orc.topk_indices(s, M)
        if T <= M:
            assert got.tolist() == list(range(T))
            continue
        best = max(itertools.combinations(range(T), M), key=lambda c: sum(keys[list(c)]))
        assert got.tolist() == sorted(best)


def test_ties_keep_highest_indices():
    """One query row with a zero query attends uniformly: W_i = Hq / T for all
    i; under either alpha every deep score ties and the newest tokens win."""
    rng = np.random.default_rng(8)
    T0, Hq = 9, 4
    _, kc, vc, kn, vn = _rand_inputs(rng, T0, 1, Hq, 2, 8)
    _, w = orc.chunk_attention(np.zeros((1, Hq, 8)), kc, vc, kn, vn)
    np.testing.assert_allclose(w, np.full(T0 + 1, Hq / (T0 + 1)), rtol=1e-14)
    for alpha in (0, 1):
        a = orc.attention_importance(w, T0, 1, alpha)
        assert orc.topk_indices(a, 4).tolist() == [6, 7, 8, 9]


def test_fifo_closed_form_all_shallow_lambda_zero():
    """Shallow layers with lambda 0 reduce to FIFO: keep the newest M tokens."""
    rng = np.random.default_rng(9)
    L, T0, C, Hq, Hkv, d = 3, 20, 6, 4, 2, 8
    caches, chunks = [], []
    for _ in range(L):
        q, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
        caches.append(orc.LayerCache(kc, vc, np.arange(T0)))
        chunks.append({"q": q, "k": kn, "v": vn, "pos": np.arange(T0, T0 + C)})
    budgets = [5, 12, 26]
    cfg = orc.OracleConfig(budgets=budgets, classes=[orc.SHALLOW] * L, lambdas=[0.0] * L)
    res = orc.stream_step(caches, chunks, cfg)
    T = T0 + C
    for l in range(L):
        assert res["kept"][l].tolist() == list(range(max(0, T - budgets[l]), T))


def test_budget_at_least_T_keeps_everything_and_query_sees_full_cache():
    rng = np.random.default_rng(10)
    L, T0, C, Hq, Hkv, d = 2, 12, 5, 4, 2, 8
    caches, chunks = [], []
    for _ in range(L):
        q, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
        caches.append(orc.LayerCache(kc, vc, np.arange(T0)))
        chunks.append({"q": q, "k": kn, "v": vn, "pos": np.arange(T0, T0 + C)})
    res = orc.stream_step(caches, chunks, orc.OracleConfig(budgets=[T0 + C, 100]))
    for l in range(L):
        assert res["kept"][l].tolist() == list(range(T0 + C))
        np.testing.assert_array_equal(res["caches"][l].k, np.concatenate([caches[l].k,
                                                                          chunks[l]["k"]]))
    qq, _, _, kq, vq = _rand_inputs(rng, 0, 4, Hq, Hkv, d)
    o = orc.query_attention(res["caches"][0], qq, kq, vq)
    full_k = np.concatenate([caches[0].k, chunks[0]["k"], kq]).transpose(1, 0, 2)
    full_v = np.concatenate([caches[0].v, chunks[0]["v"], vq]).transpose(1, 0, 2)
    T = T0 + C + 4
    mask = torch.arange(T)[None, :] <= (T0 + C + torch.arange(4))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(qq).permute(1, 0, 2),
        torch.from_numpy(full_k).repeat_interleave(2, dim=0),
        torch.from_numpy(full_v).repeat_interleave(2, dim=0), attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)


def test_kept_set_invariants_and_stream_lengths():
    """|I| = min(T, M), I strictly ascending, kept positions a strictly
    increasing subset of the candidates; over a stream from an empty cache the
    length after step s is min(C (s+1), M)."""
    rng = np.random.default_rng(11)
    L, C, Hq, Hkv, d, M = 4, 5, 4, 2, 8, 12
    caches = [orc.LayerCache(np.zeros((0, Hkv, d)), np.zeros((0, Hkv, d)),
                             np.zeros(0, dtype=np.int64)) for _ in range(L)]
    for s in range(6):
        chunks = []
        for _ in range(L):
            q, _, _, kn, vn = _rand_inputs(rng, 0, C, Hq, Hkv, d)
            chunks.append({"q": q, "k": kn, "v": vn, "pos": np.arange(C * s, C * s + C)})
        res = orc.stream_step(caches, chunks, orc.OracleConfig(budgets=[M] * L))
        for l in range(L):
            idx = res["kept"][l]
            T = res["appended"][l].k.shape[0]
            assert len(idx) == min(T, M)
            assert np.all(np.diff(idx) > 0)
            p = res["caches"][l].pos
            assert np.all(np.diff(p) > 0)
            assert set(p.tolist()) <= set(res["appended"][l].pos.tolist())
            assert len(p) == min(C * (s + 1), M)
        caches = res["caches"]


def test_lambda_zero_makes_layers_independent():
    rng = np.random.default_rng(12)
    L, T0, C, Hq, Hkv, d = 3, 16, 6, 4, 2, 8
    caches, chunks = [], []
    for _ in range(L):
        q, kc, vc, kn, vn = _rand_inputs(rng, T0, C, Hq, Hkv, d)
        caches.append(orc.LayerCache(kc, vc, np.arange(T0)))
        chunks.append({"q": q, "k": kn, "v": vn, "pos": np.arange(T0, T0 + C)})
    cfg = orc.OracleConfig(budgets=[10] * L, classes=[orc.MIDDLE, orc.DEEP, orc.DEEP],
                           lambdas=[0.0] * L)
    res = orc.stream_step(caches, chunks, cfg)
    for l in range(L):
        np.testing.assert_array_equal(res["smoothed"][l], res["scores"][l])
        alone = orc.stream_step([caches[l]], [chunks[l]], orc.OracleConfig(
            budgets=[10], classes=[[orc.MIDDLE, orc.DEEP, orc.DEEP][l]], lambdas=[0.0]))
        if l == 0:
            continue   # omega depends on the partition; layer 0 alone is its own span
        assert res["kept"][l].tolist() == alone["kept"][0].tolist()
