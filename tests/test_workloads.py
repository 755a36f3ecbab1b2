"""The seeded input generators: deterministic, bfloat16 rounding as torch does
it, rotary embedding norm-preserving, positions and budgets as stated."""
import numpy as np
import torch

from paper_2601_14724_amd import workloads as wk


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 3,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.0078125, 65504.0], np.float32)])
    ours = wk.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(wk.bf16_bits_to_f64(ours),
                                  torch.from_numpy(x).to(torch.bfloat16).double().numpy())


def test_generators_are_deterministic_and_shaped():
    wl = wk.scaled(wk.WORKLOADS["c3_7b_28layer"], init_len=64, chunk=16, n_layers=2,
                   budgets=(32, 40))
    a, b = wk.gen_chunk(wl, 0, 1), wk.gen_chunk(wl, 0, 1)
    for key in ("q", "k", "v", "pos"):
        np.testing.assert_array_equal(a[key], b[key])
    assert a["q"].shape == (16, 28, 128) and a["k"].shape == (16, 4, 128)
    assert a["pos"].tolist() == list(range(64, 80))
    c = wk.gen_cache(wl, 0)
    assert c["k"].shape == (64, 4, 128) and c["pos"].tolist() == list(range(64))
    assert not np.array_equal(wk.gen_chunk(wl, 0, 0)["q"], a["q"])


def test_rope_preserves_pair_norms():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 3, 8))
    y = wk.rope_f64(x, np.arange(5) * 1000)
    np.testing.assert_allclose(x[..., :4] ** 2 + x[..., 4:] ** 2,
                               y[..., :4] ** 2 + y[..., 4:] ** 2, rtol=1e-12)
    np.testing.assert_allclose(wk.rope_f64(x, np.zeros(5, dtype=np.int32)), x)


def test_workload_table():
    c3 = wk.WORKLOADS["c3_7b_28layer"]
    assert c3.budgets[0] == 2048 and c3.budgets[-1] == 6144 and sum(c3.budgets) == 114675
    c5 = wk.WORKLOADS["c5_7b_long"]
    assert c5.budgets[0] == 4096 and c5.budgets[-1] == 16384 and sum(c5.budgets) == 286708
    assert c5.query_positions().tolist()[0] == 35904
    c4 = wk.WORKLOADS["c4_7b_stream64"]
    assert c4.chunk_positions(3).tolist()[0] == 3 * 784
