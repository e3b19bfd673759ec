"""Seeded input generator: shapes, recipes, determinism, bf16 rounding."""
import numpy as np
import torch

from paper_2512_23068_amd import inputs


def test_recipes_and_shapes():
    for cfg in inputs.CONFIGS:
        p = inputs.make_params(cfg)
        D, N = cfg.d_inner, cfg.d_state
        assert p["A"].shape == (D, N) and p["W_B"].shape == (D, N) and p["W_C"].shape == (D, N)
        assert p["w_delta"].shape == (D,) and p["b_delta"].shape == (D,)
        assert np.all(p["A"] < 0)
        v = np.logaddexp(0.0, p["b_delta"].astype(np.float64))
        assert np.all(v >= cfg.delta_lo * (1 - 1e-5)) and np.all(v <= cfg.delta_hi * (1 + 1e-5))
        if cfg.a_kind == "s4d":
            assert np.array_equal(p["A"][3], -np.arange(1, N + 1, dtype=np.float32))
        if cfg.a_kind == "stiff":
            assert p["A"].min() < -500 and p["A"].max() > -1.5


def test_small_workload_values_and_determinism():
    cfg = inputs.get_config("tiny")
    a = inputs.make_inputs(cfg, threads=1)
    b = inputs.make_inputs(cfg, threads=4)
    assert np.array_equal(a["x"], b["x"]) and np.array_equal(a["dx"], b["dx"])
    assert a["x"].shape == (1, 1024, 16) and a["dx"].shape == (1, 1, 1024, 16)
    assert a["dx"][0, 0, 0, 0] == 1.0 and np.count_nonzero(a["dx"]) == 1
    c = inputs.make_inputs(cfg.with_(seqlen=700, dx_kind="normal", n_dirs=3), threads=3)
    assert c["x"].shape == (1, 700, 16) and c["dx"].shape == (3, 1, 700, 16)
    assert np.array_equal(c["x"], a["x"][:, :700])   # block seeding: prefix-stable
    assert abs(c["dx"].std() - 1) < 0.05


def test_bf16_rounding_matches_torch_rne():
    g = np.random.default_rng(0)
    v = (g.standard_normal(100000) * np.exp(g.uniform(-10, 10, 100000))).astype(np.float32)
    ours = inputs.bf16_bits_to_f32(inputs.round_to_bf16_bits(v))
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


def test_bf16_workload_values_are_bf16():
    cfg = inputs.get_config("stiff128k").with_(seqlen=64, d_inner=128)
    x = inputs.make_x(cfg)
    assert np.array_equal(x, inputs.bf16_bits_to_f32(inputs.round_to_bf16_bits(x)).reshape(x.shape))


def test_empty_sequences():
    """Every generator gives empty arrays of the right shapes for L = 0."""
    ssm = inputs.make_inputs(inputs.get_config("mamba130m").with_(seqlen=0, d_inner=8, n_dirs=2))
    assert ssm["x"].shape == (1, 0, 8) and ssm["dx"].shape == (2, 1, 0, 8)
    assert inputs.make_adjoint(inputs.get_config("mamba130m").with_(seqlen=0, d_inner=8)).shape == (1, 0, 8)
    la = inputs.make_la_inputs(inputs.LA_BY_NAME["la_tiny"].with_(seqlen=0, n_dirs=2))
    assert la["q"].shape == (1, 2, 0, 16) and la["dv"].shape == (2, 1, 2, 0, 64)
