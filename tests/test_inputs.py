"""The shared seeded input generator: determinism, shapes, bf16 rounding."""
import numpy as np
import torch

from moe_inputs import (CONFIGS, as_f64, bf16_bits_to_f32, bf16_round_bits, get_config,
                        make_inputs, to_torch)


def test_bf16_rounding_matches_torch(rng):
    v = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, -3.5e-39], np.float32)])
    ours = bf16_round_bits(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(bf16_bits_to_f32(ours), torch.from_numpy(v).to(torch.bfloat16).float().numpy())


def test_deterministic_and_shaped():
    cfg = get_config("tiny")
    a, b = make_inputs(cfg), make_inputs(cfg)
    for key in a:
        if a[key] is None:
            assert b[key] is None
        else:
            assert np.array_equal(a[key], b[key])
    assert a["x"].shape == (256, 64) and a["w_gate"].shape == (64, 4)
    assert a["w1"].shape == (4, 64, 128) and a["w2"].shape == (4, 128, 64) and a["w3"] is None
    assert a["x"].dtype == np.float32
    s = get_config("fine", T=64, M=32, H=16)
    i = make_inputs(s)
    assert i["x"].dtype == np.uint16 and i["w3"].shape == (64, 32, 16)
    assert abs(as_f64(i["w1"]).std() - 0.02) < 0.002
    assert np.array_equal(to_torch(i["x"]).float().numpy(), as_f64(i["x"]).astype(np.float32))


def test_block_seeding_is_thread_count_independent(monkeypatch):
    import moe_inputs
    cfg = get_config("balanced", H=4096 + 8)     # several blocks of draws
    ref = make_inputs(cfg, with_dy=False)["w1"]
    monkeypatch.setattr(moe_inputs, "_workers", lambda: 1)
    assert np.array_equal(make_inputs(cfg, with_dy=False)["w1"], ref)


def test_zipf_bias():
    cfg = CONFIGS["skewed"]
    b = make_inputs(cfg.replace(T=8, M=8, H=8))["bias"]
    rho = np.exp(-b.astype(np.float64) / 1.2)
    assert sorted(np.round(rho).astype(int).tolist()) == list(range(1, cfg.E + 1))
