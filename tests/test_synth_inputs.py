"""The seeded input generator: shapes, determinism, bf16 exactness, unit norms."""
import numpy as np

from lact_synth import CONFIGS, bf16_bits, make_cotangents, make_inputs, round_to_bf16


def test_bf16_rounding_is_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 0.0], np.float32)
    # halfway cases round to even mantissa
    r = round_to_bf16(x)
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == 1.0 + 2 ** -6 and r[3] == 1.0
    assert r[4] == -2.5 and r[5] == 0.0
    assert bf16_bits(np.array([np.nan], np.float32))[0] == 0x7FC0


def test_shapes_and_recipe():
    cfg = CONFIGS["tiny_fp32"]
    a = make_inputs(cfg, 0)
    assert a["q"].shape == (2, 1024, 64) and a["k"].shape == (2, 1024, 64)
    assert a["W1"].shape == (2, 64, 64) and a["W2"].shape == (2, 64, 64)
    assert a["eta"].shape == (2, 1024) and np.all(a["eta"] > 0)
    np.testing.assert_allclose(np.linalg.norm(a["q"], axis=-1), 1.0, rtol=1e-5)
    for w in ("W1", "W2", "W3"):
        np.testing.assert_allclose(np.linalg.norm(a[w], axis=-1), 1.0, rtol=1e-5)
    b = make_inputs(cfg, 0)
    for key in a:
        assert np.array_equal(a[key], b[key])
    c = make_inputs(cfg, 1)
    assert not np.array_equal(a["q"], c["q"])


def test_bf16_workload_values_are_representable():
    cfg = CONFIGS["video"].with_(H=2, n_kv=300, n_q=300)
    a = make_inputs(cfg, 0)
    for key in ("q", "k", "v"):
        assert np.array_equal(round_to_bf16(a[key]), a[key])
    np.testing.assert_allclose(np.linalg.norm(a["k"], axis=-1), 1.0, atol=1e-2)


def test_weights_repeat_over_batch():
    cfg = CONFIGS["lm32k"].with_(n_kv=64, n_q=64, d=64, h=64)
    a = make_inputs(cfg, 0)
    assert np.array_equal(a["W1"][0], a["W1"][4]) and not np.array_equal(a["W1"][0], a["W1"][1])
    sub = make_inputs(cfg, 0, heads=[5, 6])
    assert np.array_equal(sub["W2"][0], a["W2"][5])


def test_momentum_factor_draw():
    cfg = CONFIGS["lm32k_mom"].with_(n_kv=256, n_q=256, d=64, h=64)
    a = make_inputs(cfg, 0)
    b = make_inputs(cfg.with_(momentum=0), 0)
    assert "beta" not in b and a["beta"].shape == (16, 256) and a["beta"].dtype == np.float32
    assert np.all((a["beta"] > 0) & (a["beta"] < 1)) and abs(a["beta"].mean() - 0.5) < 0.02
    for key in b:                       # the other draws do not move
        assert np.array_equal(a[key], b[key])


def test_cotangent_draw():
    cfg = CONFIGS["lm32k"].with_(name="ct", B=1, H=2, d=64, h=64, n_kv=100, n_q=130, chunk=64, linear=1)
    a, b = make_cotangents(cfg, 5), make_cotangents(cfg, 5)
    assert a["do"].shape == (2, 130, 64) and a["dW"].shape == (2, 64, 64)
    assert np.array_equal(a["do"], b["do"]) and np.array_equal(a["dW"], b["dW"])
    assert np.array_equal(round_to_bf16(a["do"]), a["do"])
    assert not np.array_equal(make_cotangents(cfg, 6)["do"], a["do"])
    # the forward's inputs do not move when cotangents are drawn
    assert np.array_equal(make_inputs(cfg, 5)["q"], make_inputs(cfg, 5)["q"])
    assert abs(float(np.std(a["do"])) * 8.0 - 1.0) < 0.05
