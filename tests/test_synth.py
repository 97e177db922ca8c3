"""The seeded input generator: determinism, shapes, storage types and set recipes."""
import numpy as np
import torch

from synth import get_config, make_layer, uniform_head_sets, zipf_mlp_sets
from synth.gen import positions


def test_selection_sizes_follow_floor_rule():
    assert get_config("opt125m_b1").k_mlp == 307
    assert get_config("opt6.7b_b1").k_mlp == 1310
    assert get_config("opt66b_b1").k_mlp == 1843
    assert get_config("opt175b_b1").k_mlp == 2457


def test_layer_is_deterministic_and_typed():
    cfg = get_config("small_f16")
    a = make_layer(cfg, 3)
    b = make_layer(cfg, 3)
    c = make_layer(cfg, 4)
    for k in a:
        assert torch.equal(a[k], b[k]), k
    assert not torch.equal(a["W1T"], c["W1T"])
    assert a["W1T"].dtype == torch.float16 and a["x"].dtype == torch.float32
    assert a["K"].shape == (1, cfg.H, cfg.L, cfg.dh)
    assert a["BT_m"].shape == (cfg.N, cfg.r)
    assert int(a["pos"][0]) == cfg.L - 1
    # N(0, 0.02^2) weights
    assert abs(float(a["W1T"].float().std()) - 0.02) < 1e-3


def test_batch_sets_and_positions():
    cfg = get_config("opt175b_b32")
    pos = positions(cfg, 4)
    assert pos.shape == (32,) and pos.min() >= 511 and pos.max() <= 2047
    hs = uniform_head_sets(cfg, 4)
    assert hs.shape == (32, 32) and np.all(np.diff(hs, axis=1) > 0)
    ms = zipf_mlp_sets(cfg, 4)
    assert ms.shape == (32, 2457) and np.all(np.diff(ms, axis=1) > 0)
    U = np.unique(ms)
    # Zipf-skewed popularity: the union is far below the uniform expectation
    # (about 1 - (1 - 0.05)^32 = 81 % of N) yet far above one set.
    assert 2457 * 4 < U.size < 0.7 * cfg.N
    assert np.array_equal(zipf_mlp_sets(cfg, 4), ms)
