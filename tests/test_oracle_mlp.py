"""Pins for the oracle's sparsified MLP (Eq. (1), Section 2.3).

Each check ties the oracle to something other than itself: the dense computation
(full index set), a second formulation (mask form), additivity over disjoint sets,
exact no-op of ReLU-zero neurons, a library routine for the dense layer, brute force
over every subset on a tiny shape, and the folded-Gaussian fact of Appendix G.3.
"""
import itertools

import numpy as np
import pytest
import torch

from oracle import dejavu as O


def _mlp(rng, d, N, bias=True):
    W1T = rng.normal(0, 0.02, (N, d))
    W2T = rng.normal(0, 0.02, (N, d))
    b1 = rng.normal(0, 0.02, N) if bias else None
    b2 = rng.normal(0, 0.02, d) if bias else None
    y = rng.normal(0, 1.0, d)
    return y, W1T, b1, W2T, b2


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


@pytest.mark.parametrize("bias", [False, True])
def test_full_set_equals_dense(bias):
    rng = np.random.default_rng(1)
    y, W1T, b1, W2T, b2 = _mlp(rng, 40, 96, bias)
    full = O.mlp_sparse(y, W1T, b1, W2T, b2, np.arange(96))
    dense = O.mlp_dense(y, W1T, b1, W2T, b2)
    assert _rel(full, dense) < 1e-12


def test_dense_matches_torch_linear_relu():
    rng = np.random.default_rng(2)
    y, W1T, b1, W2T, b2 = _mlp(rng, 33, 70)
    # torch.nn.functional.linear(x, W, b) = x W^T + b; the second layer's weight in
    # nn.Linear layout is W^2 = W2T^T.
    t = torch.nn.functional.linear(torch.tensor(y), torch.tensor(W1T), torch.tensor(b1))
    t = torch.nn.functional.linear(torch.relu(t), torch.tensor(W2T.T.copy()), torch.tensor(b2))
    assert _rel(O.mlp_dense(y, W1T, b1, W2T, b2), t.numpy()) < 1e-13


def test_gather_form_equals_mask_form():
    rng = np.random.default_rng(3)
    y, W1T, b1, W2T, b2 = _mlp(rng, 64, 200)
    S = np.sort(rng.choice(200, 37, replace=False))
    assert _rel(O.mlp_sparse(y, W1T, b1, W2T, b2, S),
                O.mlp_sparse_masked(y, W1T, b1, W2T, b2, S)) < 1e-13


def test_additivity_over_disjoint_sets_and_empty_set():
    rng = np.random.default_rng(4)
    y, W1T, b1, W2T, b2 = _mlp(rng, 48, 120)
    perm = rng.permutation(120)
    S1, S2 = np.sort(perm[:30]), np.sort(perm[30:75])
    f1 = O.mlp_sparse(y, W1T, b1, W2T, b2, S1)
    f2 = O.mlp_sparse(y, W1T, b1, W2T, b2, S2)
    f12 = O.mlp_sparse(y, W1T, b1, W2T, b2, np.sort(np.concatenate([S1, S2])))
    assert _rel(f12, f1 + f2 - b2) < 1e-12
    assert np.array_equal(O.mlp_sparse(y, W1T, b1, W2T, b2, []), b2)


def test_relu_zero_neuron_is_an_exact_noop():
    rng = np.random.default_rng(5)
    y, W1T, b1, W2T, b2 = _mlp(rng, 32, 64)
    z = W1T @ y + b1
    dead = np.nonzero(z <= 0)[0]
    live = np.nonzero(z > 0)[0]
    S = np.sort(live[:10])
    base = O.mlp_sparse(y, W1T, b1, W2T, b2, S)
    Splus = np.sort(np.concatenate([S, dead[:5]]))
    assert O.mlp_sparse(y, W1T, b1, W2T, b2, Splus).tobytes() == base.tobytes()


def test_neuron_order_changes_only_rounding():
    rng = np.random.default_rng(6)
    y, W1T, b1, W2T, b2 = _mlp(rng, 32, 64)
    S = np.arange(0, 64, 3)
    a = O.mlp_sparse(y, W1T, b1, W2T, b2, S)
    b = O.mlp_sparse(y, W1T, b1, W2T, b2, S[::-1])
    assert _rel(a, b) < 1e-14


def test_brute_force_every_subset_tiny():
    """d = N = 8: for all 2^8 subsets, gather = mask = b2 + sum of single-neuron terms.

    Includes the structure of the worked diagram in Appendix D (neurons {0, 2}).
    """
    rng = np.random.default_rng(7)
    y, W1T, b1, W2T, b2 = _mlp(rng, 8, 8)
    singles = [O.mlp_sparse(y, W1T, b1, W2T, b2, [i]) - b2 for i in range(8)]
    for m in range(1 << 8):
        S = [i for i in range(8) if m >> i & 1]
        g = O.mlp_sparse(y, W1T, b1, W2T, b2, S)
        k = O.mlp_sparse_masked(y, W1T, b1, W2T, b2, S)
        ref = b2 + sum((singles[i] for i in S), np.zeros(8))
        assert np.allclose(g, k, rtol=0, atol=1e-15)
        assert np.allclose(g, ref, rtol=0, atol=1e-15)
    # The Appendix D example selects neurons {0, 2}.
    acts = O.mlp_activations(y, W1T, b1, [0, 2])
    expect = b2 + acts[0] * W2T[0] + acts[1] * W2T[2]
    assert np.allclose(O.mlp_sparse(y, W1T, b1, W2T, b2, [0, 2]), expect, rtol=0, atol=1e-15)


def test_best_k_subset_objective_tiny():
    """The Section 2.3 objective on a tiny shape: argmin over |S| = k of ||F_S - F||.

    A diagnostic of the definitions, not a parity target: with ReLU, keeping every
    active neuron reproduces the dense output exactly, so when k >= #active the
    optimum has zero error.
    """
    rng = np.random.default_rng(8)
    y, W1T, b1, W2T, b2 = _mlp(rng, 8, 8)
    full = O.mlp_dense(y, W1T, b1, W2T, b2)
    active = int(np.sum(W1T @ y + b1 > 0))
    k = max(active, 1)
    best = min(np.linalg.norm(O.mlp_sparse(y, W1T, b1, W2T, b2, S) - full)
               for S in itertools.combinations(range(8), k))
    assert best < 1e-15


def test_folded_gaussian_fact_half_of_relu_outputs_are_zero():
    """Fact in Appendix G.3: with Gaussian weights about half the ReLU outputs are 0."""
    rng = np.random.default_rng(9)
    d, N = 256, 20000
    W1T = rng.normal(0, 0.02, (N, d))
    y = rng.normal(0, 1.0, d)
    frac0 = np.mean(W1T @ y <= 0)
    sd = np.sqrt(0.25 / N)
    assert abs(frac0 - 0.5) < 5 * sd


# ---------------------------------------------------------------- GeLU, W4A16
def test_gelu_matches_torch_exact_gelu():
    z = np.linspace(-6, 6, 241)
    ref = torch.nn.functional.gelu(torch.tensor(z, dtype=torch.float64), approximate="none").numpy()
    assert np.allclose(O.activation(z, "gelu"), ref, rtol=1e-14, atol=1e-15)
    assert np.array_equal(O.activation(z, "relu"), np.maximum(z, 0))


@pytest.mark.parametrize("act", ["relu", "gelu"])
def test_gelu_mlp_forms_agree_and_match_torch(act):
    rng = np.random.default_rng(60)
    y, W1T, b1, W2T, b2 = _mlp(rng, 24, 40)
    W1T, W2T = W1T * 50, W2T * 50       # pre-activations of order 1: GeLU away from its linear part
    S = np.sort(rng.choice(40, 13, replace=False))
    assert _rel(O.mlp_sparse(y, W1T, b1, W2T, b2, S, act), O.mlp_sparse_masked(y, W1T, b1, W2T, b2, S, act)) < 1e-13
    assert _rel(O.mlp_sparse(y, W1T, b1, W2T, b2, range(40), act), O.mlp_dense(y, W1T, b1, W2T, b2, act)) < 1e-13
    f = torch.nn.functional
    h = f.linear(torch.tensor(y), torch.tensor(W1T), torch.tensor(b1))
    h = f.gelu(h, approximate="none") if act == "gelu" else f.relu(h)
    ref = (h @ torch.tensor(W2T) + torch.tensor(b2)).numpy()
    assert _rel(O.mlp_dense(y, W1T, b1, W2T, b2, act), ref) < 1e-13


def test_dequant_q4_hand_values():
    """Byte 0x80 holds q = 0 (low nibble, even element) and q = 8 (high nibble): -8 s, 0.
    Byte 0xF3: q = 3 then 15: -5 s, 7 s. The second block of 32 uses its own scale."""
    packed = np.zeros((1, 32), dtype=np.uint8)       # d = 64: two blocks
    packed[0, 0] = 0x80
    packed[0, 1] = 0xF3
    packed[0, 16] = 0x9A                              # element 32: q = 10, element 33: q = 9
    packed[0, 2:16] = 0x88
    packed[0, 17:] = 0x88
    scales = np.array([[0.5, 2.0]], dtype=np.float16)
    w = O.dequant_q4(packed, scales, 64)[0]
    assert w[:4].tolist() == [-4.0, 0.0, -2.5, 3.5]
    assert w[32:34].tolist() == [4.0, 2.0]
    assert np.count_nonzero(w) == 5


def test_quantizer_and_dequant_round_trip_within_half_a_step():
    """synth.quantize_q4 (the input format) against the oracle's dequantisation: every
    weight is reproduced within half its block's step (round to nearest), codes fit 4
    bits, and the largest magnitude of each block maps to +-7 steps."""
    from synth import quantize_q4
    rng = np.random.default_rng(61)
    W = torch.tensor(rng.normal(0, 0.02, (5, 96)), dtype=torch.float16)
    packed, scales = quantize_q4(W)
    assert packed.dtype == torch.uint8 and packed.shape == (5, 48) and scales.shape == (5, 3)
    deq = O.dequant_q4(packed.numpy(), scales.numpy(), 96)
    step = np.repeat(scales.numpy().astype(np.float64), 32, axis=1)
    err = np.abs(deq - W.numpy().astype(np.float64))
    assert (err <= 0.5 * step * (1 + 1e-3) + 1e-12).all()
    assert np.allclose(np.abs(deq).reshape(5, 3, 32).max(axis=-1), 7 * scales.numpy().astype(np.float64))
    assert np.array_equal(O.dequant_q4_rows(packed.numpy(), scales.numpy(), 96, [3, 1]), deq[[3, 1]])
