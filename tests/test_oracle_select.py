"""Pins for the oracle's predictor and set selection (Sections 4.1-4.2, Algorithm 1).

Top-k is checked by brute force over every subset on tiny shapes, against
torch.topk where scores are distinct, and on ties. The threshold rule is checked by
its defining property and by invariance under a monotone map (the sigmoid).
The two-layer predictor is checked against a chain of nn.Linear maps and by
associativity, which catches a transposed factor.
"""
import itertools

import numpy as np
import pytest
import torch

from oracle import dejavu as O


@pytest.mark.parametrize("n,k", [(6, 2), (8, 3), (10, 5), (12, 1), (7, 7)])
def test_topk_maximises_score_sum_brute_force(n, k):
    rng = np.random.default_rng(n * 100 + k)
    s = rng.normal(size=n)
    best = max(itertools.combinations(range(n), k), key=lambda S: sum(s[i] for i in S))
    got = O.select_topk(s, k)
    assert list(got) == sorted(best)
    # Unique optimum when scores are distinct: every other subset is strictly worse.
    top = sum(s[i] for i in best)
    assert sum(1 for S in itertools.combinations(range(n), k)
               if abs(sum(s[i] for i in S) - top) < 1e-15) == 1


def test_topk_matches_torch_topk_on_distinct_scores():
    rng = np.random.default_rng(20)
    s = rng.normal(size=3000)
    ref = np.sort(torch.topk(torch.tensor(s), 307).indices.numpy())
    assert np.array_equal(O.select_topk(s, 307), ref)


def test_topk_ties_lower_index_wins_and_edge_sizes():
    s = np.array([1.0, 3.0, 2.0, 3.0, 2.0, 2.0, 0.0])
    assert list(O.select_topk(s, 1)) == [1]
    assert list(O.select_topk(s, 2)) == [1, 3]
    assert list(O.select_topk(s, 3)) == [1, 2, 3]
    assert list(O.select_topk(s, 4)) == [1, 2, 3, 4]
    assert list(O.select_topk(s, 0)) == []
    assert list(O.select_topk(s, 7)) == list(range(7))
    with pytest.raises(ValueError):
        O.select_topk(s, 8)


def test_threshold_rule_and_monotone_invariance():
    rng = np.random.default_rng(21)
    s = rng.normal(size=500)
    t = 0.8
    S = O.select_threshold(s, t)
    assert np.all(s[S] >= t)
    rest = np.setdiff1d(np.arange(500), S)
    assert np.all(s[rest] < t)
    sig = 1 / (1 + np.exp(-s))
    assert np.array_equal(O.select_threshold(sig, 1 / (1 + np.exp(-t))), S)
    assert np.array_equal(O.select_topk(sig, 40), O.select_topk(s, 40))
    # Inclusive at equality (Algorithm 1 labels m_r(x) >= t as positive).
    assert list(O.select_threshold(np.array([0.5, 0.2, 0.5]), 0.5)) == [0, 2]


def test_predictor_matches_linear_chain_and_associativity():
    rng = np.random.default_rng(22)
    d, r, n = 37, 11, 53
    AT = rng.normal(size=(r, d))
    BT = rng.normal(size=(n, r))
    x = rng.normal(size=d)
    # nn.Linear(d, r) has weight [r, d] = AT; nn.Linear(r, n) has weight [n, r] = BT.
    ref = torch.nn.functional.linear(torch.nn.functional.linear(torch.tensor(x), torch.tensor(AT)),
                                     torch.tensor(BT)).numpy()
    s = O.predictor_scores(x, AT, BT)
    assert s.shape == (n,)
    assert np.allclose(s, ref, rtol=1e-13, atol=1e-13)
    # (x A) B = x (A B), with A = AT^T and B = BT^T.
    assert np.allclose(s, x @ (AT.T @ BT.T), rtol=1e-12, atol=1e-12)
    # A one-hot input picks column j of A B.
    e = np.zeros(d)
    e[5] = 1.0
    assert np.allclose(O.predictor_scores(e, AT, BT), (AT.T @ BT.T)[5], rtol=1e-13, atol=1e-13)
    # Batched rows are independent.
    X = rng.normal(size=(3, d))
    Sb = O.predictor_scores(X, AT, BT)
    for b in range(3):
        assert np.allclose(Sb[b], O.predictor_scores(X[b], AT, BT), rtol=1e-13, atol=1e-13)
