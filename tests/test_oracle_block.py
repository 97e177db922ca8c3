"""Pins for the oracle's layer norm, layer recurrences (Section 4.3, Appendix C.3) and batch union.

Layer norm against torch; the sparse layer with every head and neuron selected
against the dense layer; predicted sets against explicitly passed ones; look-ahead vs
sequential inputs to the neuron predictor; the union of Section 5.2 / Appendix C.1.
"""
import numpy as np
import pytest
import torch

from oracle import dejavu as O


def _layer(rng, d=24, N=48, H=4, dh=6, cap=9, r=5):
    attn = {n: rng.normal(0, 0.2, (H * dh, d)) for n in ("Wq", "Wk", "Wv", "WoT")}
    attn.update(bq=rng.normal(0, 0.1, H * dh), bk=rng.normal(0, 0.1, H * dh),
                bv=rng.normal(0, 0.1, H * dh), bo=rng.normal(0, 0.1, d))
    mlp = dict(W1T=rng.normal(0, 0.2, (N, d)), b1=rng.normal(0, 0.1, N),
               W2T=rng.normal(0, 0.2, (N, d)), b2=rng.normal(0, 0.1, d))
    K = rng.normal(size=(H, cap, dh))
    V = rng.normal(size=(H, cap, dh))
    ph = dict(AT=rng.normal(size=(r, d)), BT=rng.normal(size=(H, r)))
    pm = dict(AT=rng.normal(size=(r, d)), BT=rng.normal(size=(N, r)))
    ln = dict(g1=1 + rng.normal(0, 0.1, d), be1=rng.normal(0, 0.1, d),
              g2=1 + rng.normal(0, 0.1, d), be2=rng.normal(0, 0.1, d), eps=1e-5)
    return attn, mlp, K, V, ph, pm, ln


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def test_layer_norm_matches_torch_and_none_is_identity():
    rng = np.random.default_rng(30)
    x = rng.normal(3.0, 2.0, (4, 50))
    g = rng.normal(1, 0.1, 50)
    b = rng.normal(0, 0.1, 50)
    ref = torch.nn.functional.layer_norm(torch.tensor(x), (50,), torch.tensor(g), torch.tensor(b),
                                         eps=1e-5).numpy()
    assert np.allclose(O.layer_norm(x, g, b, 1e-5), ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(O.layer_norm(x, None, None), x)


def test_full_sets_reproduce_dense_recurrence():
    rng = np.random.default_rng(31)
    attn, mlp, K, V, _, _, ln = _layer(rng)
    y = rng.normal(size=24)
    for lnx in (None, ln):
        sp = O.sparse_block(y, attn, mlp, K, V, 6, 0.4, S_A=np.arange(4), S_M=np.arange(48), ln=lnx)
        dense = O.dense_block(y, attn, mlp, K, V, 6, 0.4, ln=lnx)
        assert _rel(sp["out"], dense) < 1e-13
    # Without normalisation the layer is literally y + MHA(y), then + MLP(y~).
    sp = O.sparse_block(y, attn, mlp, K, V, 6, 0.4, S_A=np.arange(4), S_M=np.arange(48))
    yt = y + O.mha_dense_einsum(y, attn, K, V, 6, 0.4)
    assert _rel(sp["out"], yt + O.mlp_dense(yt, mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"])) < 1e-13


@pytest.mark.parametrize("mode", ["lookahead", "sequential"])
def test_predicted_sets_equal_explicit_sets(mode):
    rng = np.random.default_rng(32)
    attn, mlp, K, V, ph, pm, ln = _layer(rng)
    y = rng.normal(size=24)
    r = O.sparse_block(y, attn, mlp, K, V, 8, 0.4, pred_h=ph, pred_m=pm, k_heads=2, k_mlp=10,
                       ln=ln, mode=mode)
    assert len(r["S_A"]) == 2 and len(r["S_M"]) == 10
    assert np.all(np.diff(r["S_A"]) > 0) and np.all(np.diff(r["S_M"]) > 0)
    x1 = O.layer_norm(y, ln["g1"], ln["be1"])
    src = x1 if mode == "lookahead" else O.layer_norm(r["y_tilde"], ln["g2"], ln["be2"])
    assert np.array_equal(r["S_M"], O.select_topk(O.predictor_scores(src, pm["AT"], pm["BT"]), 10))
    assert np.array_equal(r["S_A"], O.select_topk(O.predictor_scores(x1, ph["AT"], ph["BT"]), 2))
    again = O.sparse_block(y, attn, mlp, K, V, 8, 0.4, S_A=r["S_A"], S_M=r["S_M"], ln=ln)
    assert np.array_equal(again["out"], r["out"])


def test_union_and_batched_forms():
    rng = np.random.default_rng(33)
    attn, mlp, K, V, _, _, _ = _layer(rng)
    Y = rng.normal(size=(3, 24))
    sets = [np.sort(rng.choice(48, 7, replace=False)) for _ in range(3)]
    U = O.union_of_sets(sets)
    assert np.array_equal(U, np.unique(np.concatenate(sets)))
    un = O.mlp_batch(Y, mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], sets, "union")
    mk = O.mlp_batch(Y, mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], sets, "masked")
    for b in range(3):
        assert _rel(un[b], O.mlp_sparse_masked(Y[b], mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], U)) < 1e-13
        assert _rel(mk[b], O.mlp_sparse_masked(Y[b], mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], sets[b])) < 1e-13
    Kb = np.stack([K, K * 0.5, -K])
    Vb = np.stack([V, V, V * 2])
    hs = [[0, 2], [1], [3, 1]]
    out, Kn, _ = O.mha_batch(Y, attn, Kb, Vb, [3, 8, 0], [sorted(h) for h in hs], 0.3)
    for b, p in enumerate([3, 8, 0]):
        ref, Kr, _, _ = O.mha_sparse(Y[b], attn, Kb[b], Vb[b], p, sorted(hs[b]), 0.3)
        assert np.array_equal(out[b], ref) and np.array_equal(Kn[b], Kr)


@pytest.mark.parametrize("step", [1, 5, 2048])
def test_union_rows_matrix_form_equals_gather_form(step):
    """mlp_union_rows (slices of neurons as matrix products, the form used to check the
    batch-32 union MLP at full size) against mlp_sparse one neuron at a time, and against
    the mask form; a dropped bias, a wrong slice bound or a transposed factor would
    differ."""
    rng = np.random.default_rng(34)
    _, mlp, *_ = _layer(rng, N=48)
    Y = rng.normal(size=(5, 24))
    sets = [np.sort(rng.choice(48, 9, replace=False)) for _ in range(5)]
    U = O.union_of_sets(sets)
    got = O.mlp_union_rows(Y, mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], U, rows_per_step=step)
    for b in range(5):
        ref = O.mlp_sparse(Y[b], mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], U)
        assert _rel(got[b], ref) < 1e-13
        assert _rel(got[b], O.mlp_sparse_masked(Y[b], mlp["W1T"], mlp["b1"], mlp["W2T"], mlp["b2"], U)) < 1e-13
    # no biases, fp16 storage: the rows are upcast exactly
    W1 = mlp["W1T"].astype(np.float16)
    W2 = mlp["W2T"].astype(np.float16)
    got = O.mlp_union_rows(Y, W1, None, W2, None, U, rows_per_step=step)
    assert _rel(got[2], O.mlp_sparse(Y[2], W1, None, W2, None, U)) < 1e-13
    # the empty union leaves b2
    assert np.array_equal(O.mlp_union_rows(Y, W1, None, W2, mlp["b2"], [])[3], mlp["b2"])


def _stack(rng, L, **kw):
    layers = []
    for _ in range(L):
        attn, mlp, K, V, ph, pm, ln = _layer(rng, **kw)
        layers.append(dict(attn=attn, mlp=mlp, K=K, V=V, pos=6, pred_h=ph, pred_m=pm, ln=ln))
    return layers


def test_lookahead_one_layer_is_the_single_layer_call():
    """With one layer the look-ahead recurrence is the single-layer look-ahead call:
    both sets from LN1(y) of that layer (reading R8)."""
    rng = np.random.default_rng(35)
    (lay,) = _stack(rng, 1)
    y = rng.normal(size=24)
    r = O.lookahead_layers(y, [lay], 0.4, 2, 9)
    ref = O.sparse_block(y, lay["attn"], lay["mlp"], lay["K"], lay["V"], 6, 0.4, pred_h=lay["pred_h"],
                         pred_m=lay["pred_m"], k_heads=2, k_mlp=9, ln=lay["ln"], mode="lookahead")
    assert np.array_equal(r["out"], ref["out"])
    assert np.array_equal(r["S_A"][0], ref["S_A"]) and np.array_equal(r["S_M"][0], ref["S_M"])
    assert np.array_equal(r["K_new"][0], ref["K_new"])


@pytest.mark.parametrize("L", [2, 4])
def test_lookahead_full_sets_are_the_dense_recurrence(L):
    """Every head and neuron selected: L look-ahead layers equal L dense layers applied in
    turn, each on its own cache."""
    rng = np.random.default_rng(36)
    layers = _stack(rng, L)
    y = rng.normal(size=24)
    r = O.lookahead_layers(y, layers, 0.4, 4, 48)
    ref = y
    for lay in layers:
        ref = O.dense_block(ref, lay["attn"], lay["mlp"], lay["K"], lay["V"], 6, 0.4, ln=lay["ln"])
    assert _rel(r["out"], ref) < 1e-12
    assert len(r["y"]) == L + 1 and np.array_equal(r["y"][0], y)


def test_lookahead_sets_come_from_the_previous_layers_input():
    """A construction whose sets are known in closed form: each predictor reads
    coordinates 0-3 of its input (AT selects them, BT is the identity), so its top-2 are
    the two largest of those coordinates. y_0 ranks coordinates 0, 1 first; layer 0's
    MLP bias flips the order, so y_1 ranks 2, 3 first. S^1 is predicted from layer 0's
    input, hence {0, 1}; S^2 from layer 1's input, hence {2, 3}. (A predictor fed the
    layer's own input would give {2, 3} for S^1.)"""
    rng = np.random.default_rng(37)
    layers = _stack(rng, 3, d=24, N=4, H=4, dh=6, r=4)
    for l, lay in enumerate(layers):
        for p in ("pred_h", "pred_m"):
            AT = np.zeros((4, 24))
            AT[np.arange(4), np.arange(4)] = 1.0
            lay[p] = dict(AT=AT, BT=np.eye(4))
        for n in ("Wq", "Wk", "Wv", "WoT"):
            lay["attn"][n] = lay["attn"][n] * 1e-3
        lay["attn"]["bo"] = np.zeros(24)
        lay["mlp"]["W2T"] = lay["mlp"]["W2T"] * 1e-3
        lay["mlp"]["b2"] = np.zeros(24)
        lay["ln"].update(g1=np.ones(24), be1=np.zeros(24))
    layers[0]["mlp"]["b2"][:4] = [-20.0, -20.0, 20.0, 20.0]
    y = np.concatenate([[5.0, 4.0, -3.0, -4.0], rng.normal(0, 0.1, 20)])
    r = O.lookahead_layers(y, layers, 0.4, 2, 2)
    want = [[0, 1], [0, 1], [2, 3]]
    assert [s.tolist() for s in r["S_A"]] == want
    assert [s.tolist() for s in r["S_M"]] == want
    assert np.argsort(-r["y"][1][:4])[:2].tolist() == [2, 3]
