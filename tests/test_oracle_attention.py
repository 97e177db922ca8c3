"""Pins for the oracle's sparsified MHA (Eq. (2) and D_i, Section 2.3; KV step of Section 4.2).

Closed forms (one token, equal keys, zero scale, one-hot query on orthogonal keys),
a library routine (torch's scaled-dot-product attention in float64 on the CPU), an
independent dense formulation (einsum over all heads), additivity over head sets,
brute force over every head subset on a tiny shape, and the cache contract.
"""
import numpy as np
import pytest
import torch

from oracle import dejavu as O


def _attn(rng, d, H, dh, bias=True):
    a = {n: rng.normal(0, 0.3, (H * dh, d)) for n in ("Wq", "Wk", "Wv", "WoT")}
    if bias:
        for n in ("bq", "bk", "bv"):
            a[n] = rng.normal(0, 0.1, H * dh)
        a["bo"] = rng.normal(0, 0.1, d)
    return a


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def test_single_token_returns_value():
    rng = np.random.default_rng(10)
    q, k, v = rng.normal(size=(3, 16))
    out = O.attention_head(q, k[None], v[None], 0.25)
    assert np.allclose(out, v, rtol=0, atol=1e-15)


def test_equal_keys_and_zero_scale_give_mean_value():
    rng = np.random.default_rng(11)
    q = rng.normal(size=8)
    V = rng.normal(size=(9, 8))
    K_eq = np.tile(rng.normal(size=8), (9, 1))
    assert np.allclose(O.attention_head(q, K_eq, V, 0.7), V.mean(0), rtol=0, atol=1e-14)
    K = rng.normal(size=(9, 8))
    assert np.allclose(O.attention_head(q, K, V, 0.0), V.mean(0), rtol=0, atol=1e-14)


def test_one_hot_query_on_orthogonal_keys():
    """q = e_m, keys c*e_t: only key m scores c*scale, the n-1 others score 0."""
    n, c, scale = 6, 3.0, 0.5
    K = c * np.eye(n)
    V = np.arange(n * n, dtype=float).reshape(n, n)
    q = np.zeros(n)
    q[2] = 1.0
    big = np.exp(c * scale)
    p = np.full(n, 1.0 / (big + n - 1))
    p[2] = big / (big + n - 1)
    assert np.allclose(O.attention_head(q, K, V, scale), p @ V, rtol=1e-14, atol=0)


@pytest.mark.parametrize("scale", [1.0, 0.125])
def test_head_matches_torch_sdpa(scale):
    rng = np.random.default_rng(12)
    q = rng.normal(size=32)
    K = rng.normal(size=(50, 32))
    V = rng.normal(size=(50, 32))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q)[None, None], torch.tensor(K)[None], torch.tensor(V)[None], scale=scale)
    assert _rel(O.attention_head(q, K, V, scale), ref[0, 0].numpy()) < 1e-13


def test_all_heads_equal_dense_einsum_and_cache_update():
    rng = np.random.default_rng(13)
    d, H, dh, cap, pos = 24, 4, 6, 10, 7
    a = _attn(rng, d, H, dh)
    K = rng.normal(size=(H, cap, dh))
    V = rng.normal(size=(H, cap, dh))
    y = rng.normal(size=d)
    out, Kn, Vn, heads = O.mha_sparse(y, a, K, V, pos, range(H), 1 / np.sqrt(dh))
    dense = O.mha_dense_einsum(y, a, K, V, pos, 1 / np.sqrt(dh))
    assert _rel(out, dense) < 1e-13
    # Rows other than pos are untouched; row pos holds the fresh keys/values.
    mask = np.ones(cap, bool)
    mask[pos] = False
    assert np.array_equal(Kn[:, mask], K[:, mask]) and np.array_equal(Vn[:, mask], V[:, mask])
    for i in range(H):
        assert np.allclose(Kn[i, pos], a["Wk"][i * dh:(i + 1) * dh] @ y + a["bk"][i * dh:(i + 1) * dh])


def test_non_selected_heads_keep_their_cache_rows():
    rng = np.random.default_rng(14)
    d, H, dh, cap, pos = 16, 5, 4, 8, 3
    a = _attn(rng, d, H, dh)
    K = rng.normal(size=(H, cap, dh))
    V = rng.normal(size=(H, cap, dh))
    _, Kn, Vn, _ = O.mha_sparse(rng.normal(size=d), a, K, V, pos, [1, 4], 0.5)
    for i in (0, 2, 3):
        assert Kn[i].tobytes() == K[i].tobytes() and Vn[i].tobytes() == V[i].tobytes()


def test_head_additivity_and_brute_force_tiny():
    """H = 4: every head subset equals bo + the sum of its single-head terms.

    Includes the Appendix D diagram's head set {0, 3}.
    """
    rng = np.random.default_rng(15)
    d, H, dh, cap, pos = 8, 4, 2, 3, 2
    a = _attn(rng, d, H, dh)
    K = rng.normal(size=(H, cap, dh))
    V = rng.normal(size=(H, cap, dh))
    y = rng.normal(size=d)
    singles = [O.mha_sparse(y, a, K, V, pos, [i], 0.7)[0] - a["bo"] for i in range(H)]
    for m in range(1 << H):
        S = [i for i in range(H) if m >> i & 1]
        out = O.mha_sparse(y, a, K, V, pos, S, 0.7)[0]
        assert np.allclose(out, a["bo"] + sum((singles[i] for i in S), np.zeros(d)),
                           rtol=0, atol=1e-13)
    out03, _, _, heads = O.mha_sparse(y, a, K, V, pos, [0, 3], 0.7)
    expect = a["bo"] + heads[0] @ a["WoT"][0:2] + heads[3] @ a["WoT"][6:8]
    assert np.allclose(out03, expect, rtol=0, atol=1e-14)


def test_pos_zero_attends_only_the_fresh_token():
    rng = np.random.default_rng(16)
    d, H, dh, cap = 12, 3, 4, 5
    a = _attn(rng, d, H, dh, bias=False)
    K = rng.normal(size=(H, cap, dh))
    V = rng.normal(size=(H, cap, dh))
    y = rng.normal(size=d)
    out, _, _, heads = O.mha_sparse(y, a, K, V, 0, [2], 1.0)
    v2 = a["Wv"][8:12] @ y
    assert np.allclose(heads[2], v2, rtol=0, atol=1e-14)
    assert np.allclose(out, v2 @ a["WoT"][8:12], rtol=0, atol=1e-14)


def _kv_layer(rng, d=16, H=5, dh=4, cap=12):
    attn = {n: rng.normal(0, 0.3, (H * dh, d)) for n in ("Wq", "Wk", "Wv", "WoT")}
    attn.update(bq=rng.normal(0, 0.1, H * dh), bk=rng.normal(0, 0.1, H * dh), bv=rng.normal(0, 0.1, H * dh),
                bo=rng.normal(0, 0.1, d))
    return attn


def test_kvfill_decode_equals_a_run_with_every_heads_cache_written():
    """Section 4.2's missing-KV rule over 10 tokens with changing head sets: each step's
    output is the output of a run in which every head's key and value were written at
    every token (same arithmetic, computed when the head is next selected instead of
    at its own token), bit for bit; and every selected head's cache is complete."""
    rng = np.random.default_rng(40)
    d, H, dh, cap, T = 16, 5, 4, 12, 10
    attn = _kv_layer(rng, d, H, dh, cap)
    K = np.zeros((H, cap, dh))
    V = np.zeros((H, cap, dh))
    Y = np.zeros((cap, d))
    valid = np.zeros((H, cap), dtype=bool)
    Kf, Vf = K.copy(), V.copy()                       # the reference: all heads written
    for pos in range(T):
        y = rng.normal(size=d)
        S = np.sort(rng.choice(H, 2, replace=False))
        out, K, V, Y, valid = O.mha_sparse_kvfill(y, attn, K, V, Y, valid, pos, S, 0.5)
        _, Kf, Vf, _ = O.mha_sparse(y, attn, Kf, Vf, pos, range(H), 0.5)   # writes all heads' rows
        ref, _, _, _ = O.mha_sparse(y, attn, Kf, Vf, pos, S, 0.5)
        assert np.array_equal(out, ref), pos
        for h in S:
            assert valid[h, :pos + 1].all()
            assert np.array_equal(K[h, :pos + 1], Kf[h, :pos + 1]) and np.array_equal(V[h, :pos + 1], Vf[h, :pos + 1])
        for h in set(range(H)) - set(S.tolist()):
            assert not valid[h, pos]
        assert np.array_equal(Y[pos], y)


def test_kvfill_with_a_complete_cache_is_the_plain_sparse_attention():
    """Nothing missing: the rule reduces to mha_sparse (nothing recomputed)."""
    rng = np.random.default_rng(41)
    attn = _kv_layer(rng)
    K = rng.normal(size=(5, 12, 4))
    V = rng.normal(size=(5, 12, 4))
    Y = rng.normal(size=(12, 16))
    valid = np.ones((5, 12), dtype=bool)
    y = rng.normal(size=16)
    out, Kn, Vn, Yn, vn = O.mha_sparse_kvfill(y, attn, K, V, Y, valid, 7, [1, 3], 0.5)
    ref, Kr, Vr, _ = O.mha_sparse(y, attn, K, V, 7, [1, 3], 0.5)
    assert np.array_equal(out, ref) and np.array_equal(Kn, Kr) and np.array_equal(Vn, Vr)
    assert np.array_equal(Yn[:7], Y[:7]) and vn[[1, 3], 7].all() and not vn[[0, 2, 4], 7].any()


def test_kvfill_only_touches_missing_rows_of_selected_heads():
    """A missing row is recomputed from the kept input of its own token, and only for a
    selected head; present rows are never rewritten (they keep whatever they hold)."""
    rng = np.random.default_rng(42)
    attn = _kv_layer(rng)
    K = np.full((5, 12, 4), 7.0)
    V = np.full((5, 12, 4), -7.0)
    Y = rng.normal(size=(12, 16))
    valid = np.ones((5, 12), dtype=bool)
    valid[2, 3] = valid[4, 5] = False
    y = rng.normal(size=16)
    _, Kn, Vn, _, vn = O.mha_sparse_kvfill(y, attn, K, V, Y, valid, 6, [2], 0.5)
    k3 = (np.asarray(attn["Wk"])[8:12] @ Y[3]) + attn["bk"][8:12]
    assert np.allclose(Kn[2, 3], k3, rtol=1e-14) and vn[2, 3]
    assert (Kn[4, 5] == 7.0).all() and not vn[4, 5]                  # head 4 not selected: still missing
    rows = [(h, t) for h in range(5) for t in range(6) if (h, t) != (2, 3)]
    assert all((Kn[h, t] == 7.0).all() and (Vn[h, t] == -7.0).all() for h, t in rows)


def test_kvfill_keeps_the_input_in_the_storage_type():
    """Reading R18: with a half-precision keep, Y[pos] is the input rounded to the
    nearest half (ties to even, checked on values exactly between two halves), and a
    row filled later is the projection of that rounded input, not of the exact one."""
    rng = np.random.default_rng(43)
    attn = _kv_layer(rng)
    H, cap, dh, d = 5, 12, 4, 16
    K = np.zeros((H, cap, dh))
    V = np.zeros((H, cap, dh))
    Y = np.zeros((cap, d))
    valid = np.zeros((H, cap), dtype=bool)
    y = rng.normal(size=d)
    y[0] = 1.0 + 2.0 ** -11          # halfway between 1 and 1 + 2^-10: ties to even, 1.0
    y[1] = 1.0 + 3.0 * 2.0 ** -11    # halfway between 1 + 2^-10 and 1 + 2^-9: ties to even, 1 + 2^-9
    _, K, V, Y, valid = O.mha_sparse_kvfill(y, attn, K, V, Y, valid, 0, [0], 0.5, y_keep=np.float16)
    assert Y[0, 0] == 1.0 and Y[0, 1] == 1.0 + 2.0 ** -9
    assert np.array_equal(Y[0], y.astype(np.float16).astype(np.float64))
    assert (np.abs(Y[0] - y) <= 2.0 ** -11 * np.maximum(np.abs(y), 2.0 ** -14)).all()   # half an ulp
    # head 3 was not selected at token 0; at token 1 it is, and fills row 0 from Y[0]
    y1 = rng.normal(size=d)
    _, K, V, Y, valid = O.mha_sparse_kvfill(y1, attn, K, V, Y, valid, 1, [3], 0.5, y_keep=np.float16)
    k0 = np.asarray(attn["Wk"])[12:16] @ Y[0] + attn["bk"][12:16]
    k0_exact = np.asarray(attn["Wk"])[12:16] @ y + attn["bk"][12:16]
    assert np.allclose(K[3, 0], k0, rtol=1e-14) and not np.allclose(K[3, 0], k0_exact, rtol=1e-9)
