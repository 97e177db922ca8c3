"""GPU parity of the batched path (B > 1 sequences, one token each, on the matrix cores)
against the fp64 oracle on the same seeded inputs.

The MLP runs on the union of the sequences' neuron sets (Section 5.2) or, masked, on
each sequence's own set; attention keeps a head set, a cache and a position per
sequence. Outputs: max relative L2 error <= 2e-3 per sequence. The batched path rounds
its MFMA operands (x-hat, ReLU outputs, attention outputs) to fp16, whose relative
error (2^-11 per operand, uncorrelated over thousands of terms) stays an order of
magnitude inside that bound. Cache rows of non-selected heads stay bit-identical.
"""
import numpy as np
import pytest
import torch

from oracle import dejavu as O
from paper_2310_17157_amd import binding as Bd
from paper_2310_17157_amd.workload import layer_objects
from synth import get_config, make_layer, uniform_head_sets, zipf_mlp_sets
from tests.gpu_util import REL_TOL, check_topk_set, host, oracle_attn, oracle_ln, oracle_mlp, rel_l2

pytestmark = pytest.mark.gpu


def _sync():
    torch.cuda.synchronize()


def _cfg(name, B=None):
    cfg = get_config(name)
    if B is not None and B != cfg.B:
        cfg = cfg.with_(B=B, name=f"{cfg.name}_B{B}")
    return cfg


def _mlp(t, biases=True):
    return Bd.MLP(t["W1T"], t["W2T"], t["b1"] if biases else None, t["b2"] if biases else None)


# ------------------------------------------------------------------------ MLP
@pytest.mark.parametrize("B", [2, 8, 17, 32])
@pytest.mark.parametrize("mode", ["union", "masked"])
def test_batch_mlp_per_sequence_sets(B, mode):
    cfg = _cfg("small_b8", B)
    t = make_layer(cfg, 21, device="cuda", biases=True, with_predictors=False)
    sets = zipf_mlp_sets(cfg, 21)
    idx = torch.tensor(sets, dtype=torch.int32, device="cuda")
    bm = Bd.DV_MLP_UNION if mode == "union" else Bd.DV_MLP_MASKED
    out = Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1, batch_mode=bm, flags=Bd.DV_VALIDATE)
    _sync()
    m = oracle_mlp(t)
    ref = O.mlp_batch(host(t["x"]), m["W1T"], m["b1"], m["W2T"], m["b2"], [s.tolist() for s in sets], mode)
    got = host(out)
    for b in range(B):
        assert rel_l2(got[b], ref[b]) < REL_TOL, (b, rel_l2(got[b], ref[b]))


@pytest.mark.parametrize("offset", [1, 2, 3])
@pytest.mark.parametrize("mode", ["union", "masked"])
def test_batch_mlp_sets_at_any_word_offset(offset, mode):
    """Index sets that start 4, 8 or 12 bytes into a 16-byte block (a view into a larger
    buffer) give the same output, bit for bit, as the same sets at an aligned address."""
    cfg = _cfg("small_b8", 17)
    t = make_layer(cfg, 26, device="cuda", biases=True, with_predictors=False)
    sets = zipf_mlp_sets(cfg, 26)
    idx = torch.tensor(sets, dtype=torch.int32, device="cuda")
    buf = torch.full((sets.size + 8,), -7, dtype=torch.int32, device="cuda")
    view = buf[offset:offset + sets.size].view(sets.shape)
    view.copy_(idx)
    assert view.data_ptr() % 16 == 4 * offset
    bm = Bd.DV_MLP_UNION if mode == "union" else Bd.DV_MLP_MASKED
    a = Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1, batch_mode=bm)
    b = Bd.dv_sparse_mlp(_mlp(t), t["x"], view, idx_per_seq=1, batch_mode=bm)
    _sync()
    assert torch.equal(a, b)


@pytest.mark.parametrize("mode", ["union", "masked"])
def test_batch_mlp_largest_neuron_count(mode):
    """n = 131072, the largest neuron count of the batched path (the union kernel's
    per-neuron marks then take 128 KB of LDS): per-sequence outputs match the oracle."""
    cfg = _cfg("small_b8", 4).with_(name="n131072_b4", N=131072, k_mlp=3000)
    t = make_layer(cfg, 27, device="cuda", biases=True, with_predictors=False)
    sets = zipf_mlp_sets(cfg, 27)
    idx = torch.tensor(sets, dtype=torch.int32, device="cuda")
    bm = Bd.DV_MLP_UNION if mode == "union" else Bd.DV_MLP_MASKED
    out = Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1, batch_mode=bm, flags=Bd.DV_VALIDATE)
    _sync()
    U = np.unique(sets)
    W1, W2, b1 = host(t["W1T"])[U], host(t["W2T"])[U], host(t["b1"])[U]   # the union's rows only
    pos = {int(u): i for i, u in enumerate(U)}
    local = [np.array([pos[int(v)] for v in s_], dtype=np.int64).tolist() for s_ in sets]
    ref = O.mlp_batch(host(t["x"]), W1, b1, W2, host(t["b2"]), local, mode)
    got = host(out)
    for b in range(cfg.B):
        assert rel_l2(got[b], ref[b]) < REL_TOL, (b, rel_l2(got[b], ref[b]))


def test_batch_mlp_union_differs_from_masked():
    """The two batch semantics give different outputs (the union adds other sequences' neurons)."""
    cfg = _cfg("small_b8")
    t = make_layer(cfg, 22, device="cuda", biases=True, with_predictors=False)
    idx = torch.tensor(zipf_mlp_sets(cfg, 22), dtype=torch.int32, device="cuda")
    u = Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1, batch_mode=Bd.DV_MLP_UNION)
    m = Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1, batch_mode=Bd.DV_MLP_MASKED)
    _sync()
    assert rel_l2(host(u)[0], host(m)[0]) > 10 * REL_TOL


def test_batch_mlp_shared_set_and_full_set():
    cfg = _cfg("small_b8")
    t = make_layer(cfg, 23, device="cuda", biases=True, with_predictors=False)
    m = oracle_mlp(t)
    x = host(t["x"])
    S = np.sort(np.random.default_rng(23).permutation(cfg.N)[: cfg.k_mlp]).astype(np.int32)
    out = Bd.dv_sparse_mlp(_mlp(t), t["x"], torch.tensor(S, device="cuda"), idx_per_seq=0)
    full = Bd.dv_sparse_mlp(_mlp(t), t["x"], torch.arange(cfg.N, dtype=torch.int32, device="cuda"), idx_per_seq=0)
    _sync()
    for b in range(cfg.B):
        assert rel_l2(host(out)[b], O.mlp_sparse(x[b], m["W1T"], m["b1"], m["W2T"], m["b2"], S)) < REL_TOL
        assert rel_l2(host(full)[b], O.mlp_dense(x[b], m["W1T"], m["b1"], m["W2T"], m["b2"])) < REL_TOL


def test_batch_mlp_empty_set_is_bias():
    cfg = _cfg("small_b8")
    t = make_layer(cfg, 24, device="cuda", biases=True, with_predictors=False)
    idx = torch.zeros((cfg.B, 0), dtype=torch.int32, device="cuda")
    out = Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1)
    _sync()
    for b in range(cfg.B):
        assert np.array_equal(host(out)[b].astype(np.float32), host(t["b2"]).astype(np.float32))


def test_batch_mlp_rejects_bad_sets_under_validate():
    cfg = _cfg("small_b8")
    t = make_layer(cfg, 25, device="cuda", with_predictors=False)
    sets = zipf_mlp_sets(cfg, 25)
    sets[3, 5] = sets[3, 4]          # duplicate -> not strictly ascending
    idx = torch.tensor(sets, dtype=torch.int32, device="cuda")
    with pytest.raises(Bd.DvError) as e:
        Bd.dv_sparse_mlp(_mlp(t), t["x"], idx, idx_per_seq=1, flags=Bd.DV_VALIDATE)
    assert e.value.status == Bd.DV_ERR_INDEX


# ------------------------------------------------------------------ attention
def _check_attn(cfg, t, heads, out, K0, V0, biases=True):
    a = oracle_attn(t, biases)
    pos = [int(p) for p in t["pos"]]
    ref, Kn, Vn = O.mha_batch(host(t["x"]), a, K0, V0, pos, [h.tolist() for h in heads], 1.0 / np.sqrt(cfg.dh))
    got = host(out)
    K1, V1 = host(t["K"]), host(t["V"])
    for b in range(cfg.B):
        assert rel_l2(got[b], ref[b]) < REL_TOL, (b, rel_l2(got[b], ref[b]))
        for h in range(cfg.H):
            if h in set(heads[b].tolist()):
                for C1, Cn in ((K1, Kn), (V1, Vn)):
                    assert rel_l2(C1[b, h, pos[b]], Cn[b, h, pos[b]]) < 2e-3
            else:
                assert np.array_equal(K1[b, h, pos[b]], K0[b, h, pos[b]])
                assert np.array_equal(V1[b, h, pos[b]], V0[b, h, pos[b]])
        # every other position of every head is untouched
        mask = np.ones(K1.shape[2], dtype=bool)
        mask[pos[b]] = False
        assert np.array_equal(K1[b][:, mask], K0[b][:, mask])
        assert np.array_equal(V1[b][:, mask], V0[b][:, mask])


@pytest.mark.parametrize("B", [2, 8, 32])
@pytest.mark.parametrize("kv_scale", [1.0, 30.0])
def test_batch_attn(B, kv_scale):
    cfg = _cfg("small_b8", B)
    t = make_layer(cfg, 31, device="cuda", biases=True, kv_scale=kv_scale)
    K0, V0 = host(t["K"]).copy(), host(t["V"]).copy()
    heads = uniform_head_sets(cfg, 31)
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    out = Bd.dv_sparse_attn(attn, t["x"], kv, torch.tensor(heads, device="cuda"), 1.0 / np.sqrt(cfg.dh),
                            flags=Bd.DV_VALIDATE)
    _sync()
    _check_attn(cfg, t, heads, out, K0, V0)


@pytest.mark.parametrize("kvd", ["f16", "f32"])
def test_batch_attn_widest_heads(kvd):
    """Heads of 256 on the batched path, with an fp16 or an fp32 cache."""
    cfg = _cfg("small_b8", 4).with_(name=f"dh256_b4_{kvd}", d=1024, H=6, dh=256, k_heads=3, kvdtype=kvd)
    t = make_layer(cfg, 34, device="cuda", biases=True)
    K0, V0 = host(t["K"]).copy(), host(t["V"]).copy()
    heads = uniform_head_sets(cfg, 34)
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    out = Bd.dv_sparse_attn(attn, t["x"], kv, torch.tensor(heads, device="cuda"), 1.0 / np.sqrt(cfg.dh))
    _sync()
    _check_attn(cfg, t, heads, out, K0, V0)


def test_batch_attn_all_heads_and_pos0():
    cfg = _cfg("small_b8").with_(k_heads=10, L_range=(1, 2))
    t = make_layer(cfg, 32, device="cuda", biases=True)
    K0, V0 = host(t["K"]).copy(), host(t["V"]).copy()
    heads = np.tile(np.arange(cfg.H, dtype=np.int32), (cfg.B, 1))
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    out = Bd.dv_sparse_attn(attn, t["x"], kv, torch.tensor(heads, device="cuda"), 1.0 / np.sqrt(cfg.dh))
    _sync()
    assert min(int(p) for p in t["pos"]) == 0
    _check_attn(cfg, t, heads, out, K0, V0)


def test_batch_attn_no_heads_is_bias():
    cfg = _cfg("small_b8")
    t = make_layer(cfg, 33, device="cuda", biases=True)
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    out = Bd.dv_sparse_attn(attn, t["x"], kv, torch.zeros((cfg.B, 0), dtype=torch.int32, device="cuda"), 0.1)
    _sync()
    for b in range(cfg.B):
        assert np.array_equal(host(out)[b].astype(np.float32), host(t["bo"]).astype(np.float32))


# ---------------------------------------------------------------------- layer
def _check_block(cfg, t, out, hs, ms, K0, V0, mode, batch_mode):
    """Sets against the oracle's scores (near-ties allowed); the output against the oracle
    layer rerun on the GPU's sets with the same batch semantics."""
    a, m, ln = oracle_attn(t), oracle_mlp(t), oracle_ln(t)
    x = host(t["x"])
    pos = [int(p) for p in t["pos"]]
    hs, ms = host(hs), host(ms)
    scale = 1.0 / np.sqrt(cfg.dh)
    AT_h, BT_h, AT_m, BT_m = (host(t[k]) for k in ("AT_h", "BT_h", "AT_m", "BT_m"))
    U = O.union_of_sets([s.tolist() for s in ms])
    got = host(out)
    for b in range(cfg.B):
        xh = O.layer_norm(x[b], ln["g1"], ln["be1"], ln["eps"])
        check_topk_set(hs[b], O.predictor_scores(xh, AT_h, BT_h), cfg.k_heads)
        S_M = U if batch_mode == "union" else ms[b]
        r = O.sparse_block(x[b], a, m, K0[b], V0[b], pos[b], scale, S_A=hs[b], S_M=S_M, ln=ln)
        if mode == "lookahead":
            s_m = O.predictor_scores(xh, AT_m, BT_m)
        else:
            s_m = O.predictor_scores(O.layer_norm(r["y_tilde"], ln["g2"], ln["be2"], ln["eps"]), AT_m, BT_m)
        check_topk_set(ms[b], s_m, cfg.k_mlp)
        assert rel_l2(got[b], r["out"]) < REL_TOL, (b, rel_l2(got[b], r["out"]))


@pytest.mark.parametrize("B", [8, 32])
@pytest.mark.parametrize("mode", ["lookahead", "sequential"])
@pytest.mark.parametrize("batch_mode", ["union", "masked"])
def test_batch_block(B, mode, batch_mode):
    cfg = _cfg("small_b8", B)
    t = make_layer(cfg, 41, device="cuda", biases=True, ln_random=True)
    K0, V0 = host(t["K"]).copy(), host(t["V"]).copy()
    attn, mlp, ph, pm, kv, ln = layer_objects(t, cfg.H)
    out, hs, ms = Bd.dv_sparse_block(attn, mlp, ph, pm, ln, kv, t["x"], cfg.k_heads, cfg.k_mlp,
                                     1.0 / np.sqrt(cfg.dh),
                                     mode=Bd.DV_LOOKAHEAD if mode == "lookahead" else Bd.DV_SEQUENTIAL,
                                     batch_mode=Bd.DV_MLP_UNION if batch_mode == "union" else Bd.DV_MLP_MASKED)
    _sync()
    _check_block(cfg, t, out, hs, ms, K0, V0, mode, batch_mode)


def test_batch_block_deterministic():
    cfg = _cfg("small_b8")
    t = make_layer(cfg, 42, device="cuda", biases=True, ln_random=True)
    attn, mlp, ph, pm, kv, ln = layer_objects(t, cfg.H)
    outs = []
    for _ in range(2):
        o, h, m = Bd.dv_sparse_block(attn, mlp, ph, pm, ln, kv, t["x"], cfg.k_heads, cfg.k_mlp, 0.1)
        outs.append((o.clone(), h.clone(), m.clone()))
    _sync()
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)


# ------------------------------------------------------------ OPT-175B, batch 32
@pytest.fixture(scope="module")
def b32():
    cfg = get_config("opt175b_b32")
    t = make_layer(cfg, 4, device="cuda", biases=False)
    return cfg, t


@pytest.mark.parametrize("mode", ["union", "masked"])
def test_opt175b_b32_mlp_every_sequence(b32, mode):
    """The batch-32 MLP at full size: every one of the 32 sequences against the oracle,
    on the union of the Zipf sets (Section 5.2) or on each sequence's own set."""
    cfg, t = b32
    sets = zipf_mlp_sets(cfg, 4)
    idx = torch.tensor(sets, dtype=torch.int32, device="cuda")
    bm = Bd.DV_MLP_UNION if mode == "union" else Bd.DV_MLP_MASKED
    out = Bd.dv_sparse_mlp(_mlp(t, biases=False), t["x"], idx, idx_per_seq=1, batch_mode=bm)
    _sync()
    W1T, W2T = host(t["W1T"]), host(t["W2T"])
    x = host(t["x"])
    got = host(out)
    if mode == "union":
        U = O.union_of_sets([s.tolist() for s in sets])
        assert 20000 < len(U) < 30000
        ref = O.mlp_union_rows(x, W1T, None, W2T, None, U)
    else:
        ref = np.stack([O.mlp_sparse(x[b], W1T, None, W2T, None, sets[b]) for b in range(cfg.B)])
    errs = [rel_l2(got[b], ref[b]) for b in range(cfg.B)]
    assert max(errs) < REL_TOL, (int(np.argmax(errs)), max(errs))


def _u16(a):
    return np.ascontiguousarray(a).view(np.uint16) if a.dtype == np.float16 else np.ascontiguousarray(a).view(np.uint32)


def test_opt175b_b32_attention_every_sequence(b32):
    """Batch-32 attention at full size: every sequence's output against the oracle, its
    fresh keys and values at its own position, and the cache contract for the whole
    cache (only rows pos[b] of the heads sequence b selected change, bit for bit)."""
    cfg, t = b32
    heads = uniform_head_sets(cfg, 4)
    pos = [int(p) for p in t["pos"]]
    assert 511 <= min(pos) and max(pos) <= 2047
    K0, V0 = host(t["K"]).copy(), host(t["V"]).copy()
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H, biases=False)
    out = Bd.dv_sparse_attn(attn, t["x"], kv, torch.tensor(heads, device="cuda"), 1.0 / np.sqrt(cfg.dh))
    _sync()
    a = oracle_attn(t, biases=False)
    x = host(t["x"])
    got = host(out)
    Kg, Vg = host(t["K"]), host(t["V"])
    allowed = np.zeros(Kg.shape[:3], dtype=bool)
    errs = []
    for b in range(cfg.B):
        ref, Kn, Vn, _ = O.mha_sparse(x[b], a, K0[b], V0[b], pos[b], heads[b], 1.0 / np.sqrt(cfg.dh))
        errs.append(rel_l2(got[b], ref))
        for h in heads[b]:
            assert rel_l2(Kg[b, h, pos[b]].astype(np.float64), Kn[h, pos[b]]) < REL_TOL, (b, h)
            assert rel_l2(Vg[b, h, pos[b]].astype(np.float64), Vn[h, pos[b]]) < REL_TOL, (b, h)
            allowed[b, h, pos[b]] = True
    assert max(errs) < REL_TOL, (int(np.argmax(errs)), max(errs))
    for C, C0 in ((Kg, K0), (Vg, V0)):
        changed = (_u16(C) != _u16(C0)).any(axis=-1)
        assert not (changed & ~allowed).any(), np.argwhere(changed & ~allowed)[:5]


def test_opt175b_b32_deterministic(b32):
    """Two identical batch-32 attention + union-MLP steps give bitwise identical outputs
    (every split sum runs in a fixed order)."""
    cfg, t = b32
    heads = torch.tensor(uniform_head_sets(cfg, 4), device="cuda")
    idx = torch.tensor(zipf_mlp_sets(cfg, 4), dtype=torch.int32, device="cuda")
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H, biases=False)
    outs = []
    for _ in range(2):
        a_out = Bd.dv_sparse_attn(attn, t["x"], kv, heads, 1.0 / np.sqrt(cfg.dh))
        m_out = Bd.dv_sparse_mlp(_mlp(t, biases=False), a_out, idx, idx_per_seq=1)
        outs.append((a_out.clone(), m_out.clone()))
    _sync()
    for u, v in zip(outs[0], outs[1]):
        assert torch.equal(u, v)
