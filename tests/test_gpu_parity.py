"""GPU parity: every C-ABI entry point against the fp64 oracle on the same seeded inputs.

Outputs: max relative L2 error <= 2e-3 (fp16 weights, fp32 accumulation). Sets:
bit-exact up to predictor-score near-ties within 1e-3 (relative) of the k-th score.
Cache: rows of non-selected heads (and all other positions) untouched, bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import dejavu as O
from paper_2310_17157_amd import binding as Bd
from paper_2310_17157_amd.workload import layer_objects
from synth import get_config
from tests.gpu_util import (REL_TOL, check_topk_set, host, layer, near_tie_band, oracle_attn, oracle_ln,
                            oracle_mlp, rel_l2)

pytestmark = pytest.mark.gpu

SMALL = ["small_f32", "small_f16", "opt125m_b1"]


def _sync():
    torch.cuda.synchronize()


# ----------------------------------------------------------------- predictors
@pytest.mark.parametrize("name", SMALL + ["opt6.7b_b1", "opt175b_b1"])
def test_predict_mlp_topk(name):
    cfg, t = layer(name, 11, with_dense=False)
    pred = Bd.Predictor(t["AT_m"], t["BT_m"])
    scores = torch.empty((1, cfg.N), dtype=torch.float32, device="cuda")
    idx, cnt = Bd.dv_predict_mlp(pred, t["x"], cfg.k_mlp, scores=scores)
    _sync()
    s_or = O.predictor_scores(host(t["x"])[0], host(t["AT_m"]), host(t["BT_m"]))
    assert rel_l2(host(scores)[0], s_or) < 1e-4
    check_topk_set(host(idx)[0], s_or, cfg.k_mlp)
    assert int(cnt[0]) == cfg.k_mlp


@pytest.mark.parametrize("name", SMALL + ["opt175b_b1"])
def test_predict_heads_topk(name):
    cfg, t = layer(name, 12, with_dense=False)
    pred = Bd.Predictor(t["AT_h"], t["BT_h"])
    idx, _ = Bd.dv_predict_heads(pred, t["x"], cfg.k_heads)
    _sync()
    s_or = O.predictor_scores(host(t["x"])[0], host(t["AT_h"]), host(t["BT_h"]))
    check_topk_set(host(idx)[0], s_or, cfg.k_heads)


@pytest.mark.parametrize("name", ["small_f16", "opt125m_b1"])
def test_predict_threshold(name):
    cfg, t = layer(name, 13, with_dense=False)
    pred = Bd.Predictor(t["AT_m"], t["BT_m"])
    s_or = O.predictor_scores(host(t["x"])[0], host(t["AT_m"]), host(t["BT_m"]))
    thr = float(np.sort(s_or)[::-1][cfg.k_mlp // 2])
    idx, cnt = Bd.dv_predict_mlp(pred, t["x"], mode=Bd.DV_SELECT_THRESHOLD, thresh=thr)
    _sync()
    n = int(cnt[0])
    g = host(idx)[0][:n].tolist()
    assert g == sorted(set(g))
    o = set(O.select_threshold(s_or, thr).tolist())
    scale = max(abs(thr), float(np.sqrt(np.mean(s_or ** 2))))
    band = set(np.nonzero(np.abs(s_or - thr) <= 1e-3 * scale)[0].tolist())
    assert (set(g) ^ o) <= band


def test_predict_batch_rows_are_independent():
    cfg, t = layer("small_f16", 14, with_dense=False)
    x = torch.randn((5, cfg.d), device="cuda") * 0.02
    pred = Bd.Predictor(t["AT_m"], t["BT_m"])
    idx, _ = Bd.dv_predict_mlp(pred, x, cfg.k_mlp)
    _sync()
    for b in range(5):
        s_or = O.predictor_scores(host(x)[b], host(t["AT_m"]), host(t["BT_m"]))
        check_topk_set(host(idx)[b], s_or, cfg.k_mlp)


def test_topk_ties_and_edge_sizes():
    """Exact ties in the scores: lower index first. k = n and k = 0 edge sizes."""
    d, r, n = 64, 8, 300
    AT = torch.zeros((r, d), dtype=torch.float32, device="cuda")
    AT[0, 0] = 1.0
    BT = torch.zeros((n, r), dtype=torch.float32, device="cuda")
    vals = torch.tensor([float((i * 7) % 5) for i in range(n)], device="cuda")   # many exact ties
    BT[:, 0] = vals
    x = torch.zeros((1, d), dtype=torch.float32, device="cuda")
    x[0, 0] = 1.0
    pred = Bd.Predictor(AT, BT)
    s = vals.cpu().double().numpy()
    for k in (1, 37, 60, 61, 150, 299, 300):
        idx, _ = Bd.dv_predict_mlp(pred, x, k)
        _sync()
        assert host(idx)[0].tolist() == O.select_topk(s, k).tolist(), k
    idx, cnt = Bd.dv_predict_mlp(pred, x, 0, cap_idx=1)
    _sync()
    assert int(cnt[0]) == 0


@pytest.mark.parametrize("n", [96, 1024, 1025, 3000])
def test_select_paths_agree_with_oracle(n):
    """Score vectors up to 1024 are ranked in LDS, longer ones by the radix select: both
    give the oracle's set, with exact ties to the lower index, in top-k and threshold
    mode (the threshold count may exceed the capacity; the first cap members are kept)."""
    d, r = 64, 8
    AT = torch.zeros((r, d), dtype=torch.float32, device="cuda")
    AT[0, 0] = 1.0
    BT = torch.zeros((n, r), dtype=torch.float32, device="cuda")
    vals = torch.tensor([float((i * 13) % 11) - 5.0 for i in range(n)], device="cuda")   # ties, both signs
    BT[:, 0] = vals
    x = torch.zeros((1, d), dtype=torch.float32, device="cuda")
    x[0, 0] = 1.0
    pred = Bd.Predictor(AT, BT)
    s = vals.cpu().double().numpy()
    for k in (1, n // 3, n - 1, n):
        idx, cnt = Bd.dv_predict_heads(pred, x, k)
        _sync()
        assert host(idx)[0].tolist() == O.select_topk(s, k).tolist(), (n, k)
        assert int(cnt[0]) == k, (n, k)
    full = O.select_threshold(s, 2.0).tolist()
    cap = max(1, len(full) // 2)
    idx, cnt = Bd.dv_predict_heads(pred, x, mode=Bd.DV_SELECT_THRESHOLD, thresh=2.0, cap_idx=cap)
    _sync()
    assert int(cnt[0]) == len(full)
    assert host(idx)[0][:cap].tolist() == full[:cap]


def test_select_register_path_large_sets():
    """Register-resident selection (n <= 49152) of sets too large to stage in LDS
    (more than 8128 members) is written straight to memory: top-k with and without a
    tie at the boundary, and threshold mode with the count above the capacity."""
    n = 40000
    d, r = 64, 8
    AT = torch.zeros((r, d), dtype=torch.float32, device="cuda")
    AT[0, 0] = 1.0
    BT = torch.zeros((n, r), dtype=torch.float32, device="cuda")
    vals = torch.tensor([float((i * 37) % 1009) - 500.0 for i in range(n)], device="cuda")
    BT[:, 0] = vals
    x = torch.zeros((1, d), dtype=torch.float32, device="cuda")
    x[0, 0] = 1.0
    pred = Bd.Predictor(AT, BT)
    s = vals.cpu().double().numpy()
    for k in (8128, 8129, 9000, 20000, 39999):
        idx, cnt = Bd.dv_predict_mlp(pred, x, k)
        _sync()
        assert host(idx)[0].tolist() == O.select_topk(s, k).tolist(), k
        assert int(cnt[0]) == k, k
    full = O.select_threshold(s, 0.0).tolist()
    assert len(full) > 8128
    cap = len(full) - 7
    idx, cnt = Bd.dv_predict_mlp(pred, x, mode=Bd.DV_SELECT_THRESHOLD, thresh=0.0, cap_idx=cap)
    _sync()
    assert int(cnt[0]) == len(full)
    assert host(idx)[0][:cap].tolist() == full[:cap]


def test_select_streaming_path_agrees_with_oracle():
    """More than 49152 scores do not fit the registers of one workgroup: the radix
    select streams them from memory in every pass. Exact ties, top-k and threshold."""
    n = 100000
    d, r = 64, 8
    AT = torch.zeros((r, d), dtype=torch.float32, device="cuda")
    AT[0, 0] = 1.0
    BT = torch.zeros((n, r), dtype=torch.float32, device="cuda")
    vals = torch.tensor([float((i * 37) % 1009) - 500.0 for i in range(n)], device="cuda")
    BT[:, 0] = vals
    x = torch.zeros((1, d), dtype=torch.float32, device="cuda")
    x[0, 0] = 1.0
    pred = Bd.Predictor(AT, BT)
    s = vals.cpu().double().numpy()
    for k in (1, 5000, n - 1, n):
        idx, cnt = Bd.dv_predict_mlp(pred, x, k)
        _sync()
        assert host(idx)[0].tolist() == O.select_topk(s, k).tolist(), k
        assert int(cnt[0]) == k, k
    full = O.select_threshold(s, 400.0).tolist()
    cap = len(full) - 7
    idx, cnt = Bd.dv_predict_mlp(pred, x, mode=Bd.DV_SELECT_THRESHOLD, thresh=400.0, cap_idx=cap)
    _sync()
    assert int(cnt[0]) == len(full)
    assert host(idx)[0][:cap].tolist() == full[:cap]


# ------------------------------------------------------------------ sparse MLP
@pytest.mark.parametrize("name", SMALL + ["opt6.7b_b1", "opt66b_b1", "opt175b_b1"])
def test_sparse_mlp(name):
    cfg, t = layer(name, 21, biases=True)
    _, mlp, *_ = layer_objects(t, cfg.H)
    rng = np.random.default_rng(21)
    S = np.sort(rng.choice(cfg.N, cfg.k_mlp, replace=False)).astype(np.int32)
    idx = torch.tensor(S, device="cuda")
    x = torch.randn((1, cfg.d), device="cuda")
    out = Bd.dv_sparse_mlp(mlp, x, idx)
    _sync()
    om = oracle_mlp(t)
    ref = O.mlp_sparse(host(x)[0], om["W1T"], om["b1"], om["W2T"], om["b2"], S)
    assert rel_l2(host(out)[0], ref) < REL_TOL


def test_sparse_mlp_full_set_is_dense_and_empty_set_is_bias():
    cfg, t = layer("small_f16", 22, biases=True)
    _, mlp, *_ = layer_objects(t, cfg.H)
    x = torch.randn((1, cfg.d), device="cuda")
    om = oracle_mlp(t)
    out = Bd.dv_sparse_mlp(mlp, x, torch.arange(cfg.N, dtype=torch.int32, device="cuda"))
    _sync()
    assert rel_l2(host(out)[0], O.mlp_dense(host(x)[0], om["W1T"], om["b1"], om["W2T"], om["b2"])) < REL_TOL
    out = Bd.dv_sparse_mlp(mlp, x, torch.empty(0, dtype=torch.int32, device="cuda"))
    _sync()
    assert np.array_equal(host(out)[0], host(t["b2"]))


def test_validate_flag_rejects_bad_sets():
    cfg, t = layer("small_f16", 23)
    _, mlp, *_ = layer_objects(t, cfg.H)
    x = torch.randn((1, cfg.d), device="cuda")
    for bad in ([5, 3, 9], [1, 1, 2], [0, 2, cfg.N]):
        with pytest.raises(Bd.DvError) as e:
            Bd.dv_sparse_mlp(mlp, x, torch.tensor(bad, dtype=torch.int32, device="cuda"), flags=Bd.DV_VALIDATE)
        assert e.value.status == 6
    Bd.dv_sparse_mlp(mlp, x, torch.tensor([0, 2, 7], dtype=torch.int32, device="cuda"), flags=Bd.DV_VALIDATE)


# ------------------------------------------------------------ sparse attention
def _attn_case(name, seed, heads=None, pos=None, kv_scale=1.0):
    cfg, t = layer(name, seed, biases=True, kv_scale=kv_scale)
    if pos is not None:
        t["pos"] = torch.tensor([pos], dtype=torch.int32)
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    rng = np.random.default_rng(seed)
    if heads is None:
        heads = np.sort(rng.choice(cfg.H, cfg.k_heads, replace=False)).astype(np.int32)
    heads = np.asarray(heads, dtype=np.int32)
    x = torch.randn((1, cfg.d), device="cuda")
    K0, V0 = host(t["K"])[0].copy(), host(t["V"])[0].copy()
    out = Bd.dv_sparse_attn(attn, x, kv, torch.tensor(heads, device="cuda").reshape(1, -1),
                            1.0 / np.sqrt(cfg.dh))
    _sync()
    p = int(t["pos"][0])
    ref, Kn, Vn, _ = O.mha_sparse(host(x)[0], oracle_attn(t), K0, V0, p, heads, 1.0 / np.sqrt(cfg.dh))
    return cfg, t, heads, p, out, ref, K0, V0, Kn, Vn


@pytest.mark.parametrize("name", SMALL + ["opt6.7b_b1", "opt66b_b1", "opt175b_b1"])
def test_sparse_attn(name):
    cfg, t, heads, p, out, ref, K0, V0, Kn, Vn = _attn_case(name, 31)
    assert rel_l2(host(out)[0], ref) < REL_TOL
    Kg, Vg = host(t["K"])[0], host(t["V"])[0]
    for h in range(cfg.H):
        if h in heads:
            assert rel_l2(Kg[h, p].astype(np.float64), Kn[h, p]) < REL_TOL
            assert rel_l2(Vg[h, p].astype(np.float64), Vn[h, p]) < REL_TOL
            rows = np.arange(Kg.shape[1]) != p
            assert Kg[h, rows].tobytes() == K0[h, rows].tobytes()
            assert Vg[h, rows].tobytes() == V0[h, rows].tobytes()
        else:
            assert Kg[h].tobytes() == K0[h].tobytes() and Vg[h].tobytes() == V0[h].tobytes()


@pytest.mark.parametrize("wd,kvd", [("f16", "f16"), ("f32", "f32"), ("f16", "f32")])
def test_sparse_attn_widest_heads_and_cache_types(wd, kvd):
    """Heads of 256, the widest head the attention kernel takes, with each pairing of
    weight and cache types (an fp32 cache beside fp16 weights included)."""
    cfg = get_config("small_f16").with_(name=f"dh256_{wd}_{kvd}", d=1024, H=6, dh=256, L=300, k_heads=3,
                                        wdtype=wd, kvdtype=kvd)
    _, t, heads, p, out, ref, K0, V0, Kn, Vn = _attn_case(cfg, 33)
    assert rel_l2(host(out)[0], ref) < REL_TOL
    Kg, Vg = host(t["K"])[0], host(t["V"])[0]
    for h in heads:
        assert rel_l2(Kg[h, p].astype(np.float64), Kn[h, p]) < REL_TOL
        assert rel_l2(Vg[h, p].astype(np.float64), Vn[h, p]) < REL_TOL


def test_sparse_attn_peaky_scores_and_first_position():
    # Large logits exercise the max-subtracted softmax and the split-KV combine.
    cfg, t, heads, p, out, ref, *_ = _attn_case("small_f16", 32, kv_scale=30.0)
    assert rel_l2(host(out)[0], ref) < REL_TOL
    # pos = 0: each head attends only to its fresh key, so H_i = v_i.
    cfg, t, heads, p, out, ref, *_ = _attn_case("small_f32", 33, pos=0)
    assert rel_l2(host(out)[0], ref) < REL_TOL


def test_sparse_attn_long_context_multi_subchunk():
    """4000 attended positions for one head: each workgroup walks several sub-chunks
    (online softmax) and the split count stays within the combine limit."""
    from synth import get_config
    cfg = get_config("small_f16").with_(L=4000, k_heads=1)
    from synth import make_layer
    t = make_layer(cfg, 36, device="cuda", biases=True, kv_scale=4.0)
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    x = torch.randn((1, cfg.d), device="cuda")
    K0, V0 = host(t["K"])[0].copy(), host(t["V"])[0].copy()
    out = Bd.dv_sparse_attn(attn, x, kv, torch.tensor([[7]], dtype=torch.int32, device="cuda"), 0.09)
    _sync()
    ref, *_ = O.mha_sparse(host(x)[0], oracle_attn(t), K0, V0, cfg.L - 1, [7], 0.09)
    assert rel_l2(host(out)[0], ref) < REL_TOL


def test_sparse_attn_all_heads_and_no_heads():
    cfg, t, heads, p, out, ref, *_ = _attn_case("small_f16", 34, heads=list(range(10)))
    assert rel_l2(host(out)[0], ref) < REL_TOL
    cfg, t = layer("small_f16", 35, biases=True)
    attn, _, _, _, kv, _ = layer_objects(t, cfg.H)
    out = Bd.dv_sparse_attn(attn, torch.randn((1, cfg.d), device="cuda"), kv,
                            torch.empty((1, 0), dtype=torch.int32, device="cuda"), 0.1)
    _sync()
    assert np.array_equal(host(out)[0], host(t["bo"]))


# --------------------------------------------------------------- decoder layer
def _block(name, seed, mode, biases=True, ln=True, k_heads=None, k_mlp=None):
    cfg, t = layer(name, seed, biases=biases, ln_random=ln)
    attn, mlp, ph, pm, kv, lnp = layer_objects(t, cfg.H, use_ln=True, biases=biases)
    kh = k_heads or cfg.k_heads
    km = k_mlp or cfg.k_mlp
    K0, V0 = host(t["K"])[0].copy(), host(t["V"])[0].copy()
    x = t["x"]
    scale = 1.0 / np.sqrt(cfg.dh)
    out, hs, ms = Bd.dv_sparse_block(attn, mlp, ph, pm, lnp, kv, x, kh, km, scale, mode=mode)
    _sync()
    y = host(x)[0]
    lno = oracle_ln(t)
    gh, gm = host(hs)[0], host(ms)[0]
    # Sets first (predictor parity), then arithmetic with the GPU's own sets.
    x1 = O.layer_norm(y, lno["g1"], lno["be1"])
    s_h = O.predictor_scores(x1, host(t["AT_h"]), host(t["BT_h"]))
    check_topk_set(gh, s_h, kh)
    r = O.sparse_block(y, oracle_attn(t, biases), oracle_mlp(t, biases), K0, V0, int(t["pos"][0]), scale,
                       S_A=gh, S_M=gm, ln=lno)
    src = x1 if mode == Bd.DV_LOOKAHEAD else O.layer_norm(r["y_tilde"], lno["g2"], lno["be2"])
    s_m = O.predictor_scores(src, host(t["AT_m"]), host(t["BT_m"]))
    check_topk_set(gm, s_m, km)
    g = host(out)[0]
    assert rel_l2(g - y, r["out"] - y) < REL_TOL
    assert rel_l2(g, r["out"]) < REL_TOL
    check_cache_contract(host(t["K"])[0], host(t["V"])[0], K0, V0, r["K_new"], r["V_new"], gh, int(t["pos"][0]))
    return cfg, t, out, hs, ms, r


def check_cache_contract(Kg, Vg, K0, V0, Kn, Vn, heads, p):
    """Section 4.2: only row p of the selected heads changes (bit for bit elsewhere), and
    it holds the fresh key / value."""
    allowed = np.zeros(Kg.shape[:2], dtype=bool)
    for h in heads:
        allowed[h, p] = True
        assert rel_l2(Kg[h, p].astype(np.float64), Kn[h, p]) < REL_TOL, h
        assert rel_l2(Vg[h, p].astype(np.float64), Vn[h, p]) < REL_TOL, h
    for C, C0 in ((Kg, K0), (Vg, V0)):
        bits = np.uint16 if C.dtype == np.float16 else np.uint32
        changed = (np.ascontiguousarray(C).view(bits) != np.ascontiguousarray(C0).view(bits)).any(axis=-1)
        assert not (changed & ~allowed).any(), np.argwhere(changed & ~allowed)[:5]


@pytest.mark.parametrize("name", SMALL)
@pytest.mark.parametrize("mode", [0, 1])
def test_sparse_block(name, mode):
    _block(name, 41, mode)


def test_sparse_block_all_heads_all_neurons_is_dense():
    cfg, t = layer("small_f32", 42, biases=True, ln_random=True)
    attn, mlp, ph, pm, kv, lnp = layer_objects(t, cfg.H)
    K0, V0 = host(t["K"])[0].copy(), host(t["V"])[0].copy()
    out, _, _ = Bd.dv_sparse_block(attn, mlp, ph, pm, lnp, kv, t["x"], cfg.H, cfg.N, 0.3)
    _sync()
    ref = O.dense_block(host(t["x"])[0], oracle_attn(t), oracle_mlp(t), K0, V0, int(t["pos"][0]), 0.3,
                        ln=oracle_ln(t))
    y = host(t["x"])[0]
    assert rel_l2(host(out)[0] - y, ref - y) < REL_TOL


def test_sparse_block_is_deterministic():
    cfg, t = layer("small_f16", 43, biases=True, ln_random=True)
    attn, mlp, ph, pm, kv, lnp = layer_objects(t, cfg.H)
    outs = []
    for _ in range(2):
        out, hs, ms = Bd.dv_sparse_block(attn, mlp, ph, pm, lnp, kv, t["x"], cfg.k_heads, cfg.k_mlp, 0.1)
        _sync()
        outs.append((host(out).tobytes(), host(hs).tobytes(), host(ms).tobytes()))
    assert outs[0] == outs[1]


def test_sparse_block_full_size_is_deterministic():
    """Two identical OPT-175B-shaped block calls give bitwise identical outputs and sets:
    the row-axpy split sums (10 row splits over 24 column spans, the last split of each
    span to arrive adds them) run in split order whatever the arrival order."""
    cfg, t = layer("opt175b_b1", 49, biases=True, ln_random=True)
    attn, mlp, ph, pm, kv, lnp = layer_objects(t, cfg.H)
    outs = []
    for _ in range(3):
        out, hs, ms = Bd.dv_sparse_block(attn, mlp, ph, pm, lnp, kv, t["x"], cfg.k_heads, cfg.k_mlp,
                                         1.0 / np.sqrt(cfg.dh))
        _sync()
        outs.append((host(out).tobytes(), host(hs).tobytes(), host(ms).tobytes()))
    assert outs[0] == outs[1] == outs[2]


def test_sparse_block_at_the_width_limit():
    """d = 16000, the widest input the row-dot kernels stage: with many rows per
    workgroup their LDS passes 64 KB (QKV over 16 heads x 128 rows of each projection,
    fc1 over 6000 neurons, the predictors' hidden layer at rank 3000)."""
    cfg = get_config("small_f16").with_(name="d16000", d=16000, N=8192, H=32, dh=128, L=64, r=3000,
                                        k_mlp=6000, k_heads=16)
    _block(cfg, 45, Bd.DV_LOOKAHEAD)


def test_sparse_block_at_the_rank_limit():
    """Predictor rank 16000 for both predictors: the score launch stages both hidden
    vectors, 128 KB of LDS."""
    cfg = get_config("small_f16").with_(name="r16000", d=256, N=512, H=4, dh=64, L=40, r=16000,
                                        k_mlp=100, k_heads=2)
    _block(cfg, 46, Bd.DV_LOOKAHEAD)


def test_sparse_block_neuron_selection_streams_past_49152():
    """65536 neurons: the neuron top-k hosted in the QKV launch streams the scores
    (more than one workgroup's registers hold)."""
    cfg = get_config("small_f16").with_(name="n65536", d=256, N=65536, H=4, dh=64, L=40, r=64,
                                        k_mlp=3000, k_heads=2)
    _block(cfg, 47, Bd.DV_LOOKAHEAD)


@pytest.mark.parametrize("name", ["opt6.7b_b1", "opt66b_b1", "opt175b_b1"])
def test_sparse_block_full_size(name):
    """The full-size layers, at the launch configuration the benchmark times."""
    _block(name, 44, Bd.DV_LOOKAHEAD)


def test_sparse_block_full_size_sequential():
    """OPT-175B shape in sequential mode: the neuron predictor reads LN2(y~) after the
    out-projection and selects 2457 of 49152 neurons in a launch of its own."""
    _block("opt175b_b1", 48, Bd.DV_SEQUENTIAL)
