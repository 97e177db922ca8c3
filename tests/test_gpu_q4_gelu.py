"""GPU parity of the Section 5.2 variants: 4-bit weights (W4A16, dv_sparse_mlp_q4) and
the GeLU activation (dv_mlp.act, batch 1 and the batched path), against the fp64
oracle (oracle.dejavu.dequant_q4_rows and mlp_sparse with the same activation) on the
same stored codes and scales."""
import numpy as np
import pytest
import torch

from oracle import dejavu as O
from paper_2310_17157_amd import binding as Bd
from synth import get_config, make_layer, quantize_q4, zipf_mlp_sets
from tests.gpu_util import REL_TOL, host, oracle_mlp, rel_l2

pytestmark = pytest.mark.gpu


def _q4_layer(d, N, seed, biases=True):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    W1 = (torch.randn((N, d), generator=g, device="cuda") * 0.02).half()
    W2 = (torch.randn((N, d), generator=g, device="cuda") * 0.02).half()
    P1, S1 = quantize_q4(W1)
    P2, S2 = quantize_q4(W2)
    b1 = torch.randn(N, generator=g, device="cuda") * 0.02 if biases else None
    b2 = torch.randn(d, generator=g, device="cuda") * 0.02 if biases else None
    return P1, S1, P2, S2, b1, b2


@pytest.mark.parametrize("d,N,k,act", [(1312, 5000, 501, "relu"), (1312, 5000, 501, "gelu"), (256, 700, 700, "relu"),
                                       (12288, 49152, 2457, "relu"), (12288, 49152, 2457, "gelu")])
def test_q4_sparse_mlp(d, N, k, act):
    P1, S1, P2, S2, b1, b2 = _q4_layer(d, N, 140 + d % 97)
    m = Bd.MLPQ4(P1, S1, P2, S2, b1, b2, act=Bd.DV_ACT_GELU if act == "gelu" else Bd.DV_ACT_RELU)
    rng = np.random.default_rng(141)
    S = np.sort(rng.choice(N, k, replace=False)).astype(np.int32)
    x = torch.randn((1, d), device="cuda")
    out = Bd.dv_sparse_mlp_q4(m, x, torch.tensor(S, device="cuda"))
    torch.cuda.synchronize()
    W1 = O.dequant_q4_rows(host(P1), host(S1), d, S)
    W2 = O.dequant_q4_rows(host(P2), host(S2), d, S)
    ref = O.mlp_sparse(host(x)[0], W1, host(b1)[S], W2, host(b2), range(k), act)
    assert rel_l2(host(out)[0], ref) < REL_TOL


def test_q4_empty_set_is_bias_and_determinism():
    P1, S1, P2, S2, b1, b2 = _q4_layer(512, 300, 150)
    m = Bd.MLPQ4(P1, S1, P2, S2, b1, b2)
    x = torch.randn((1, 512), device="cuda")
    out = Bd.dv_sparse_mlp_q4(m, x, torch.empty(0, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert np.array_equal(host(out)[0], host(b2))
    idx = torch.arange(0, 300, 3, dtype=torch.int32, device="cuda")
    a = Bd.dv_sparse_mlp_q4(m, x, idx).clone()
    b = Bd.dv_sparse_mlp_q4(m, x, idx)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_q4_full_size_is_deterministic():
    """The OPT-175B set: ten row splits per 512-column span, added by the last split to
    arrive; two calls agree bit for bit."""
    P1, S1, P2, S2, b1, b2 = _q4_layer(12288, 49152, 151)
    m = Bd.MLPQ4(P1, S1, P2, S2, b1, b2)
    x = torch.randn((1, 12288), device="cuda")
    rng = np.random.default_rng(152)
    idx = torch.tensor(np.sort(rng.choice(49152, 2457, replace=False)).astype(np.int32), device="cuda")
    a = Bd.dv_sparse_mlp_q4(m, x, idx).clone()
    b = Bd.dv_sparse_mlp_q4(m, x, idx)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["small_f16", "small_f32", "opt175b_b1"])
def test_gelu_sparse_mlp(name):
    cfg = get_config(name)
    t = make_layer(cfg, 160, device="cuda", biases=True, with_predictors=False)
    mlp = Bd.MLP(t["W1T"], t["W2T"], t["b1"], t["b2"], act=Bd.DV_ACT_GELU)
    rng = np.random.default_rng(161)
    S = np.sort(rng.choice(cfg.N, cfg.k_mlp, replace=False)).astype(np.int32)
    x = torch.randn((1, cfg.d), device="cuda")
    out = Bd.dv_sparse_mlp(mlp, x, torch.tensor(S, device="cuda"))
    torch.cuda.synchronize()
    om = oracle_mlp(t)
    ref = O.mlp_sparse(host(x)[0], om["W1T"], om["b1"], om["W2T"], om["b2"], S, "gelu")
    assert rel_l2(host(out)[0], ref) < REL_TOL


@pytest.mark.parametrize("mode", ["union", "masked"])
def test_gelu_batched_mlp(mode):
    cfg = get_config("small_b8")
    t = make_layer(cfg, 170, device="cuda", biases=True, with_predictors=False)
    sets = zipf_mlp_sets(cfg, 170)
    mlp = Bd.MLP(t["W1T"], t["W2T"], t["b1"], t["b2"], act=Bd.DV_ACT_GELU)
    out = Bd.dv_sparse_mlp(mlp, t["x"], torch.tensor(sets, dtype=torch.int32, device="cuda"), idx_per_seq=1,
                           batch_mode=Bd.DV_MLP_UNION if mode == "union" else Bd.DV_MLP_MASKED)
    torch.cuda.synchronize()
    om = oracle_mlp(t)
    U = O.union_of_sets([s.tolist() for s in sets])
    for b in range(cfg.B):
        S = U if mode == "union" else sets[b]
        ref = O.mlp_sparse(host(t["x"])[b], om["W1T"], om["b1"], om["W2T"], om["b2"], S, "gelu")
        assert rel_l2(host(out)[b], ref) < REL_TOL, b
