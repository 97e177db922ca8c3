"""GPU parity of dv_sparse_attn_kvfill, the missing-KV rule of Section 4.2, over several
decode steps with changing head sets: each step's output against the fp64 oracle
(oracle.dejavu.mha_sparse_kvfill, run step by step on its own state), the validity
marks bit for bit, the filled cache rows of the selected heads, and the outputs of a
run whose cache holds every head's key and value at every token. The kept inputs Y are
stored in the cache's type (reading R18): fp16 caches keep them rounded to nearest even,
which the oracle models with its y_keep argument."""
import numpy as np
import pytest
import torch

from oracle import dejavu as O
from paper_2310_17157_amd import binding as Bd
from synth import get_config, make_layer
from tests.gpu_util import REL_TOL, host, oracle_attn, rel_l2

pytestmark = pytest.mark.gpu


def _keep(Y):
    """The oracle's storage type for the kept inputs: that of the GPU's Y."""
    return np.float16 if Y.dtype == torch.float16 else None


def _head_schedule(rng, H, k, T, starve=None):
    sets = []
    for s in range(T):
        pool = [h for h in range(H) if not (starve is not None and h == starve and s < T - 1)]
        S = np.sort(rng.choice(pool, min(k, len(pool)), replace=False))
        if starve is not None and s == T - 1 and starve not in S:
            S = np.sort(np.concatenate([S[:-1], [starve]]))
        sets.append(S.astype(np.int32))
    return sets


# The fill lists the missing positions into the workspace when k_heads * (pos + 1)
# ints fit in 32 * d; at this shape (8 heads x 1600 positions > 32 x 384) every fill
# workgroup lists its head's positions itself instead.
UNLISTED = get_config("small_f16").with_(name="kvfill_unlisted", d=384, N=1536, H=12, dh=32, L=1600, r=32,
                                         k_mlp=150, k_heads=8)


@pytest.mark.parametrize("name,T,empty_step", [("small_f16", 12, 5), ("small_f32", 10, None), ("opt175b_b1", 8, None),
                                               ("unlisted", 8, 3)])
def test_kvfill_decode_steps_against_oracle(name, T, empty_step):
    cfg = UNLISTED if name == "unlisted" else get_config(name)
    t = make_layer(cfg, 120, device="cuda", biases=True)
    attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], cfg.H, t["bq"], t["bk"], t["bv"], t["bo"])
    cap, d, H = cfg.kv_cap, cfg.d, cfg.H
    p0 = cap - T                                  # the prompt filled rows 0..p0-1 of every head
    kv = Bd.KVCache(t["K"], t["V"], [p0])
    Y = torch.zeros((cap, d), dtype=t["K"].dtype, device="cuda")
    Y[:p0] = torch.randn((p0, d), device="cuda")
    valid = torch.zeros((H, cap), dtype=torch.uint8, device="cuda")
    valid[:, :p0] = 1
    rng = np.random.default_rng(121)
    sets = _head_schedule(rng, H, cfg.k_heads, T, starve=0)   # head 0 misses every step but the last
    if empty_step is not None:
        sets[empty_step] = np.zeros(0, dtype=np.int32)
    a = oracle_attn(t)
    Ko, Vo = host(t["K"])[0].astype(np.float64), host(t["V"])[0].astype(np.float64)
    Yo, vo = host(Y).astype(np.float64), host(valid).astype(bool)
    scale = 1.0 / np.sqrt(cfg.dh)
    for s in range(T):
        pos = p0 + s
        kv.set_pos([pos])
        x = torch.randn((1, d), device="cuda")
        out = Bd.dv_sparse_attn_kvfill(attn, x, kv, Y, valid, torch.tensor(sets[s], device="cuda"), scale)
        torch.cuda.synchronize()
        ref, Ko, Vo, Yo, vo = O.mha_sparse_kvfill(host(x)[0], a, Ko, Vo, Yo, vo, pos, sets[s], scale,
                                                  y_keep=_keep(Y))
        assert rel_l2(host(out)[0], ref) < REL_TOL, (s, rel_l2(host(out)[0], ref))
        assert np.array_equal(host(valid).astype(bool), vo), s
        assert np.array_equal(host(Y)[pos].astype(np.float64), Yo[pos])   # rounded to nearest even
        Kg, Vg = host(t["K"])[0], host(t["V"])[0]
        for h in sets[s]:
            assert rel_l2(Kg[h, :pos + 1].astype(np.float64), Ko[h, :pos + 1]) < REL_TOL, (s, h)
            assert rel_l2(Vg[h, :pos + 1].astype(np.float64), Vo[h, :pos + 1]) < REL_TOL, (s, h)


def test_kvfill_equals_a_cache_with_every_head_written():
    """The same steps against a second cache in which every head writes its key and
    value at every token (dv_sparse_attn over all heads, then over the selected ones):
    the outputs agree within the tolerance."""
    cfg = get_config("small_f16")
    t = make_layer(cfg, 130, device="cuda", biases=True)
    attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], cfg.H, t["bq"], t["bk"], t["bv"], t["bo"])
    cap, d, H, T = cfg.kv_cap, cfg.d, cfg.H, 10
    p0 = cap - T
    K2, V2 = t["K"].clone(), t["V"].clone()
    kv = Bd.KVCache(t["K"], t["V"], [p0])
    kv2 = Bd.KVCache(K2, V2, [p0])
    Y = torch.zeros((cap, d), dtype=t["K"].dtype, device="cuda")
    valid = torch.zeros((H, cap), dtype=torch.uint8, device="cuda")
    valid[:, :p0] = 1
    rng = np.random.default_rng(131)
    scale = 1.0 / np.sqrt(cfg.dh)
    allh = torch.arange(H, dtype=torch.int32, device="cuda").view(1, -1)
    for s in range(T):
        kv.set_pos([p0 + s])
        kv2.set_pos([p0 + s])
        S = torch.tensor(np.sort(rng.choice(H, cfg.k_heads, replace=False)).astype(np.int32), device="cuda")
        x = torch.randn((1, d), device="cuda")
        out = Bd.dv_sparse_attn_kvfill(attn, x, kv, Y, valid, S, scale)
        Bd.dv_sparse_attn(attn, x, kv2, allh, scale)
        ref = Bd.dv_sparse_attn(attn, x, kv2, S.view(1, -1), scale)
        torch.cuda.synchronize()
        assert rel_l2(host(out)[0], host(ref)[0]) < REL_TOL, s


@pytest.mark.parametrize("name,M,wd,kvd", [("small_f16", 70, None, None), ("opt175b_b1", 150, None, None),
                                           ("small_f16", 40, "f16", "f32"), ("small_f16", 40, "f32", "f16")])
def test_kvfill_heads_missing_many_positions(name, M, wd, kvd):
    """Selected heads missing far more positions than one workgroup slice takes per
    group (4 positions x 4 slices), some contiguous and some scattered: every slice
    runs several groups, and the filled rows and the output match the oracle. Also
    with mixed weight and cache types (the kept inputs follow the cache's type)."""
    cfg = get_config(name)
    if wd is not None:
        cfg = cfg.with_(name=f"{name}_{wd}_{kvd}", wdtype=wd, kvdtype=kvd)
    t = make_layer(cfg, 140, device="cuda", biases=True)
    attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], cfg.H, t["bq"], t["bk"], t["bv"], t["bo"])
    cap, d, H = cfg.kv_cap, cfg.d, cfg.H
    pos = cap - 1
    kv = Bd.KVCache(t["K"], t["V"], [pos])
    Y = torch.zeros((cap, d), dtype=t["K"].dtype, device="cuda")
    Y[:pos] = torch.randn((pos, d), device="cuda")
    rng = np.random.default_rng(141)
    vh = np.ones((H, cap), dtype=np.uint8)
    vh[:, pos:] = 0
    vh[0, pos - M:pos] = 0                                       # a long contiguous gap
    vh[1, rng.choice(pos, M, replace=False)] = 0                 # scattered
    vh[2, rng.choice(pos, 5, replace=False)] = 0                 # a few
    valid = torch.tensor(vh, device="cuda")
    S = np.array(sorted({0, 1, 2} | set(rng.choice(np.arange(3, H), cfg.k_heads - 3, replace=False).tolist())),
                 dtype=np.int32)
    a = oracle_attn(t)
    Ko, Vo = host(t["K"])[0].astype(np.float64), host(t["V"])[0].astype(np.float64)
    Yo, vo = host(Y).astype(np.float64), vh.astype(bool)
    scale = 1.0 / np.sqrt(cfg.dh)
    x = torch.randn((1, d), device="cuda")
    out = Bd.dv_sparse_attn_kvfill(attn, x, kv, Y, valid, torch.tensor(S, device="cuda"), scale)
    torch.cuda.synchronize()
    ref, Ko, Vo, Yo, vo = O.mha_sparse_kvfill(host(x)[0], a, Ko, Vo, Yo, vo, pos, S, scale, y_keep=_keep(Y))
    assert rel_l2(host(out)[0], ref) < REL_TOL
    assert np.array_equal(host(valid).astype(bool), vo)
    Kg, Vg = host(t["K"])[0], host(t["V"])[0]
    for h in S:
        assert rel_l2(Kg[h, :pos + 1].astype(np.float64), Ko[h, :pos + 1]) < REL_TOL, h
        assert rel_l2(Vg[h, :pos + 1].astype(np.float64), Vo[h, :pos + 1]) < REL_TOL, h
    for h in (0, 1, 2):   # the filled rows themselves, not only the whole head
        miss = np.flatnonzero(vh[h, :pos] == 0)
        assert rel_l2(Kg[h, miss].astype(np.float64), Ko[h, miss]) < REL_TOL, h
        assert rel_l2(Vg[h, miss].astype(np.float64), Vo[h, miss]) < REL_TOL, h


def test_kvfill_is_deterministic():
    """The same decode steps from the same starting state, twice: outputs, filled cache
    rows, kept inputs and marks are bitwise identical (the fill adds its column halves in
    a fixed order, and every workgroup of a head lists its missing positions in order)."""
    cfg = get_config("opt175b_b1")
    t = make_layer(cfg, 150, device="cuda", biases=True)
    attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], cfg.H, t["bq"], t["bk"], t["bv"], t["bo"])
    cap, d, H, T = cfg.kv_cap, cfg.d, cfg.H, 6
    p0 = cap - T
    K0, V0 = t["K"].clone(), t["V"].clone()
    Y0 = torch.randn((cap, d), device="cuda").to(t["K"].dtype)
    v0 = torch.ones((H, cap), dtype=torch.uint8, device="cuda")
    v0[:, p0:] = 0
    v0[:, p0 - 40:p0:3] = 0                      # scattered gaps in every head
    rng = np.random.default_rng(151)
    sets = [torch.tensor(np.sort(rng.choice(H, cfg.k_heads, replace=False)).astype(np.int32), device="cuda")
            for _ in range(T)]
    xs = [torch.randn((1, d), device="cuda") for _ in range(T)]
    runs = []
    for _ in range(2):
        K, V, Y, valid = K0.clone(), V0.clone(), Y0.clone(), v0.clone()
        kv = Bd.KVCache(K, V, [p0])
        outs = []
        for s in range(T):
            kv.set_pos([p0 + s])
            outs.append(Bd.dv_sparse_attn_kvfill(attn, xs[s], kv, Y, valid, sets[s], 1.0 / np.sqrt(cfg.dh)))
        torch.cuda.synchronize()
        runs.append([host(o).tobytes() for o in outs] + [host(a).tobytes() for a in (K, V, Y, valid)])
    assert runs[0] == runs[1]


@pytest.mark.parametrize("name", ["small_f16", "opt175b_b1"])
def test_kvfill_from_the_first_token(name):
    """Decode from an empty cache (pos = 0, nothing valid yet) for a few tokens with
    changing head sets: at pos 0 nothing is missing and the listing is empty; at later
    tokens a newly selected head is missing every earlier row."""
    cfg = get_config(name)
    t = make_layer(cfg, 160, device="cuda", biases=True)
    attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], cfg.H, t["bq"], t["bk"], t["bv"], t["bo"])
    cap, d, H, T = cfg.kv_cap, cfg.d, cfg.H, 4
    kv = Bd.KVCache(t["K"], t["V"], [0])
    Y = torch.zeros((cap, d), dtype=t["K"].dtype, device="cuda")
    valid = torch.zeros((H, cap), dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(161)
    sets = _head_schedule(rng, H, cfg.k_heads, T)
    a = oracle_attn(t)
    Ko, Vo = host(t["K"])[0].astype(np.float64), host(t["V"])[0].astype(np.float64)
    Yo, vo = host(Y).astype(np.float64), host(valid).astype(bool)
    scale = 1.0 / np.sqrt(cfg.dh)
    for pos in range(T):
        kv.set_pos([pos])
        x = torch.randn((1, d), device="cuda")
        out = Bd.dv_sparse_attn_kvfill(attn, x, kv, Y, valid, torch.tensor(sets[pos], device="cuda"), scale)
        torch.cuda.synchronize()
        ref, Ko, Vo, Yo, vo = O.mha_sparse_kvfill(host(x)[0], a, Ko, Vo, Yo, vo, pos, sets[pos], scale,
                                                  y_keep=_keep(Y))
        assert rel_l2(host(out)[0], ref) < REL_TOL, pos
        assert np.array_equal(host(valid).astype(bool), vo), pos
        Kg, Vg = host(t["K"])[0], host(t["V"])[0]
        for h in sets[pos]:
            assert rel_l2(Kg[h, :pos + 1].astype(np.float64), Ko[h, :pos + 1]) < REL_TOL, (pos, h)
            assert rel_l2(Vg[h, :pos + 1].astype(np.float64), Vo[h, :pos + 1]) < REL_TOL, (pos, h)
