"""Helpers for the GPU parity tests: seeded layers on the device, the same values for
the oracle on the host, and the parity rules (relative L2 error and set equality up
to predictor-score near-ties)."""
import numpy as np
import torch

from synth import get_config, make_layer, to_numpy64

REL_TOL = 2e-3         # max relative L2 error of an output vector (fp16 weights, fp32 accumulation)
NEAR_TIE = 1e-3        # relative band around the k-th score inside which set membership may differ


def layer(cfg_name, seed, **kw):
    """A seeded layer on the GPU for a named configuration (or a Config)."""
    cfg = get_config(cfg_name) if isinstance(cfg_name, str) else cfg_name
    return cfg, make_layer(cfg, seed, device="cuda", **kw)


def host(t):
    """Stored values on the host: fp16 stays fp16 (the oracle upcasts rows exactly)."""
    if t is None:
        return None
    a = t.detach().cpu()
    return a.numpy() if a.dtype in (torch.float16, torch.int32, torch.int64) else a.to(torch.float64).numpy()


def oracle_attn(t, biases=True):
    d = {k: host(t[k]) for k in ("Wq", "Wk", "Wv", "WoT")}
    if biases:
        d.update({k: host(t[k]) for k in ("bq", "bk", "bv", "bo")})
    return d


def oracle_mlp(t, biases=True):
    d = {"W1T": host(t["W1T"]), "W2T": host(t["W2T"])}
    if biases:
        d.update(b1=host(t["b1"]), b2=host(t["b2"]))
    return d


def oracle_ln(t):
    return dict(g1=host(t["g1"]), be1=host(t["be1"]), g2=host(t["g2"]), be2=host(t["be2"]), eps=1e-5)


def rel_l2(gpu, ref):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-300))


def near_tie_band(scores, k):
    """Indices whose score is within NEAR_TIE (relative) of the oracle's k-th largest."""
    s = np.asarray(scores, dtype=np.float64)
    tau = np.sort(s)[::-1][k - 1]
    scale = max(abs(tau), float(np.sqrt(np.mean(s * s))))
    return set(np.nonzero(np.abs(s - tau) <= NEAR_TIE * scale)[0].tolist())


def check_topk_set(gpu_set, oracle_scores, k):
    """|G| = |O| = k, G ascending and unique, and G xor O inside the near-tie band."""
    from oracle import dejavu as O
    g = [int(v) for v in np.asarray(gpu_set).reshape(-1)]
    assert len(g) == k
    assert all(a < b for a, b in zip(g, g[1:])), "GPU set not strictly ascending"
    o = set(O.select_topk(oracle_scores, k).tolist())
    diff = set(g) ^ o
    band = near_tie_band(oracle_scores, k)
    assert diff <= band, f"set mismatch outside the near-tie band: {sorted(diff - band)[:10]}"
    return len(diff), len(band)
