"""Seeded input generator.

Recipe (every draw is float32 from one torch.Generator seeded with `seed`, in this
fixed order, then cast with round-to-nearest-even to the storage type):

  x      [B][d]            ~ N(0, 0.02^2), kept float32
  Wq, Wk, Wv [H*dh][d]     ~ N(0, 0.02^2)   (nn.Linear layout: head i = rows i*dh..)
  WoT    [H*dh][d]         ~ N(0, 0.02^2)   (output projection stored transposed, by head)
  W1T    [N][d]            ~ N(0, 0.02^2)   (neuron i's input weights, a contiguous row)
  W2T    [N][d]            ~ N(0, 0.02^2)   (second linear layer stored transposed)
  AT_h [r][d], BT_h [H][r] ~ N(0, 0.02^2)   (head predictor factors)
  AT_m [r][d], BT_m [N][r] ~ N(0, 0.02^2)   (neuron predictor factors)
  K, V  [B][H][cap][dh]    ~ N(0, 1) * kv_scale (K only) cast to the KV type
  then, only when requested: biases ~ N(0, 0.02^2) (otherwise zero), and layer-norm
  gamma ~ 1 + N(0, 0.1^2), beta ~ N(0, 0.1^2) (otherwise gamma = 1, beta = 0).

Index sets that are inputs rather than predictions (the batch-32 workload) are drawn
on the CPU from their own generator, so they do not depend on the device.
"""
from typing import Dict, Optional

import numpy as np
import torch

from .configs import Config

_TORCH_DT = {"f32": torch.float32, "f16": torch.float16}


def _draw(g, shape, std, dtype, device):
    t = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        t.mul_(std)
    return t.to(_TORCH_DT[dtype]) if dtype != "f32" else t


def make_layer(cfg: Config, seed: int, device="cpu", *, biases: bool = False,
               ln_random: bool = False, kv_scale: float = 1.0,
               with_predictors: bool = True, with_dense: bool = True) -> Dict[str, torch.Tensor]:
    """Draw one synthetic decoder layer plus its input and KV cache.

    with_dense=False skips the attention/MLP weights (predictor-only tests);
    with_predictors=False skips the predictor factors.
    """
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(int(seed))
    d, N, H, dh, r, B = cfg.d, cfg.N, cfg.H, cfg.dh, cfg.r, cfg.B
    wd = cfg.wdtype
    out: Dict[str, torch.Tensor] = {}
    out["x"] = _draw(g, (B, d), 0.02, "f32", dev)
    if with_dense:
        for name in ("Wq", "Wk", "Wv", "WoT"):
            out[name] = _draw(g, (H * dh, d), 0.02, wd, dev)
        out["W1T"] = _draw(g, (N, d), 0.02, wd, dev)
        out["W2T"] = _draw(g, (N, d), 0.02, wd, dev)
    if with_predictors:
        out["AT_h"] = _draw(g, (r, d), 0.02, wd, dev)
        out["BT_h"] = _draw(g, (H, r), 0.02, wd, dev)
        out["AT_m"] = _draw(g, (r, d), 0.02, wd, dev)
        out["BT_m"] = _draw(g, (N, r), 0.02, wd, dev)
    if with_dense:
        cap = cfg.kv_cap
        K = _draw(g, (B, H, cap, dh), 1.0, "f32", dev)
        if kv_scale != 1.0:
            K.mul_(kv_scale)
        out["K"] = K.to(_TORCH_DT[cfg.kvdtype]) if cfg.kvdtype != "f32" else K
        out["V"] = _draw(g, (B, H, cap, dh), 1.0, cfg.kvdtype, dev)
        zeros = lambda n: torch.zeros(n, dtype=torch.float32, device=dev)
        if biases:
            for name, n in (("bq", H * dh), ("bk", H * dh), ("bv", H * dh), ("bo", d),
                            ("b1", N), ("b2", d)):
                out[name] = _draw(g, (n,), 0.02, "f32", dev)
        else:
            for name, n in (("bq", H * dh), ("bk", H * dh), ("bv", H * dh), ("bo", d),
                            ("b1", N), ("b2", d)):
                out[name] = zeros(n)
        if ln_random:
            out["g1"] = 1.0 + _draw(g, (d,), 0.1, "f32", dev)
            out["be1"] = _draw(g, (d,), 0.1, "f32", dev)
            out["g2"] = 1.0 + _draw(g, (d,), 0.1, "f32", dev)
            out["be2"] = _draw(g, (d,), 0.1, "f32", dev)
        else:
            out["g1"] = torch.ones(d, dtype=torch.float32, device=dev)
            out["be1"] = zeros(d)
            out["g2"] = torch.ones(d, dtype=torch.float32, device=dev)
            out["be2"] = zeros(d)
        out["pos"] = torch.tensor(positions(cfg, seed), dtype=torch.int32)
    return out


def positions(cfg: Config, seed: int) -> np.ndarray:
    """Decode position per sequence (attended length = pos + 1).

    Batch 1: pos = L - 1. Batch > 1: L_b ~ U{lo..hi} from a CPU generator keyed on
    the seed, pos_b = L_b - 1.
    """
    if cfg.B == 1 or cfg.L_range is None:
        return np.full(cfg.B, cfg.L - 1, dtype=np.int32)
    rng = np.random.default_rng([int(seed), 0x4C])
    lo, hi = cfg.L_range
    return (rng.integers(lo, hi + 1, size=cfg.B) - 1).astype(np.int32)


def uniform_head_sets(cfg: Config, seed: int) -> np.ndarray:
    """Per-sequence head sets: k_heads of H drawn uniformly without replacement, ascending."""
    rng = np.random.default_rng([int(seed), 0x48])
    sets = [np.sort(rng.permutation(cfg.H)[: cfg.k_heads]) for _ in range(cfg.B)]
    return np.stack(sets).astype(np.int32)


def zipf_mlp_sets(cfg: Config, seed: int, s: Optional[float] = None) -> np.ndarray:
    """Per-sequence neuron sets with Zipf(s)-skewed popularity, ascending.

    A seeded permutation assigns each neuron a popularity rank rho(i) in 1..N with
    weight rho(i)^-s; each sequence draws k_mlp neurons without replacement in
    proportion to those weights (Gumbel-top-k: the k largest log w_i + Gumbel_i).
    """
    s = cfg.zipf_s if s is None else s
    rng = np.random.default_rng([int(seed), 0x5A])
    rho = rng.permutation(cfg.N) + 1
    logw = -s * np.log(rho.astype(np.float64))
    sets = []
    for _ in range(cfg.B):
        gumbel = -np.log(-np.log(rng.random(cfg.N)))
        keys = logw + gumbel
        top = np.argpartition(-keys, cfg.k_mlp - 1)[: cfg.k_mlp]
        sets.append(np.sort(top))
    return np.stack(sets).astype(np.int32)


def to_numpy64(t: torch.Tensor) -> np.ndarray:
    """Exact upcast of stored values (fp16, including subnormals, or fp32) to float64."""
    return t.detach().to("cpu").to(torch.float64).numpy()


def quantize_q4(W: torch.Tensor, block: int = 32):
    """4-bit weights in blocks of `block` elements of a row, for W4A16 inputs: per block
    an fp16 scale s = max|w| / 7 (1 for an all-zero block) and codes
    q = clamp(round(w / s), -8, 7) + 8 in [0, 15], two per byte (low nibble first).
    Returns (packed uint8 [rows, d/2], scales fp16 [rows, d/block]) on W's device."""
    rows, d = W.shape
    assert d % block == 0 and block % 2 == 0
    w = W.float().view(rows, d // block, block)
    s = (w.abs().amax(dim=-1) / 7.0).half()
    s = torch.where(s == 0, torch.ones_like(s), s)
    q = torch.clamp(torch.round(w / s.float()[..., None]), -8, 7).to(torch.int32) + 8
    q = q.view(rows, d)
    packed = (q[:, 0::2] | (q[:, 1::2] << 4)).to(torch.uint8)
    return packed.contiguous(), s.contiguous()
