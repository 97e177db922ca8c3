"""Algorithmic bytes and FLOPs of the decode hot path (what the method must move).

Per layer and token, with s_w the weight element size and s_kv the KV element size:
  dense attention weights   4 d^2 s_w bytes, 8 d^2 FLOP     (Table 2, Section 2.2)
  dense MLP weights         2 d N s_w bytes, 4 d N FLOP     (16 d^2 at N = 4d)
  sparse MLP (rows of W1T and W2T for S_M)      k * 2 d s_w
  sparse attention weights (Wq, Wk, Wv, WoT rows of S_A)   k_h * 4 d_h d s_w
  KV read for S_A (pos + 1 positions, keys and values)     k_h * 2 L d_h s_kv
  predictor factors (AT_h, BT_h, AT_m, BT_m)    (d r + r H + d r + r N) s_w
Activations, biases and layer-norm parameters are below 0.1 % and are not counted.
"""
from dataclasses import dataclass


@dataclass(frozen=True)
class Bytes:
    mlp: int
    attn_w: int
    kv: int
    pred_h: int
    pred_m: int

    @property
    def attn(self) -> int:
        return self.attn_w + self.kv

    @property
    def block(self) -> int:
        return self.mlp + self.attn

    @property
    def pred(self) -> int:
        return self.pred_h + self.pred_m

    @property
    def total(self) -> int:
        return self.block + self.pred


def dense_attention_flops(d: int) -> int:
    return 8 * d * d


def dense_attention_bytes(d: int, s_w: int) -> int:
    return 4 * d * d * s_w


def dense_mlp_flops(d: int, N: int) -> int:
    return 4 * d * N


def dense_mlp_bytes(d: int, N: int, s_w: int) -> int:
    return 2 * d * N * s_w


def sparse_mlp_bytes(d: int, k: int, s_w: int) -> int:
    return 2 * k * d * s_w


def sparse_attn_weight_bytes(d: int, dh: int, k_heads: int, s_w: int) -> int:
    return 4 * k_heads * dh * d * s_w


def kv_bytes(dh: int, k_heads: int, attended: int, s_kv: int) -> int:
    return 2 * k_heads * attended * dh * s_kv


def predictor_bytes(d: int, r: int, n_out: int, s_w: int) -> int:
    return (d * r + r * n_out) * s_w


def layer_bytes(cfg, attended=None) -> Bytes:
    """Algorithmic bytes for one token of a batch-1 workload `cfg` (a synth Config)."""
    L = cfg.L if attended is None else attended
    return Bytes(
        mlp=sparse_mlp_bytes(cfg.d, cfg.k_mlp, cfg.wbytes),
        attn_w=sparse_attn_weight_bytes(cfg.d, cfg.dh, cfg.k_heads, cfg.wbytes),
        kv=kv_bytes(cfg.dh, cfg.k_heads, L, cfg.kvbytes),
        pred_h=predictor_bytes(cfg.d, cfg.r, cfg.H, cfg.wbytes),
        pred_m=predictor_bytes(cfg.d, cfg.r, cfg.N, cfg.wbytes),
    )


def batch_bytes(cfg, union_size: int, head_union: int, attended_per_seq_heads: int) -> dict:
    """Algorithmic bytes of one batch step: union MLP rows, union head weights, per-(b, h) KV."""
    return dict(
        mlp=sparse_mlp_bytes(cfg.d, union_size, cfg.wbytes),
        attn_w=sparse_attn_weight_bytes(cfg.d, cfg.dh, head_union, cfg.wbytes),
        kv=2 * attended_per_seq_heads * cfg.dh * cfg.kvbytes,
    )
