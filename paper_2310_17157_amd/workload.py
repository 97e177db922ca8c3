"""Wrap a layer's tensors (as drawn by the seeded generator) into binding objects."""
from typing import Dict

import torch

from .binding import LN, MLP, Attn, KVCache, Predictor


def layer_objects(t: Dict[str, torch.Tensor], H: int, use_ln: bool = True, biases: bool = True):
    """Return (attn, mlp, pred_h, pred_m, kv, ln) views of the tensors in `t`."""
    attn = Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], H,
                t.get("bq") if biases else None, t.get("bk") if biases else None,
                t.get("bv") if biases else None, t.get("bo") if biases else None)
    mlp = MLP(t["W1T"], t["W2T"], t.get("b1") if biases else None, t.get("b2") if biases else None)
    pred_h = Predictor(t["AT_h"], t["BT_h"])
    pred_m = Predictor(t["AT_m"], t["BT_m"])
    kv = KVCache(t["K"], t["V"], [int(p) for p in t["pos"]])
    ln = LN(t["g1"], t["be1"], t["g2"], t["be2"], 1e-5) if use_ln else None
    return attn, mlp, pred_h, pred_m, kv, ln
