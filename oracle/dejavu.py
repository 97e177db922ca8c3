"""Plain fp64 CPU oracle of the Deja Vu decode hot path (arXiv 2310.17157).

TEST INFRASTRUCTURE ONLY. This module exists to check the HIP library. Only the
test-suite, the package's smoke check and the CPU-baseline leg of the benchmark may
import it; the library and its Python binding never do, and it imports nothing from
them. It is slow on purpose: every function is the paper's definition written out
in float64 NumPy, with no blocking, fusion or reordering beyond what the definition
states, so that it can be checked against the paper by eye.

Where it follows the paper
  * Sparsified MLP, Section 2.3 "Problem Formulation", Eq. (1):
        MLP_{S_M}(y) = sigma(y W^1_{S_M}) (W^2_{S_M})^T, sigma = ReLU.
    Neuron i is column i of W^1 and W^2; it is stored here as row i of W1T = (W^1)^T
    and W2T = (W^2)^T (the transposed storage of Section 4.4 "Memory coalescing").
  * Sparsified MHA, Section 2.3, Eq. (2) and the definition of D_i:
        MHA_{S_A}(y) = sum_{i in S_A} H_i(y) W^O_i,
        H_i(y) = D_i(y)^{-1} exp(y W^Q_i (W^K_i)^T X^T) X W^V_i,
        D_i(y) = exp(y W^Q_i (W^K_i)^T X^T) 1_n.
    At decode time X W^K_i and X W^V_i are the cached keys and values of head i.
  * Sparsity predictors, Section 4.1 "Design" and Section 4.2 "Approach": a small
    two-layer fully connected network per block whose output scores neurons (or
    heads, one class per head) for the set S_M (S_A).
  * Layer recurrences, Section 4.3 (sequential form and look-ahead form) and the
    residual form of Appendix C.3 (y~ = y + MHA(y), y^ = y~ + MLP(y~)), with the
    normalisation before each block noted in Appendix B.
  * Batch union, Section 5.2 and Appendix C.1: the sparse GEMM runs on the union of
    the sets of the sequences in the batch.

Readings where the paper is silent or loose (each is also listed in the design notes):
  R1  Eq. (2) has no 1/sqrt(d_h); an explicit `scale` argument carries it (1 reproduces
      Eq. (2) literally).
  R2  The formulas have no biases; OPT layers do. Biases are optional and added once
      (b1 per neuron before sigma; b2, bo once per output).
  R3  X holds the past tokens and the current one: attention covers cache rows
      0..pos-1 and the fresh key/value at pos.
  R4  sigma is ReLU (OPT) by default; GeLU (BLOOM) is the other choice Section 2.3
      names (see R16).
  R5  The predictor is the linear low-rank map s = (x A) B with A = AT^T (d x r),
      B = BT^T (r x n): no hidden activation, no bias.
  R6  The rule from scores to a set: top-k of the raw scores (ties: lower index
      first), or the threshold rule {i : s_i >= t} of Algorithm 1. Sets are
      returned ascending.
  R7  Pre-LN placement with biased variance; a missing LN is the identity.
  R8  Look-ahead: both sets come from the attention block's input LN1(y) of the same
      layer; sequential: S_M comes from LN2(y~).
  R9  Batch > 1: the MLP runs on the union U of the per-sequence sets for every
      sequence ("union"), or on each sequence's own set ("masked"); attention uses
      each sequence's own head set and its own position.
  R15 4-bit weights (Section 5.2, W4A16; the paper fixes no format): each row in
      blocks of 32 elements with one fp16 scale per block, element = scale * (q - 8)
      for a 4-bit code q, two codes per byte, the even element in the low nibble.
  R16 GeLU is the exact form x * Phi(x) with the normal CDF written through erf.
  R17 Cross-layer look-ahead (Section 4.3): the sets of layer l+1 come from layer
      l+1's own predictors (they score its heads and neurons) applied to layer l's
      normalised input LN1^l(y_l); layer 0's sets from its predictors on LN1^0(y_0).
  R18 Missing keys and values (Section 4.2): the kept per-token input is the
      attention block's normalised input (what the keys and values are computed
      from), stored in the cache's type (an fp16 cache keeps it rounded to the
      nearest half, like the keys and values themselves); a head selected now gets
      its missing rows from it before it attends.

Parity pins: every function here is checked in tests/test_oracle_*.py against
something other than itself (closed forms, brute force on tiny shapes, invariants,
library routines for special cases, and the values printed in Tables 1-2).
"""
import math
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=F64)


# --------------------------------------------------------------------------- LN
def layer_norm(x, gamma=None, beta=None, eps: float = 1e-5) -> np.ndarray:
    """Layer normalisation over the last axis (biased variance), reading R7.

    gamma is None means no normalisation at all (identity), which is the literal
    form of the residual recurrences.
    """
    x = _f64(x)
    if gamma is None:
        return x.copy()
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps)
    y = y * _f64(gamma)
    if beta is not None:
        y = y + _f64(beta)
    return y


# ------------------------------------------------------------------- predictors
def predictor_scores(x, AT, BT) -> np.ndarray:
    """Scores of the two-layer predictor (Section 4.1 "Design", reading R5).

    x: [d] or [B, d]; AT: [r, d] (row m = column m of A); BT: [n, r] (row i = column
    i of B). Returns s = (x A) B with shape [n] or [B, n].
    """
    x = _f64(x)
    A = _f64(AT).T          # d x r
    Bm = _f64(BT).T         # r x n
    hidden = x @ A          # first layer
    return hidden @ Bm      # second layer


def select_topk(s, k: int) -> np.ndarray:
    """S = the k highest-scoring indices (reading R6), ascending.

    Order by (-s_i, i) so that among equal scores the lower index wins.
    """
    s = _f64(s)
    n = s.shape[0]
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    order = sorted(range(n), key=lambda i: (-s[i], i))
    return np.array(sorted(order[:k]), dtype=np.int64)


def select_threshold(s, t: float) -> np.ndarray:
    """S = {i : s_i >= t} (the labelling rule of Algorithm 1), ascending."""
    s = _f64(s)
    return np.array([i for i in range(s.shape[0]) if s[i] >= t], dtype=np.int64)


# -------------------------------------------------------------------------- MLP
_erf = np.vectorize(math.erf, otypes=[F64])


def activation(z, act: str = "relu") -> np.ndarray:
    """sigma of Eq. (1): ReLU (OPT, reading R4) or GeLU, x * Phi(x) with the normal CDF
    Phi(x) = (1 + erf(x / sqrt 2)) / 2 (the exact form, not a tanh approximation)."""
    z = _f64(z)
    if act == "relu":
        return np.maximum(z, 0.0)
    if act == "gelu":
        return 0.5 * z * (1.0 + _erf(z / math.sqrt(2.0)))
    raise ValueError(act)


def mlp_dense(y, W1T, b1, W2T, b2, act: str = "relu") -> np.ndarray:
    """Dense MLP: sigma(y W^1 + b1) (W^2)^T + b2."""
    y = _f64(y)
    z = y @ _f64(W1T).T
    if b1 is not None:
        z = z + _f64(b1)
    a = activation(z, act)
    out = a @ _f64(W2T)
    if b2 is not None:
        out = out + _f64(b2)
    return out


def mlp_sparse(y, W1T, b1, W2T, b2, S, act: str = "relu") -> np.ndarray:
    """Eq. (1): sum over i in S of sigma(y . W^1_i + b1_i) * W^2_i, plus b2 once.

    Gather form: one neuron at a time, in the order S lists them.
    y: [d] (one token). Returns [d].
    """
    y = _f64(y)
    W1T = np.asarray(W1T)
    W2T = np.asarray(W2T)
    d = y.shape[0]
    out = np.zeros(d, dtype=F64) if b2 is None else _f64(b2).copy()
    for i in S:
        i = int(i)
        z = float(np.dot(y, _f64(W1T[i])))
        if b1 is not None:
            z += float(b1[i])
        a = (z if z > 0.0 else 0.0) if act == "relu" else float(activation(z, act))
        out += a * _f64(W2T[i])
    return out


def mlp_sparse_masked(y, W1T, b1, W2T, b2, S, act: str = "relu") -> np.ndarray:
    """Eq. (1) in mask form: (ReLU(y W^1 + b1) * 1_S) (W^2)^T + b2.

    An independent formulation of mlp_sparse (dense products, then a 0/1 mask).
    """
    y = _f64(y)
    mask = np.zeros(np.asarray(W1T).shape[0], dtype=F64)
    mask[np.asarray(S, dtype=np.int64)] = 1.0
    z = y @ _f64(W1T).T
    if b1 is not None:
        z = z + _f64(b1)
    a = activation(z, act) * mask
    out = a @ _f64(W2T)
    if b2 is not None:
        out = out + _f64(b2)
    return out


def mlp_activations(y, W1T, b1, S) -> np.ndarray:
    """ReLU(y . W^1_i + b1_i) for i in S, in S order (the first half of Eq. (1))."""
    y = _f64(y)
    W1T = np.asarray(W1T)
    out = np.empty(len(S), dtype=F64)
    for j, i in enumerate(S):
        z = float(np.dot(y, _f64(W1T[int(i)])))
        if b1 is not None:
            z += float(b1[int(i)])
        out[j] = z if z > 0.0 else 0.0
    return out


# ----------------------------------------------------------- 4-bit weights (W4A16)
Q4_BLOCK = 32   # elements per scale (reading R15)


def dequant_q4(packed, scales, d: int) -> np.ndarray:
    """Rows of 4-bit weights (Section 5.2 "Compatibility with Quantization", W4A16;
    format of reading R15): element j of a row is scales[j // 32] * (q_j - 8), where q_j
    is the low 4 bits of byte j // 2 for even j and the high 4 bits for odd j.
    packed: [rows, d/2] uint8; scales: [rows, d/32] (fp16 values). Returns [rows, d] fp64."""
    packed = np.asarray(packed, dtype=np.uint8)
    rows = packed.shape[0]
    q = np.empty((rows, d), dtype=F64)
    q[:, 0::2] = packed & 15          # even elements: low nibbles
    q[:, 1::2] = packed >> 4          # odd elements: high nibbles
    s = np.repeat(_f64(scales), Q4_BLOCK, axis=1)    # element j -> scale of block j // 32
    return s * (q - 8.0)


def dequant_q4_rows(packed, scales, d: int, rows) -> np.ndarray:
    """dequant_q4 of the listed rows only (a gathered set), in list order."""
    rows = [int(i) for i in rows]
    return dequant_q4(np.asarray(packed)[rows], np.asarray(scales)[rows], d)


# -------------------------------------------------------------------- attention
def head_projection(y, W, b, i: int, dh: int) -> np.ndarray:
    """y W_i for head i, where W is stored [H*dh, d] and head i is rows i*dh..(i+1)*dh."""
    y = _f64(y)
    rows = _f64(np.asarray(W)[i * dh:(i + 1) * dh])
    v = rows @ y
    if b is not None:
        v = v + _f64(b)[i * dh:(i + 1) * dh]
    return v


def attention_head(q, Kh, Vh, scale: float) -> np.ndarray:
    """H_i of Eq. (2) for one head at decode time.

    q: [dh]; Kh, Vh: [n, dh] (keys X W^K_i and values X W^V_i of all n attended tokens).
    D_i^{-1} exp(sigma) is computed as exp(sigma - max sigma) / sum exp(sigma - max sigma),
    which is the same number.
    """
    q = _f64(q)
    Kh = _f64(Kh)
    Vh = _f64(Vh)
    sigma = scale * (Kh @ q)                 # [n]
    e = np.exp(sigma - sigma.max())
    D = e.sum()
    return (e / D) @ Vh                      # [dh]


def mha_sparse(y, attn: Dict, K, V, pos: int, S_A, scale: float
               ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, Dict[int, np.ndarray]]:
    """Sparsified MHA (Section 2.3) for one token, with the KV-cache step of Section 4.2.

    attn: Wq, Wk, Wv, WoT ([H*dh, d]) and optional bq, bk, bv ([H*dh]), bo ([d]);
    K, V: [H, cap, dh] cache of this sequence (read only; copies are returned).
    For every selected head i the fresh key/value are written at row `pos` (only for
    the selected heads, Section 4.2) and attention covers rows 0..pos (reading R3).
    Returns (out [d], K_new, V_new, {i: H_i(y)}).
    """
    y = _f64(y)
    H, cap, dh = np.asarray(K).shape
    K_new = _f64(K).copy()
    V_new = _f64(V).copy()
    d = y.shape[0]
    bo = attn.get("bo")
    out = np.zeros(d, dtype=F64) if bo is None else _f64(bo).copy()
    heads = {}
    WoT = np.asarray(attn["WoT"])
    for i in S_A:
        i = int(i)
        q = head_projection(y, attn["Wq"], attn.get("bq"), i, dh)
        k = head_projection(y, attn["Wk"], attn.get("bk"), i, dh)
        v = head_projection(y, attn["Wv"], attn.get("bv"), i, dh)
        K_new[i, pos] = k
        V_new[i, pos] = v
        Hi = attention_head(q, K_new[i, :pos + 1], V_new[i, :pos + 1], scale)
        heads[i] = Hi
        out += Hi @ _f64(WoT[i * dh:(i + 1) * dh])      # H_i(y) W^O_i
    return out, K_new, V_new, heads


def mha_sparse_kvfill(y, attn: Dict, K, V, Y, valid, pos: int, S_A, scale: float, y_keep=None):
    """Sparsified MHA for one token with the missing-KV rule of Section 4.2 ("Approach").

    Keys and values are computed only for the selected heads, so a head that was not
    selected at some past token has no cache row there. The token's attention input y
    is kept for every token (Y[pos] = y); when a head is selected, the rows it is
    missing are computed from the kept inputs (K[h, t] = Y[t] W^K_h + b, likewise V)
    before the head attends, and marked present. valid[h, t] is True where row t of
    head h holds that token's key and value; after the call it is True for every row
    0..pos of the selected heads and False at pos for the others.
    y_keep: the storage type of the kept inputs (reading R18: the cache's type); None
    keeps y exactly, np.float16 keeps y rounded to the nearest half (ties to even), as
    an fp16 store of it holds.
    Y: [cap, d]; valid: [H, cap] bool (neither is modified; copies are returned).
    Returns (out [d], K_new, V_new, Y_new, valid_new).
    """
    y = _f64(y)
    H, cap, dh = np.asarray(K).shape
    K_fill = _f64(K).copy()
    V_fill = _f64(V).copy()
    Y_new = _f64(Y).copy()
    valid_new = np.asarray(valid, dtype=bool).copy()
    Y_new[pos] = y if y_keep is None else y.astype(y_keep).astype(np.float64)
    for i in S_A:
        i = int(i)
        for t in range(pos):
            if not valid_new[i, t]:
                K_fill[i, t] = head_projection(Y_new[t], attn["Wk"], attn.get("bk"), i, dh)
                V_fill[i, t] = head_projection(Y_new[t], attn["Wv"], attn.get("bv"), i, dh)
                valid_new[i, t] = True
    out, K_new, V_new, _ = mha_sparse(y, attn, K_fill, V_fill, pos, S_A, scale)
    sel = set(int(i) for i in S_A)
    for i in range(H):
        valid_new[i, pos] = i in sel
    return out, K_new, V_new, Y_new, valid_new


def mha_dense_einsum(y, attn: Dict, K, V, pos: int, scale: float) -> np.ndarray:
    """Dense multi-head attention written as textbook batched tensor algebra.

    An independent formulation: all heads at once with einsum over [H, T, dh].
    """
    y = _f64(y)
    H, cap, dh = np.asarray(K).shape
    d = y.shape[0]

    def proj(W, b):
        t = np.einsum("od,d->o", _f64(W), y)
        if b is not None:
            t = t + _f64(b)
        return t.reshape(H, dh)

    q = proj(attn["Wq"], attn.get("bq"))
    k = proj(attn["Wk"], attn.get("bk"))
    v = proj(attn["Wv"], attn.get("bv"))
    Kc = np.concatenate([_f64(K)[:, :pos], k[:, None, :]], axis=1)    # [H, T, dh]
    Vc = np.concatenate([_f64(V)[:, :pos], v[:, None, :]], axis=1)
    logits = scale * np.einsum("hd,htd->ht", q, Kc)
    logits = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(logits)
    p = p / p.sum(axis=1, keepdims=True)
    o = np.einsum("ht,htd->hd", p, Vc)                                 # [H, dh]
    out = np.einsum("hd,hde->e", o, _f64(attn["WoT"]).reshape(H, dh, d))
    bo = attn.get("bo")
    if bo is not None:
        out = out + _f64(bo)
    return out


# ------------------------------------------------------------------------ block
def sparse_block(y, attn: Dict, mlp: Dict, K, V, pos: int, scale: float, *,
                 S_A=None, S_M=None, pred_h: Optional[Dict] = None,
                 pred_m: Optional[Dict] = None, k_heads: Optional[int] = None,
                 k_mlp: Optional[int] = None, ln: Optional[Dict] = None,
                 mode: str = "lookahead") -> Dict:
    """One decoder layer for one token with contextual sparsity (Section 4.3).

    y~ = y + MHA_{S_A}(LN1(y)); y^ = y~ + MLP_{S_M}(LN2(y~)).
    Sets are taken as given when S_A / S_M are passed; otherwise they are predicted:
    S_A = top-k_heads(SP_A(LN1(y))); S_M = top-k_mlp(SP_M(LN1(y))) in look-ahead mode
    or top-k_mlp(SP_M(LN2(y~))) in sequential mode (reading R8).
    Returns a dict with out, y_tilde, attn_out, mlp_out, S_A, S_M, K_new, V_new and
    the predictor scores used.
    """
    ln = ln or {}
    y = _f64(y)
    x1 = layer_norm(y, ln.get("g1"), ln.get("be1"), ln.get("eps", 1e-5))
    res = {}
    if S_A is None:
        s_h = predictor_scores(x1, pred_h["AT"], pred_h["BT"])
        S_A = select_topk(s_h, k_heads)
        res["scores_h"] = s_h
    if S_M is None and mode == "lookahead":
        s_m = predictor_scores(x1, pred_m["AT"], pred_m["BT"])
        S_M = select_topk(s_m, k_mlp)
        res["scores_m"] = s_m
    attn_out, K_new, V_new, _ = mha_sparse(x1, attn, K, V, pos, S_A, scale)
    y_t = y + attn_out
    x2 = layer_norm(y_t, ln.get("g2"), ln.get("be2"), ln.get("eps", 1e-5))
    if S_M is None:
        s_m = predictor_scores(x2, pred_m["AT"], pred_m["BT"])
        S_M = select_topk(s_m, k_mlp)
        res["scores_m"] = s_m
    mlp_out = mlp_sparse(x2, mlp["W1T"], mlp.get("b1"), mlp["W2T"], mlp.get("b2"), S_M)
    res.update(out=y_t + mlp_out, y_tilde=y_t, attn_out=attn_out, mlp_out=mlp_out,
               S_A=np.asarray(S_A), S_M=np.asarray(S_M), K_new=K_new, V_new=V_new)
    return res


def lookahead_layers(y, layers: Sequence[Dict], scale: float, k_heads: int, k_mlp: int,
                     S0: Optional[Tuple] = None) -> Dict:
    """Several decoder layers with the cross-layer look-ahead of Section 4.3 ("Approach").

    The sets used by layer l come from its predictors applied to the normalised input of
    the layer before it, so that they can be computed while that layer runs:
        S^0     = (top-k_heads(SP_A^0(x_0)), top-k_mlp(SP_M^0(x_0))),  x_0 = LN1^0(y_0)
        S^{l+1} = (top-k_heads(SP_A^{l+1}(x_l)), top-k_mlp(SP_M^{l+1}(x_l))), x_l = LN1^l(y_l)
        y_{l+1} = sparse_block_l(y_l; S^l)
    (the paper writes the predictor that produces S^{l+1} from y_l as SP^l; here it is
    stored with layer l+1, whose heads and neurons it scores, reading R17). S0, if given,
    replaces the prediction of S^0. layers[l] holds attn, mlp, K, V (the layer's cache
    of this sequence), pos, pred_h and pred_m ({AT, BT}) and ln.
    Returns {out, y: [y_0..y_L], S_A, S_M (per layer), K_new, V_new (per layer)}.
    """
    y = _f64(y)

    def predict(layer, x):
        s_h = predictor_scores(x, layer["pred_h"]["AT"], layer["pred_h"]["BT"])
        s_m = predictor_scores(x, layer["pred_m"]["AT"], layer["pred_m"]["BT"])
        return select_topk(s_h, k_heads), select_topk(s_m, k_mlp)

    def norm1(layer, v):
        ln = layer.get("ln") or {}
        return layer_norm(v, ln.get("g1"), ln.get("be1"), ln.get("eps", 1e-5))

    sets = S0 if S0 is not None else predict(layers[0], norm1(layers[0], y))
    res = {"y": [y], "S_A": [], "S_M": [], "K_new": [], "V_new": []}
    for l, layer in enumerate(layers):
        nxt = predict(layers[l + 1], norm1(layer, y)) if l + 1 < len(layers) else None
        r = sparse_block(y, layer["attn"], layer["mlp"], layer["K"], layer["V"], layer["pos"], scale,
                         S_A=sets[0], S_M=sets[1], ln=layer.get("ln"))
        res["S_A"].append(np.asarray(sets[0]))
        res["S_M"].append(np.asarray(sets[1]))
        res["K_new"].append(r["K_new"])
        res["V_new"].append(r["V_new"])
        y = r["out"]
        res["y"].append(y)
        sets = nxt
    res["out"] = y
    return res


def dense_block(y, attn: Dict, mlp: Dict, K, V, pos: int, scale: float,
                ln: Optional[Dict] = None) -> np.ndarray:
    """The dense layer: y~ = y + MHA(LN1(y)), y^ = y~ + MLP(LN2(y~))."""
    ln = ln or {}
    y = _f64(y)
    x1 = layer_norm(y, ln.get("g1"), ln.get("be1"), ln.get("eps", 1e-5))
    y_t = y + mha_dense_einsum(x1, attn, K, V, pos, scale)
    x2 = layer_norm(y_t, ln.get("g2"), ln.get("be2"), ln.get("eps", 1e-5))
    return y_t + mlp_dense(x2, mlp["W1T"], mlp.get("b1"), mlp["W2T"], mlp.get("b2"))


# ------------------------------------------------------------------------ batch
def union_of_sets(sets: Sequence[Sequence[int]]) -> np.ndarray:
    """U = union of the per-sequence sets (Section 5.2, Appendix C.1), ascending."""
    u = set()
    for s in sets:
        u.update(int(i) for i in s)
    return np.array(sorted(u), dtype=np.int64)


def mlp_batch(Y, W1T, b1, W2T, b2, sets, mode: str = "union") -> np.ndarray:
    """Batched sparse MLP (reading R9). Y: [B, d]; sets: per-sequence S_M^b.

    union: every sequence uses U; masked: sequence b uses its own S_M^b.
    """
    Y = _f64(Y)
    if mode == "union":
        U = union_of_sets(sets)
        return np.stack([mlp_sparse(Y[b], W1T, b1, W2T, b2, U) for b in range(Y.shape[0])])
    return np.stack([mlp_sparse(Y[b], W1T, b1, W2T, b2, sets[b]) for b in range(Y.shape[0])])


def mlp_union_rows(Y, W1T, b1, W2T, b2, U, rows_per_step: int = 2048, act: str = "relu") -> np.ndarray:
    """Eq. (1) on the rows U for every sequence of a batch, as matrix products.

    out[b] = b2 + sum_{i in U} ReLU(Y[b] . W^1_i + b1_i) W^2_i, taken over slices of U
    (rows_per_step neurons at a time, so that a slice of fp16 rows upcast to float64
    stays small). The same sum as mlp_sparse for each sequence, grouped by slices
    of neurons instead of one neuron at a time. Y: [B, d]; returns [B, d].
    """
    Y = _f64(Y)
    W1T = np.asarray(W1T)
    W2T = np.asarray(W2T)
    U = np.asarray(U, dtype=np.int64)
    out = np.zeros((Y.shape[0], W1T.shape[1]), dtype=F64)
    if b2 is not None:
        out += _f64(b2)
    for c0 in range(0, U.shape[0], rows_per_step):
        rows = U[c0:c0 + rows_per_step]
        z = Y @ _f64(W1T[rows]).T                 # [B, rows]
        if b1 is not None:
            z = z + _f64(b1)[rows]
        out += activation(z, act) @ _f64(W2T[rows])
    return out


def mha_batch(Y, attn: Dict, K, V, pos: Sequence[int], head_sets, scale: float):
    """Batched sparse MHA: sequence b uses its own head set, cache K[b], V[b] and pos[b].

    Returns (out [B, d], K_new [B, H, cap, dh], V_new).
    """
    Y = _f64(Y)
    outs, Ks, Vs = [], [], []
    for b in range(Y.shape[0]):
        o, Kn, Vn, _ = mha_sparse(Y[b], attn, np.asarray(K)[b], np.asarray(V)[b],
                                  int(pos[b]), head_sets[b], scale)
        outs.append(o)
        Ks.append(Kn)
        Vs.append(Vn)
    return np.stack(outs), np.stack(Ks), np.stack(Vs)
