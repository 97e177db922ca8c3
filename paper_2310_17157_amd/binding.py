"""ctypes binding of libdejavu_hip.so (the C ABI declared in include/dv.h).

Argument marshalling only: torch tensors supply device memory and the current
stream; every step of the computation runs in the library's HIP kernels. The
library is loaded from this package directory and nothing else is tried: if it is
missing, loading raises (there is no CPU fallback).

Entry points keep the C names: dv_predict_mlp, dv_predict_heads, dv_sparse_mlp,
dv_sparse_attn, dv_sparse_block. Each takes the tensors, allocates outputs and the
workspace with torch when they are not given, calls the C function on the current
stream and raises DvError on a non-zero status.
"""
import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_size_t, c_uint32, c_void_p
from dataclasses import dataclass
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdejavu_hip.so")

DV_F32, DV_F16, DV_Q4 = 0, 1, 2
DV_ACT_RELU, DV_ACT_GELU = 0, 1
DV_SELECT_TOPK, DV_SELECT_THRESHOLD = 0, 1
DV_LOOKAHEAD, DV_SEQUENTIAL = 0, 1
DV_MLP_UNION, DV_MLP_MASKED = 0, 1
DV_DETERMINISTIC, DV_VALIDATE = 1, 2
(DV_OK, DV_ERR_NULL, DV_ERR_SHAPE, DV_ERR_DTYPE, DV_ERR_ALIGN, DV_ERR_WORKSPACE, DV_ERR_INDEX, DV_ERR_HIP,
 DV_ERR_UNSUPPORTED, DV_ERR_ARG) = range(10)

STATUS = {0: "DV_OK", 1: "DV_ERR_NULL", 2: "DV_ERR_SHAPE", 3: "DV_ERR_DTYPE", 4: "DV_ERR_ALIGN",
          5: "DV_ERR_WORKSPACE", 6: "DV_ERR_INDEX", 7: "DV_ERR_HIP", 8: "DV_ERR_UNSUPPORTED",
          9: "DV_ERR_ARG"}


class DvError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn}: {STATUS.get(status, status)} ({msg})")
        self.status = status


class CPredictor(ctypes.Structure):
    _fields_ = [("d", c_int32), ("r", c_int32), ("n_out", c_int32), ("wtype", c_int32),
                ("AT", c_void_p), ("BT", c_void_p)]


class CMlp(ctypes.Structure):
    _fields_ = [("d", c_int32), ("n", c_int32), ("wtype", c_int32), ("act", c_int32),
                ("W1T", c_void_p), ("b1", c_void_p), ("W2T", c_void_p), ("b2", c_void_p)]


class CMlpQ4(ctypes.Structure):
    _fields_ = [("d", c_int32), ("n", c_int32), ("act", c_int32), ("reserved", c_int32),
                ("W1T", c_void_p), ("S1", c_void_p), ("b1", c_void_p),
                ("W2T", c_void_p), ("S2", c_void_p), ("b2", c_void_p)]


class CAttn(ctypes.Structure):
    _fields_ = [("d", c_int32), ("H", c_int32), ("dh", c_int32), ("wtype", c_int32),
                ("Wq", c_void_p), ("Wk", c_void_p), ("Wv", c_void_p),
                ("bq", c_void_p), ("bk", c_void_p), ("bv", c_void_p),
                ("WoT", c_void_p), ("bo", c_void_p)]


class CKV(ctypes.Structure):
    _fields_ = [("B", c_int32), ("H", c_int32), ("dh", c_int32), ("cap", c_int32),
                ("ktype", c_int32), ("reserved", c_int32), ("K", c_void_p), ("V", c_void_p),
                ("pos", POINTER(c_int32))]


class CLN(ctypes.Structure):
    _fields_ = [("g1", c_void_p), ("be1", c_void_p), ("g2", c_void_p), ("be2", c_void_p),
                ("eps", c_float)]


class CLayer(ctypes.Structure):
    _fields_ = [("attn", CAttn), ("mlp", CMlp), ("pa", CPredictor), ("pm", CPredictor), ("ln", CLN), ("kv", CKV)]


_PRED_ARGS = [POINTER(CPredictor), c_void_p, c_int32, c_int32, c_int32, c_float, c_void_p, c_int32,
              c_void_p, c_void_p, c_void_p, c_size_t, c_uint32, c_void_p]
_SIGS = {
    "dv_status_string": (c_char_p, [c_int32]),
    "dv_set_launch_events": (c_int32, [POINTER(c_void_p), c_int32, POINTER(c_int32), c_char_p]),
    "dv_launch_label": (c_char_p, [c_int32]),
    "dv_abi_version": (c_int32, []),
    "dv_stream_read": (c_int32, [c_void_p, c_size_t, c_void_p, c_void_p]),
    "dv_sparse_mlp_q4_workspace_bytes": (c_size_t, [POINTER(CMlpQ4), c_int32]),
    "dv_sparse_mlp_q4": (c_int32, [POINTER(CMlpQ4), c_void_p, c_void_p, c_int32, c_void_p, c_void_p, c_size_t,
                                   c_uint32, c_void_p]),
    "dv_sparse_attn_kvfill": (c_int32, [POINTER(CAttn), c_void_p, POINTER(CKV), c_void_p, c_void_p, c_void_p,
                                        c_int32, c_float, c_void_p, c_void_p, c_size_t, c_uint32, c_void_p]),
    "dv_sparse_decode_workspace_bytes": (c_size_t, [POINTER(CLayer), c_int32, c_int32, c_int32]),
    "dv_sparse_decode": (c_int32, [POINTER(CLayer), c_int32, c_void_p, c_void_p, c_int32, c_int32, c_float,
                                   c_void_p, c_void_p, c_void_p, c_size_t, c_uint32, c_void_p]),
    "dv_sparse_block_noalloc": (c_int32, [POINTER(CAttn), POINTER(CMlp), POINTER(CPredictor), POINTER(CPredictor),
                                          POINTER(CLN), POINTER(CKV), c_void_p, c_void_p, c_int32, c_int32,
                                          c_int32, c_int32, c_int32, c_float, c_void_p, c_void_p, c_uint32,
                                          c_void_p]),
    "dv_predict_workspace_bytes": (c_size_t, [POINTER(CPredictor), c_int32]),
    "dv_predict_mlp": (c_int32, _PRED_ARGS),
    "dv_predict_heads": (c_int32, _PRED_ARGS),
    "dv_sparse_mlp_workspace_bytes": (c_size_t, [POINTER(CMlp), c_int32, c_int32, c_int32]),
    "dv_sparse_mlp": (c_int32, [POINTER(CMlp), c_void_p, c_int32, c_void_p, c_int32, c_int32, c_int32,
                                c_void_p, c_void_p, c_size_t, c_uint32, c_void_p]),
    "dv_sparse_attn_workspace_bytes": (c_size_t, [POINTER(CAttn), POINTER(CKV), c_int32, c_int32]),
    "dv_sparse_attn": (c_int32, [POINTER(CAttn), c_void_p, c_int32, POINTER(CKV), c_void_p, c_int32,
                                 c_float, c_void_p, c_void_p, c_size_t, c_uint32, c_void_p]),
    "dv_sparse_block_workspace_bytes": (c_size_t, [POINTER(CAttn), POINTER(CMlp), POINTER(CPredictor),
                                                   POINTER(CPredictor), POINTER(CKV), c_int32, c_int32,
                                                   c_int32]),
    "dv_sparse_block": (c_int32, [POINTER(CAttn), POINTER(CMlp), POINTER(CPredictor), POINTER(CPredictor),
                                  POINTER(CLN), POINTER(CKV), c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                  c_int32, c_int32, c_float, c_void_p, c_void_p, c_void_p, c_size_t,
                                  c_uint32, c_void_p]),
}

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises OSError if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise OSError(f"{path} not found: build it with `python -m paper_2310_17157_amd.build`")
        lib = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def lib_path() -> str:
    return LIB_PATH


# ------------------------------------------------------------------ helpers
def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _wtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float16:
        return DV_F16
    if t.dtype == torch.float32:
        return DV_F32
    raise TypeError(f"unsupported storage dtype {t.dtype}")


_F32 = (torch.float32,)
_I32 = (torch.int32,)
_STORE = (torch.float16, torch.float32)


def _tensor(name, t, dtypes, ndim=None, shape=None, optional=False, dev=True):
    """Argument check before anything reaches the library: dtype, rank, shape,
    contiguity and device. The kernels read raw pointers, so a wrong dtype or a strided
    view would be read as something else (or past its end)."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, not {type(t).__name__}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}; expected {' or '.join(str(d) for d in dtypes)}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D, got shape {tuple(t.shape)}")
    if shape is not None and any(w is not None and w != g for w, g in zip(shape, t.shape)):
        raise ValueError(f"{name} has shape {tuple(t.shape)}; expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dev:
        _gpu(name, t)


def _gpu(name, *ts):
    for t in ts:
        if t is not None and t.device.type != "cuda":
            raise ValueError(f"{name} must be a GPU tensor, not on {t.device}")


def _wsarg(ws):
    """(pointer, bytes) of a workspace: a contiguous uint8 GPU tensor."""
    _tensor("ws", ws, (torch.uint8,), 1)
    return ws.data_ptr(), ws.numel()


def _same_dtype(name, *ts):
    ds = {t.dtype for t in ts if t is not None}
    if len(ds) > 1:
        raise TypeError(f"{name}: all weights must share one dtype, got {sorted(str(d) for d in ds)}")


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check(fn: str, st: int):
    if st != 0:
        raise DvError(fn, st, load().dv_status_string(st).decode())


def _workspace(nbytes: int, device) -> torch.Tensor:
    # 256-byte alignment: torch's caching allocator returns 512-byte aligned blocks.
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


@dataclass
class Predictor:
    """Two-layer low-rank predictor: AT [r][d], BT [n_out][r] (same storage dtype)."""
    AT: torch.Tensor
    BT: torch.Tensor

    def c(self) -> CPredictor:
        # checked and built once per set of tensors (calls are on the hot path)
        key = tuple(id(t) for t in (self.AT, self.BT,))
        if getattr(self, "_ck", None) != key:
            _tensor("Predictor.AT", self.AT, _STORE, 2, dev=False)
            r, d = self.AT.shape
            _tensor("Predictor.BT", self.BT, _STORE, 2, (None, r), dev=False)
            _same_dtype("Predictor", self.AT, self.BT)
            _gpu(type(self).__name__, self.AT, self.BT)
            self._cs = CPredictor(d, r, self.BT.shape[0], _wtype(self.AT), _ptr(self.AT), _ptr(self.BT))
            self._ck = key
        return self._cs


@dataclass
class MLP:
    W1T: torch.Tensor
    W2T: torch.Tensor
    b1: Optional[torch.Tensor] = None
    b2: Optional[torch.Tensor] = None
    act: int = DV_ACT_RELU

    def c(self) -> CMlp:
        # checked and built once per set of tensors (calls are on the hot path)
        key = tuple(id(t) for t in (self.W1T, self.W2T, self.b1, self.b2,)) + (self.act,)
        if getattr(self, "_ck", None) != key:
            _tensor("MLP.W1T", self.W1T, _STORE, 2, dev=False)
            n, d = self.W1T.shape
            _tensor("MLP.W2T", self.W2T, _STORE, 2, (n, d), dev=False)
            _same_dtype("MLP", self.W1T, self.W2T)
            _tensor("MLP.b1", self.b1, _F32, 1, (n,), optional=True, dev=False)
            _tensor("MLP.b2", self.b2, _F32, 1, (d,), optional=True, dev=False)
            _gpu(type(self).__name__, self.W1T, self.W2T, self.b1, self.b2)
            self._cs = CMlp(d, n, _wtype(self.W1T), int(self.act), _ptr(self.W1T), _ptr(self.b1), _ptr(self.W2T),
                            _ptr(self.b2))
            self._ck = key
        return self._cs


@dataclass
class MLPQ4:
    """4-bit MLP weights (W4A16): W1T, W2T [n][d/2] uint8 codes (even element in the low
    nibble), S1, S2 [n][d/32] fp16 block scales; element = scale * (code - 8)."""
    W1T: torch.Tensor
    S1: torch.Tensor
    W2T: torch.Tensor
    S2: torch.Tensor
    b1: Optional[torch.Tensor] = None
    b2: Optional[torch.Tensor] = None
    act: int = DV_ACT_RELU

    def c(self) -> CMlpQ4:
        key = tuple(id(t) for t in (self.W1T, self.S1, self.W2T, self.S2, self.b1, self.b2)) + (self.act,)
        if getattr(self, "_ck", None) != key:
            _tensor("MLPQ4.W1T", self.W1T, (torch.uint8,), 2, dev=False)
            n, h = self.W1T.shape
            d = 2 * h
            _tensor("MLPQ4.W2T", self.W2T, (torch.uint8,), 2, (n, h), dev=False)
            _tensor("MLPQ4.S1", self.S1, (torch.float16,), 2, (n, d // 32), dev=False)
            _tensor("MLPQ4.S2", self.S2, (torch.float16,), 2, (n, d // 32), dev=False)
            _tensor("MLPQ4.b1", self.b1, _F32, 1, (n,), optional=True, dev=False)
            _tensor("MLPQ4.b2", self.b2, _F32, 1, (d,), optional=True, dev=False)
            _gpu("MLPQ4", self.W1T, self.S1, self.W2T, self.S2, self.b1, self.b2)
            self._cs = CMlpQ4(d, n, int(self.act), 0, _ptr(self.W1T), _ptr(self.S1), _ptr(self.b1), _ptr(self.W2T),
                              _ptr(self.S2), _ptr(self.b2))
            self._ck = key
        return self._cs


@dataclass
class Attn:
    Wq: torch.Tensor
    Wk: torch.Tensor
    Wv: torch.Tensor
    WoT: torch.Tensor
    H: int
    bq: Optional[torch.Tensor] = None
    bk: Optional[torch.Tensor] = None
    bv: Optional[torch.Tensor] = None
    bo: Optional[torch.Tensor] = None

    def c(self) -> CAttn:
        # checked and built once per set of tensors (calls are on the hot path)
        key = tuple(id(t) for t in (self.Wq, self.Wk, self.Wv, self.WoT, self.bq, self.bk, self.bv, self.bo, self.H,))
        if getattr(self, "_ck", None) != key:
            _tensor("Attn.Wq", self.Wq, _STORE, 2, dev=False)
            hd, d = self.Wq.shape
            if self.H <= 0 or hd % self.H:
                raise ValueError(f"Attn: {hd} projection rows do not split into H = {self.H} heads")
            for nm in ("Wk", "Wv", "WoT"):
                _tensor(f"Attn.{nm}", getattr(self, nm), _STORE, 2, (hd, d), dev=False)
            _same_dtype("Attn", self.Wq, self.Wk, self.Wv, self.WoT)
            for nm in ("bq", "bk", "bv"):
                _tensor(f"Attn.{nm}", getattr(self, nm), _F32, 1, (hd,), optional=True, dev=False)
            _tensor("Attn.bo", self.bo, _F32, 1, (d,), optional=True, dev=False)
            _gpu(type(self).__name__, self.Wq, self.Wk, self.Wv, self.WoT, self.bq, self.bk, self.bv, self.bo)
            self._cs = CAttn(d, self.H, hd // self.H, _wtype(self.Wq), _ptr(self.Wq), _ptr(self.Wk), _ptr(self.Wv),
                         _ptr(self.bq), _ptr(self.bk), _ptr(self.bv), _ptr(self.WoT), _ptr(self.bo))
            self._ck = key
        return self._cs


class KVCache:
    """K, V [B][H][cap][dh] device tensors and the host positions pos[B]."""

    def __init__(self, K: torch.Tensor, V: torch.Tensor, pos):
        self.K, self.V = K, V
        self._pos = (c_int32 * K.shape[0])(*[int(p) for p in pos])

    def set_pos(self, pos):
        """Move to new decode positions (the struct handed to the library keeps pointing
        at the same host array)."""
        for b, p in enumerate(pos):
            self._pos[b] = int(p)

    def c(self) -> CKV:
        # checked and built once per set of tensors (calls are on the hot path)
        key = tuple(id(t) for t in (self.K, self.V, self._pos,))
        if getattr(self, "_ck", None) != key:
            _tensor("KVCache.K", self.K, _STORE, 4, dev=False)
            _tensor("KVCache.V", self.V, _STORE, 4, tuple(self.K.shape), dev=False)
            _same_dtype("KVCache", self.K, self.V)
            B, H, cap, dh = self.K.shape
            _gpu(type(self).__name__, self.K, self.V)
            self._cs = CKV(B, H, dh, cap, _wtype(self.K), 0, _ptr(self.K), _ptr(self.V),
                       ctypes.cast(self._pos, POINTER(c_int32)))
            self._ck = key
        return self._cs


@dataclass
class LN:
    g1: Optional[torch.Tensor] = None
    be1: Optional[torch.Tensor] = None
    g2: Optional[torch.Tensor] = None
    be2: Optional[torch.Tensor] = None
    eps: float = 1e-5

    def c(self) -> CLN:
        # checked and built once per set of tensors (calls are on the hot path)
        key = tuple(id(t) for t in (self.g1, self.be1, self.g2, self.be2, self.eps,))
        if getattr(self, "_ck", None) != key:
            for nm in ("g1", "be1", "g2", "be2"):
                _tensor(f"LN.{nm}", getattr(self, nm), _F32, 1, optional=True, dev=False)
            _gpu(type(self).__name__, self.g1, self.be1, self.g2, self.be2)
            self._cs = CLN(_ptr(self.g1), _ptr(self.be1), _ptr(self.g2), _ptr(self.be2), self.eps)
            self._ck = key
        return self._cs


# ------------------------------------------------------------- entry points
def _predict(fn, pred: Predictor, x, k=0, mode=DV_SELECT_TOPK, thresh=0.0, idx=None, count=None,
             scores=None, cap_idx=None, ws=None, flags=0, stream=None):
    lib = load()
    cp = pred.c()
    _tensor("x", x, _F32, 2, (None, cp.d), dev=False)
    B = x.shape[0]
    _tensor("idx", idx, _I32, 2, (B, None), optional=True, dev=False)
    _tensor("count", count, _I32, 1, (B,), optional=True, dev=False)
    _tensor("scores", scores, _F32, 2, (B, cp.n_out), optional=True, dev=False)
    _gpu("arguments", x, idx, count, scores)
    if cap_idx is None:
        cap_idx = k if mode == DV_SELECT_TOPK else cp.n_out
    if idx is None:
        idx = torch.empty((B, max(cap_idx, 1)), dtype=torch.int32, device=x.device)
    if count is None:
        count = torch.empty(B, dtype=torch.int32, device=x.device)
    if ws is None:
        ws = _workspace(lib.dv_predict_workspace_bytes(ctypes.byref(cp), B), x.device)
    st = getattr(lib, fn)(ctypes.byref(cp), _ptr(x), B, mode, k, thresh, _ptr(idx), cap_idx, _ptr(count),
                          _ptr(scores), *_wsarg(ws), flags, _stream(stream))
    _check(fn, st)
    return idx, count


def dv_predict_mlp(pred: Predictor, x, k=0, **kw):
    """S_M per sequence from s = (x A) B: top-k (default) or threshold. Returns (idx, count)."""
    return _predict("dv_predict_mlp", pred, x, k, **kw)


def dv_predict_heads(pred: Predictor, x, k=0, **kw):
    """S_A per sequence from the head predictor. Returns (idx, count)."""
    return _predict("dv_predict_heads", pred, x, k, **kw)


def dv_sparse_mlp(mlp: MLP, x, idx, idx_per_seq=0, batch_mode=DV_MLP_UNION, out=None, ws=None,
                  flags=0, stream=None):
    """out[b] = MLP_S(x[b]) (Eq. (1)), without residual."""
    lib = load()
    cm = mlp.c()
    _tensor("x", x, _F32, 2, (None, cm.d), dev=False)
    B = x.shape[0]
    _tensor("idx", idx, _I32, dev=False)
    n_idx = idx.shape[-1]
    if idx_per_seq and idx.numel() != B * n_idx:
        raise ValueError(f"idx holds {idx.numel()} entries; per-sequence sets need B x n_idx = {B * n_idx}")
    _tensor("out", out, _F32, 2, (B, cm.d), optional=True, dev=False)
    _gpu("arguments", x, idx, out)
    if out is None:
        out = torch.empty((B, cm.d), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = _workspace(lib.dv_sparse_mlp_workspace_bytes(ctypes.byref(cm), B, n_idx, idx_per_seq), x.device)
    st = lib.dv_sparse_mlp(ctypes.byref(cm), _ptr(x), B, _ptr(idx), n_idx, idx_per_seq, batch_mode,
                           _ptr(out), *_wsarg(ws), flags, _stream(stream))
    _check("dv_sparse_mlp", st)
    return out


def dv_sparse_attn(attn: Attn, x, kv: KVCache, heads, scale, out=None, ws=None, flags=0, stream=None):
    """out[b] = bo + sum_{i in S_A^b} H_i(x[b]) W^O_i (Eq. (2)); updates the cache rows at pos."""
    lib = load()
    ca, ck = attn.c(), kv.c()
    _tensor("x", x, _F32, 2, (None, ca.d), dev=False)
    B = x.shape[0]
    _tensor("heads", heads, _I32, dev=False)
    n_heads = heads.shape[-1]
    if heads.numel() != B * n_heads:
        raise ValueError(f"heads holds {heads.numel()} entries; expected B x n_heads = {B * n_heads}")
    _tensor("out", out, _F32, 2, (B, ca.d), optional=True, dev=False)
    _gpu("arguments", x, heads, out)
    if out is None:
        out = torch.empty((B, ca.d), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = _workspace(lib.dv_sparse_attn_workspace_bytes(ctypes.byref(ca), ctypes.byref(ck), B, n_heads),
                        x.device)
    st = lib.dv_sparse_attn(ctypes.byref(ca), _ptr(x), B, ctypes.byref(ck), _ptr(heads), n_heads, scale,
                            _ptr(out), *_wsarg(ws), flags, _stream(stream))
    _check("dv_sparse_attn", st)
    return out


def dv_sparse_mlp_q4(mlp: MLPQ4, x, idx, out=None, ws=None, flags=0, stream=None):
    """out = MLP_S(x) with 4-bit weights (Section 5.2, W4A16), one token."""
    lib = load()
    cm = mlp.c()
    _tensor("x", x, _F32, 2, (1, cm.d), dev=False)
    _tensor("idx", idx, _I32, dev=False)
    n_idx = idx.shape[-1]
    _tensor("out", out, _F32, 2, (1, cm.d), optional=True, dev=False)
    _gpu("arguments", x, idx, out)
    if out is None:
        out = torch.empty((1, cm.d), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = _workspace(lib.dv_sparse_mlp_q4_workspace_bytes(ctypes.byref(cm), n_idx), x.device)
    st = lib.dv_sparse_mlp_q4(ctypes.byref(cm), _ptr(x), _ptr(idx), n_idx, _ptr(out), *_wsarg(ws), flags,
                              _stream(stream))
    _check("dv_sparse_mlp_q4", st)
    return out


def dv_sparse_attn_kvfill(attn: Attn, x, kv: KVCache, Y, valid, heads, scale, out=None, ws=None, flags=0,
                          stream=None):
    """dv_sparse_attn for one sequence with the missing-KV rule of Section 4.2: Y [cap][d]
    keeps every token's attention input in the cache's dtype (fp16 or fp32, like K and
    V), valid [H][cap] uint8 marks the cache rows that hold their token's key and value
    (both updated in place)."""
    lib = load()
    ca, ck = attn.c(), kv.c()
    _tensor("x", x, _F32, 2, (1, ca.d), dev=False)
    _tensor("Y", Y, (kv.K.dtype,), 2, (ck.cap, ca.d), dev=False)
    _tensor("valid", valid, (torch.uint8,), 2, (ca.H, ck.cap), dev=False)
    _tensor("heads", heads, _I32, dev=False)
    n_heads = heads.shape[-1]
    if heads.numel() != n_heads:
        raise ValueError("heads: one sequence's set")
    _tensor("out", out, _F32, 2, (1, ca.d), optional=True, dev=False)
    _gpu("arguments", x, Y, valid, heads, out)
    if out is None:
        out = torch.empty((1, ca.d), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = _workspace(lib.dv_sparse_attn_workspace_bytes(ctypes.byref(ca), ctypes.byref(ck), 1, n_heads), x.device)
    st = lib.dv_sparse_attn_kvfill(ctypes.byref(ca), _ptr(x), ctypes.byref(ck), _ptr(Y), _ptr(valid), _ptr(heads),
                                   n_heads, scale, _ptr(out), *_wsarg(ws), flags, _stream(stream))
    _check("dv_sparse_attn_kvfill", st)
    return out


def dv_sparse_block(attn: Attn, mlp: MLP, pred_h: Predictor, pred_m: Predictor, ln: Optional[LN],
                    kv: KVCache, x, k_heads, k_mlp, scale, mode=DV_LOOKAHEAD, batch_mode=DV_MLP_UNION,
                    out=None, heads_out=None, idx_out=None, ws=None, flags=0, stream=None):
    """One decoder layer with contextual sparsity (Section 4.3). Returns (out, heads, idx)."""
    lib = load()
    ca, cm, cph, cpm, ck = attn.c(), mlp.c(), pred_h.c(), pred_m.c(), kv.c()
    cl = ln.c() if ln is not None else None
    _tensor("x", x, _F32, 2, (None, ca.d), dev=False)
    B = x.shape[0]
    _tensor("out", out, _F32, 2, (B, ca.d), optional=True, dev=False)
    _tensor("heads_out", heads_out, _I32, 2, (B, k_heads), optional=True, dev=False)
    _tensor("idx_out", idx_out, _I32, 2, (B, k_mlp), optional=True, dev=False)
    _gpu("arguments", x, out, heads_out, idx_out)
    if out is None:
        out = torch.empty_like(x)
    if heads_out is None:
        heads_out = torch.empty((B, k_heads), dtype=torch.int32, device=x.device)
    if idx_out is None:
        idx_out = torch.empty((B, k_mlp), dtype=torch.int32, device=x.device)
    if ws is None:
        ws = _workspace(block_workspace_bytes(attn, mlp, pred_h, pred_m, kv, B, k_heads, k_mlp), x.device)
    st = lib.dv_sparse_block(ctypes.byref(ca), ctypes.byref(cm), ctypes.byref(cph), ctypes.byref(cpm),
                             ctypes.byref(cl) if cl is not None else None, ctypes.byref(ck), _ptr(x),
                             _ptr(out), B, k_heads, k_mlp, mode, batch_mode, scale, _ptr(heads_out),
                             _ptr(idx_out), *_wsarg(ws), flags, _stream(stream))
    _check("dv_sparse_block", st)
    return out, heads_out, idx_out


def _layers_c(layers):
    """layers: sequence of (attn, mlp, pred_h, pred_m, kv, ln) tuples -> a dv_layer array."""
    arr = (CLayer * len(layers))()
    for i, (attn, mlp, ph, pm, kv, ln) in enumerate(layers):
        arr[i] = CLayer(attn.c(), mlp.c(), ph.c(), pm.c(), ln.c() if ln is not None else CLN(None, None, None, None,
                                                                                                 1e-5), kv.c())
    return arr


def decode_workspace_bytes(layers, k_heads, k_mlp) -> int:
    arr = _layers_c(layers)
    return load().dv_sparse_decode_workspace_bytes(arr, len(layers), k_heads, k_mlp)


def dv_sparse_decode(layers, x, k_heads, k_mlp, scale, out=None, heads_out=None, idx_out=None, ws=None,
                     flags=0, stream=None, _arr=None):
    """Several layers for one token with the cross-layer look-ahead (Section 4.3): the
    sets of layer l+1 are predicted from layer l's input inside layer l's launches.
    layers: sequence of (attn, mlp, pred_h, pred_m, kv, ln). Returns
    (out, heads [L, k_heads], idx [L, k_mlp])."""
    lib = load()
    arr = _arr if _arr is not None else _layers_c(layers)
    L = len(layers)
    d = arr[0].attn.d
    _tensor("x", x, _F32, 2, (1, d), dev=False)
    _tensor("out", out, _F32, 2, (1, d), optional=True, dev=False)
    _tensor("heads_out", heads_out, _I32, 2, (L, k_heads), optional=True, dev=False)
    _tensor("idx_out", idx_out, _I32, 2, (L, k_mlp), optional=True, dev=False)
    _gpu("arguments", x, out, heads_out, idx_out)
    if out is None:
        out = torch.empty_like(x)
    if heads_out is None:
        heads_out = torch.empty((L, k_heads), dtype=torch.int32, device=x.device)
    if idx_out is None:
        idx_out = torch.empty((L, k_mlp), dtype=torch.int32, device=x.device)
    if ws is None:
        ws = _workspace(lib.dv_sparse_decode_workspace_bytes(arr, L, k_heads, k_mlp), x.device)
    st = lib.dv_sparse_decode(arr, L, _ptr(x), _ptr(out), k_heads, k_mlp, scale, _ptr(heads_out), _ptr(idx_out),
                              *_wsarg(ws), flags, _stream(stream))
    _check("dv_sparse_decode", st)
    return out, heads_out, idx_out


STATIC_SCRATCH_BYTES = 16 << 20   # DV_STATIC_SCRATCH_BYTES


def dv_sparse_block_noalloc(attn: Attn, mlp: MLP, pred_h: Predictor, pred_m: Predictor, ln: Optional[LN],
                            kv: KVCache, x, k_heads, k_mlp, scale, out, heads_out, idx_out,
                            mode=DV_LOOKAHEAD, batch_mode=DV_MLP_UNION, flags=0, stream=None):
    """dv_sparse_block without a workspace (the library's own per-device scratch); the
    outputs must be given, since this call allocates nothing."""
    lib = load()
    ca, cm, cph, cpm, ck = attn.c(), mlp.c(), pred_h.c(), pred_m.c(), kv.c()
    cl = ln.c() if ln is not None else None
    _tensor("x", x, _F32, 2, (None, ca.d), dev=False)
    B = x.shape[0]
    _tensor("out", out, _F32, 2, (B, ca.d), dev=False)
    _tensor("heads_out", heads_out, _I32, 2, (B, k_heads), optional=True, dev=False)
    _tensor("idx_out", idx_out, _I32, 2, (B, k_mlp), optional=True, dev=False)
    _gpu("arguments", x, out, heads_out, idx_out)
    st = lib.dv_sparse_block_noalloc(ctypes.byref(ca), ctypes.byref(cm), ctypes.byref(cph), ctypes.byref(cpm),
                                     ctypes.byref(cl) if cl is not None else None, ctypes.byref(ck), _ptr(x),
                                     _ptr(out), B, k_heads, k_mlp, mode, batch_mode, scale, _ptr(heads_out),
                                     _ptr(idx_out), flags, _stream(stream))
    _check("dv_sparse_block_noalloc", st)
    return out, heads_out, idx_out


def block_workspace_bytes(attn, mlp, pred_h, pred_m, kv, B, k_heads, k_mlp) -> int:
    lib = load()
    ca, cm, cph, cpm, ck = attn.c(), mlp.c(), pred_h.c(), pred_m.c(), kv.c()
    return lib.dv_sparse_block_workspace_bytes(ctypes.byref(ca), ctypes.byref(cm), ctypes.byref(cph),
                                               ctypes.byref(cpm), ctypes.byref(ck), B, k_heads, k_mlp)


def mlp_workspace_bytes(mlp, B, n_idx, idx_per_seq=0) -> int:
    cm = mlp.c()
    return load().dv_sparse_mlp_workspace_bytes(ctypes.byref(cm), B, n_idx, idx_per_seq)


def attn_workspace_bytes(attn, kv, B, n_heads) -> int:
    ca, ck = attn.c(), kv.c()
    return load().dv_sparse_attn_workspace_bytes(ctypes.byref(ca), ctypes.byref(ck), B, n_heads)


def predict_workspace_bytes(pred, B) -> int:
    cp = pred.c()
    return load().dv_predict_workspace_bytes(ctypes.byref(cp), B)


def dv_stream_read(buf: torch.Tensor, sink: torch.Tensor, nbytes: Optional[int] = None, stream=None):
    """One plain contiguous read of `nbytes` (default: all) of `buf`: the measured
    bandwidth ceiling the gathered kernels are compared with."""
    if not isinstance(buf, torch.Tensor) or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous tensor")
    _tensor("sink", sink, _F32)
    _gpu("buf", buf)
    n = buf.numel() * buf.element_size() if nbytes is None else int(nbytes)
    if n > buf.numel() * buf.element_size():
        raise ValueError("nbytes exceeds the buffer")
    _check("dv_stream_read", load().dv_stream_read(buf.data_ptr(), n, sink.data_ptr(), _stream(stream)))


# --------------------------------------------------------- per-launch timing
_HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000   # hipEventDisableSystemFence


class LaunchTimer:
    """Per-launch times of the library's entry points from HIP events.

    Arms dv_set_launch_events with `n_pairs` event pairs created through the HIP
    runtime; after a call (and a synchronisation) `times_ms()` returns
    [(label, milliseconds)] for each launch of that call: from the start of the
    launch's first kernel to the end of its last, as stamped by the kernels'
    own dispatches on the stream the library launched on.
    """

    def __init__(self, n_pairs: int = 16, only: Optional[str] = None):
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreateWithFlags.argtypes = [POINTER(c_void_p), ctypes.c_uint]
        self._hip.hipEventElapsedTime.argtypes = [POINTER(c_float), c_void_p, c_void_p]
        self._hip.hipEventSynchronize.argtypes = [c_void_p]
        self._hip.hipEventDestroy.argtypes = [c_void_p]
        self.n = n_pairs
        self.events = (c_void_p * (2 * n_pairs))()
        for i in range(2 * n_pairs):
            ev = c_void_p()
            # timing-only events: no system-scope fence (cache write-back and
            # invalidation) when recorded, which would stall the next launch
            if self._hip.hipEventCreateWithFlags(ctypes.byref(ev), _HIP_EVENT_DISABLE_SYSTEM_FENCE) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.events[i] = ev
        self.n_launched = c_int32(0)
        self.only = only.encode() if only else None
        self.labels = []

    def arm(self):
        _check("dv_set_launch_events",
               load().dv_set_launch_events(self.events, self.n, ctypes.byref(self.n_launched), self.only))

    def disarm(self):
        lib = load()
        labels = [lib.dv_launch_label(i).decode() for i in range(self.n_launched.value)]
        if self.only is not None:
            labels = [l for l in labels if l == self.only.decode()]
        self.labels = labels[: self.n]
        lib.dv_set_launch_events(None, 0, None, None)

    def times_ms(self):
        out = []
        for i in range(len(self.labels)):
            a, b = self.events[2 * i], self.events[2 * i + 1]
            self._hip.hipEventSynchronize(b)
            ms = c_float(0.0)
            if self._hip.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
                raise RuntimeError("hipEventElapsedTime failed")
            out.append((self.labels[i], ms.value))
        return out

    def close(self):
        load().dv_set_launch_events(None, 0, None, None)
        for i in range(2 * self.n):
            self._hip.hipEventDestroy(self.events[i])
