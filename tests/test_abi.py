"""The C ABI without a GPU: the library loads, exports every function include/dv.h
declares, and rejects bad arguments on the host before any device call.

Pointers here are fake (aligned, non-NULL integers). Every call below fails host
validation, so no HIP API is reached.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2310_17157_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dv.h")
FAKE = 0x10000000          # 256-byte aligned fake device address


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dv_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return B.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert {"dv_predict_mlp", "dv_predict_heads", "dv_sparse_mlp", "dv_sparse_attn",
            "dv_sparse_block"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", B.lib_path()], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (dv_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        assert hasattr(lib, n)


def test_status_strings_and_version(lib):
    assert lib.dv_abi_version() == 1
    for s in range(10):
        assert lib.dv_status_string(s)
    assert lib.dv_status_string(99) == b"unknown status"


def _mlp(d=64, n=128, wtype=B.DV_F16):
    return B.CMlp(d, n, wtype, 0, FAKE, None, FAKE, None)


def _call_mlp(lib, m, x=FAKE, Bn=1, idx=FAKE, n_idx=8, per_seq=0, mode=0, out=FAKE, ws=FAKE,
              ws_bytes=1 << 30, flags=0):
    return lib.dv_sparse_mlp(ctypes.byref(m) if m is not None else None, x, Bn, idx, n_idx, per_seq, mode,
                             out, ws, ws_bytes, flags, None)


def test_sparse_mlp_validation(lib):
    assert _call_mlp(lib, None) == 1                                   # NULL
    assert _call_mlp(lib, _mlp(), x=None) == 1
    assert _call_mlp(lib, _mlp(wtype=7)) == 3                         # dtype
    assert _call_mlp(lib, _mlp(d=60)) == 4                            # fp16 row not 16-byte multiple
    assert _call_mlp(lib, _mlp(), x=FAKE + 4) == 4                    # misaligned x
    assert _call_mlp(lib, _mlp(), n_idx=129) == 2                     # k > n
    assert _call_mlp(lib, _mlp(), Bn=0) == 2
    assert _call_mlp(lib, _mlp(), per_seq=2) == 9
    bad_act = _mlp()
    bad_act.act = 2
    assert _call_mlp(lib, bad_act) == 9                                # unknown activation
    assert _call_mlp(lib, _mlp(), mode=5) == 9
    assert _call_mlp(lib, _mlp(), flags=1 << 7) == 9
    assert _call_mlp(lib, _mlp(), ws=None) == 5
    assert _call_mlp(lib, _mlp(), ws=FAKE + 16) == 5
    assert _call_mlp(lib, _mlp(), ws_bytes=16) == 5
    m = _mlp()
    need = lib.dv_sparse_mlp_workspace_bytes(ctypes.byref(m), 1, 8, 0)
    assert need > 0 and need % 256 == 0
    assert _call_mlp(lib, _mlp(), ws_bytes=need - 1) == 5


def _attn(d=64, H=4, dh=16):
    return B.CAttn(d, H, dh, B.DV_F16, FAKE, FAKE, FAKE, None, None, None, FAKE, None)


def _kv(Bn=1, H=4, dh=16, cap=10, pos=(3,)):
    arr = (ctypes.c_int32 * len(pos))(*pos)
    kv = B.CKV(Bn, H, dh, cap, B.DV_F16, 0, FAKE, FAKE, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)))
    kv._keep = arr
    return kv


def test_sparse_attn_validation(lib):
    a, kv = _attn(), _kv()
    call = lambda a=a, kv=kv, n_heads=2, scale=0.25, ws_bytes=1 << 30, x=FAKE: lib.dv_sparse_attn(
        ctypes.byref(a), x, 1, ctypes.byref(kv), FAKE, n_heads, scale, FAKE, FAKE, ws_bytes, 0, None)
    assert call(x=None) == 1
    assert call(n_heads=5) == 2                                       # more heads than H
    assert call(kv=_kv(pos=(10,))) == 2                               # pos >= cap
    assert call(kv=_kv(pos=(-1,))) == 2
    assert call(kv=_kv(H=3)) == 2                                     # cache/head mismatch
    assert call(kv=_kv(dh=4)) == 2
    assert call(scale=float("nan")) == 9
    assert call(ws_bytes=0) == 5
    need = lib.dv_sparse_attn_workspace_bytes(ctypes.byref(a), ctypes.byref(kv), 1, 2)
    assert need > 0 and call(ws_bytes=need - 256) == 5


def test_predict_and_block_validation(lib):
    p = B.CPredictor(64, 16, 128, B.DV_F16, FAKE, FAKE)
    call = lambda p=p, k=8, mode=0, cap=8, x=FAKE: lib.dv_predict_mlp(
        ctypes.byref(p), x, 1, mode, k, 0.0, FAKE, cap, FAKE, None, FAKE, 1 << 30, 0, None)
    assert call(x=None) == 1
    assert call(k=129) == 2
    assert call(cap=4) == 2                                           # cap_idx < k
    assert call(mode=3) == 9
    assert call(p=B.CPredictor(64, 12, 128, B.DV_F16, FAKE, FAKE)) == 4   # r % 8 != 0
    assert lib.dv_predict_workspace_bytes(ctypes.byref(p), 1) > 0

    a, m, kv = _attn(), _mlp(), _kv()
    ph = B.CPredictor(64, 16, 4, B.DV_F16, FAKE, FAKE)
    pm = B.CPredictor(64, 16, 128, B.DV_F16, FAKE, FAKE)
    blk = lambda ph=ph, pm=pm, kh=2, km=8, mode=0, ws_bytes=1 << 30: lib.dv_sparse_block(
        ctypes.byref(a), ctypes.byref(m), ctypes.byref(ph), ctypes.byref(pm), None, ctypes.byref(kv),
        FAKE, FAKE + 4096, 1, kh, km, mode, 0, 0.25, None, None, FAKE, ws_bytes, 0, None)
    assert blk(ph=B.CPredictor(64, 16, 5, B.DV_F16, FAKE, FAKE)) == 2   # head predictor n_out != H
    assert blk(kh=0) == 2
    assert blk(km=129) == 2
    assert blk(mode=4) == 9
    assert blk(pm=B.CPredictor(64, 16, 128, B.DV_F32, FAKE, FAKE)) == 3  # predictor dtypes differ
    assert blk(ws_bytes=1) == 5


def test_batched_path_limits(lib):
    """B > 1 runs on the matrix cores: up to 32 sequences, fp16 weights; the rest is
    DV_ERR_UNSUPPORTED before any device work."""
    assert _call_mlp(lib, _mlp(), Bn=33, per_seq=1) == B.DV_ERR_UNSUPPORTED
    assert _call_mlp(lib, _mlp(wtype=B.DV_F32), Bn=2, per_seq=1) == B.DV_ERR_UNSUPPORTED
    assert _call_mlp(lib, _mlp(), Bn=2, per_seq=1, ws=None) == B.DV_ERR_WORKSPACE
    # the union marks one byte per neuron in LDS: up to 131072 neurons at B > 1
    assert _call_mlp(lib, _mlp(n=131073), Bn=2, per_seq=1) == B.DV_ERR_UNSUPPORTED
    assert _call_mlp(lib, _mlp(n=131072), Bn=2, per_seq=1, ws=None) == B.DV_ERR_WORKSPACE
    m = _mlp()
    one = lib.dv_sparse_mlp_workspace_bytes(ctypes.byref(m), 1, 8, 1)
    many = lib.dv_sparse_mlp_workspace_bytes(ctypes.byref(m), 32, 8, 1)
    assert many > one > 0 and many % 256 == 0
    a = _attn()
    kv33 = _kv(Bn=33, pos=tuple([3] * 33))
    assert lib.dv_sparse_attn(ctypes.byref(a), FAKE, 33, ctypes.byref(kv33), FAKE, 2, 0.25, FAKE, FAKE,
                              1 << 30, 0, None) == B.DV_ERR_UNSUPPORTED
    kv2 = _kv(Bn=2, pos=(3, 9))
    assert lib.dv_sparse_attn_workspace_bytes(ctypes.byref(a), ctypes.byref(kv2), 2, 2) > 0


def test_binding_rejects_bad_tensors_before_the_library():
    """The binding checks dtype, shape, contiguity and device of every tensor before a
    pointer reaches the C ABI (CPU tensors here: every case fails in Python)."""
    import torch
    h16 = lambda *s: torch.zeros(*s, dtype=torch.float16)
    f32 = lambda *s: torch.zeros(*s, dtype=torch.float32)
    # a weight struct whose matrices differ in dtype
    with pytest.raises(TypeError):
        B.MLP(h16(8, 16), f32(8, 16)).c()
    with pytest.raises(TypeError):
        B.Attn(h16(8, 16), h16(8, 16), f32(8, 16), h16(8, 16), 2).c()
    with pytest.raises(TypeError):
        B.Predictor(h16(4, 16), f32(8, 4)).c()
    with pytest.raises(TypeError):
        B.KVCache(h16(1, 2, 4, 8), f32(1, 2, 4, 8), [0]).c()
    # fp16 biases, wrong shapes, a transposed (non-contiguous) view
    with pytest.raises(TypeError):
        B.MLP(h16(8, 16), h16(8, 16), b1=h16(8)).c()
    with pytest.raises(ValueError):
        B.MLP(h16(8, 16), h16(8, 16), b2=f32(15)).c()
    with pytest.raises(ValueError):
        B.MLP(h16(16, 8).t(), h16(8, 16)).c()
    with pytest.raises(ValueError):
        B.Attn(h16(9, 16), h16(9, 16), h16(9, 16), h16(9, 16), 2).c()      # 9 rows, 2 heads
    # CPU tensors of the right dtype are rejected as not on the GPU
    with pytest.raises(ValueError, match="GPU"):
        B.MLP(h16(8, 16), h16(8, 16)).c()
    # entry-point arguments: an int64 index set, an fp16 input
    class _M(B.MLP):
        def c(self):
            return B.CMlp(16, 8, B.DV_F16, 0, FAKE, None, FAKE, None)
    m = _M(h16(8, 16), h16(8, 16))
    with pytest.raises(TypeError, match="int32"):
        B.dv_sparse_mlp(m, f32(1, 16).cuda() if torch.cuda.is_available() else f32(1, 16),
                        torch.tensor([1, 2], dtype=torch.int64))
    with pytest.raises(TypeError, match="float32"):
        B.dv_sparse_mlp(m, h16(1, 16), torch.tensor([1, 2], dtype=torch.int32))


def test_noalloc_block_rejects_what_its_scratch_cannot_hold(lib):
    """dv_sparse_block_noalloc has a fixed scratch of DV_STATIC_SCRATCH_BYTES per device:
    a layer whose workspace would exceed it is rejected before any device call (here a
    neuron predictor scoring 2^23 neurons needs 32 MB of scores alone)."""
    a, kv = _attn(), _kv()
    n = 1 << 23
    m = _mlp(n=n)
    ph = B.CPredictor(64, 16, 4, B.DV_F16, FAKE, FAKE)
    pm = B.CPredictor(64, 16, n, B.DV_F16, FAKE, FAKE)
    need = lib.dv_sparse_block_workspace_bytes(ctypes.byref(a), ctypes.byref(m), ctypes.byref(ph),
                                               ctypes.byref(pm), ctypes.byref(kv), 1, 2, 8)
    assert need > B.STATIC_SCRATCH_BYTES
    st = lib.dv_sparse_block_noalloc(ctypes.byref(a), ctypes.byref(m), ctypes.byref(ph), ctypes.byref(pm), None,
                                     ctypes.byref(kv), FAKE, FAKE + 4096, 1, 2, 8, 0, 0, 0.25, None, None, 0, None)
    assert st == B.DV_ERR_WORKSPACE
    hdr = open(HEADER).read()
    assert f"#define DV_STATIC_SCRATCH_BYTES (16u << 20)" in hdr and B.STATIC_SCRATCH_BYTES == 16 << 20


C_PROGRAM = r"""
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "dv.h"

/* A C caller of the library: the header compiles as C99 and the entry points link and
 * reject bad arguments on the host (no device is touched). */
int main(void) {
  dv_mlp m;
  float *x = (float *)(uintptr_t)0x10000000u;
  int32_t *idx = (int32_t *)(uintptr_t)0x10000000u;
  void *ws = (void *)(uintptr_t)0x10000000u;
  size_t need;
  if (dv_abi_version() != 1) return 1;
  if (strcmp(dv_status_string(DV_OK), dv_status_string(DV_ERR_NULL)) == 0) return 2;
  memset(&m, 0, sizeof m);
  m.d = 64;
  m.n = 128;
  m.wtype = DV_F16;
  m.act = DV_ACT_RELU;
  m.W1T = x;
  m.W2T = x;
  if (dv_sparse_mlp(NULL, x, 1, idx, 8, 0, 0, x, ws, 1u << 30, 0, NULL) != DV_ERR_NULL) return 3;
  if (dv_sparse_mlp(&m, x, 1, idx, 129, 0, 0, x, ws, 1u << 30, 0, NULL) != DV_ERR_SHAPE) return 4;
  need = dv_sparse_mlp_workspace_bytes(&m, 1, 8, 0);
  if (need == 0 || need % 256 != 0) return 5;
  if (dv_sparse_mlp(&m, x, 1, idx, 8, 0, 0, x, ws, need - 1, 0, NULL) != DV_ERR_WORKSPACE) return 6;
  printf("c caller ok\n");
  return 0;
}
"""


def test_header_compiles_as_c_and_links(tmp_path):
    """include/dv.h is a C header: a C99 program (-Wall -Wextra -Werror -pedantic) compiles
    against it, links the library and gets the documented host-side statuses."""
    src = tmp_path / "caller.c"
    exe = tmp_path / "caller"
    src.write_text(C_PROGRAM)
    libdir = os.path.dirname(B.lib_path())
    libname = os.path.basename(B.lib_path())
    cc = subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I",
                         os.path.join(ROOT, "include"), str(src), "-o", str(exe), os.path.join(libdir, libname),
                         "-Wl,-rpath," + libdir], capture_output=True, text=True)
    assert cc.returncode == 0, cc.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0, (run.returncode, run.stdout, run.stderr)
    assert "c caller ok" in run.stdout
