"""GPU: the per-launch timing hook (dv_set_launch_events) that the benchmark's
per-kernel figures come from.

Each timed launch's events are stamped by its kernels' own dispatches; the intervals
must cover every launch of a call once, in launch order and without overlap, and
arming the hook must not change any result.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2310_17157_amd import binding as Bd
from paper_2310_17157_amd.workload import layer_objects
from tests.gpu_util import host, layer

pytestmark = pytest.mark.gpu

BLOCK_LAUNCHES = {"pred_hidden", "pred_scores", "qkv", "attn", "oproj", "fc1", "fc2"}


def _call(cfg, objs, x):
    attn, mlp, ph, pm, kv, lnp = objs
    return Bd.dv_sparse_block(attn, mlp, ph, pm, lnp, kv, x, cfg.k_heads, cfg.k_mlp, 1.0 / np.sqrt(cfg.dh))


def _gap_ms(timer, i):
    """Time from the end of timed launch i to the start of launch i + 1."""
    ms = ctypes.c_float(0.0)
    assert timer._hip.hipEventElapsedTime(ctypes.byref(ms), timer.events[2 * i + 1], timer.events[2 * i + 2]) == 0
    return ms.value


@pytest.mark.parametrize("name", ["opt125m_b1", "opt175b_b1"])
def test_launch_events_cover_every_launch_in_order(name):
    cfg, t = layer(name, 71, biases=True, ln_random=True)
    objs = layer_objects(t, cfg.H)
    ref = [host(a).tobytes() for a in _call(cfg, objs, t["x"])]
    torch.cuda.synchronize()
    timer = Bd.LaunchTimer(32)
    try:
        timer.arm()
        outs = _call(cfg, objs, t["x"])
        timer.disarm()
        torch.cuda.synchronize()
        times = timer.times_ms()
        labels = [lab for lab, _ in times]
        assert BLOCK_LAUNCHES <= set(labels), labels
        assert len(labels) == timer.n_launched.value
        for lab, ms in times:
            assert 0.0 < ms < 1000.0, (lab, ms)
        for i in range(len(times) - 1):
            assert _gap_ms(timer, i) >= -1e-3, (labels[i], labels[i + 1])
    finally:
        timer.close()
    # timing changes no result (the call repeats the same cache writes)
    assert [host(a).tobytes() for a in outs] == ref


def test_launch_events_only_one_label():
    cfg, t = layer("opt125m_b1", 72, biases=True, ln_random=True)
    objs = layer_objects(t, cfg.H)
    timer = Bd.LaunchTimer(4, only="qkv")
    try:
        for _ in range(2):
            timer.arm()
            _call(cfg, objs, t["x"])
            timer.disarm()
            torch.cuda.synchronize()
            times = timer.times_ms()
            assert [lab for lab, _ in times] == ["qkv"]
            assert 0.0 < times[0][1] < 1000.0
    finally:
        timer.close()
