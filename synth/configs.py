"""Workload shapes: OPT-shaped single decoder layers at decode time.

The five full-size workloads are OPT-125m/6.7B/66B/175B layer shapes at batch 1 and
the OPT-175B shape at batch 32. Selection sizes use k = floor(p * N) for the MLP
(computed in integers so that 8% of 16384 is 1310 and 5% of 49152 is 2457) and an
exact head count. The smaller shapes below them are parity cases: small enough for
the fp64 oracle to finish in seconds, ragged on purpose (d, N, L not multiples of
any tile size) so that tails are exercised.
"""
from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class Config:
    name: str
    d: int            # model width d
    N: int            # MLP neurons (4d in OPT)
    H: int            # attention heads h
    dh: int           # head width d_h
    L: int            # attended positions per sequence at batch 1 (cache rows 0..L-1, pos = L-1)
    r: int            # predictor rank (hidden width of the two-layer predictor)
    k_mlp: int        # |S_M| per sequence
    k_heads: int      # |S_A| per sequence
    wdtype: str       # "f32" or "f16": weights, predictor factors
    kvdtype: str      # "f32" or "f16": KV cache
    B: int = 1
    L_range: Optional[Tuple[int, int]] = None   # batch>1: per-sequence L ~ U{lo..hi}
    zipf_s: Optional[float] = None              # batch>1: neuron popularity exponent
    cap: Optional[int] = None                   # KV capacity; default = max attended length
    desc: str = ""

    @property
    def kv_cap(self) -> int:
        if self.cap is not None:
            return self.cap
        return self.L_range[1] if self.L_range else self.L

    @property
    def wbytes(self) -> int:
        return 4 if self.wdtype == "f32" else 2

    @property
    def kvbytes(self) -> int:
        return 4 if self.kvdtype == "f32" else 2

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


def _kfloor(num: int, den: int, n: int) -> int:
    return (num * n) // den


CONFIGS = {
    # Full-size workloads (OPT layer shapes).
    "opt125m_b1": Config("opt125m_b1", d=768, N=3072, H=12, dh=64, L=128, r=64,
                         k_mlp=_kfloor(10, 100, 3072), k_heads=4, wdtype="f32", kvdtype="f32",
                         desc="OPT-125m-shaped layer, batch 1, fp32, MLP top-10%, 4 of 12 heads"),
    "opt6.7b_b1": Config("opt6.7b_b1", d=4096, N=16384, H=32, dh=128, L=1024, r=1000,
                         k_mlp=_kfloor(8, 100, 16384), k_heads=12, wdtype="f16", kvdtype="f16",
                         desc="OPT-6.7B-shaped layer, batch 1, fp16 weights, MLP top-8%, 12 of 32 heads"),
    "opt66b_b1": Config("opt66b_b1", d=9216, N=36864, H=72, dh=128, L=2048, r=1000,
                        k_mlp=_kfloor(5, 100, 36864), k_heads=24, wdtype="f16", kvdtype="f16",
                        desc="OPT-66B-shaped layer, batch 1, fp16 weights, MLP top-5%, 24 of 72 heads"),
    "opt175b_b1": Config("opt175b_b1", d=12288, N=49152, H=96, dh=128, L=2048, r=1000,
                         k_mlp=_kfloor(5, 100, 49152), k_heads=32, wdtype="f16", kvdtype="f16",
                         desc="OPT-175B-shaped layer, batch 1, fp16 weights, MLP top-5%, 32 of 96 heads"),
    "opt175b_b32": Config("opt175b_b32", d=12288, N=49152, H=96, dh=128, L=2048, r=1000,
                          k_mlp=_kfloor(5, 100, 49152), k_heads=32, wdtype="f16", kvdtype="f16",
                          B=32, L_range=(512, 2048), zipf_s=1.1,
                          desc="OPT-175B-shaped layer, batch 32, per-sequence L~U[512,2048], "
                               "Zipf(1.1) neuron sets (union MLP), 32 of 96 heads per sequence"),
    # Parity cases: ragged, several tiles, oracle-fast.
    "tiny": Config("tiny", d=8, N=8, H=4, dh=2, L=3, r=4, k_mlp=2, k_heads=2,
                   wdtype="f32", kvdtype="f32", desc="brute-force shape"),
    "small_f32": Config("small_f32", d=392, N=1000, H=7, dh=56, L=77, r=40, k_mlp=101, k_heads=3,
                        wdtype="f32", kvdtype="f32", desc="ragged fp32 parity case"),
    "small_f16": Config("small_f16", d=1288, N=5000, H=10, dh=128, L=333, r=200, k_mlp=501,
                        k_heads=4, wdtype="f16", kvdtype="f16", desc="ragged fp16 parity case"),
    "small_b8": Config("small_b8", d=1288, N=5000, H=10, dh=128, L=333, r=200, k_mlp=501,
                       k_heads=4, wdtype="f16", kvdtype="f16", B=8, L_range=(40, 333), zipf_s=1.1,
                       desc="ragged fp16 batch-8 parity case"),
}


def get_config(name: str) -> Config:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS)}") from None
