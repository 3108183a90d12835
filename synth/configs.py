"""The five prefill workloads, as seeded synthetic inputs.

The paper evaluates real LLaMA / Qwen / Vicuna activations on LongEval and
LV-Eval; none of those models or datasets are used here.  Seeded synthetic
tensors with the shapes below stand in for them:

  1k-mha-d64     B=1, 2/2 heads, d=64, L=1024, tile 64x64, g=1, Bernoulli(0.5)
  8k-gqa         B=1, 32/8 heads, d=128, L=8192, tile 128x64, g=1, Bernoulli(0.5),
                 K outlier channels
  32k-gqa        B=1, 32/8, d=128, L=32768, tile 128x64, g=4, Bernoulli(0.75),
                 K outlier channels
  128k-gqa       B=1, 32/8, d=128, L=131072, tile 128x64, g=16, structured mask
                 (FP16 on the 256-key sink and within 4096 tokens of the
                 diagonal, INT8 elsewhere), K outlier channels
  64k-b4-gqa     B=4, 64/8, d=128, L=65536, tile 128x64, g=8, three masks:
                 all-FP16, all-INT8, Bernoulli(0.5)

Values are N(0,1) drawn in float32 and rounded to float16; "outlier channels"
are ceil(1% of d) K channels per KV head, picked by seed, multiplied by 8.
All workloads are causal self-attention with scale 1/sqrt(d).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np


@dataclass(frozen=True)
class MaskSpec:
    kind: str              # "bernoulli" | "all_fp16" | "all_int8" | "sink_band"
    p_int8: float = 0.0    # for "bernoulli"
    sink_keys: int = 0     # for "sink_band"
    band_tokens: int = 0   # for "sink_band"

    @property
    def label(self) -> str:
        if self.kind == "bernoulli":
            return f"bern{self.p_int8:g}"
        if self.kind == "sink_band":
            return f"sink{self.sink_keys}_band{self.band_tokens}"
        return self.kind


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    index: int
    B: int
    Hq: int
    Hk: int
    d: int
    L: int
    block_m: int
    block_n: int
    group_size: int
    masks: tuple = field(default_factory=tuple)
    k_outliers: bool = False
    causal: bool = True

    @property
    def seed(self) -> int:
        return 20260 + self.index

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def Lq(self) -> int:
        return self.L

    @property
    def Lk(self) -> int:
        return self.L

    @property
    def T_m(self) -> int:
        return math.ceil(self.Lq / self.block_m)

    @property
    def T_n(self) -> int:
        return math.ceil(self.Lk / self.block_n)

    @property
    def T_mask(self) -> int:
        return math.ceil(self.T_n / self.group_size)

    @property
    def words_per_row(self) -> int:
        return max(1, math.ceil(self.T_mask / 64))

    def legal_pairs(self) -> int:
        """Number of legal (query, key) pairs summed over batch and query heads."""
        if self.causal:
            off = self.Lk - self.Lq
            per_head = int(np.clip(np.arange(self.Lq, dtype=np.int64) + off + 1, 0, self.Lk).sum())
        else:
            per_head = self.Lq * self.Lk
        return self.B * self.Hq * per_head

    def with_(self, **kw) -> "WorkloadConfig":
        return replace(self, **kw)


WORKLOADS = {
    "1k-mha-d64": WorkloadConfig("1k-mha-d64", 1, B=1, Hq=2, Hk=2, d=64, L=1024, block_m=64,
                                 block_n=64, group_size=1, masks=(MaskSpec("bernoulli", 0.5),)),
    "8k-gqa": WorkloadConfig("8k-gqa", 2, B=1, Hq=32, Hk=8, d=128, L=8192, block_m=128,
                             block_n=64, group_size=1, masks=(MaskSpec("bernoulli", 0.5),),
                             k_outliers=True),
    "32k-gqa": WorkloadConfig("32k-gqa", 3, B=1, Hq=32, Hk=8, d=128, L=32768, block_m=128,
                              block_n=64, group_size=4, masks=(MaskSpec("bernoulli", 0.75),),
                              k_outliers=True),
    "128k-gqa": WorkloadConfig("128k-gqa", 4, B=1, Hq=32, Hk=8, d=128, L=131072, block_m=128,
                               block_n=64, group_size=16,
                               masks=(MaskSpec("sink_band", sink_keys=256, band_tokens=4096),),
                               k_outliers=True),
    "64k-b4-gqa": WorkloadConfig("64k-b4-gqa", 5, B=4, Hq=64, Hk=8, d=128, L=65536, block_m=128,
                                 block_n=64, group_size=8,
                                 masks=(MaskSpec("all_fp16"), MaskSpec("all_int8"),
                                        MaskSpec("bernoulli", 0.5))),
}


def workload(name: str) -> WorkloadConfig:
    return WORKLOADS[name]


def small_workload(name: str, *, B=1, Hq=2, Hk=1, d=128, L=300, block_m=128, block_n=64,
                   group_size=1, mask=MaskSpec("bernoulli", 0.5), k_outliers=False,
                   causal=True, index=100) -> WorkloadConfig:
    """A small ad-hoc workload for tests (ragged lengths, odd groupings)."""
    return WorkloadConfig(name, index, B=B, Hq=Hq, Hk=Hk, d=d, L=L, block_m=block_m,
                          block_n=block_n, group_size=group_size, masks=(mask,),
                          k_outliers=k_outliers, causal=causal)
