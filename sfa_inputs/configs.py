"""The five synthetic workloads: shapes of the paper's GPT-2 and Qwen3
attention (head dims 64 and 128; Qwen3-style 4:1 grouped KV heads), a
skewed-support stress case and a sparse-code KV-cache decode step.

Workload `tiny` is small enough for the oracle to finish in a second;
`qwen3_32k` is the headline forward workload."""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str              # "fwd" or "decode"
    B: int
    Hq: int
    Hkv: int
    n: int                 # sequence length (fwd) or cached context length (decode)
    d: int
    k: int
    causal: bool
    seed: int
    v_bf16: bool           # V (and the decode V cache) stored as bf16
    o_bf16: bool           # output stored as bf16
    zipf_s: float = 0.0    # >0: supports drawn with Zipf(s) popularity
    note: str = ""

    @property
    def scale(self) -> float:
        return 1.0 / (self.d ** 0.5)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny", "fwd", 1, 1, 1, 256, 64, 8, True, 1, False, False,
                 note="fp32 V and O"),
        Workload("gpt2s", "fwd", 8, 12, 12, 1024, 64, 16, True, 2, True, True,
                 note="GPT-2 small attention shape"),
        Workload("qwen3_32k", "fwd", 1, 32, 8, 32768, 128, 16, True, 3, True, True,
                 note="Qwen3-like GQA 4:1, 32K context"),
        Workload("zipf_128k", "fwd", 1, 8, 8, 131072, 128, 8, True, 4, True, True,
                 zipf_s=1.1, note="Zipf(1.1) feature popularity, 128K context"),
        Workload("decode_64k", "decode", 64, 32, 8, 65536, 128, 16, False, 5, True, True,
                 note="one new token per sequence over a 64K sparse-code cache"),
    ]
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
