"""The five decode workloads (shapes only; no arithmetic of the method).

Each entry names the model shape it imitates, the context length, the ladder
profile and which parts of the hot path it exercises.
"""
from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    id: int
    name: str
    B: int
    Hq: int
    Hkv: int
    T: int
    D: int = 128
    block: int = 64
    profile: str = "graded"     # "tiny" | "graded" | "exact"
    page: int = 0               # Quest page size (0 = dense read)
    topk: int = 0               # Quest pages per KV head
    rd_percent: int = 0         # exact residual fraction in percent of T
    dynamic_steps: int = 0      # decode steps with append + demote


TINY = Workload(1, "tiny graded dense, 8q/2kv, T=2048", B=1, Hq=8, Hkv=2, T=2048, profile="tiny")
LLAMA16K = Workload(2, "Llama-3-8B-shaped graded dense, 32q/8kv, T=16384", B=1, Hq=32, Hkv=8, T=16384)
QUEST32K = Workload(3, "Compressed-Quest, 32q/8kv, T=32768, page 16, top-128", B=1, Hq=32, Hkv=8,
                    T=32768, page=16, topk=128)
RD128K = Workload(4, "Qwen2.5-7B-shaped graded+RD, 28q/4kv, B=8, T=131072, 2% residual", B=8, Hq=28,
                  Hkv=4, T=131072, rd_percent=2)
QUEST1M = Workload(5, "1M-token Compressed-Quest + demotion, 32q/8kv, T=1048576, page 16, top-256", B=1,
                   Hq=32, Hkv=8, T=1048576, page=16, topk=256, dynamic_steps=64)
# the Quest point at 128k context (workload 3's shapes at T=131072)
QUEST128K = Workload(3, "Compressed-Quest, 32q/8kv, T=131072, page 16, top-128", B=1, Hq=32, Hkv=8,
                     T=131072, page=16, topk=128)

ALL = {w.id: w for w in (TINY, LLAMA16K, QUEST32K, RD128K, QUEST1M)}
