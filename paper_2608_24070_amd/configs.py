"""The five synthetic workloads (LLaMA-2 shaped layers) used by the tests and the benchmark.

Ranks follow the SLiM setup: adapter rank = 10% of the smaller layer dimension, here
rounded down to a multiple of 64. Layer shapes are those of LLaMA-2 7B/13B/70B linear
layers. Inputs are synthetic (see ``synth``).
"""
from dataclasses import dataclass, field


def rank_for(n: int, k: int) -> int:
    return 64 * int(0.1 * min(n, k) // 64)


@dataclass(frozen=True)
class Layer:
    name: str
    n: int          # output features (rows of W)
    k: int          # input features (reduction length)
    r: int          # adapter rank


@dataclass(frozen=True)
class Workload:
    key: str
    layers: tuple
    ms: tuple                      # row counts of X (tokens) exercised
    xdtype: str = "bf16"
    seeds: tuple = (0,)
    backward: bool = False
    note: str = ""


TINY = Workload("tiny", (Layer("tiny", 512, 512, 32),), (16,), xdtype="fp16",
                note="16x512 fp16 input, 512x512 weight, rank 32")
DECODE = Workload("decode", (Layer("decode", 4096, 4096, rank_for(4096, 4096)),), (1, 4, 16),
                  note="decode-shaped: M in {1,4,16}, 4096x4096 weight, rank 384")
PREFILL = Workload("prefill", (Layer("up_proj", 11008, 4096, rank_for(11008, 4096)),), (2048,),
                   note="LLaMA-2-7B MLP up-projection, M = 2048, rank 384 (+ fp16 with 1% outlier channels x20)")
BLOCK13B = Workload("block13b", tuple(
    Layer(nm, n, k, rank_for(n, k)) for nm, n, k in [
        ("q", 5120, 5120), ("k", 5120, 5120), ("v", 5120, 5120), ("o", 5120, 5120),
        ("gate", 13824, 5120), ("up", 13824, 5120), ("down", 5120, 13824)]), (4096,),
    note="LLaMA-2-13B block, 7 linears in sequence at M = 4096, rank 512")
MLP70B = Workload("mlp70b", (Layer("mlp70b", 28672, 8192, 512),), (1, 16, 512, 8192), seeds=(0, 1, 2),
                  backward=True, note="LLaMA-2-70B MLP shape 28672x8192, rank 512, forward and double-pruned dX")

ALL = {w.key: w for w in (TINY, DECODE, PREFILL, BLOCK13B, MLP70B)}
