"""The draft-tree workloads the library is measured and tested on: Qwen2.5-7B and
-32B decoder-layer projection shapes (public model dimensions) at the token
counts of a speculative draft tree, with the bit widths and group sizes used for
the substitutes."""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Proj:
    name: str
    K: int  # input features
    N: int  # output features


QWEN7B = (Proj("q", 3584, 3584), Proj("k", 3584, 512), Proj("v", 3584, 512),
          Proj("o", 3584, 3584), Proj("gate", 3584, 18944), Proj("up", 3584, 18944),
          Proj("down", 18944, 3584))
QWEN32B = (Proj("q", 5120, 5120), Proj("k", 5120, 1024), Proj("v", 5120, 1024),
           Proj("o", 5120, 5120), Proj("gate", 5120, 27648), Proj("up", 5120, 27648),
           Proj("down", 27648, 5120))


def fused_layer(projs):
    """The per-layer launch plan: q|k|v and gate|up share their input, so each
    pair/triple is one launch over concatenated columns; 7 projections -> 4 launches."""
    by = {p.name: p for p in projs}
    return (Proj("qkv", by["q"].K, by["q"].N + by["k"].N + by["v"].N),
            by["o"],
            Proj("gate_up", by["gate"].K, by["gate"].N + by["up"].N),
            by["down"])


@dataclass(frozen=True)
class Workload:
    key: str
    description: str
    projs: tuple
    bits: int
    group: int
    ms: tuple
    layers: int = 1
    outlier_frac: float = 0.0
    fused: bool = False


WORKLOADS = {
    "tiny": Workload("tiny", "tiny qlinear K=256 N=512, 4-bit g64", (Proj("tiny", 256, 512),),
                     4, 64, (1, 4)),
    "qwen7b_mlp": Workload("qwen7b_mlp", "Qwen2.5-7B-shaped MLP projections, 4-bit g128",
                           (Proj("gate", 3584, 18944), Proj("up", 3584, 18944),
                            Proj("down", 18944, 3584)), 4, 128, (1, 8, 32, 64)),
    "qwen7b_mlp_draft": Workload("qwen7b_mlp_draft", "Qwen2.5-7B-shaped MLP projections, 4-bit g128, "
                                 "at small draft batches (Sec. 5.1 draws k = 6 leaves per pass)",
                                 (Proj("gate", 3584, 18944), Proj("up", 3584, 18944),
                                  Proj("down", 18944, 3584)), 4, 128, (2, 4, 6, 8)),
    "qwen7b_stack": Workload("qwen7b_stack", "Qwen2.5-7B-shaped 28-layer substitute stack, "
                             "4-bit g128", QWEN7B, 4, 128, (64,), layers=28, fused=True),
    "qwen32b_stack": Workload("qwen32b_stack", "Qwen2.5-32B-shaped 64-layer substitute stack, "
                              "3-bit g128", QWEN32B, 3, 128, (1, 16, 64, 128), layers=64,
                              fused=True),
    "qwen32b_2bit": Workload("qwen32b_2bit", "Qwen2.5-32B-shaped 64-layer stack, 2-bit g64, "
                             "1% outlier channels x20", QWEN32B, 2, 64, (128,), layers=64,
                             outlier_frac=0.01, fused=True),
}


def weight_bytes(N: int, K: int, bits: int, group: int) -> int:
    """Algorithmic weight bytes of one projection: packed codes + fp16 scale + fp16 zero."""
    return N * K * bits // 8 + 4 * N * (K // group)
