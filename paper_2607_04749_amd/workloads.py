"""Model shapes and the five resharding workloads.

A workload is a model, a source (TP, PP) configuration, a target one, and
which ranks run at real shape.  "full" workloads keep every source and every
target rank in one GPU's memory (all packs, in-memory routing, all unpacks);
"share" workloads run one source rank's pack and one target rank's unpack at
real shape, with the other sources that feed that target packed beforehand.

States per logical element: bf16 parameter, fp32 master, fp32 Adam m, fp32
Adam v (14 bytes), seeded from N(0, 0.02), with v = |N(0, 1e-4)|.
"""
from __future__ import annotations

from dataclasses import dataclass, field

GPT = 0
LLAMA = 1
LAYERS_ONLY = 1  # model flag: layer tensors only (no embeddings, final norm or head)

KINDS = ("param_bf16", "master_f32", "adam_m_f32", "adam_v_f32")
ESIZE = (2, 4, 4, 4)
BYTES_PER_ELEM = sum(ESIZE)


@dataclass(frozen=True)
class ModelShape:
    arch: int
    num_layers: int
    hidden: int
    num_heads: int
    num_kv_heads: int
    ffn_hidden: int
    vocab: int
    max_pos: int
    tied: int
    flags: int = 0

    def astuple(self):
        return (self.arch, self.num_layers, self.hidden, self.num_heads, self.num_kv_heads,
                self.ffn_hidden, self.vocab, self.max_pos, self.tied, self.flags)


@dataclass(frozen=True)
class Parallel:
    tp: int
    pp: int
    dp: int = 1

    @property
    def world(self) -> int:
        return self.tp * self.pp * self.dp

    def astuple(self):
        return (self.tp, self.pp, self.dp)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    src: Parallel
    dst: Parallel
    mode: str  # "full" or "share"
    seed: int
    pack_rank: int = 0
    unpack_rank: int = 0
    note: str = field(default="")


TINY_GPT = ModelShape(GPT, 4, 256, 4, 4, 1024, 1024, 128, 1)
GPT_1_3B = ModelShape(GPT, 24, 2048, 16, 16, 8192, 50304, 2048, 1)
LLAMA_7B = ModelShape(LLAMA, 32, 4096, 32, 32, 11008, 32000, 0, 0)
LLAMA_13B = ModelShape(LLAMA, 40, 5120, 40, 40, 13824, 32000, 0, 0)
LLAMA_70B = ModelShape(LLAMA, 80, 8192, 64, 8, 28672, 32000, 0, 0)

SEED_BASE = 0xE7C00000

WORKLOADS = {
    "tiny-gpt": Workload("tiny-gpt", TINY_GPT, Parallel(2, 2), Parallel(4, 1), "full",
                         SEED_BASE + 0, note="TP2xPP2 -> TP4xPP1, all 4 sources and 4 targets"),
    "gpt-1.3b": Workload("gpt-1.3b", GPT_1_3B, Parallel(4, 2), Parallel(2, 4), "full",
                         SEED_BASE + 1, note="TP4xPP2 -> TP2xPP4, full 8->8 emulation"),
    "llama-7b": Workload("llama-7b", LLAMA_7B, Parallel(8, 1), Parallel(4, 1), "share",
                         SEED_BASE + 2, note="TP8 -> TP4 scale-in, pack src 0, unpack dst 0"),
    "llama-13b": Workload("llama-13b", LLAMA_13B, Parallel(4, 2), Parallel(8, 2), "share",
                          SEED_BASE + 3, note="TP4xPP2 -> TP8xPP2 scale-out, pack src 0, unpack dst 0"),
    "llama-70b": Workload("llama-70b", LLAMA_70B, Parallel(8, 8), Parallel(8, 4), "share",
                          SEED_BASE + 4, note="TP8xPP8 -> TP8xPP4, pack src 0, unpack dst 0"),
}

ORDER = ("tiny-gpt", "gpt-1.3b", "llama-7b", "llama-13b", "llama-70b")
