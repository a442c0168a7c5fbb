"""The five synthetic staging workloads (shapes, sharding, budgets, seeds).

Plain data: decoder shapes and the value recipe of each workload.  Sizes follow
the decoder families the paper's evaluation uses (an 8B-class model, Sec. 5
"Experimental Setup"); the shapes are synthetic stand-ins, not any released
checkpoint.
"""
from __future__ import annotations

from dataclasses import dataclass

MiB = 1 << 20
GiB = 1 << 30


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    # decoder shape
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    # staging layout
    train_shards: int          # W: flat fp32 training shards
    tp: int                    # T: rollout tensor-parallel ranks
    chunk_bytes: int           # B: byte budget of one staged chunk
    moment_chunk_bytes: int = 0  # Bm: bounded host chunk for Adam moments (0: none)
    specials_frac: float = 0.0   # fraction of weights replaced by cast-stressing values
    generator: str = "numpy"     # "numpy" (host, PCG64) or "torch" (device Philox)

    @property
    def model(self) -> tuple[int, int, int, int, int, int, int]:
        return (self.n_layers, self.hidden, self.n_q_heads, self.n_kv_heads, self.head_dim, self.ffn, self.vocab)


TINY = Workload("tiny", 0, 2, 256, 4, 4, 64, 688, 2048, train_shards=4, tp=2, chunk_bytes=256 * 1024)
HALF_B = Workload("0.5b", 1, 24, 896, 14, 2, 64, 4864, 151936, train_shards=8, tp=1, chunk_bytes=64 * MiB,
                  specials_frac=0.001)
EIGHT_B = Workload("8b", 2, 32, 4096, 32, 8, 128, 14336, 128256, train_shards=8, tp=4, chunk_bytes=256 * MiB,
                   generator="torch")
THIRTY_TWO_B = Workload("32b", 3, 64, 5120, 40, 8, 128, 27648, 152064, train_shards=1, tp=8, chunk_bytes=GiB,
                        generator="torch")
EIGHT_B_ADAM = Workload("8b_adam", 4, 32, 4096, 32, 8, 128, 14336, 128256, train_shards=8, tp=4,
                        chunk_bytes=256 * MiB, moment_chunk_bytes=512 * MiB, generator="torch")

ALL = (TINY, HALF_B, EIGHT_B, THIRTY_TWO_B, EIGHT_B_ADAM)
BY_NAME = {w.name: w for w in ALL}
