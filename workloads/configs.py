"""The synthetic workloads, as specifications the generator turns into bytes.

Shapes are Llama-3-8B attention shapes (32 query heads, 8 KV heads,
head_dim 128, block size 16) except the tiny fp32 decode case. Every
sequence length range is inclusive. Each workload has its own seed.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence

SEED_BASE = 260823658


@dataclass(frozen=True)
class BatchSpec:
    """One attention call's worth of synthetic input.

    ``seq_lens`` are total context lengths *including* the new tokens of the
    call; ``q_lens`` are the new (query) tokens per sequence, so a decode
    sequence has ``q_len == 1`` and a prefill chunk of ``n`` tokens over
    ``c`` cached tokens has ``seq_len == c + n``.
    """

    name: str
    dtype: str                      # "f32" or "bf16": storage and input type
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    seed: int
    # Either fixed lengths or an inclusive uniform range with a count.
    fixed_seq_lens: Optional[Sequence[int]] = None
    rand_count: int = 0
    rand_lo: int = 0
    rand_hi: int = 0
    # Sequences whose lengths and chunk sizes are fixed and placed before
    # the random ones: tuples (seq_len, q_len).
    fixed_prefix: Sequence[tuple] = field(default_factory=tuple)
    q_len_rand: int = 1             # q_len of every random / fixed_seq_lens sequence
    num_blocks: Optional[int] = None  # pool size; None -> 1.1x rule
    max_num_batched_tokens: Optional[int] = None

    @property
    def scale(self) -> float:
        return 1.0 / (self.head_dim ** 0.5)


def pool_blocks_rule(total_blocks: int) -> int:
    """Pool size: the blocks the batch needs plus 10% free, rounded up to a
    whole number of 2 MiB granules' worth of blocks (32 blocks of 64 KiB at
    the Llama shapes)."""
    want = -(-total_blocks * 11 // 10)
    return -(-want // 32) * 32


# Tiny paged decode in fp32: 4 sequences, GQA 2:1, head_dim 64.
TINY_DECODE_F32 = BatchSpec(name="tiny_decode_f32", dtype="f32", num_q_heads=4, num_kv_heads=2,
                            head_dim=64, block_size=16, seed=SEED_BASE + 1,
                            fixed_seq_lens=(37, 64, 101, 130), num_blocks=64)
# Llama-3-8B-shaped decode layer, bf16: 256 sequences, lengths U[512, 4096].
DECODE_B256 = BatchSpec(name="decode_b256_l512_4096_bf16", dtype="bf16", num_q_heads=32,
                        num_kv_heads=8, head_dim=128, block_size=16, seed=SEED_BASE + 2,
                        rand_count=256, rand_lo=512, rand_hi=4096)
# Mixed chunked-prefill step: the last 8192-token chunk of a 32768-token
# prompt (24576 cached tokens) plus 128 decode sequences U[1024, 8192].
MIXED_STEP = BatchSpec(name="mixed_chunk8192_ctx24576_plus_decode128_bf16", dtype="bf16",
                       num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=16,
                       seed=SEED_BASE + 3, fixed_prefix=((32768, 8192),),
                       rand_count=128, rand_lo=1024, rand_hi=8192,
                       max_num_batched_tokens=8192 + 128)
# Chunk-size equivalence: one 32768-token prompt, prefilled whole.
PREFILL_L32768 = BatchSpec(name="prefill_l32768_bf16", dtype="bf16", num_q_heads=32,
                           num_kv_heads=8, head_dim=128, block_size=16, seed=SEED_BASE + 4,
                           fixed_prefix=((32768, 32768),), num_blocks=2272,
                           max_num_batched_tokens=32768)

WORKLOADS = {s.name: s for s in (TINY_DECODE_F32, DECODE_B256, MIXED_STEP, PREFILL_L32768)}


# Elastic-pool decode workload (32 layers, base + elastic handle per layer).
@dataclass(frozen=True)
class ElasticSpec:
    name: str = "elastic_decode_32l_b512_l8192_32768_bf16"
    num_layers: int = 32
    num_q_heads: int = 32
    num_kv_heads: int = 8
    head_dim: int = 128
    block_size: int = 16
    batch: int = 512
    len_lo: int = 8192
    len_hi: int = 32768
    elastic_bytes_total: int = 3 << 30          # 3 GiB over all layers
    base_blocks: int = 96768                    # 6 GiB - 96 MiB per layer
    elastic_fraction: float = 0.15              # share of block references that are elastic ids
    seed: int = SEED_BASE + 5

    @property
    def block_bytes(self) -> int:
        return 2 * self.num_kv_heads * self.block_size * self.head_dim * 2

    @property
    def elastic_bytes_per_layer(self) -> int:
        return self.elastic_bytes_total // self.num_layers

    @property
    def elastic_blocks(self) -> int:
        return self.elastic_bytes_per_layer // self.block_bytes

    @property
    def scale(self) -> float:
        return 1.0 / (self.head_dim ** 0.5)


ELASTIC = ElasticSpec()
