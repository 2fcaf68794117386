"""The synthetic KV-cache workloads.

Each config fixes the cache shape (layers, heads, head dim, block size, 16-bit
type), the batch, the distribution of sequence lengths, the fraction of
logical blocks that live in the memory slice, and the seed. Seeds are
27040 + the workload's index.
"""
from dataclasses import dataclass, field
from typing import Tuple


@dataclass(frozen=True)
class KVConfig:
    name: str
    layers: int
    q_heads: int
    kv_heads: int
    head_dim: int
    dtype: str                 # "f16" or "bf16"
    block_size: int            # tokens per KV block
    batch: int
    lens: Tuple                # ("uniform", lo, hi) inclusive, or
                               # ("lognormal", median, sigma, lo, hi)
    slice_frac: float          # fraction of each layer's logical blocks in the slice
    seed: int
    extra: dict = field(default_factory=dict, compare=False)

    @property
    def elem_bytes(self) -> int:
        return 2

    @property
    def block_bytes(self) -> int:
        """Bytes of one layer-block: K and V of block_size tokens, all KV heads."""
        return 2 * self.block_size * self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads

    def scaled(self, **kw) -> "KVConfig":
        d = dict(self.__dict__)
        d.update(kw)
        return KVConfig(**d)


# Tiny parity case: one layer, MHA, fp16, half of the blocks in the slice.
TINY = KVConfig("tiny", 1, 8, 8, 128, "f16", 16, 8, ("uniform", 64, 512), 0.5, 27040)

# Llama-3-8B-shaped KV cache: GQA 32/8, bf16, block 16, batch 64, len U[1024,4096].
LLAMA8B = KVConfig("llama3-8b-kv", 32, 32, 8, 128, "bf16", 16, 64,
                   ("uniform", 1024, 4096), 0.3, 27041)

# One GPU's share of a 70B-shaped layer at tensor-parallel degree 8: 8 q heads,
# 1 KV head, block 32, batch 128, lognormal lengths (median 2048, sigma 1.0,
# clipped to [128, 16384]), half the blocks in the slice.
L70B_TP8 = KVConfig("llama-70b-tp8-share", 80, 8, 1, 128, "bf16", 32, 128,
                    ("lognormal", 2048, 1.0, 128, 16384), 0.5, 27042)

# Bursty elastic trace on the 8B-shaped cache: 200 steps of a random walk of the
# slice fraction in [0, 0.7], lend/reclaim of 1-25 % of the lent blocks per step.
BURSTY = LLAMA8B.scaled(name="bursty-8b", slice_frac=0.3, seed=27043,
                        extra={"steps": 200, "frac_max": 0.7,
                               "step_frac": (0.01, 0.25)})

# Copy-throughput stress: 8 KV heads, fp16, block sizes 16/64/256, up to 2^20
# blocks capped at 100 GiB of KV, 60 % slice-resident.
STRESS = KVConfig("stress", 1, 8, 8, 128, "f16", 16, 1, ("uniform", 0, 0), 0.6, 27044,
                  extra={"block_sizes": (16, 64, 256), "max_blocks": 1 << 20,
                         "max_kv_bytes": 100 << 30})

CONFIGS = {c.name: c for c in (TINY, LLAMA8B, L70B_TP8, BURSTY, STRESS)}
