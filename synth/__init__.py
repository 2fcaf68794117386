"""Seeded synthetic inputs shaped like the paper's LLM-serving KV caches.

This package draws random numbers and lays out workload structure (sequence
lengths, which logical KV blocks sit in the memory slice, the order blocks are
allocated in, the K/V/q values). It holds none of the method's arithmetic: no
block movement, no bookkeeping of ownership, no attention. Both the CPU oracle
tests and the GPU path take their inputs from here; neither side imports the
other.

The workloads stand in for the paper's serving setting (LLaMA/OPT models on
ShareGPT/Alpaca request streams, evaluation section), whose datasets and
weights are not used: only the KV-cache shapes and length mixes are modelled.
"""
from .configs import KVConfig, CONFIGS, TINY, LLAMA8B, L70B_TP8, BURSTY, STRESS
from .gen import (
    seq_lens, placement, BlockPlacement, round_to_16bit, random_16bit,
    q_values, element_index, pack_block, unpack_block, LAYOUT_ATTN, LAYOUT_NHD, NAN16,
)

__all__ = [
    "KVConfig", "CONFIGS", "TINY", "LLAMA8B", "L70B_TP8", "BURSTY", "STRESS",
    "seq_lens", "placement", "BlockPlacement", "round_to_16bit", "random_16bit",
    "q_values", "element_index", "pack_block", "unpack_block",
    "LAYOUT_ATTN", "LAYOUT_NHD", "NAN16",
]
