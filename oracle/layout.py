"""Byte layout of one layer-block (oracle's own statement of the format).

A layer-block holds the keys and values of ``block_size`` consecutive tokens of
one sequence, for every KV head of one layer (the paper's "KV cache blocks",
inherited from vLLM, section 4.2.1). The K half comes first, then the V half.

ATTN layout (the local paged cache, read by decode attention):
    K as [kv_head][token][channel]      (one contiguous row per token and head)
    V as [kv_head][channel][token]      (transposed: one row per channel)
NHD layout (token-major, an optional layout of the slice):
    K as [token][kv_head][channel]
    V as [token][kv_head][channel]

Elements are 16-bit (fp16 or bf16) patterns. Decoding is a reshape plus an axis
transpose; values are upcast exactly to float64 by ``to_float64``.
"""
import numpy as np

LAYOUT_ATTN = 0
LAYOUT_NHD = 1


def block_bytes(kv_heads: int, head_dim: int, block_size: int, elem_bytes: int = 2) -> int:
    return 2 * block_size * kv_heads * head_dim * elem_bytes


def decode_block(block_u8, layout: int, kv_heads: int, head_dim: int, block_size: int):
    """bytes -> (K, V), each a uint16 array [kv_head][token][channel]."""
    e = np.frombuffer(np.ascontiguousarray(block_u8).tobytes(), dtype=np.uint16)
    n = block_size * kv_heads * head_dim
    k, v = e[:n], e[n:2 * n]
    if layout == LAYOUT_ATTN:
        K = k.reshape(kv_heads, block_size, head_dim)
        V = v.reshape(kv_heads, head_dim, block_size).transpose(0, 2, 1)
    elif layout == LAYOUT_NHD:
        K = k.reshape(block_size, kv_heads, head_dim).transpose(1, 0, 2)
        V = v.reshape(block_size, kv_heads, head_dim).transpose(1, 0, 2)
    else:
        raise ValueError(f"unknown layout {layout}")
    return np.array(K), np.array(V)


def encode_block(K, V, layout: int) -> np.ndarray:
    """(K, V) uint16 [kv_head][token][channel] -> bytes of one layer-block."""
    K = np.asarray(K, dtype=np.uint16)
    V = np.asarray(V, dtype=np.uint16)
    if layout == LAYOUT_ATTN:
        k = K.reshape(-1)
        v = V.transpose(0, 2, 1).reshape(-1)
    elif layout == LAYOUT_NHD:
        k = K.transpose(1, 0, 2).reshape(-1)
        v = V.transpose(1, 0, 2).reshape(-1)
    else:
        raise ValueError(f"unknown layout {layout}")
    return np.concatenate([k, v]).view(np.uint8).copy()


def convert_block(block_u8, src_layout: int, dst_layout: int, kv_heads: int, head_dim: int,
                  block_size: int) -> np.ndarray:
    """Re-lay one block from one layout into another (same logical K and V)."""
    if src_layout == dst_layout:
        return np.array(block_u8, dtype=np.uint8, copy=True)
    K, V = decode_block(block_u8, src_layout, kv_heads, head_dim, block_size)
    return encode_block(K, V, dst_layout)


def to_float64(bits, dtype: str) -> np.ndarray:
    """Exact value of 16-bit patterns as float64 (fp16 or bf16)."""
    bits = np.asarray(bits, dtype=np.uint16)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    raise ValueError(dtype)
