"""Float64 paged decode attention.

The paper runs vLLM's attention and states no formula; the hot path needs the
textbook scaled dot-product attention of one new query token per sequence over
that sequence's cached tokens, read through its block table:

    for sequence b and query head h (kv head g = h // (Hq / Hkv), the grouped
    query convention):
        s_t = (q . k_t) * scale            for t < len_b, scale = 1/sqrt(D)
        w_t = exp(s_t - max_t s_t)
        o   = sum_t w_t v_t / sum_t w_t
    len_b == 0 gives o = 0.

Token t of sequence b is row t % block_size of the block
block_table[b][t // block_size]. Keys, values and queries are the exact
float64 values of their 16-bit inputs.
"""
import numpy as np

from .layout import LAYOUT_ATTN, decode_block, to_float64


def _gather_sequence(read_block, row_ids, n_tokens, kv_heads, head_dim, block_size):
    """K, V of one sequence as uint16 [kv_head][n_tokens][channel]."""
    nblk = -(-n_tokens // block_size)
    Ks, Vs = [], []
    for j in range(nblk):
        K, V = decode_block(read_block(int(row_ids[j])), LAYOUT_ATTN, kv_heads, head_dim,
                            block_size)
        Ks.append(K)
        Vs.append(V)
    K = np.concatenate(Ks, axis=1)[:, :n_tokens]
    V = np.concatenate(Vs, axis=1)[:, :n_tokens]
    return K, V


def contiguous_decode_attention(q, K, V, scale=None):
    """One sequence, contiguous cache. q float64 [Hq][D]; K, V float64
    [Hkv][n][D]. Returns float64 [Hq][D]."""
    Hq, D = q.shape
    Hkv, n, _ = K.shape
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    out = np.zeros((Hq, D), dtype=np.float64)
    if n == 0:
        return out
    G = Hq // Hkv
    for h in range(Hq):
        g = h // G
        s = (K[g] @ q[h]) * scale
        w = np.exp(s - s.max())
        out[h] = (w @ V[g]) / w.sum()
    return out


def paged_decode_attention(q16, block_table, seq_lens, read_block, kv_heads, head_dim,
                           block_size, dtype, scale=None):
    """q16: uint16 [B][Hq][D] patterns; block_table int [B][maxblk] of local
    block ids; seq_lens int [B]; read_block(id) -> bytes of that local block
    (ATTN layout). Returns float64 [B][Hq][D]."""
    q = to_float64(q16, dtype)
    B, Hq, D = q.shape
    out = np.zeros((B, Hq, D), dtype=np.float64)
    for b in range(B):
        n = int(seq_lens[b])
        if n == 0:
            continue
        K, V = _gather_sequence(read_block, block_table[b], n, kv_heads, head_dim, block_size)
        out[b] = contiguous_decode_attention(q[b], to_float64(K, dtype), to_float64(V, dtype),
                                             scale)
    return out
