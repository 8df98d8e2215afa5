"""Rotary position embedding and paged-KV multi-query attention.

The serving engine keeps the KV cache in fixed-size blocks addressed through a
per-sequence block table (PagedAttention, the vLLM cache the paper's rollout
engines use, Sec. 2 and its citation of Kwon et al. 2023). In the verify step the
1+k new positions of sequence b sit at positions ctx_b .. ctx_b+k; their keys and
values are written into the cache first, and query j attends to keys 0..ctx_b+j
(causal inside the draft window). Grouped-query attention: query head h reads kv
head h // (Hq / Hkv). Scores are scaled by 1/sqrt(D), softmax in float64 here.

Cache layouts (blocks of 16 tokens): K [num_blocks, Hkv, 16, D], V [num_blocks,
Hkv, D, 16]. Position p of sequence b lives in block block_table[b, p // 16],
slot p % 16.

RoPE (not fixed by the paper; the common rotate-half form): pairs (i, i + D/2),
inverse frequency theta^(-2i/D), angle = position * inv_freq, all in float64.
"""
import numpy as np


def rope_angles(positions, D, theta):
    i = np.arange(D // 2, dtype=np.float64)
    inv_freq = np.power(np.float64(theta), -2.0 * i / D)
    return np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]


def apply_rope(x, positions, theta):
    """x [..., n, H, D] with positions [n] (x's leading token axis) -> rotated float64."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    ang = rope_angles(positions, D, theta)          # [n, D/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., : D // 2], x[..., D // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def gather_kv(k_cache, v_cache, block_table_row, n_pos, kv_head, block_size=16):
    """Keys/values of positions 0..n_pos-1 of one sequence and kv head -> [n_pos, D] each."""
    pos = np.arange(n_pos)
    blk = np.asarray(block_table_row)[pos // block_size]
    slot = pos % block_size
    K = k_cache[blk, kv_head, slot, :]
    V = v_cache[blk, kv_head, :, slot]
    return np.asarray(K, np.float64), np.asarray(V, np.float64)


def attend(q, K, V):
    """Plain softmax attention of query rows q [r, D] over keys/values [n, D]."""
    D = q.shape[-1]
    s = (q @ K.T) / np.sqrt(D)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ V


def paged_attention(q, k_cache, v_cache, block_tables, context_lens, k, block_size=16):
    """q [B*(1+k), Hq, D] float64 (token index b*(1+k)+j). k_cache/v_cache: widened
    float64 caches already holding the new positions. Returns [B*(1+k), Hq, D]."""
    q = np.asarray(q, np.float64)
    T, Hq, D = q.shape
    B = len(context_lens)
    Hkv = k_cache.shape[1]
    G = Hq // Hkv
    out = np.zeros_like(q)
    for b in range(B):
        ctx = int(context_lens[b])
        for h in range(Hkv):
            K, V = gather_kv(k_cache, v_cache, block_tables[b], ctx + k + 1, h, block_size)
            for j in range(k + 1):
                t = b * (k + 1) + j
                n = ctx + j + 1
                out[t, h * G:(h + 1) * G] = attend(q[t, h * G:(h + 1) * G], K[:n], V[:n])
    return out


def dense_causal_attention(q, keys, values, ctx, k):
    """Second, independent routine for the same quantity on contiguous K/V: builds the
    full score matrix of the 1+k queries with an explicit causal mask (no paging).
    q [1+k, G, D]; keys/values [ctx+k+1, D]."""
    q = np.asarray(q, np.float64)
    n = ctx + k + 1
    D = q.shape[-1]
    out = np.zeros_like(q)
    for g in range(q.shape[1]):
        s = (q[:, g, :] @ np.asarray(keys, np.float64).T) / np.sqrt(D)   # [1+k, n]
        mask = np.arange(n)[None, :] > (ctx + np.arange(k + 1))[:, None]
        s = np.where(mask, -np.inf, s)
        w = np.exp(s - s.max(axis=1, keepdims=True))
        w /= w.sum(axis=1, keepdims=True)
        out[:, g, :] = w @ np.asarray(values, np.float64)
    return out
