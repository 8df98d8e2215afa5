"""Shared test plumbing: numpy views of generated tensors for the oracle, device copies for
the library, and the oracle's config dict for a workload. No arithmetic of the method."""
import numpy as np
import torch


def host(t):
    """numpy array of a tensor's stored values: bf16 as uint16 bit patterns, fp8 as uint8."""
    if t is None:
        return None
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dev(t):
    return None if t is None else t.cuda().contiguous()


def oracle_cfg(w):
    return dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=w.n_layers,
                n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta, block_size=16)


def layer_host(lw):
    return {k: host(v) for k, v in lw.items()}


def model_from(w, layers, head, molt):
    return molt.Model([{k: dev(v) for k, v in lw.items()} for lw in layers],
                      None if head is None else {k: dev(v) for k, v in head.items()},
                      n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                      top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta)


def max_abs(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64)))) if np.size(a) else 0.0


def tiled_layout(mat_bytes):
    """The library's tiled expert-weight layout, from its definition in include/molt.h
    (molt_pack_weights), written with numpy index arithmetic: mat_bytes [rows, row_bytes]
    uint8 -> flat uint8 of the size with rows padded (zeros) to a multiple of 32."""
    rows, rb = mat_bytes.shape
    pad = (-rows) % 32
    if pad:   # zero rows up to a multiple of 32
        mat_bytes = np.concatenate([mat_bytes, np.zeros((pad, rb), np.uint8)])
        rows += pad
    r = np.arange(rows)[:, None]
    j = np.arange(rb)[None, :]
    off = ((r // 32) * (rb // 128) + j // 128) * 4096 + ((j % 64) // 16) * 1024 \
        + (((j % 128) // 64) * 32 + r % 32) * 16 + j % 16
    out = np.empty(rows * rb, np.uint8)
    out[off.ravel()] = mat_bytes.ravel()
    return out
