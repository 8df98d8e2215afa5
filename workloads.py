"""Seeded synthetic workloads for the speculative-decoding verify step.

This module only draws random inputs: weights, KV-cache contents, block tables,
context lengths, draft tokens, draft distributions and acceptance uniforms. It
holds none of the verify step's arithmetic, and both the CPU oracle and the GPU
library consume what it produces (the oracle through host copies).

The shapes follow the method's statement of the problem: a mixture-of-experts
policy whose serving engine verifies ``k`` speculative tokens per sequence
(Sec. 4.1, table of scaling controls: number of speculative tokens, zero
disables) over a paged KV cache, at temperature 1 with no truncation (Sec. 5.3,
Sec. 5.4). The paper's own datasets and checkpoints are not used: every tensor
below is random, seeded per (workload, tensor, layer).

Layouts (row-major, all shared with the C-ABI):
  embed, lm_head      [V, d]             act dtype
  attn_norm, moe_norm [d] fp32,  final_norm [d] fp32
  w_qkv               [(Hq + 2 Hkv) D, d] (rows: q heads, then k heads, then v heads)
  w_o                 [d, Hq D]
  w_router            [E, d]
  w_gate_up           [E, 2F, d]  rows 0..F-1 gate, F..2F-1 up
  w_down              [E, d, F]
  s_gate_up, s_down   [E, 2F], [E, d] fp32 per-output-channel scales (fp8 only)
  k_cache             [num_blocks, Hkv, 16, D]   (16 tokens of one head contiguous)
  v_cache             [num_blocks, Hkv, D, 16]   (token index fastest)
"""
from __future__ import annotations

import dataclasses
import hashlib
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_experts: int
    top_k: int
    d_ff: int
    vocab: int
    batch: int
    k: int
    ctx_lo: int
    ctx_hi: int
    dtype: str = "bf16"          # activations, attention weights, KV cache: "f32" | "bf16"
    expert_dtype: str = "bf16"   # "f32" | "bf16" | "fp8"
    full_model: bool = False     # embedding + LM head + sampler around the layers
    zipf: Optional[float] = None  # router bias exponent (popularity ~ rank^-zipf)
    draft: str = "uniform"       # "uniform" | "perturbed" (q = softmax(target + N(0, sigma^2)))
    draft_sigma: float = 0.5
    weight_std: float = 0.02
    block_size: int = 16
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6

    @property
    def tokens_per_step(self) -> int:
        return self.batch * (1 + self.k)

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# Tiny fp32 decoder: every part of the step, small enough for the oracle in seconds.
TINY_FP32 = Workload(
    name="tiny_fp32", n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
    n_experts=8, top_k=2, d_ff=512, vocab=2048, batch=4, k=3, ctx_lo=64, ctx_hi=128,
    dtype="f32", expert_dtype="f32", full_model=True, draft="uniform")

# One verify layer at a 35B-A3B-like MoE shape.
LAYER_BF16 = Workload(
    name="layer_bf16", n_layers=1, d_model=2048, n_q_heads=32, n_kv_heads=4, head_dim=128,
    n_experts=128, top_k=8, d_ff=768, vocab=151936, batch=64, k=4, ctx_lo=4096, ctx_hi=4096)

# The same layer with long, variable agent contexts (attention-bandwidth bound).
LONG_CTX_BF16 = LAYER_BF16.scaled(name="long_ctx_bf16", batch=16, ctx_lo=32768, ctx_hi=65536)

# Full-depth verify step: 48 layers + LM head + sampler.
FULL_DEPTH_BF16 = LAYER_BF16.scaled(
    name="full_depth_bf16", n_layers=48, batch=128, k=4, ctx_lo=8192, ctx_hi=8192,
    full_model=True, draft="perturbed", draft_sigma=0.5)

# fp8 experts with Zipf(1.2)-skewed routing.
FP8_ZIPF = LAYER_BF16.scaled(name="fp8_zipf", batch=256, k=8, ctx_lo=2048, ctx_hi=2048,
                             expert_dtype="fp8", zipf=1.2)

WORKLOADS = {w.name: w for w in (TINY_FP32, LAYER_BF16, LONG_CTX_BF16, FULL_DEPTH_BF16, FP8_ZIPF)}


# ----------------------------------------------------------------------------------------
# seeding
# ----------------------------------------------------------------------------------------

def _seed(*parts) -> int:
    h = hashlib.sha256("/".join(str(p) for p in parts).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def rng(seed: int, *parts, device="cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(seed, *parts))
    return g


def torch_dtype(name: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}[name]


def _normal(shape, std, g, device, dtype):
    # drawn in fp32 and stored in the workload's dtype (bf16 storage rounds once)
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(dtype)


# ----------------------------------------------------------------------------------------
# paged-KV layout
# ----------------------------------------------------------------------------------------

@dataclass
class KVLayout:
    context_lens: np.ndarray      # [B] int32: tokens already cached
    block_tables: np.ndarray      # [B, max_blocks] int32 (-1 = unused)
    num_blocks: int
    block_size: int


def make_kv_layout(w: Workload, seed: int, spare_blocks: int = 0, extra_tokens: int = 0) -> KVLayout:
    """Context lengths uniform in [ctx_lo, ctx_hi] and a seeded permutation of physical
    blocks; every sequence owns enough blocks for its context plus the 1+k new tokens (plus
    extra_tokens: the draft head writes up to k - 1 positions past them)."""
    g = np.random.Generator(np.random.Philox(_seed(seed, w.name, "ctx")))
    B, bs = w.batch, w.block_size
    ctx = g.integers(w.ctx_lo, w.ctx_hi + 1, size=B).astype(np.int32)
    need = (ctx.astype(np.int64) + w.k + 1 + extra_tokens + bs - 1) // bs
    max_blocks = int(need.max())
    total = int(need.sum()) + spare_blocks
    perm = g.permutation(total).astype(np.int32)
    bt = np.full((B, max_blocks), -1, dtype=np.int32)
    pos = 0
    for b in range(B):
        n = int(need[b])
        bt[b, :n] = perm[pos:pos + n]
        pos += n
    return KVLayout(context_lens=ctx, block_tables=bt, num_blocks=total, block_size=bs)


def make_kv_cache(w: Workload, layout: KVLayout, seed: int, layer: int, device="cpu"):
    """Random N(0,1) K and V contents for one layer (every slot, used or not)."""
    nb, H, D, bs = layout.num_blocks, w.n_kv_heads, w.head_dim, layout.block_size
    dt = torch_dtype(w.dtype)
    kc = _normal((nb, H, bs, D), 1.0, rng(seed, w.name, "kcache", layer, device=device), device, dt)
    vc = _normal((nb, H, D, bs), 1.0, rng(seed, w.name, "vcache", layer, device=device), device, dt)
    return kc, vc


def empty_kv_cache(w: Workload, layout: KVLayout, device="cpu"):
    nb, H, D, bs = layout.num_blocks, w.n_kv_heads, w.head_dim, layout.block_size
    dt = torch_dtype(w.dtype)
    return (torch.zeros(nb, H, bs, D, dtype=dt, device=device),
            torch.zeros(nb, H, D, bs, dtype=dt, device=device))


# ----------------------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------------------

def make_fp8_weights(shape, std, g, device):
    """A synthetic fp8 checkpoint: N(0, std^2) weights quantised per output channel (every
    row of the last axis): s = amax / 448, codes = e4m3fn(w / s) by torch's float8_e4m3fn
    conversion (round to nearest even; |w / s| <= 448 up to one rounding, which rounds to
    448). Returns (uint8 codes, f32 scales of shape[:-1])."""
    wt = torch.randn(*shape, generator=g, device=device, dtype=torch.float32).mul_(std)
    s = wt.abs().amax(dim=-1) / 448.0
    s = torch.where(s > 0, s, torch.ones_like(s))
    codes = (wt / s.unsqueeze(-1)).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, s


def make_layer_weights(w: Workload, seed: int, layer: int, device="cpu") -> dict:
    d, Hq, Hkv, D, E, F = w.d_model, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_experts, w.d_ff
    dt = torch_dtype(w.dtype)
    std = w.weight_std
    out = {
        "attn_norm": torch.ones(d, dtype=torch.float32, device=device),
        "moe_norm": torch.ones(d, dtype=torch.float32, device=device),
        "w_qkv": _normal(((Hq + 2 * Hkv) * D, d), std, rng(seed, w.name, "wqkv", layer, device=device), device, dt),
        "w_o": _normal((d, Hq * D), std, rng(seed, w.name, "wo", layer, device=device), device, dt),
        "w_router": _normal((E, d), std, rng(seed, w.name, "wrouter", layer, device=device), device, dt),
    }
    if w.expert_dtype == "fp8":
        out["w_gate_up"], out["s_gate_up"] = make_fp8_weights(
            (E, 2 * F, d), std, rng(seed, w.name, "wgu", layer, device=device), device)
        out["w_down"], out["s_down"] = make_fp8_weights(
            (E, d, F), std, rng(seed, w.name, "wd", layer, device=device), device)
    else:
        edt = torch_dtype(w.expert_dtype)
        out["w_gate_up"] = _normal((E, 2 * F, d), std, rng(seed, w.name, "wgu", layer, device=device), device, edt)
        out["w_down"] = _normal((E, d, F), std, rng(seed, w.name, "wd", layer, device=device), device, edt)
        out["s_gate_up"] = None
        out["s_down"] = None
    if w.zipf is not None:
        # popularity ~ rank^-zipf: bias_e = -zipf * log(rank(e)), ranks a seeded permutation
        g = np.random.Generator(np.random.Philox(_seed(seed, w.name, "zipf", layer)))
        ranks = g.permutation(E) + 1
        out["router_bias"] = torch.tensor(-w.zipf * np.log(ranks), dtype=torch.float32, device=device)
    else:
        out["router_bias"] = None
    return out


def make_head_weights(w: Workload, seed: int, device="cpu") -> dict:
    dt = torch_dtype(w.dtype)
    return {
        "embed": _normal((w.vocab, w.d_model), w.weight_std, rng(seed, w.name, "embed", device=device), device, dt),
        "lm_head": _normal((w.vocab, w.d_model), w.weight_std, rng(seed, w.name, "lmhead", device=device), device, dt),
        "final_norm": torch.ones(w.d_model, dtype=torch.float32, device=device),
    }


def make_mtp_weights(w: Workload, seed: int, device="cpu") -> dict:
    """MTP draft head: norms of the embedding and hidden halves, eh_proj [d, 2d] (input
    [RMSNorm(e); RMSNorm(h)]), one decoder layer of the target's shape (seeded as layer
    n_layers) and the head's output norm. Norm gains are 1 + N(0, 0.1^2) so that the halves
    and the output norm are told apart."""
    d = w.d_model
    g = rng(seed, w.name, "mtp_norms", device=device)
    gains = 1.0 + 0.1 * torch.randn(3, d, generator=g, device=device, dtype=torch.float32)
    return {
        "enorm": gains[0].contiguous(), "hnorm": gains[1].contiguous(),
        "final_norm": gains[2].contiguous(),
        "eh_proj": _normal((d, 2 * d), w.weight_std, rng(seed, w.name, "mtp_eh", device=device),
                           device, torch_dtype(w.dtype)),
        "layer": make_layer_weights(w, seed, w.n_layers, device=device),
    }


# ----------------------------------------------------------------------------------------
# step inputs
# ----------------------------------------------------------------------------------------

def make_hidden(w: Workload, seed: int, T: Optional[int] = None, device="cpu") -> torch.Tensor:
    """Residual-stream input of a layer-only workload: N(0,1) fp32 [T, d]."""
    T = w.tokens_per_step if T is None else T
    return torch.randn(T, w.d_model, generator=rng(seed, w.name, "hidden", device=device),
                       device=device, dtype=torch.float32)


def make_prompts(w: Workload, layout: KVLayout, seed: int) -> list:
    """Uniform prompt tokens that fill each sequence's context (for a prefill)."""
    g = np.random.Generator(np.random.Philox(_seed(seed, w.name, "prompt")))
    return [g.integers(0, w.vocab, size=int(c)).astype(np.int32) for c in layout.context_lens]


def make_step_tokens(w: Workload, seed: int) -> np.ndarray:
    """[B, 1+k] int32: the last emitted token, then k drafts, uniform over the vocabulary."""
    g = np.random.Generator(np.random.Philox(_seed(seed, w.name, "tokens")))
    return g.integers(0, w.vocab, size=(w.batch, 1 + w.k)).astype(np.int32)


def make_uniforms(B: int, k: int, seed: int, tag="u", device="cpu") -> torch.Tensor:
    """[B, k+1] fp32 uniforms in [0, 1): k acceptance tests, then one for the final token."""
    return torch.rand(B, k + 1, generator=rng(seed, tag, B, k, device=device), device=device,
                      dtype=torch.float32)


def make_softmax_q(B: int, k: int, V: int, seed: int, tag="q", device="cpu") -> torch.Tensor:
    """Draft distributions: softmax of seeded N(0,1) logits, [B, k, V] fp32 (library softmax)."""
    z = torch.randn(B, k, V, generator=rng(seed, tag, B, k, V, device=device), device=device)
    return torch.softmax(z, dim=-1)


def make_logits(B: int, rows: int, V: int, seed: int, std: float = 1.0, tag="logits", device="cpu"):
    z = torch.randn(B, rows, V, generator=rng(seed, tag, B, rows, V, device=device), device=device)
    if std != 1.0:
        z.mul_(std)
    return z
