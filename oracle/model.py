"""The target model's forward pass over the 1+k verify positions, and the full step.

The verify step of MTP speculative decoding (Sec. 4.1 control table: number of
speculative tokens, zero disables; Sec. 5.4: the MTP head's drafts are verified
by the target): each sequence b feeds its last emitted token and k drafts at
positions ctx_b .. ctx_b+k through a pre-norm MoE decoder:
    x = Embed[token]                                   (float32 residual stream)
    per layer:  x += Attn(RMSNorm(x))  ;  x += MoE(RMSNorm(x))
    logits = RMSNorm(x) W_lm^T                         (float32)
then applies the speculative accept rule (sampler.spec_accept) and records the
expert routes of every layer (routing replay, Sec. 4.1).

Rounding points (the method's bf16 reading, shared with the GPU path): RMSNorm
outputs, q/k/v after RoPE, the attention output and the SwiGLU product are stored
in the activation dtype (bf16; float32 for the f32 model); projections produce
float32; the residual stream is float32. RMSNorm: x / sqrt(mean(x^2) + eps) * g.
"""
import numpy as np

from . import attention, codecs, moe, sampler


def rmsnorm(x, g, eps):
    x = np.asarray(x, dtype=np.float64)
    r = 1.0 / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(g, dtype=np.float64)


def widen_cache(c, dtype):
    c = np.asarray(c)
    if dtype == "bf16":
        return codecs.bf16_bits_to_f32(c).astype(np.float64)
    return c.astype(np.float32).astype(np.float64)


def attention_block(x, lw, kcache, vcache, block_tables, context_lens, k, cfg):
    """x [T, d] float32 (T = B(1+k)); kcache/vcache float64 arrays, updated in place."""
    act = cfg["dtype"]
    Hq, Hkv, D = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    T = x.shape[0]
    B = len(context_lens)
    y = moe.round_act(rmsnorm(x, lw["attn_norm"], cfg["rms_eps"]), act)
    Wqkv = moe.widen(lw["w_qkv"], act)
    qkv = (y @ Wqkv.T).astype(np.float32).astype(np.float64)
    q = qkv[:, : Hq * D].reshape(T, Hq, D)
    kk = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D)
    vv = qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D)
    pos = np.array([int(context_lens[b]) + j for b in range(B) for j in range(k + 1)])
    q = moe.round_act(attention.apply_rope(q, pos, cfg["rope_theta"]), act)
    kk = moe.round_act(attention.apply_rope(kk, pos, cfg["rope_theta"]), act)
    vv = moe.round_act(vv, act)
    bs = cfg.get("block_size", 16)
    for t in range(T):
        b, p = t // (k + 1), pos[t]
        blk = block_tables[b][p // bs]
        kcache[blk, :, p % bs, :] = kk[t]
        vcache[blk, :, :, p % bs] = vv[t]
    o = attention.paged_attention(q, kcache, vcache, block_tables, context_lens, k, bs)
    o = moe.round_act(o.reshape(T, Hq * D), act)
    Wo = moe.widen(lw["w_o"], act)
    return (x.astype(np.float64) + (o @ Wo.T).astype(np.float32)).astype(np.float32)


def moe_block(x, lw, cfg, replay_ids=None):
    act = cfg["dtype"]
    y = moe.round_act(rmsnorm(x, lw["moe_norm"], cfg["rms_eps"]), act)
    r = moe.moe_layer(y, moe.widen(lw["w_router"], act), lw["w_gate_up"], lw["w_down"],
                      cfg["top_k"], act, cfg["expert_dtype"], lw.get("s_gate_up"),
                      lw.get("s_down"), lw.get("router_bias"), replay_ids)
    return (x.astype(np.float64) + r["out"].astype(np.float64)).astype(np.float32), r


def decoder_forward(x, get_layer, caches, block_tables, context_lens, k, cfg):
    """Runs every layer. get_layer(l) -> layer weight dict; caches[l] = (k, v) float64.
    Returns the final residual stream and per-layer routing results."""
    routes = []
    for l in range(cfg["n_layers"]):
        lw = get_layer(l)
        kc, vc = caches[l]
        x = attention_block(x, lw, kc, vc, block_tables, context_lens, k, cfg)
        x, r = moe_block(x, lw, cfg)
        routes.append(r)
    return x, routes


def embed(tokens, head, cfg):
    E = moe.widen(head["embed"], cfg["dtype"])
    return E[np.asarray(tokens).reshape(-1)].astype(np.float32)


def lm_logits(x, head, cfg):
    y = moe.round_act(rmsnorm(x, head["final_norm"], cfg["rms_eps"]), cfg["dtype"])
    return (y @ moe.widen(head["lm_head"], cfg["dtype"]).T).astype(np.float32)


def verify_step(tokens, get_layer, head, caches, block_tables, context_lens, cfg,
                draft_probs, uniforms):
    """tokens [B, 1+k] (last emitted token then k drafts). Returns logits [B, 1+k, V],
    the sampler outputs and the route records [L, T, K]."""
    tokens = np.asarray(tokens)
    B, kp1 = tokens.shape
    k = kp1 - 1
    x = embed(tokens, head, cfg)
    x, routes = decoder_forward(x, get_layer, caches, block_tables, context_lens, k, cfg)
    logits = lm_logits(x, head, cfg).reshape(B, kp1, -1)
    s = sampler.spec_accept(logits, tokens[:, 1:], uniforms, draft_probs)
    s["logits"] = logits
    s["routes"] = np.stack([r["ids"] for r in routes]) if routes else None
    s["route_margin"] = np.stack([r["margin"] for r in routes]) if routes else None
    s["route_order_margin"] = np.stack([r["order_margin"] for r in routes]) if routes else None
    return s


def prefill(prompts, get_layer, head, caches, block_tables, cfg):
    """Fills the caches with each prompt's keys/values (positions 0..len-1), one
    sequence at a time: a causal forward with an empty context and a window equal
    to the prompt."""
    for b, prompt in enumerate(prompts):
        n = len(prompt)
        x = embed(np.asarray(prompt)[None, :], head, cfg)
        decoder_forward(x, get_layer, caches, [block_tables[b]], [0], n - 1, cfg)
