"""Behavior-log-prob recompute with routing replay: the actor's pass over the tokens the
serving engine emitted (test infrastructure, like the rest of this package).

Rollout routing replay records the expert choices made during generation and reuses them
in the actor; token alignment, route alignment and numerical-consistency diagnostics
accompany it (Sec. 4.1). The trace carries the token IDs the engine returned and their
behavior log-probabilities (Sec. 4.2, Eq. 1). The recompute scores given tokens with the
target model:
    x = Embed[tokens], the decoder layers with each MoE layer's experts taken from the
    replayed routes (their weights still come from the router: a softmax over the router
    logits of the given experts), logits = RMSNorm(x) W_lm^T, and for row j of sequence b
    with target token y = targets[b, j]:  lp = (l_y - m) - ln S  (m, S as in the sampler);
    a target outside [0, V) scores NaN.
Without replay the router chooses (a plain recompute). On the weights that generated the
tokens, the recompute with the recorded routes reproduces the recorded behavior
log-probabilities.
"""
import numpy as np

from . import model, sampler


def score_tokens(tokens, targets, get_layer, head, caches, block_tables, context_lens, cfg,
                 replay=None):
    """tokens, targets [B, 1+k] (rows at positions context_lens[b] + j); caches[l] = (k, v)
    float64 (updated in place with the window's keys and values); replay [L, B(1+k), K] or
    None. Returns dict: logprobs [B, 1+k] f32, logits [B, 1+k, V] f32, routes [L, T, K]."""
    tokens = np.asarray(tokens)
    B, kp1 = tokens.shape
    x = model.embed(tokens, head, cfg)
    routes = []
    for l in range(cfg["n_layers"]):
        lw = get_layer(l)
        kc, vc = caches[l]
        x = model.attention_block(x, lw, kc, vc, block_tables, context_lens, kp1 - 1, cfg)
        x, r = model.moe_block(x, lw, cfg, None if replay is None else np.asarray(replay)[l])
        routes.append(r["ids"])
    logits = model.lm_logits(x, head, cfg).reshape(B, kp1, -1)
    V = logits.shape[-1]
    m, S = sampler.row_stats(logits)
    y = np.asarray(targets).astype(np.int64)
    ok = (y >= 0) & (y < V)
    ly = np.take_along_axis(logits.astype(np.float64), np.where(ok, y, 0)[..., None], axis=-1)[..., 0]
    lp = np.where(ok, (ly - m) - np.log(S), np.nan).astype(np.float32)
    return {"logprobs": lp, "logits": logits, "routes": np.stack(routes)}
