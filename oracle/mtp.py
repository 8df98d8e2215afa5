"""MTP draft head: the drafts and draft distributions that the verify step checks
(test infrastructure, like the rest of this package).

The rollout engines speculate with the checkpoint's multi-token-prediction (MTP) head
(Sec. 4.1 control table: number of speculative tokens, zero disables; Sec. 5.4: enabling
the MTP head shortens the generation stage about five-fold). The paper does not print the
head. It is read here as the MTP module of DeepSeek-V3 (Sec. 2.2 of that report), run by
the serving engine as a one-layer draft model that shares the target's embedding and LM
head:
    y  = [RMSNorm(Emb(t); g_e) ; RMSNorm(h; g_h)]        each half rounded to the act dtype
    x  = y W_eh^T                                        f32, W_eh [d, 2d]
    x  = DecoderLayer(x)                                 the target's layer structure: pre-norm
                                                         attention over the head's own paged
                                                         KV cache, then the routed MoE
    logits = RMSNorm(x; g_f) W_lm^T,  q = softmax(logits)
Row (h_p, token at p+1) sits at cache position p and predicts the token at p+2.

After a verify step of sequence b (context c_b; tokens x_0..x_k at positions c_b..c_b+k;
n_b accepted drafts; the emitted token y_b, the bonus or replacement, at position
c_b + n_b + 1) one draft step runs (after a prefill the catch-up window is the prompt's
instead of k+1 rows, with n_b = its length - 1 and y_b the token sampled from its logits):
  * catch-up: k+1 rows per sequence at positions c_b + j, j = 0..k, with h = the target's
    final residual stream (before its final norm) at row j and token x_{j+1} for j < n_b,
    y_b for j >= n_b. Row n_b predicts draft 1. Rows past n_b carry rejected drafts' hidden
    states; their outputs are not used and their cache entries are rewritten later.
  * drafting: draft i+1 (i = 1..k-1) from one row per sequence at position c_b + n_b + i,
    with h = the head's previous output (pre-norm) and token = draft i.
Each draft is drawn from q with the verify step's integer inverse CDF (sampler's
fixed_point_draw with r = p) and one uniform; the greedy variant takes the first argmax of
the logits and returns no q (the verify step then reads q as one-hot at the draft).
"""
import numpy as np

from . import model, moe, sampler


def head_input(tokens, h, mtp, head, cfg):
    """x = [RMSNorm(Emb(t)); RMSNorm(h)] W_eh^T for rows (tokens [T], h [T, d])."""
    act = cfg["dtype"]
    e = model.embed(np.asarray(tokens).reshape(-1), head, cfg)
    ye = moe.round_act(model.rmsnorm(e, mtp["enorm"], cfg["rms_eps"]), act)
    yh = moe.round_act(model.rmsnorm(h, mtp["hnorm"], cfg["rms_eps"]), act)
    y = np.concatenate([ye, yh], axis=1)
    return (y @ moe.widen(mtp["eh_proj"], act).T).astype(np.float32)


def head_layer(x, mtp, kcache, vcache, block_tables, context_lens, k, cfg):
    """The head's decoder layer on rows b*(k+1)+j at positions context_lens[b] + j.
    Returns the rows and their route-set margins (the router's gap at the top-K boundary)."""
    x = model.attention_block(x, mtp["layer"], kcache, vcache, block_tables, context_lens, k, cfg)
    x, r = model.moe_block(x, mtp["layer"], cfg)
    return x, r["margin"]


def head_logits(x, mtp, head, cfg):
    return model.lm_logits(x, {"final_norm": mtp["final_norm"], "lm_head": head["lm_head"]}, cfg)


def mtp_draft(hidden, tokens, n_accepted, next_tokens, mtp, head, kcache, vcache, block_tables,
              context_lens, cfg, uniforms=None, forced=None, k=None):
    """hidden [B W, d] f32 (the verify step's final residual stream: W = 1+k; or a prefill's,
    W = its window, with n_accepted = lens - 1); tokens [B, W]; k drafts (default W - 1);
    n_accepted [B]; next_tokens [B]; kcache/vcache: the head's cache as float64 arrays
    (updated in place); uniforms [B, k] (None: greedy drafts). forced [B, k]: feed these
    tokens to the following rows instead of the drawn drafts (teacher forcing, to compare
    every step on its own).

    Returns dict: drafts [B, k] int32, q [B, k, V] float64 (None when greedy), logits
    [B, k, V] f32, h [B, k, d] f32 (the head's output row behind each draft), margin [B, k]
    (the draw's margin relative to its total mass; greedy: the gap between the two largest
    logits), route_margin [B, k] (the route-set margin of the head row behind each draft: a
    near-tie there lets rounding pick another expert set)."""
    tokens = np.asarray(tokens)
    B, kp1 = tokens.shape                      # kp1: the catch-up window W
    k = kp1 - 1 if k is None else k
    n = np.asarray(n_accepted).astype(np.int64)
    nxt = np.asarray(next_tokens).astype(np.int64)
    ctx = np.asarray(context_lens).astype(np.int64)
    # catch-up rows
    row_tok = np.array([[tokens[b, j + 1] if j < n[b] else nxt[b] for j in range(kp1)]
                        for b in range(B)]).reshape(-1)
    x = head_input(row_tok, np.asarray(hidden, np.float32), mtp, head, cfg)
    x, rm = head_layer(x, mtp, kcache, vcache, block_tables, ctx, kp1 - 1, cfg)
    h = x[np.arange(B) * kp1 + n]
    drafts = np.zeros((B, k), np.int32)
    logits_all, qs, hs, margins = [], [], [], np.zeros((B, k))
    route_margin = np.zeros((B, k))
    route_margin[:, 0] = rm[np.arange(B) * kp1 + n]
    for i in range(k):
        lg = head_logits(h, mtp, head, cfg)                   # [B, V] f32
        logits_all.append(lg)
        hs.append(h)
        if uniforms is None:
            d = np.argmax(lg, axis=1)
            top2 = np.sort(lg.astype(np.float64), axis=1)[:, -2:]
            margins[:, i] = top2[:, 1] - top2[:, 0]
        else:
            m, S = sampler.row_stats(lg)
            p = np.exp(lg.astype(np.float64) - m[:, None]) / S[:, None]
            d, _, mg = sampler.fixed_point_draw(p, np.asarray(uniforms, np.float32)[:, i])
            qs.append(p)
            margins[:, i] = mg
        drafts[:, i] = d
        if i + 1 == k:
            break
        tok = np.asarray(forced)[:, i] if forced is not None else d
        x = head_input(tok, h, mtp, head, cfg)
        x, rm = head_layer(x, mtp, kcache, vcache, block_tables, ctx + n + i + 1, 0, cfg)
        route_margin[:, i + 1] = rm
        h = x
    return {"drafts": drafts, "q": None if uniforms is None else np.stack(qs, axis=1),
            "logits": np.stack(logits_all, axis=1), "h": np.stack(hs, axis=1), "margin": margins,
            "route_margin": route_margin}
