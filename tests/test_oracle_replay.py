"""Pins of the oracle's behavior-log-prob recompute with routing replay (oracle/replay.py):

* the scores are torch's log_softmax of the logits at the targets (a library routine);
* on the weights that generated them, the recompute of the emitted tokens with the recorded
  routes reproduces the verify step's recorded behavior log-probabilities and logits (the
  identity of the training contract, Eq. 1, and route alignment);
* replaying the routes the router itself chose changes nothing; replaying other routes
  changes the logits, unless every expert is the same (then any routes give the plain
  forward, because the replayed weights still sum to one);
* targets outside the vocabulary score NaN.
"""
import numpy as np
import torch

import workloads
from oracle import model, replay


def _tiny(seed=0, batch=3, k=3, layers=2):
    w = workloads.TINY_FP32.scaled(batch=batch, k=k, ctx_lo=20, ctx_hi=40, n_layers=layers)
    cfg = dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=w.n_layers, n_q_heads=w.n_q_heads,
               n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps,
               rope_theta=w.rope_theta, block_size=16)
    layout = workloads.make_kv_layout(w, seed)
    lw = [{k_: (None if v is None else v.numpy()) for k_, v in
           workloads.make_layer_weights(w, seed, l).items()} for l in range(w.n_layers)]
    head = {k_: v.numpy() for k_, v in workloads.make_head_weights(w, seed).items()}
    caches = [tuple(model.widen_cache(c.numpy(), w.dtype) for c in workloads.empty_kv_cache(w, layout))
              for _ in range(w.n_layers)]
    model.prefill(workloads.make_prompts(w, layout, seed), lambda l: lw[l], head, caches,
                  layout.block_tables, cfg)
    return w, cfg, layout, lw, head, caches


def _copy(caches):
    return [(a.copy(), b.copy()) for a, b in caches]


def _score(s, tokens, targets, rep=None, lw=None):
    w, cfg, layout, lw0, head, caches = s
    lw = lw0 if lw is None else lw
    return replay.score_tokens(tokens, targets, lambda l: lw[l], head, _copy(caches),
                               layout.block_tables, layout.context_lens, cfg, rep)


def test_scores_are_log_softmax_at_targets():
    s = _tiny(seed=1)
    w = s[0]
    toks = workloads.make_step_tokens(w, 2)
    g = np.random.default_rng(3)
    targets = g.integers(0, w.vocab, toks.shape)
    targets[0, 1] = -1
    targets[1, 2] = w.vocab
    r = _score(s, toks, targets)
    ref = torch.log_softmax(torch.from_numpy(r["logits"].astype(np.float64)), dim=-1)
    ok = (targets >= 0) & (targets < w.vocab)
    want = torch.gather(ref, -1, torch.from_numpy(np.where(ok, targets, 0))[..., None])[..., 0].numpy()
    np.testing.assert_allclose(r["logprobs"][ok], want[ok], rtol=1e-6, atol=1e-6)
    assert np.isnan(r["logprobs"][~ok]).all()


def test_replay_reproduces_recorded_behavior_logprobs():
    s = _tiny(seed=4)
    w, cfg, layout, lw, head, caches = s
    toks = workloads.make_step_tokens(w, 5)
    q = workloads.make_softmax_q(w.batch, w.k, w.vocab, 6).numpy()
    u = workloads.make_uniforms(w.batch, w.k, 7).numpy()
    v = model.verify_step(toks, lambda l: lw[l], head, _copy(caches), layout.block_tables,
                          layout.context_lens, cfg, q, u)
    # the emitted tokens as targets of their rows (-1 past each sequence's emitted token)
    r = _score(s, toks, v["tokens"], rep=v["routes"])
    np.testing.assert_array_equal(r["routes"], v["routes"])
    np.testing.assert_allclose(r["logits"], v["logits"], rtol=0, atol=0)
    emitted = v["tokens"] >= 0
    np.testing.assert_allclose(r["logprobs"][emitted], v["logprobs"][emitted], rtol=0, atol=0)
    assert np.isnan(r["logprobs"][~emitted]).all()


def test_replaying_own_routes_is_the_plain_forward():
    s = _tiny(seed=8)
    w = s[0]
    toks = workloads.make_step_tokens(w, 9)
    tg = np.roll(toks, -1, axis=1)
    plain = _score(s, toks, tg)
    again = _score(s, toks, tg, rep=plain["routes"])
    np.testing.assert_array_equal(plain["logits"], again["logits"])
    # other routes: different logits
    other = (plain["routes"] + 1) % w.n_experts
    moved = _score(s, toks, tg, rep=other)
    assert np.abs(moved["logits"] - plain["logits"]).max() > 1e-3
    np.testing.assert_array_equal(moved["routes"], other)


def test_identical_experts_make_routes_irrelevant():
    s = _tiny(seed=10, layers=1)
    w = s[0]
    lw = [dict(s[3][0])]
    lw[0]["w_gate_up"] = np.repeat(lw[0]["w_gate_up"][:1], w.n_experts, axis=0)
    lw[0]["w_down"] = np.repeat(lw[0]["w_down"][:1], w.n_experts, axis=0)
    toks = workloads.make_step_tokens(w, 11)
    tg = np.roll(toks, -1, axis=1)
    plain = _score(s, toks, tg, lw=lw)
    rng = np.random.default_rng(12)
    T = w.batch * (w.k + 1)
    rep = np.stack([np.stack([rng.permutation(w.n_experts)[:w.top_k] for _ in range(T)])])
    moved = _score(s, toks, tg, rep=rep, lw=lw)
    np.testing.assert_allclose(moved["logits"], plain["logits"], rtol=1e-6, atol=1e-7)
