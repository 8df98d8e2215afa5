"""Pins of the oracle's MTP draft head (oracle/mtp.py):

* wiring of the two input halves: with eh_proj = [0 | I] and a layer whose outputs are zero
  (w_o = 0, w_down = 0) the head's logits are the target LM head's logits of the verify
  step's hidden row n_b (the row that produced the emitted token); with eh_proj = [I | 0]
  they are the LM head's logits of the emitted token's embedding, and each later draft's
  logits those of the previous draft's embedding;
* catch-up and drafting agree: draft 2 of a step equals draft 1 of a step whose catch-up
  already contains draft 1 (one more accepted token, the head's own output as its hidden
  row), which fixes the drafting rows' positions, cache use and hidden-state recurrence;
* rejected drafts and the hidden rows behind them do not influence any output;
* the greedy variant takes the argmax of the sampled variant's q.
"""
import numpy as np
import pytest

import workloads
from oracle import model, mtp as omtp
from helpers import host, layer_host, oracle_cfg


def _setup(seed=0, B=4, k=3, n=None):
    w = workloads.TINY_FP32.scaled(n_layers=1, batch=B, k=k)
    layout = workloads.make_kv_layout(w, seed, extra_tokens=k)
    head = {kk: host(v) for kk, v in workloads.make_head_weights(w, seed).items()}
    mt = workloads.make_mtp_weights(w, seed)
    mtp = {kk: host(v) for kk, v in mt.items() if kk != "layer"}
    mtp["layer"] = layer_host(mt["layer"])
    kc, vc = workloads.make_kv_cache(w, layout, seed, w.n_layers)
    cache = (model.widen_cache(host(kc), w.dtype), model.widen_cache(host(vc), w.dtype))
    hidden = host(workloads.make_hidden(w, seed))
    tokens = workloads.make_step_tokens(w, seed)
    g = np.random.default_rng(seed)
    n = g.integers(0, k + 1, B) if n is None else np.asarray(n)
    nxt = g.integers(0, w.vocab, B)
    u = host(workloads.make_uniforms(B, k - 1, seed, tag="mtp_u"))
    cfg = oracle_cfg(w)
    return dict(w=w, layout=layout, head=head, mtp=mtp, cache=cache, hidden=hidden,
                tokens=tokens, n=n, nxt=nxt, u=u, cfg=cfg)


def _run(s, uniforms="default", **over):
    a = dict(s, **over)
    kc, vc = (c.copy() for c in a["cache"])
    u = a["u"] if isinstance(uniforms, str) else uniforms
    return omtp.mtp_draft(a["hidden"], a["tokens"], a["n"], a["nxt"], a["mtp"], a["head"], kc, vc,
                          a["layout"].block_tables, a["layout"].context_lens, a["cfg"], uniforms=u,
                          forced=a.get("forced"))


def _silent_layer(mtp):
    lay = dict(mtp["layer"])
    lay["w_o"] = np.zeros_like(lay["w_o"])
    lay["w_down"] = np.zeros_like(lay["w_down"])
    return lay


def _no_eps(s):
    # RMSNorm is then idempotent (with eps the head's second normalisation rescales by
    # 1/sqrt(1 - eps/mean(x^2)), 0.1% for embedding rows of rms 0.02)
    s["cfg"] = dict(s["cfg"], rms_eps=0.0)
    return s


def test_hidden_half_reproduces_target_head():
    s = _no_eps(_setup(seed=1))
    d, k = s["w"].d_model, s["w"].k
    mtp = dict(s["mtp"], layer=_silent_layer(s["mtp"]), hnorm=np.ones(d, np.float32),
               final_norm=np.ones(d, np.float32),
               eh_proj=np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1).astype(np.float32))
    out = _run(s, mtp=mtp)
    rows = np.arange(s["w"].batch) * (k + 1) + s["n"]
    ref = model.lm_logits(s["hidden"][rows], s["head"], s["cfg"])
    np.testing.assert_allclose(out["logits"][:, 0], ref, rtol=1e-5, atol=1e-6)
    # later drafts: the head's own output renormalised again, the same logits
    for i in range(1, k):
        np.testing.assert_allclose(out["logits"][:, i], ref, rtol=1e-5, atol=1e-6)


def test_embedding_half_follows_emitted_token_and_drafts():
    s = _no_eps(_setup(seed=2))
    d, k = s["w"].d_model, s["w"].k
    mtp = dict(s["mtp"], layer=_silent_layer(s["mtp"]), enorm=np.ones(d, np.float32),
               final_norm=np.ones(d, np.float32),
               eh_proj=np.concatenate([np.eye(d), np.zeros((d, d))], axis=1).astype(np.float32))
    for u in ("default", None):
        out = _run(s, uniforms=u, mtp=mtp)
        prev = s["nxt"]
        for i in range(k):
            ref = model.lm_logits(model.embed(prev, s["head"], s["cfg"]), s["head"], s["cfg"])
            np.testing.assert_allclose(out["logits"][:, i], ref, rtol=1e-5, atol=1e-6)
            prev = out["drafts"][:, i]


@pytest.mark.parametrize("seed,i,n", [(3, 1, [0, 1, 2, 1]), (4, 1, [2, 0, 1, 0]),
                                       (7, 2, [0, 1, 1, 0])])
def test_catch_up_agrees_with_drafting(seed, i, n):
    """Draft i+1 of a step equals draft 1 of the same step with i more accepted tokens: y_b,
    drafts 1..i-1 in the verify slots, draft i as the emitted token, and the head's own
    outputs behind drafts 1..i as the hidden rows of those slots."""
    k = 3
    s = _setup(seed=seed, k=k, n=np.array(n))
    a = _run(s)
    B = s["w"].batch
    tokens2 = s["tokens"].copy()
    hidden2 = s["hidden"].copy()
    for b in range(B):
        nb = s["n"][b]
        fed = [s["nxt"][b]] + [a["drafts"][b, j] for j in range(i - 1)]
        for j in range(i):
            tokens2[b, nb + 1 + j] = fed[j]
            hidden2[b * (k + 1) + nb + 1 + j] = a["h"][b, j]
    u2 = np.roll(s["u"], -i, axis=1)
    b2 = _run(s, tokens=tokens2, hidden=hidden2, n=s["n"] + i, nxt=a["drafts"][:, i - 1], u=u2)
    ok = b2["margin"][:, 0] > 1e-9
    assert ok.sum() >= B - 1
    np.testing.assert_array_equal(b2["drafts"][ok, 0], a["drafts"][ok, i])
    np.testing.assert_allclose(b2["logits"][:, 0], a["logits"][:, i], rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(b2["q"][:, 0], a["q"][:, i], rtol=1e-5, atol=1e-9)


def test_rejected_rows_do_not_matter():
    k = 3
    s = _setup(seed=5, k=k, n=np.array([0, 3, 1, 2]))
    a = _run(s)
    tokens2 = s["tokens"].copy()
    hidden2 = s["hidden"].copy()
    g = np.random.default_rng(9)
    for b in range(s["w"].batch):
        nb = s["n"][b]
        tokens2[b, nb + 1:] = g.integers(0, s["w"].vocab, k - nb)
        hidden2[b * (k + 1) + nb + 1:(b + 1) * (k + 1)] = g.normal(size=(k - nb, s["w"].d_model))
    b2 = _run(s, tokens=tokens2, hidden=hidden2)
    np.testing.assert_array_equal(a["drafts"], b2["drafts"])
    np.testing.assert_allclose(a["q"], b2["q"], rtol=0, atol=1e-12)


def test_greedy_is_argmax_of_q():
    s = _setup(seed=6, k=1)
    a = _run(s, uniforms=np.full((s["w"].batch, 1), 0.5, np.float32))
    g = _run(s, uniforms=None)
    np.testing.assert_array_equal(g["drafts"][:, 0], np.argmax(a["q"][:, 0], axis=1))
    np.testing.assert_allclose(a["q"].sum(axis=-1), 1.0, atol=1e-12)
