"""GPU parity of the behavior-log-prob recompute with routing replay (molt_score_tokens):

* the consistency diagnostic: after a GPU verify step, scoring its tokens with its emitted
  tokens as targets and its recorded routes as replay reproduces the recorded logits and
  behavior log-probabilities bit for bit (NaN past each sequence's emitted token);
* against the oracle (oracle/replay.py): log-probs within 1e-4 (f32) / 4e-2 (bf16: logits
  within 2e-2 move (l_y - m) - ln S by at most twice that), with the router's own routes
  and with foreign replayed routes (every expert id shifted), where the routes used must be
  exactly the replayed ones."""
import numpy as np
import pytest
import torch

import workloads
from oracle import model as omodel, replay as oreplay
from helpers import dev, host, layer_host, max_abs, model_from, oracle_cfg

pytestmark = pytest.mark.gpu

SMALL_BF16 = workloads.LAYER_BF16.scaled(
    name="replay_small_bf16", n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128,
    n_experts=16, top_k=4, d_ff=256, vocab=8192, batch=8, k=4, ctx_lo=100, ctx_hi=700,
    full_model=True)


def _setup(molt, w, seed):
    layout = workloads.make_kv_layout(w, seed)
    layers = [workloads.make_layer_weights(w, seed, l) for l in range(w.n_layers)]
    head = workloads.make_head_weights(w, seed)
    caches = [workloads.make_kv_cache(w, layout, seed, l) for l in range(w.n_layers)]
    kv = molt.KVCache([dev(c[0]) for c in caches], [dev(c[1]) for c in caches],
                      dev(torch.from_numpy(layout.block_tables)), dev(torch.from_numpy(layout.context_lens)))
    return layout, layers, head, caches, kv, model_from(w, layers, head, molt)


def _oracle(w, layout, layers, head, caches, toks, targets, rep):
    lh = [layer_host(lw) for lw in layers]
    oc = [tuple(omodel.widen_cache(host(c), w.dtype) for c in cc) for cc in caches]
    return oreplay.score_tokens(toks, targets, lambda l: lh[l], layer_host(head), oc,
                                layout.block_tables, layout.context_lens, oracle_cfg(w), rep)


@pytest.mark.parametrize("wname", ["tiny_fp32", "small_bf16"])
def test_recompute_reproduces_verify_and_oracle(molt_lib, wname):
    molt = molt_lib
    w = workloads.TINY_FP32 if wname == "tiny_fp32" else SMALL_BF16
    seed = 41
    layout, layers, head, caches, kv, model = _setup(molt, w, seed)
    toks = workloads.make_step_tokens(w, seed)
    q = workloads.make_softmax_q(w.batch, w.k, w.vocab, seed + 1)
    u = workloads.make_uniforms(w.batch, w.k, seed + 2)
    td = dev(torch.from_numpy(toks))
    v = molt.verify_step(model, kv, td, dev(u), dev(q), want_routes=True)
    r = molt.score_tokens(model, kv, td, v["tokens"], replay_routes=v["routes"], want_logits=True,
                          want_routes=True)
    torch.cuda.synchronize()
    emitted = v["tokens"].cpu().numpy() >= 0
    np.testing.assert_array_equal(r["logits"].cpu().numpy(), v["logits"].cpu().numpy())
    np.testing.assert_array_equal(r["routes"].cpu().numpy(), v["routes"].cpu().numpy())
    lr, lv = r["logprobs"].cpu().numpy(), v["logprobs"].cpu().numpy()
    np.testing.assert_array_equal(lr[emitted], lv[emitted])
    assert np.isnan(lr[~emitted]).all()
    print(f"recompute == verify: {emitted.sum()} emitted tokens bit-exact", flush=True)
    # against the oracle, with the GPU's routes replayed on both sides (the routes are then
    # the same by construction) and with foreign routes
    tol = 1e-4 if w.dtype == "f32" else 2 * 2e-2
    targets = np.roll(toks, -1, axis=1)
    targets[:, -1] = v["tokens"].cpu().numpy()[np.arange(w.batch), v["n_accepted"].cpu().numpy()]
    routes = v["routes"].cpu().numpy()
    for name, rep in (("recorded", routes), ("shifted", (routes + 1) % w.n_experts)):
        g = molt.score_tokens(model, kv, td, dev(torch.from_numpy(targets.astype(np.int32))),
                              replay_routes=dev(torch.from_numpy(rep.astype(np.int32))), want_routes=True)
        torch.cuda.synchronize()
        o = _oracle(w, layout, layers, head, caches, toks, targets, rep)
        np.testing.assert_array_equal(g["routes"].cpu().numpy(), rep)
        err = max_abs(g["logprobs"].cpu().numpy(), o["logprobs"])
        print(f"{name} routes: max |logprob - oracle| = {err:.3e}", flush=True)
        assert err <= tol


def test_recompute_single_position(molt_lib):
    """k = 0: one position per sequence (a plain decode step's recompute)."""
    molt = molt_lib
    w = workloads.TINY_FP32.scaled(k=0)
    seed = 43
    layout, layers, head, caches, kv, model = _setup(molt, w, seed)
    toks = workloads.make_step_tokens(w, seed)
    targets = np.random.default_rng(seed).integers(0, w.vocab, toks.shape).astype(np.int32)
    g = molt.score_tokens(model, kv, dev(torch.from_numpy(toks)), dev(torch.from_numpy(targets)),
                          want_routes=True)
    torch.cuda.synchronize()
    o = _oracle(w, layout, layers, head, caches, toks, targets, None)
    clear = g["routes"].cpu().numpy() == o["routes"]
    assert clear.all()
    assert max_abs(g["logprobs"].cpu().numpy(), o["logprobs"]) <= 1e-4
