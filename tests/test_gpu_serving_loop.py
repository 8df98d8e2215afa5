"""The whole speculative serving loop on the GPU, checked step by step against the oracle run
on the same trajectory (tiny f32 decoder, B 2 with ragged prompts, k 3):

    prefill (molt_prefill) -> first token (molt_spec_accept, k = 0)
    -> draft head over the prompt window (molt_mtp_draft_window) -> k drafts with q
    -> [verify (molt_verify_step) -> draft head after the verify step (molt_mtp_draft)] x 3

with the contexts advanced by n_accepted + 1 after each verify step, the target's and the
draft head's caches shared across the calls. Every logit row and q row agrees with the
oracle within 1e-4 / 1e-5 relative, and every decision (first token, drafts, accepted
counts, emitted tokens) is the oracle's; the oracle is fed the GPU's drafts and q so that
both sides walk the same trajectory."""
import numpy as np
import pytest
import torch

import workloads
from oracle import model as omodel, mtp as omtp, sampler as osamp
from oracle.prefix import prefill_logits
from helpers import dev, host, layer_host, max_abs, model_from, oracle_cfg

pytestmark = pytest.mark.gpu


def test_prefill_draft_verify_loop(molt_lib):
    molt = molt_lib
    seed = 61
    w = workloads.TINY_FP32.scaled(batch=2, k=3, ctx_lo=0, ctx_hi=0)
    B, k, V, d = w.batch, w.k, w.vocab, w.d_model
    cfg = oracle_cfg(w)
    layers = [workloads.make_layer_weights(w, seed, l) for l in range(w.n_layers)]
    head = workloads.make_head_weights(w, seed)
    mt = workloads.make_mtp_weights(w, seed)
    model = model_from(w, layers, head, molt)
    mtp = molt.Mtp(dev(mt["enorm"]), dev(mt["hnorm"]), dev(mt["eh_proj"]),
                   {kk: dev(v) for kk, v in mt["layer"].items()}, dev(mt["final_norm"]),
                   n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                   top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta)
    lh, hh = [layer_host(lw) for lw in layers], layer_host(head)
    mh = {kk: host(v) for kk, v in mt.items() if kk != "layer"}
    mh["layer"] = layer_host(mt["layer"])
    nbps, nb = 8, 16
    bt = np.arange(nb, dtype=np.int32).reshape(B, nbps)
    btd = dev(torch.from_numpy(bt))
    zk = lambda: torch.zeros(nb, w.n_kv_heads, 16, w.head_dim, device="cuda")
    zv = lambda: torch.zeros(nb, w.n_kv_heads, w.head_dim, 16, device="cuda")
    tk, tv = [zk() for _ in range(w.n_layers)], [zv() for _ in range(w.n_layers)]
    hk, hv = [zk()], [zv()]
    ocache = [(np.zeros((nb, w.n_kv_heads, 16, w.head_dim)), np.zeros((nb, w.n_kv_heads, w.head_dim, 16)))
              for _ in range(w.n_layers)]
    ohk, ohv = np.zeros((nb, w.n_kv_heads, 16, w.head_dim)), np.zeros((nb, w.n_kv_heads, w.head_dim, 16))

    def kvs(ctx):
        c = dev(torch.from_numpy(ctx.astype(np.int32)))
        return molt.KVCache(tk, tv, btd, c), molt.KVCache(hk, hv, btd, c)

    g = np.random.default_rng(seed)
    n = 40
    lens = np.array([40, 27], np.int32)
    prompt = g.integers(0, V, (B, n)).astype(np.int32)
    ctx = np.zeros(B, np.int64)
    # prefill and the first token
    kv, hkv = kvs(ctx)
    pf = molt.prefill(model, kv, dev(torch.from_numpy(prompt)), dev(torch.from_numpy(lens)), want_hidden=True)
    u0 = workloads.make_uniforms(B, 0, seed + 1)
    first, _, _ = molt.spec_accept(pf["logits"][:, None, :].contiguous(), None, dev(u0))
    torch.cuda.synchronize()
    olog, _, ohid_all = prefill_logits(prompt, lens, lambda l: lh[l], hh, ocache, bt, ctx, cfg)
    err = max_abs(pf["logits"].cpu().numpy(), olog)
    print(f"prefill logits {err:.2e}", flush=True)
    assert err <= 1e-4
    ofirst = osamp.spec_accept(olog[:, None, :], np.zeros((B, 0), np.int64), host(u0))
    t1 = first[:, 0].cpu().numpy()
    np.testing.assert_array_equal(t1, ofirst["tokens"][:, 0])
    # draft head over the prompt window
    ud = workloads.make_uniforms(B, k - 1, seed + 2, tag="mtp_u")
    dr = molt.mtp_draft(model, mtp, hkv, pf["hidden"], dev(torch.from_numpy(prompt)),
                        dev(torch.from_numpy(lens - 1)), first[:, 0].contiguous(), dev(ud), k=k)
    torch.cuda.synchronize()
    drafts, q = dr["drafts"].cpu().numpy(), dr["draft_probs"]
    od = omtp.mtp_draft(host(pf["hidden"]), prompt, lens - 1, t1, mh, hh, ohk, ohv, bt, ctx, cfg,
                        uniforms=host(ud), forced=drafts, k=k)
    assert np.abs(q.cpu().numpy() - od["q"]).max() <= 1e-5 * od["q"].max() + 1e-9
    np.testing.assert_array_equal(drafts, od["drafts"])
    ctx = lens.astype(np.int64)
    last = t1
    for it in range(3):
        toks = np.concatenate([last[:, None], drafts], axis=1).astype(np.int32)
        u = workloads.make_uniforms(B, k, seed + 10 + it)
        kv, hkv = kvs(ctx)
        vs = molt.verify_step(model, kv, dev(torch.from_numpy(toks)), dev(u), q, want_hidden=True)
        torch.cuda.synchronize()
        ov = omodel.verify_step(toks, lambda l: lh[l], hh, ocache, bt, ctx, cfg, host(q), host(u))
        err = max_abs(vs["logits"].cpu().numpy(), ov["logits"])
        nacc = vs["n_accepted"].cpu().numpy()
        print(f"iteration {it}: verify logits {err:.2e}, n_accepted {nacc}", flush=True)
        assert err <= 1e-4
        np.testing.assert_array_equal(nacc, ov["n_accepted"])
        np.testing.assert_array_equal(vs["tokens"].cpu().numpy(), ov["tokens"])
        nxt = ov["tokens"][np.arange(B), nacc].astype(np.int32)
        ud = workloads.make_uniforms(B, k - 1, seed + 20 + it, tag="mtp_u")
        dr = molt.mtp_draft(model, mtp, hkv, vs["hidden"], dev(torch.from_numpy(toks)),
                            vs["n_accepted"], dev(torch.from_numpy(nxt)), dev(ud))
        torch.cuda.synchronize()
        drafts, q = dr["drafts"].cpu().numpy(), dr["draft_probs"]
        od = omtp.mtp_draft(host(vs["hidden"]), toks, nacc, nxt, mh, hh, ohk, ohv, bt, ctx, cfg,
                            uniforms=host(ud), forced=drafts)
        assert np.abs(q.cpu().numpy() - od["q"]).max() <= 1e-5 * od["q"].max() + 1e-9
        np.testing.assert_array_equal(drafts, od["drafts"])
        ctx = ctx + nacc + 1
        last = nxt
