"""GPU parity of the MTP draft head (molt_mtp_draft) against the oracle (oracle/mtp.py).

The oracle is teacher-forced with the GPU's drafts, so that every draft step is compared
on the same inputs: q of every step within the logits' tolerance (f32: 1e-5 relative;
bf16: logits within 2e-2 move q by at most e^(2 * 2e-2) - 1 < 5e-2 relative); drafts
bit-exact away from a draw near-tie (f32), or inside the oracle's CDF interval of the
uniform (bf16, where the CDF moves by up to ~1e-3); greedy drafts equal to the oracle's
argmax away from a logit near-tie; the head's KV cache after the step equal to the
oracle's; run-to-run determinism. The inputs come from a real GPU verify step (tiny f32
decoder, small bf16 decoder) or, at the full benchmark shape (B 128, k 4, context 8192,
vocabulary 151936), are synthetic (N(0,1) hidden rows, uniform accepted counts and
emitted tokens), with the oracle run on sampled sequences."""
import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oattn, model as omodel, mtp as omtp
from helpers import dev, host, layer_host, max_abs, model_from, oracle_cfg

pytestmark = pytest.mark.gpu

SMALL_BF16 = workloads.LAYER_BF16.scaled(
    name="mtp_small_bf16", n_layers=1, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128,
    n_experts=16, top_k=4, d_ff=256, vocab=8192, batch=8, k=4, ctx_lo=100, ctx_hi=700,
    full_model=True)


def _mtp_dev(molt, w, mt):
    return molt.Mtp(dev(mt["enorm"]), dev(mt["hnorm"]), dev(mt["eh_proj"]),
                    {k: dev(v) for k, v in mt["layer"].items()}, dev(mt["final_norm"]),
                    n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                    top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta)


def _mtp_host(mt):
    out = {k: host(v) for k, v in mt.items() if k != "layer"}
    out["layer"] = layer_host(mt["layer"])
    return out


def _setup(molt, w, seed):
    layout = workloads.make_kv_layout(w, seed, extra_tokens=w.k)
    layers = [workloads.make_layer_weights(w, seed, l) for l in range(w.n_layers)]
    head = workloads.make_head_weights(w, seed)
    mt = workloads.make_mtp_weights(w, seed)
    bt, ctx = dev(torch.from_numpy(layout.block_tables)), dev(torch.from_numpy(layout.context_lens))
    caches = [workloads.make_kv_cache(w, layout, seed, l) for l in range(w.n_layers + 1)]
    kv = molt.KVCache([dev(c[0]) for c in caches[:-1]], [dev(c[1]) for c in caches[:-1]], bt, ctx)
    hkv = molt.KVCache([dev(caches[-1][0])], [dev(caches[-1][1])], bt, ctx)
    model = model_from(w, layers, head, molt)
    return dict(w=w, layout=layout, head=head, hh=layer_host(head), mt=mt, mh=_mtp_host(mt),
                kv=kv, hkv=hkv, model=model, mtp=_mtp_dev(molt, w, mt), cfg=oracle_cfg(w))


def _verify(molt, s, seed):
    w = s["w"]
    toks = workloads.make_step_tokens(w, seed)
    q = workloads.make_softmax_q(w.batch, w.k, w.vocab, seed + 1)
    u = workloads.make_uniforms(w.batch, w.k, seed + 2)
    out = molt.verify_step(s["model"], s["kv"], dev(torch.from_numpy(toks)), dev(u), dev(q),
                           want_logits=False, want_hidden=True)
    n = out["n_accepted"]
    nxt = out["tokens"].gather(1, n.long()[:, None])[:, 0].contiguous()
    return toks, out["hidden"], n, nxt


def _oracle(s, hidden, toks, n, nxt, hcache, ud, drafts, seqs=None):
    w, layout = s["w"], s["layout"]
    bt, ctx = layout.block_tables, layout.context_lens
    if seqs is not None:   # a subset of sequences, blocks renumbered densely
        rows = [bt[b][bt[b] >= 0] for b in seqs]
        idx = np.concatenate(rows)
        bt2 = np.full((len(seqs), max(len(r) for r in rows)), -1, dtype=np.int64)
        pos = 0
        for i, r in enumerate(rows):
            bt2[i, :len(r)] = np.arange(pos, pos + len(r))
            pos += len(r)
        hcache = tuple(c[idx] for c in hcache)
        kp1 = w.k + 1
        hidden = hidden.reshape(-1, kp1, w.d_model)[seqs].reshape(-1, w.d_model)
        toks, n, nxt = toks[seqs], n[seqs], nxt[seqs]
        ud = None if ud is None else ud[seqs]
        drafts = drafts[seqs]
        bt, ctx = bt2, ctx[seqs]
    kc, vc = (omodel.widen_cache(c, w.dtype) for c in hcache)
    o = omtp.mtp_draft(hidden, toks, n, nxt, s["mh"], s["hh"], kc, vc, bt, ctx, s["cfg"],
                       uniforms=ud, forced=drafts)
    return o, kc, vc


def _check_q(qg, qo, rtol, atol):
    err = np.abs(qg.astype(np.float64) - qo)
    bad = err > rtol * qo + atol
    big = qo > 1e-6
    rel = float((err[big] / qo[big]).max()) if big.any() else 0.0
    print(f"max |q - oracle| = {err.max():.3e}, max relative {rel:.2e} where q > 1e-6", flush=True)
    assert not bad.any(), f"{bad.sum()} q entries outside tolerance"


def _drafts_in_cdf(drafts, qo, u, tol):
    """Each draft's interval [CDF(d - 1), CDF(d)) of the oracle's q holds its uniform, up to
    tol (the CDF's own movement under the logits' tolerance)."""
    B, k, V = qo.shape
    for b in range(B):
        for i in range(k):
            c = np.cumsum(qo[b, i])
            d = int(drafts[b, i])
            lo, hi = (c[d - 1] if d > 0 else 0.0), c[d]
            assert lo - tol <= u[b, i] <= hi + tol, (b, i, d, lo, hi, u[b, i])


def test_tiny_f32_after_verify(molt_lib):
    molt = molt_lib
    w = workloads.TINY_FP32
    s = _setup(molt, w, 11)
    toks, hidden, n, nxt = _verify(molt, s, 12)
    ud = workloads.make_uniforms(w.batch, w.k - 1, 13, tag="mtp_u")
    hc0 = tuple(host(c) for c in (s["hkv"].k_caches[0], s["hkv"].v_caches[0]))
    g = molt.mtp_draft(s["model"], s["mtp"], s["hkv"], hidden, dev(torch.from_numpy(toks)), n, nxt, dev(ud))
    g2 = molt.mtp_draft(s["model"], s["mtp"], s["hkv"], hidden, dev(torch.from_numpy(toks)), n, nxt, dev(ud))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(g["drafts"].cpu().numpy(), g2["drafts"].cpu().numpy())
    np.testing.assert_array_equal(g["draft_probs"].cpu().numpy(), g2["draft_probs"].cpu().numpy())
    drafts = g["drafts"].cpu().numpy()
    print(f"n_accepted {n.cpu().numpy()}, drafts {drafts.tolist()}", flush=True)
    o, kc, vc = _oracle(s, host(hidden), toks, host(n), host(nxt), hc0, host(ud), drafts)
    _check_q(g["draft_probs"].cpu().numpy(), o["q"], 1e-4, 1e-7)
    ok = o["margin"] > 1e-6
    assert ok.mean() >= 0.9
    np.testing.assert_array_equal(drafts[ok], o["drafts"][ok])
    # the head's cache: every slot the step wrote
    kg, vg = (host(c) for c in (s["hkv"].k_caches[0], s["hkv"].v_caches[0]))
    for b in range(w.batch):
        m = int(s["layout"].context_lens[b]) + w.k + int(host(n)[b]) + 1
        Kg, Vg = oattn.gather_kv(kg, vg, s["layout"].block_tables[b], m, 0)
        Ko, Vo = oattn.gather_kv(kc, vc, s["layout"].block_tables[b], m, 0)
        assert max_abs(Kg, Ko) <= 1e-4 and max_abs(Vg, Vo) <= 1e-4
    # greedy drafts
    gg = molt.mtp_draft(s["model"], s["mtp"], s["hkv"], hidden, dev(torch.from_numpy(toks)), n, nxt,
                        greedy=True)
    torch.cuda.synchronize()
    gd = gg["drafts"].cpu().numpy()
    og, _, _ = _oracle(s, host(hidden), toks, host(n), host(nxt), hc0, None, gd)
    ok = og["margin"] > 1e-4
    assert ok.mean() >= 0.9
    np.testing.assert_array_equal(gd[ok], og["drafts"][ok])


@pytest.mark.parametrize("seed", [21, 22])
def test_small_bf16_after_verify(molt_lib, seed):
    molt = molt_lib
    w = SMALL_BF16
    s = _setup(molt, w, seed)
    toks, hidden, n, nxt = _verify(molt, s, seed + 1)
    ud = workloads.make_uniforms(w.batch, w.k - 1, seed + 2, tag="mtp_u")
    hc0 = tuple(host(c) for c in (s["hkv"].k_caches[0], s["hkv"].v_caches[0]))
    g = molt.mtp_draft(s["model"], s["mtp"], s["hkv"], hidden, dev(torch.from_numpy(toks)), n, nxt, dev(ud))
    torch.cuda.synchronize()
    drafts = g["drafts"].cpu().numpy()
    print(f"n_accepted {n.cpu().numpy()}", flush=True)
    o, _, _ = _oracle(s, host(hidden), toks, host(n), host(nxt), hc0, host(ud), drafts)
    _check_q(g["draft_probs"].cpu().numpy(), o["q"], 5e-2, 1e-6)
    _drafts_in_cdf(drafts, o["q"], host(ud), 1e-3)
    assert ((drafts >= 0) & (drafts < w.vocab)).all()


# A head row whose top-K route set sits within this router-logit gap of the next expert may
# take another set under rounding (its output, and every later draft's input, then moves
# by far more than the logits' tolerance): such a row and the drafts after it are compared
# only for validity, as in the full-shape decoder test.
ROUTE_TIE = 1e-2


def test_full_shape_synthetic(molt_lib):
    """B 128, k 4, context 8192, vocabulary 151936 (the benchmark's step), one head layer;
    the oracle on six sampled sequences with n_accepted 0 to 4, each compared up to its
    first head row at a route near-tie."""
    molt = molt_lib
    w = workloads.FULL_DEPTH_BF16.scaled(n_layers=1)
    seed = 31
    layout = workloads.make_kv_layout(w, seed, extra_tokens=w.k)
    head = workloads.make_head_weights(w, seed, device="cuda")
    mt = workloads.make_mtp_weights(w, seed, device="cuda")
    bt, ctx = dev(torch.from_numpy(layout.block_tables)), dev(torch.from_numpy(layout.context_lens))
    kc, vc = workloads.make_kv_cache(w, layout, seed, 1, device="cuda")
    hkv = molt.KVCache([kc], [vc], bt, ctx)
    target = model_from(w, [mt["layer"]], head, molt)
    mtp = _mtp_dev(molt, w, mt)
    B, k, V = w.batch, w.k, w.vocab
    g = np.random.default_rng(seed)
    n = g.integers(0, k + 1, B).astype(np.int32)
    seqs = [3, 40, 77, 90, 101, 120]
    n[seqs] = [0, 2, 4, 1, 3, 0]
    nxt = g.integers(0, V, B).astype(np.int32)
    toks = workloads.make_step_tokens(w, seed)
    hidden = workloads.make_hidden(w, seed, device="cuda")
    ud = workloads.make_uniforms(B, k - 1, seed, tag="mtp_u", device="cuda")
    print("inputs built", flush=True)
    # oracle inputs first: the call rewrites the head's cache
    rows = np.concatenate([layout.block_tables[b][layout.block_tables[b] >= 0] for b in seqs])
    idx = torch.from_numpy(rows).long().cuda()
    sub = (host(kc.index_select(0, idx)), host(vc.index_select(0, idx)))
    out = molt.mtp_draft(target, mtp, hkv, hidden, dev(torch.from_numpy(toks)),
                         dev(torch.from_numpy(n)), dev(torch.from_numpy(nxt)), ud)
    torch.cuda.synchronize()
    drafts = out["drafts"].cpu().numpy()
    q = out["draft_probs"]
    assert ((drafts >= 0) & (drafts < V)).all()
    sums = q.double().sum(dim=-1).cpu().numpy()
    print(f"q row sums in [{sums.min():.8f}, {sums.max():.8f}]", flush=True)
    assert np.abs(sums - 1.0).max() < 1e-5
    # the oracle on the sampled sequences, blocks renumbered densely
    bt2 = np.full((len(seqs), max(int((layout.block_tables[b] >= 0).sum()) for b in seqs)), -1, np.int64)
    pos = 0
    for i, b in enumerate(seqs):
        m = int((layout.block_tables[b] >= 0).sum())
        bt2[i, :m] = np.arange(pos, pos + m)
        pos += m
    hh = {"embed": host(head["embed"]), "lm_head": host(head["lm_head"]), "final_norm": host(head["final_norm"])}
    okc, ovc = (omodel.widen_cache(c, w.dtype) for c in sub)
    hid = host(hidden).reshape(B, k + 1, -1)[seqs].reshape(-1, w.d_model)
    o = omtp.mtp_draft(hid, toks[seqs], n[seqs], nxt[seqs], _mtp_host(mt), hh, okc, ovc, bt2,
                       layout.context_lens[seqs], oracle_cfg(w), uniforms=host(ud)[seqs],
                       forced=drafts[seqs])
    tie = o["route_margin"] < ROUTE_TIE
    upto = np.where(tie.any(axis=1), tie.argmax(axis=1), k)   # drafts before the first near-tie
    print(f"route margins {np.array2string(o['route_margin'], precision=3)}; compared drafts per "
          f"sequence {upto.tolist()}", flush=True)
    assert upto.sum() >= 12, "too few drafts away from route near-ties"
    qg = q[seqs].cpu().numpy()
    for i in range(len(seqs)):
        if upto[i]:
            _check_q(qg[i:i + 1, :upto[i]], o["q"][i:i + 1, :upto[i]], 5e-2, 1e-6)
            _drafts_in_cdf(drafts[seqs][i:i + 1, :upto[i]], o["q"][i:i + 1, :upto[i]],
                           host(ud)[seqs][i:i + 1, :upto[i]], 1e-3)


def test_tiny_one_draft(molt_lib):
    """k = 1: the catch-up rows alone give the only draft (no drafting row)."""
    molt = molt_lib
    w = workloads.TINY_FP32.scaled(k=1)
    s = _setup(molt, w, 15)
    toks, hidden, n, nxt = _verify(molt, s, 16)
    ud = workloads.make_uniforms(w.batch, 0, 17, tag="mtp_u")
    hc0 = tuple(host(c) for c in (s["hkv"].k_caches[0], s["hkv"].v_caches[0]))
    g = molt.mtp_draft(s["model"], s["mtp"], s["hkv"], hidden, dev(torch.from_numpy(toks)), n, nxt, dev(ud))
    gg = molt.mtp_draft(s["model"], s["mtp"], s["hkv"], hidden, dev(torch.from_numpy(toks)), n, nxt, greedy=True)
    torch.cuda.synchronize()
    drafts = g["drafts"].cpu().numpy()
    o, _, _ = _oracle(s, host(hidden), toks, host(n), host(nxt), hc0, host(ud), drafts)
    _check_q(g["draft_probs"].cpu().numpy(), o["q"], 1e-4, 1e-7)
    ok = o["margin"] > 1e-6
    np.testing.assert_array_equal(drafts[ok], o["drafts"][ok])
    og, _, _ = _oracle(s, host(hidden), toks, host(n), host(nxt), hc0, None, gg["drafts"].cpu().numpy())
    ok = og["margin"] > 1e-4
    np.testing.assert_array_equal(gg["drafts"].cpu().numpy()[ok], og["drafts"][ok])
