"""GPU parity of the paged prefill (molt_prefill) and of the cache-hit re-prefill with the
session-consistent prefix cache (molt_prefix_cache_*):

* prefill of fresh, ragged prompts (a window of n rows per sequence, rows past lens[b]
  padding) against the oracle: last-row logits within 1e-4 (f32) / 2e-2 (bf16), the final
  residual rows and the keys/values written for the real positions;
* a growing agent session: the first turn is prefilled from scratch and committed; the next
  turn hits the cached full blocks and re-prefills only the new positions at context
  n_cached, and its logits match a fresh prefill of the whole conversation (GPU and
  oracle); a rewritten history hits nothing."""
import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oattn, model as omodel
from oracle.prefix import prefill_logits
from helpers import dev, host, layer_host, max_abs, model_from, oracle_cfg

pytestmark = pytest.mark.gpu

SMALL_BF16 = workloads.LAYER_BF16.scaled(
    name="prefill_small_bf16", n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128,
    n_experts=16, top_k=4, d_ff=256, vocab=8192, batch=3, k=0, ctx_lo=0, ctx_hi=0,
    full_model=True)


def _workload(name):
    return workloads.TINY_FP32.scaled(batch=3, k=0, ctx_lo=0, ctx_hi=0) if name == "tiny_fp32" else SMALL_BF16


def _model(molt, w, seed):
    layers = [workloads.make_layer_weights(w, seed, l) for l in range(w.n_layers)]
    head = workloads.make_head_weights(w, seed)
    return layers, head, model_from(w, layers, head, molt)


def _pool(w, num_blocks):
    dt = workloads.torch_dtype(w.dtype)
    return ([torch.zeros(num_blocks, w.n_kv_heads, 16, w.head_dim, dtype=dt, device="cuda") for _ in range(w.n_layers)],
            [torch.zeros(num_blocks, w.n_kv_heads, w.head_dim, 16, dtype=dt, device="cuda") for _ in range(w.n_layers)])


def _oracle_fresh(w, layers, head, toks, lens, bt, num_blocks):
    lh = [layer_host(lw) for lw in layers]
    caches = [(np.zeros((num_blocks, w.n_kv_heads, 16, w.head_dim)), np.zeros((num_blocks, w.n_kv_heads, w.head_dim, 16)))
              for _ in range(w.n_layers)]
    lg, hid, _ = prefill_logits(toks, lens, lambda l: lh[l], layer_host(head), caches, bt,
                                np.zeros(len(lens), np.int64), oracle_cfg(w))
    return lg, hid, caches


@pytest.mark.parametrize("wname", ["tiny_fp32", "small_bf16"])
def test_fresh_ragged_prefill(molt_lib, wname):
    molt = molt_lib
    w = _workload(wname)
    seed = 51
    layers, head, model = _model(molt, w, seed)
    n = 70
    lens = np.array([70, 33, 1], np.int32)
    B = len(lens)
    g = np.random.default_rng(seed)
    toks = g.integers(0, w.vocab, (B, n)).astype(np.int32)
    nbps = (n + 15) // 16
    bt = (np.arange(B * nbps).reshape(B, nbps)[:, ::-1] * 1).astype(np.int32).copy()   # reversed blocks
    kcs, vcs = _pool(w, B * nbps)
    kv = molt.KVCache(kcs, vcs, dev(torch.from_numpy(bt)), dev(torch.zeros(B, dtype=torch.int32)))
    out = molt.prefill(model, kv, dev(torch.from_numpy(toks)), dev(torch.from_numpy(lens)), want_hidden=True)
    torch.cuda.synchronize()
    lg, hid, oc = _oracle_fresh(w, layers, head, toks, lens, bt, B * nbps)
    tol = 1e-4 if w.dtype == "f32" else 2e-2
    err = max_abs(out["logits"].cpu().numpy(), lg)
    herr = max_abs(out["hidden"].cpu().numpy()[np.arange(B) * n + lens - 1], hid)
    print(f"{wname}: max |logits - oracle| = {err:.3e}, last hidden rows {herr:.3e}", flush=True)
    assert err <= tol and herr <= tol
    for l in range(w.n_layers):
        for b in range(B):
            Kg, Vg = oattn.gather_kv(omodel.widen_cache(host(kcs[l]), w.dtype),
                                     omodel.widen_cache(host(vcs[l]), w.dtype), bt[b], int(lens[b]), 0)
            Ko, Vo = oattn.gather_kv(oc[l][0], oc[l][1], bt[b], int(lens[b]), 0)
            assert max_abs(Kg, Ko) <= tol and max_abs(Vg, Vo) <= tol


@pytest.mark.parametrize("wname", ["tiny_fp32", "small_bf16"])
def test_session_reprefill_from_prefix_cache(molt_lib, wname):
    molt = molt_lib
    w = _workload(wname)
    seed = 52
    layers, head, model = _model(molt, w, seed)
    g = np.random.default_rng(seed)
    turn1 = g.integers(0, w.vocab, 70).astype(np.int32)
    turn2 = np.concatenate([turn1, g.integers(0, w.vocab, 25).astype(np.int32)])
    rewritten = turn2.copy()
    rewritten[5] = (rewritten[5] + 1) % w.vocab
    num_blocks = 32
    max_blocks = 8
    cache = molt.PrefixCache(num_blocks)
    kcs, vcs = _pool(w, num_blocks)

    def run(tokens):
        row, hit = cache.acquire(tokens, max_blocks=max_blocks)
        bt = np.full((1, max_blocks), -1, np.int32)
        bt[0, :len(row)] = row
        new = tokens[hit:]
        kv = molt.KVCache(kcs, vcs, dev(torch.from_numpy(bt)), dev(torch.tensor([hit], dtype=torch.int32)))
        out = molt.prefill(model, kv, dev(torch.from_numpy(new[None, :].copy())),
                           dev(torch.tensor([len(new)], dtype=torch.int32)))
        torch.cuda.synchronize()
        cache.commit(tokens, row)
        return out["logits"].cpu().numpy()[0], row, hit

    l1, row1, hit1 = run(turn1)
    cache.release(row1)
    l2, row2, hit2 = run(turn2)
    l3, row3, hit3 = run(rewritten)
    print(f"hits: turn 1 {hit1}, turn 2 {hit2}, rewritten {hit3}; stats {cache.stats()}", flush=True)
    assert (hit1, hit2, hit3) == (0, 64, 0)
    assert list(row2[:4]) == list(row1[:4])
    # a fresh prefill of the whole conversation, in blocks of its own
    fresh_blocks = np.arange(num_blocks - 6, num_blocks, dtype=np.int32)
    cache.release(row2)
    cache.release(row3)
    bt = np.full((1, max_blocks), -1, np.int32)
    bt[0, :6] = fresh_blocks
    kf, vf = _pool(w, num_blocks)
    kv = molt.KVCache(kf, vf, dev(torch.from_numpy(bt)), dev(torch.zeros(1, dtype=torch.int32)))
    full = molt.prefill(model, kv, dev(torch.from_numpy(turn2[None, :].copy())),
                        dev(torch.tensor([len(turn2)], dtype=torch.int32)))
    torch.cuda.synchronize()
    lf = full["logits"].cpu().numpy()[0]
    lo, _, _ = _oracle_fresh(w, layers, head, turn2[None, :], np.array([len(turn2)]), bt, num_blocks)
    tol = 1e-4 if w.dtype == "f32" else 2e-2
    e1, e2 = max_abs(l2, lf), max_abs(l2, lo[0])
    print(f"{wname}: re-prefill vs fresh GPU prefill {e1:.3e}, vs oracle {e2:.3e}", flush=True)
    assert e1 <= tol and e2 <= tol
