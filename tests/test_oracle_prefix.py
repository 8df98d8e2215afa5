"""Pins of the oracle's prefix cache and prefill window (oracle/prefix.py):

* a hand-worked session sequence on an 8-block pool (a first prompt, its extension reusing
  two full blocks, a rewritten history missing, a short prefix reusing one block, a
  16-token prompt that may not reuse its only block, an exhausted pool) and LRU eviction on
  a 4-block pool;
* invariants over random session workloads (shared base prompts, extensions, rewrites):
  reference counts equal the live rows holding a block, free and referenced blocks are
  disjoint, every block is free, referenced or evictable, hits reproduce the requested
  tokens, at least one position is always computed;
* prefill: a window split at a block boundary (prefix cached by the first window, the rest
  re-prefilled at context m) gives the same last-row logits and cache contents as one
  window over the whole prompt, and a window's last-row logits equal the sequential
  one-token decode's.
"""
import numpy as np
import pytest

import workloads
from oracle import attention, model
from oracle.prefix import BS, BlockCache, prefill_logits


def test_hand_worked_sessions():
    c = BlockCache(8)
    A = list(range(100, 140))                                  # 40 tokens
    row, hit = c.acquire(A, 40)
    assert (row, hit) == ([0, 1, 2], 0)
    c.commit(A, 40, row)                                       # 2 full blocks cached
    c.release(row)                                             # 2 freed, then 1, 0 evictable
    assert c.free == {2, 3, 4, 5, 6, 7} and c.lru == [1, 0]
    B = A + list(range(500, 510))                              # the session grows to 50
    rowB, hit = c.acquire(B, 50)
    assert (rowB, hit) == ([0, 1, 2, 3], 32) and c.lru == []
    Cc = list(A)
    Cc[5] = 9999                                               # rewritten history: no hit
    rowC, hit = c.acquire(Cc, 40)
    assert (rowC, hit) == ([4, 5, 6], 0)
    rowD, hit = c.acquire(A[:20], 20)                          # one full block of A
    assert (rowD, hit) == ([0, 7], 16) and c.ref[0] == 2
    assert c.acquire(A[:16], 16) is None                       # its only block must be computed
    assert c.ref[0] == 2 and not c.free                        # the failed acquire undid itself


def test_lru_eviction():
    c = BlockCache(4)
    A = list(range(32))
    row, _ = c.acquire(A, 32)
    c.commit(A, 32, row)
    c.release(row)
    assert c.lru == [1, 0]
    X = list(range(1000, 1048))
    rowX, hit = c.acquire(X, 48)                               # 2 free, then evict block 1
    assert (rowX, hit) == ([2, 3, 1], 0) and c.evictions == 1
    c.release(rowX)
    row2, hit = c.acquire(A + [7], 33)                         # A[:16] survived, A[:32] did not
    assert hit == 16 and row2[0] == 0


def test_failed_acquire_evicts_nothing():
    """A request larger than the free plus evictable blocks fails without dropping any
    cached prefix: on a 4-block pool holding 2 cached unreferenced blocks, an 80-token
    prompt needs 5 blocks; afterwards both entries, the free set and the eviction count
    are as before, and the cached prefix still hits."""
    c = BlockCache(4)
    A = list(range(32))
    row, _ = c.acquire(A, 32)
    c.commit(A, 32, row)
    c.release(row)
    before = (dict(c.block_of), set(c.free), list(c.lru), c.evictions)
    assert c.acquire(list(range(1000, 1080)), 80) is None
    assert (dict(c.block_of), set(c.free), list(c.lru), c.evictions) == before
    assert c.acquire(A + [7], 33)[1] == 32
    # with one of the two cached blocks referenced by a live row, 3 free + evictable
    # blocks cannot hold a 64-token prompt either; the hit block's recency alone moves
    c = BlockCache(4)
    c.commit(A, 32, c.acquire(A, 32)[0])
    c.release([0, 1])
    live, hit = c.acquire(A[:20], 20)
    assert (live, hit) == ([0, 2], 16)
    before = (dict(c.block_of), set(c.free), c.evictions)
    assert c.acquire(A[:16] + list(range(500, 548)), 64) is None
    assert (dict(c.block_of), set(c.free), c.evictions) == before and c.ref[0] == 1


def test_random_sessions_keep_invariants():
    rng = np.random.default_rng(0)
    c = BlockCache(48)
    bases = [list(rng.integers(0, 50, int(rng.integers(10, 70)))) for _ in range(4)]
    live = []                                                  # (tokens, n, row)
    for step in range(400):
        act = rng.integers(0, 3)
        if act < 2 or not live:
            toks = list(bases[rng.integers(0, 4)])
            if rng.random() < 0.5:
                toks = toks[:int(rng.integers(1, len(toks) + 1))]
            toks += list(rng.integers(0, 50, int(rng.integers(0, 40))))
            if rng.random() < 0.1 and toks:
                toks[int(rng.integers(0, len(toks)))] = 77     # a rewritten history
            n = len(toks)
            if n == 0:
                continue
            r = c.acquire(toks, n, extra=int(rng.integers(0, 8)))
            if r is None:
                continue
            row, hit = r
            assert hit % BS == 0 and hit <= n - 1
            for i in range(hit // BS):                         # hits reproduce the tokens
                assert c.key_of[row[i]] == tuple(toks[:BS * (i + 1)])
            c.commit(toks, n, row)
            live.append((toks, n, row))
        else:
            toks, n, row = live.pop(int(rng.integers(0, len(live))))
            c.release(row)
        refs = np.zeros(c.n, int)
        for _, _, row in live:
            for b in row:
                refs[b] += 1
        assert list(refs) == c.ref
        held = {b for b in range(c.n) if c.ref[b] > 0}
        assert not (held & c.free)
        assert set(c.lru) == {b for b in c.key_of if c.ref[b] == 0}
        assert len(c.free) + len(held | set(c.key_of)) == c.n
        assert set(c.key_of) == set(c.block_of.values())


def _tiny(seed=0, batch=2, n=40, layers=2):
    w = workloads.TINY_FP32.scaled(batch=batch, k=n - 1, ctx_lo=0, ctx_hi=0, n_layers=layers)
    cfg = dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=w.n_layers, n_q_heads=w.n_q_heads,
               n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps,
               rope_theta=w.rope_theta, block_size=16)
    layout = workloads.make_kv_layout(w, seed)
    lw = [{k_: (None if v is None else v.numpy()) for k_, v in
           workloads.make_layer_weights(w, seed, l).items()} for l in range(w.n_layers)]
    head = {k_: v.numpy() for k_, v in workloads.make_head_weights(w, seed).items()}
    caches = [tuple(model.widen_cache(c.numpy(), w.dtype) for c in workloads.empty_kv_cache(w, layout))
              for _ in range(w.n_layers)]
    return w, cfg, layout, lw, head, caches


@pytest.mark.parametrize("m", [16, 32])
def test_split_window_equals_whole(m):
    n = 40
    w, cfg, layout, lw, head, caches = _tiny(n=n)
    g = np.random.default_rng(1)
    toks = g.integers(0, w.vocab, (w.batch, n))
    lens = np.full(w.batch, n)
    ctx0 = np.zeros(w.batch, np.int64)
    c1 = [(a.copy(), b.copy()) for a, b in caches]
    whole, _, _ = prefill_logits(toks, lens, lambda l: lw[l], head, c1, layout.block_tables, ctx0, cfg)
    c2 = [(a.copy(), b.copy()) for a, b in caches]
    prefill_logits(toks[:, :m], np.full(w.batch, m), lambda l: lw[l], head, c2, layout.block_tables, ctx0, cfg)
    part, _, _ = prefill_logits(toks[:, m:], np.full(w.batch, n - m), lambda l: lw[l], head, c2,
                                layout.block_tables, ctx0 + m, cfg)
    np.testing.assert_allclose(part, whole, rtol=1e-5, atol=1e-6)
    for l in range(w.n_layers):
        for b in range(w.batch):
            K1, V1 = attention.gather_kv(c1[l][0], c1[l][1], layout.block_tables[b], n, 0)
            K2, V2 = attention.gather_kv(c2[l][0], c2[l][1], layout.block_tables[b], n, 0)
            np.testing.assert_allclose(K2, K1, rtol=1e-5, atol=1e-6)
            np.testing.assert_allclose(V2, V1, rtol=1e-5, atol=1e-6)


def test_window_last_row_equals_sequential_decode():
    n = 20
    w, cfg, layout, lw, head, caches = _tiny(n=n, batch=2, layers=1)
    g = np.random.default_rng(2)
    toks = g.integers(0, w.vocab, (w.batch, n))
    lens = np.array([n, 13])                                    # a ragged second sequence
    ctx0 = np.zeros(w.batch, np.int64)
    c1 = [(a.copy(), b.copy()) for a, b in caches]
    win, _, _ = prefill_logits(toks, lens, lambda l: lw[l], head, c1, layout.block_tables, ctx0, cfg)
    c2 = [(a.copy(), b.copy()) for a, b in caches]
    for j in range(n):
        last, _, _ = prefill_logits(toks[:, j:j + 1], np.ones(w.batch, int), lambda l: lw[l], head, c2,
                                    layout.block_tables, ctx0 + j, cfg)
        for b in range(w.batch):
            if j == lens[b] - 1:
                np.testing.assert_allclose(win[b], last[b], rtol=1e-5, atol=1e-6)
