"""The library's host-side prefix cache (molt_prefix_cache_*) against the oracle's block
cache (oracle/prefix.py), operation by operation on random session workloads: shared base
prompts, growing sessions, rewritten histories, small pools (eviction, exhaustion). Every
returned row and hit length, and the free / cached / referenced / evictable counts and
evictions after each operation, must be identical. Host code only: runs without a GPU."""
import numpy as np
import pytest

from oracle.prefix import BlockCache


@pytest.fixture(scope="module")
def molt():
    import paper_2607_21653_amd as m
    m.load()
    return m


def _counts(o):
    held = {b for b in range(o.n) if o.ref[b] > 0}
    return {"free": len(o.free), "cached": len(o.block_of), "referenced": len(held),
            "evictable": len(o.lru), "evictions": o.evictions}


@pytest.mark.parametrize("seed,pool", [(0, 64), (1, 24), (2, 12), (3, 200)])
def test_matches_oracle_step_by_step(molt, seed, pool):
    rng = np.random.default_rng(seed)
    o = BlockCache(pool)
    c = molt.PrefixCache(pool)
    bases = [list(rng.integers(0, 40, int(rng.integers(5, 90)))) for _ in range(5)]
    live = []
    for step in range(600):
        if rng.random() < 0.6 or not live:
            toks = list(bases[rng.integers(0, len(bases))])
            if rng.random() < 0.4:
                toks = toks[:int(rng.integers(1, len(toks) + 1))]
            toks += list(rng.integers(0, 40, int(rng.integers(0, 50))))
            if rng.random() < 0.1:
                toks[int(rng.integers(0, len(toks)))] = 99     # rewritten history
            extra = int(rng.integers(0, 20))
            mb = int(rng.integers(1, 12)) if rng.random() < 0.1 else None
            a = o.acquire(toks, len(toks), extra, max_blocks=mb)
            b = c.acquire(toks, extra_tokens=extra, max_blocks=mb)
            assert (a is None) == (b is None), (step, a, b)
            if a is not None:
                assert list(b[0]) == a[0] and b[1] == a[1], (step, a, b)
                # the session grows: commit what was prefilled
                o.commit(toks, len(toks), a[0])
                c.commit(toks, b[0])
                live.append(a[0])
                if rng.random() < 0.3:                       # a later turn extends it
                    bases.append(toks)
        else:
            row = live.pop(int(rng.integers(0, len(live))))
            o.release(row)
            c.release(np.array(row, np.int32))
        st = c.stats()
        assert {k: st[k] for k in _counts(o)} == _counts(o), step


def test_invalid_release_is_rejected(molt):
    c = molt.PrefixCache(4)
    row, _ = c.acquire(list(range(20)))
    c.release(row)
    with pytest.raises(molt.MoltError):
        c.release(row)                                      # no references left


def test_failed_acquire_changes_nothing(molt):
    """An acquire that the free and evictable blocks cannot cover returns CAPACITY before
    evicting: the cached entries, counts and evictions are unchanged and the prefix still
    hits (4-block pool, 2 cached blocks, an 80-token request)."""
    c = molt.PrefixCache(4)
    A = list(range(32))
    row, _ = c.acquire(A)
    c.commit(A, row)
    c.release(row)
    before = c.stats()
    assert c.acquire(list(range(1000, 1080))) is None
    after = c.stats()
    assert {k: after[k] for k in ("free", "cached", "referenced", "evictable", "evictions")} == \
        {k: before[k] for k in ("free", "cached", "referenced", "evictable", "evictions")}
    assert c.acquire(A + [7])[1] == 32
