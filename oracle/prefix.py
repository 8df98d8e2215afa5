"""Paged prefill with session-consistent prefix caching (test infrastructure, like the rest
of this package).

The rollout engines run with prefix caching (Sec. 4.1: prefix caching enters through the
serving engine; Sec. 5.3: every engine uses it), and an agent's growing context is
re-prefilled from the cache: session-consistent prefix caching measures a 0.05 s cache-hit
re-prefill (Sec. 5.4, table of scaling controls). Session consistency: a request reuses
cached keys/values only for a prefix whose token IDs are exactly the ones recorded (a
rewritten history or template prefix misses, Sec. 4.2). The paper gives no mechanism; it
is read here as the paged block cache of its serving engine (vLLM):

Block cache over a pool of `num_blocks` physical blocks of 16 positions.
  * A full block is identified by the whole token prefix it ends (its tokens and every
    token before them). Cached blocks form a tree: a block's cache entry lives only while
    its parent's does (dropping an entry drops the entries of every block cached under it).
  * acquire(tokens[0..n), extra): walks the longest chain of cached full blocks matching
    the prefix, at most floor((n - 1) / 16) of them (at least one position is computed, so
    the last position's logits exist); each hit block gains a reference. The sequence then
    needs ceil((n + extra) / 16) blocks in all; each missing one takes the lowest free block
    id, or, with none free, the least recently released cached block with no references is
    evicted (its entry and the entries under it dropped, their blocks freed) and the lowest
    free id taken. Returns the block table row and n_cached = 16 * hits. When the free
    and evictable blocks together cannot cover the request, nothing is evicted and the
    request fails (only the hit blocks' recency changes).
  * commit(tokens[0..n), row): every full block of the row (16 (i+1) <= n) whose prefix is
    not cached yet becomes the cached block of that prefix; a prefix already cached under
    another block keeps that block.
  * release(row): each block loses a reference, from the last block to the first; a block
    left without references becomes evictable (most recent last) if cached, else free.
Prefill of a window: the verify step's forward over tokens[b, 0..n) at positions c_b + j
(rows past lens[b] are padding: computed, their cache slots later overwritten), logits of
row lens[b] - 1.
"""
import numpy as np

from . import model

BS = 16


class BlockCache:
    def __init__(self, num_blocks):
        self.n = num_blocks
        self.ref = [0] * num_blocks
        self.key_of = {}        # block -> prefix tuple it caches
        self.block_of = {}      # prefix tuple -> block
        self.free = set(range(num_blocks))
        self.lru = []           # cached blocks without references, least recent first
        self.evictions = 0

    def _lookup(self, tokens, n):
        hits = []
        for i in range((n - 1) // BS):
            b = self.block_of.get(tuple(tokens[:BS * (i + 1)]))
            if b is None:
                break
            hits.append(b)
        return hits

    def _drop(self, key):
        """Drop the entry of `key` and of every prefix extending it."""
        for k2 in [k for k in self.block_of if len(k) >= len(key) and k[:len(key)] == key]:
            b = self.block_of.pop(k2)
            del self.key_of[b]
            if self.ref[b] == 0:
                self.lru.remove(b)
                self.free.add(b)

    def acquire(self, tokens, n, extra=0, max_blocks=None):
        tokens = [int(t) for t in tokens[:n]]
        hits = self._lookup(tokens, n)
        need = (n + extra + BS - 1) // BS
        if max_blocks is not None and need > max_blocks:
            return None
        for b in hits:
            if self.ref[b] == 0:
                self.lru.remove(b)
            self.ref[b] += 1
        row = list(hits)
        if need - len(hits) > len(self.free) + len(self.lru):
            self.release(row)              # the pool cannot hold it: undo, evict nothing
            return None
        while len(row) < need:
            if not self.free:
                self.evictions += 1
                self._drop(self.key_of[self.lru[0]])
            b = min(self.free)
            self.free.remove(b)
            self.ref[b] += 1
            row.append(b)
        return row, BS * len(hits)

    def commit(self, tokens, n, row):
        tokens = [int(t) for t in tokens[:n]]
        for i in range(n // BS):
            key = tuple(tokens[:BS * (i + 1)])
            if key in self.block_of or row[i] in self.key_of:
                continue
            self.block_of[key] = row[i]
            self.key_of[row[i]] = key

    def release(self, row):
        for b in reversed(row):
            self.ref[b] -= 1
            if self.ref[b] == 0:
                if b in self.key_of:
                    self.lru.append(b)
                else:
                    self.free.add(b)


def prefill_logits(tokens, lens, get_layer, head, caches, block_tables, context_lens, cfg):
    """tokens [B, n] (row j at position context_lens[b] + j; rows past lens[b] padding).
    Returns (logits of row lens[b] - 1 [B, V] f32, final residual rows [B, d] f32, the
    whole final residual stream [B * n, d])."""
    tokens = np.asarray(tokens)
    B, n = tokens.shape
    x = model.embed(tokens, head, cfg)
    x, _ = model.decoder_forward(x, get_layer, caches, block_tables, context_lens, n - 1, cfg)
    rows = np.arange(B) * n + np.asarray(lens) - 1
    return model.lm_logits(x[rows], head, cfg), x[rows], x
