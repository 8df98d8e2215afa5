"""The allocation-free accept (molt_spec_accept_noalloc) against molt_spec_accept with a
workspace, through the C ABI on the same seeded inputs: emitted tokens, accepted lengths
and log-probs identical bit for bit, on consecutive calls that share the library's scratch
array, each call smaller than the one before (151936-token vocabulary at B = 128, k = 4
with q; a ragged 8193-token vocabulary at B = 37, k = 3, greedy; a 16-token vocabulary at
B = 5, k = 7), and no device memory taken by the call itself."""
import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


def _inputs(B, k, V, seed, greedy):
    logits = workloads.make_logits(B, k + 1, V, seed, std=2.0)
    q = None if greedy else workloads.make_softmax_q(B, k, V, seed + 1)
    g = np.random.Generator(np.random.Philox(seed))
    drafts = g.integers(0, V, (B, k)).astype(np.int32)
    drafts[::2] = logits[::2, :k].numpy().argmax(axis=-1)     # some sequences run long
    u = workloads.make_uniforms(B, k, seed + 2)
    d = lambda t: None if t is None else t.cuda().contiguous()
    return d(logits), d(q), d(torch.from_numpy(drafts)) if k > 0 else None, d(u)


def _same(a, b):
    a, b = a.cpu(), b.cpu()
    if a.dtype == torch.float32:
        return torch.equal(torch.isnan(a), torch.isnan(b)) and torch.equal(
            torch.nan_to_num(a, nan=0.0), torch.nan_to_num(b, nan=0.0))
    return torch.equal(a, b)


def _case(lib, B, k, V, greedy, seed):
    logits, q, drafts, u = _inputs(B, k, V, seed, greedy)
    want = lib.spec_accept(logits, drafts, u, q)
    out = (torch.full((B, k + 1), -7, dtype=torch.int32, device="cuda"),
           torch.full((B,), -7, dtype=torch.int32, device="cuda"),
           torch.zeros(B, k + 1, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    lib.spec_accept_noalloc(logits, drafts, u, q, out=out)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    for name, a, b in zip(("tokens", "n_accepted", "logprobs"), out, want):
        assert _same(a, b), (B, k, V, name)
    n = out[1].cpu().numpy()
    assert ((n >= 0) & (n <= k)).all()


def test_noalloc_matches_workspace_entry_point(lib):
    for B, k, V, greedy, seed in [(128, 4, 151936, False, 11), (37, 3, 8193, True, 12),
                                  (5, 7, 16, False, 13)]:
        print(f"case B={B} k={k} V={V} greedy={greedy}", flush=True)
        _case(lib, B, k, V, greedy, seed)
