"""GPU parity of molt_paged_attention (MFMA multi-query decode attention over shuffled
paged blocks with split-KV merge) against the oracle's float64 paged attention: bf16
within 1e-2 max-abs (outputs are rounded to bf16), f32 within 1e-5; ragged contexts,
one-key and empty-context edges, k = 0, 8 drafts (72 query rows, also ragged with splits),
9 drafts with many splits and 11 (96 rows) on the 8-wavefront tiles, head dim 64, many
splits; prefill
windows longer than one 128-row query
tile (64, 41, 101 and 256 positions: several tiles, a partial last tile, tiles with splits,
an empty cached context); shuffled and contiguous block tables give bit-identical
outputs."""
import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oattn, model as omodel
from helpers import dev, host, max_abs

pytestmark = pytest.mark.gpu


def _setup(B, k, Hq, Hkv, D, ctx_lo, ctx_hi, dtype, seed):
    w = workloads.LAYER_BF16.scaled(batch=B, k=k, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D,
                                    ctx_lo=ctx_lo, ctx_hi=ctx_hi, dtype=dtype)
    layout = workloads.make_kv_layout(w, seed)
    kc, vc = workloads.make_kv_cache(w, layout, seed, 0)
    T = B * (k + 1)
    q = torch.randn(T, Hq, D, generator=workloads.rng(seed, "q")).to(workloads.torch_dtype(dtype))
    return w, layout, kc, vc, q


def _oracle(w, layout, kc, vc, q):
    out = oattn.paged_attention(omodel.widen_cache(host(q), w.dtype), omodel.widen_cache(host(kc), w.dtype),
                                omodel.widen_cache(host(vc), w.dtype), layout.block_tables,
                                layout.context_lens, w.k)
    return out.reshape(out.shape[0], -1)


def _gpu(molt, w, layout, kc, vc, q, bt=None):
    bt = layout.block_tables if bt is None else bt
    out = molt.paged_attention(dev(q), dev(kc), dev(vc), dev(torch.from_numpy(bt)),
                               dev(torch.from_numpy(layout.context_lens)), w.k)
    return out.float().cpu().numpy()


@pytest.mark.parametrize("B,k,Hq,Hkv,D,lo,hi", [
    (3, 4, 32, 4, 128, 1, 3000),        # ragged, several splits
    (2, 8, 32, 4, 128, 900, 2100),      # 72 query rows
    (3, 8, 32, 4, 128, 1, 3000),        # 72 rows, ragged, splits
    (1, 9, 32, 4, 128, 9000, 9000),     # 80 rows, many splits
    (2, 11, 32, 4, 128, 300, 2500),     # 96 rows
    (4, 0, 32, 4, 128, 0, 40),          # plain decode, empty context allowed
    (2, 3, 8, 2, 64, 200, 1500),        # head dim 64
    (1, 4, 32, 4, 128, 9000, 9000),     # 9 splits
    (2, 63, 32, 4, 128, 0, 300),        # prefill window: 8 query tiles of 64 rows, empty context allowed
    (3, 40, 16, 4, 128, 10, 700),       # G = 4: tiles of 16 positions, partial last tile
    (1, 255, 32, 4, 128, 2000, 2000),   # 32 query tiles x 4 splits
    (2, 100, 8, 2, 64, 50, 400),        # head dim 64, 7 tiles of 16 positions
    (2, 5, 64, 1, 128, 30, 500),        # G = 64: one position per 64-row tile
    (1, 3, 128, 1, 128, 100, 100),      # G = 128: one position per 128-row tile
])
def test_bf16_parity(molt_lib, B, k, Hq, Hkv, D, lo, hi):
    print(f"case B={B} k={k} Hq={Hq} Hkv={Hkv} D={D} ctx=[{lo},{hi}]", flush=True)
    w, layout, kc, vc, q = _setup(B, k, Hq, Hkv, D, lo, hi, "bf16", 100 + B + k)
    g = _gpu(molt_lib, w, layout, kc, vc, q)
    o = _oracle(w, layout, kc, vc, q)
    err = max_abs(g, o)
    print(f"max |out - oracle| = {err:.3e}", flush=True)
    assert err <= 1e-2


@pytest.mark.parametrize("B,k,lo,hi", [(4, 3, 64, 128), (2, 40, 0, 100)])
def test_f32_parity(molt_lib, B, k, lo, hi):
    w, layout, kc, vc, q = _setup(B, k, 4, 4, 64, lo, hi, "f32", 7)
    err = max_abs(_gpu(molt_lib, w, layout, kc, vc, q), _oracle(w, layout, kc, vc, q))
    assert err <= 1e-5, err


def test_shuffled_equals_contiguous(molt_lib):
    w, layout, kc, vc, q = _setup(3, 4, 32, 4, 128, 500, 2500, "bf16", 8)
    a = _gpu(molt_lib, w, layout, kc, vc, q)
    # relocate every sequence's blocks to a contiguous range
    order = [blk for b in range(w.batch) for blk in layout.block_tables[b] if blk >= 0]
    kc2, vc2 = kc[order].contiguous(), vc[order].contiguous()
    bt2 = np.full_like(layout.block_tables, -1)
    pos = 0
    for b in range(w.batch):
        n = int((layout.block_tables[b] >= 0).sum())
        bt2[b, :n] = np.arange(pos, pos + n)
        pos += n
    b2 = _gpu(molt_lib, w, layout, kc2, vc2, q, bt2)
    np.testing.assert_array_equal(a, b2)
