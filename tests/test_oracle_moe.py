"""Pins of the oracle's routing, permutation and MoE layer: a library stable sort,
all-equal logits, K = E, signed zeros, permutation invariants, the E = K = 1
reduction to a dense SwiGLU written with torch, routing replay, weights summing to
one, and identical experts collapsing the weighted sum."""
import numpy as np
import torch

from oracle import codecs, moe, routing


def test_topk_matches_stable_sort_and_ties():
    rng = np.random.default_rng(0)
    T, E, K = 200, 32, 6
    g = np.round(rng.normal(size=(T, E)) * 4) / 4          # many exact ties
    g = g.astype(np.float32)
    ids, w, _, _ = routing.topk_route(g, K)
    ref = np.argsort(-g.astype(np.float64), axis=1, kind="stable")[:, :K]
    assert (ids == ref).all()
    np.testing.assert_allclose(w.sum(axis=1), 1.0, atol=1e-6)
    full = np.exp(g - g.max(axis=1, keepdims=True))
    sel = np.take_along_axis(full, ids, axis=1)
    np.testing.assert_allclose(w, sel / sel.sum(axis=1, keepdims=True), rtol=1e-6)


def test_topk_special_cases():
    g = np.zeros((3, 8), np.float32)
    ids, w, _, _ = routing.topk_route(g, 3)
    assert (ids == [0, 1, 2]).all()
    np.testing.assert_allclose(w, 1 / 3, rtol=1e-6)
    ids, _, _, _ = routing.topk_route(np.random.default_rng(1).normal(size=(4, 8)).astype(np.float32), 8)
    assert (np.sort(ids, axis=1) == np.arange(8)).all()
    g = np.array([[-0.0, 0.0, -1.0, 0.0]], np.float32)      # -0.0 ties +0.0: lower id first
    ids, _, _, _ = routing.topk_route(g, 2)
    assert ids.tolist() == [[0, 1]]


def test_permutation_invariants():
    rng = np.random.default_rng(2)
    T, E, K = 300, 16, 4
    ids = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    counts, offsets, perm, inv = routing.permute(ids, E)
    flat = ids.reshape(-1)
    assert counts.sum() == T * K and (np.diff(offsets) == counts).all() and offsets[0] == 0
    assert sorted(perm.tolist()) == list(range(T * K))
    assert (inv[perm] == np.arange(T * K)).all()
    assert (perm == np.argsort(flat, kind="stable")).all()       # library stable sort
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert (flat[seg] == e).all() and (np.diff(seg) > 0).all()


def _bf16(a):
    return codecs.f32_to_bf16_bits(np.asarray(a, np.float32))


def test_single_expert_is_dense_swiglu():
    rng = np.random.default_rng(3)
    T, d, F = 17, 64, 48
    y = codecs.round_bf16(rng.normal(size=(T, d)))
    wr = codecs.round_bf16(rng.normal(size=(1, d)) * 0.1)
    wgu = _bf16(rng.normal(size=(1, 2 * F, d)) * 0.1)
    wd = _bf16(rng.normal(size=(1, d, F)) * 0.1)
    r = moe.moe_layer(y, wr, wgu, wd, 1, "bf16", "bf16")
    Wgu = torch.from_numpy(codecs.bf16_bits_to_f32(wgu[0]).astype(np.float64))
    Wd = torch.from_numpy(codecs.bf16_bits_to_f32(wd[0]).astype(np.float64))
    yt = torch.from_numpy(y)
    h = torch.nn.functional.silu(yt @ Wgu[:F].T) * (yt @ Wgu[F:].T)
    h = torch.from_numpy(codecs.round_bf16(h.numpy()))
    ref = (h @ Wd.T).numpy()
    np.testing.assert_allclose(r["out"], ref, rtol=1e-6, atol=1e-6)
    assert (r["weights"] == 1.0).all()


def test_identical_experts_and_replay():
    rng = np.random.default_rng(4)
    T, d, F, E, K = 9, 32, 16, 6, 3
    y = rng.normal(size=(T, d)).astype(np.float32).astype(np.float64)
    wr = rng.normal(size=(E, d)).astype(np.float32).astype(np.float64)
    one_gu = rng.normal(size=(2 * F, d)).astype(np.float32) * 0.2
    one_d = rng.normal(size=(d, F)).astype(np.float32) * 0.2
    wgu = np.broadcast_to(one_gu, (E, 2 * F, d)).copy()
    wd = np.broadcast_to(one_d, (E, d, F)).copy()
    r = moe.moe_layer(y, wr, wgu, wd, K, "f32", "f32")
    dense = moe.dense_swiglu(y, one_gu, one_d, "f32")
    np.testing.assert_allclose(r["out"], dense, rtol=1e-5, atol=1e-6)   # weights sum to 1
    replay = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    r2 = moe.moe_layer(y, wr, wgu, wd, K, "f32", "f32", replay_ids=replay)
    assert (r2["ids"] == replay).all()
    np.testing.assert_allclose(r2["weights"].sum(axis=1), 1.0, atol=1e-6)


def test_fp8_expert_is_exact_dequantised_product():
    rng = np.random.default_rng(5)
    T, d, F = 5, 64, 32
    y = codecs.round_bf16(rng.normal(size=(T, d)))
    wr = codecs.round_bf16(rng.normal(size=(1, d)))
    wgu = rng.integers(0, 256, (1, 2 * F, d)).astype(np.uint8) & 0xBF
    wd = rng.integers(0, 256, (1, d, F)).astype(np.uint8) & 0xBF
    sgu = rng.random((1, 2 * F)).astype(np.float32) * 0.05
    sd = rng.random((1, d)).astype(np.float32) * 0.05
    r = moe.moe_layer(y, wr, wgu, wd, 1, "bf16", "fp8", sgu, sd)
    # independent evaluation from dequantised float tensors
    xq, sx = codecs.fp8_quantize_rows(y.astype(np.float32))
    x_deq = codecs.fp8_decode(xq) * sx[:, None]
    Wgu = codecs.fp8_decode(wgu[0]) * sgu[0][:, None]
    a = x_deq @ Wgu.T
    h = codecs.round_bf16(a[:, :F] / (1 + np.exp(-a[:, :F])) * a[:, F:])
    hq, sh = codecs.fp8_quantize_rows(h.astype(np.float32))
    out = (codecs.fp8_decode(hq) * sh[:, None]) @ (codecs.fp8_decode(wd[0]) * sd[0][:, None]).T
    np.testing.assert_allclose(r["out"], out, rtol=1e-5, atol=1e-7)
