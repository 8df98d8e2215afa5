"""Pins of the oracle's attention, RoPE, RMSNorm and whole verify step: the paged
routine against an independent dense causal routine and torch's SDPA, one key,
identical keys, block-table shuffles, rotation invariants, unit RMS, and the
verify-equals-sequential-decode and prefill-equals-verify equivalences that fix
causal masking, KV writes and positions."""
import numpy as np
import torch

import workloads
from oracle import attention, model, moe


def _paged_setup(B=3, k=2, Hq=4, Hkv=2, D=16, ctx_lo=5, ctx_hi=40, seed=0, shuffle=True):
    rng = np.random.default_rng(seed)
    ctx = rng.integers(ctx_lo, ctx_hi + 1, B)
    need = (ctx + k + 1 + 15) // 16
    nb = int(need.sum())
    perm = rng.permutation(nb) if shuffle else np.arange(nb)
    bt = np.full((B, need.max()), -1)
    pos = 0
    for b in range(B):
        bt[b, :need[b]] = perm[pos:pos + need[b]]
        pos += need[b]
    kc = rng.normal(size=(nb, Hkv, 16, D))
    vc = rng.normal(size=(nb, Hkv, D, 16))
    q = rng.normal(size=(B * (k + 1), Hq, D))
    return q, kc, vc, bt, ctx


def test_paged_matches_dense_and_sdpa():
    B, k, Hq, Hkv, D = 3, 2, 4, 2, 16
    q, kc, vc, bt, ctx = _paged_setup(B, k, Hq, Hkv, D)
    out = attention.paged_attention(q, kc, vc, bt, ctx, k)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            K, V = attention.gather_kv(kc, vc, bt[b], ctx[b] + k + 1, h)
            qb = q[b * (k + 1):(b + 1) * (k + 1), h * G:(h + 1) * G]
            dense = attention.dense_causal_attention(qb, K, V, int(ctx[b]), k)
            np.testing.assert_allclose(out[b * (k + 1):(b + 1) * (k + 1), h * G:(h + 1) * G], dense, atol=1e-12)
            n = ctx[b] + k + 1
            mask = torch.from_numpy(np.arange(n)[None, :] <= (ctx[b] + np.arange(k + 1))[:, None])
            for g in range(G):
                ref = torch.nn.functional.scaled_dot_product_attention(
                    torch.from_numpy(qb[:, g])[None], torch.from_numpy(K)[None],
                    torch.from_numpy(V)[None], attn_mask=mask[None])
                np.testing.assert_allclose(dense[:, g], ref[0].numpy(), atol=1e-10)


def test_shuffled_blocks_equal_contiguous():
    a = _paged_setup(seed=3, shuffle=True)
    q, kc, vc, bt, ctx = a
    out1 = attention.paged_attention(q, kc, vc, bt, ctx, 2)
    # move every block to a contiguous layout and re-run
    order = [blk for b in range(len(ctx)) for blk in bt[b] if blk >= 0]
    kc2, vc2 = kc[order], vc[order]
    bt2 = np.full_like(bt, -1)
    pos = 0
    for b in range(len(ctx)):
        n = int((bt[b] >= 0).sum())
        bt2[b, :n] = np.arange(pos, pos + n)
        pos += n
    out2 = attention.paged_attention(q, kc2, vc2, bt2, ctx, 2)
    np.testing.assert_array_equal(out1, out2)


def test_single_key_and_identical_keys():
    rng = np.random.default_rng(4)
    q = rng.normal(size=(3, 8))
    K = rng.normal(size=(1, 8))
    V = rng.normal(size=(1, 8))
    np.testing.assert_allclose(attention.attend(q, K, V), np.repeat(V, 3, axis=0), atol=1e-15)
    K = np.repeat(rng.normal(size=(1, 8)), 10, axis=0)
    V = rng.normal(size=(10, 8))
    np.testing.assert_allclose(attention.attend(q, K, V), np.repeat(V.mean(0, keepdims=True), 3, 0), atol=1e-14)


def test_rope_invariants():
    rng = np.random.default_rng(5)
    D = 64
    x = rng.normal(size=(6, 1, D))
    pos = np.array([0, 1, 7, 100, 4096, 65535])
    y = attention.apply_rope(x, pos, 1e6)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    np.testing.assert_allclose(y[0], x[0], atol=0)                    # position 0: identity
    qv, kv = rng.normal(size=(1, 1, D)), rng.normal(size=(1, 1, D))
    def dot(m, n):
        return float((attention.apply_rope(qv, [m], 1e4) * attention.apply_rope(kv, [n], 1e4)).sum())
    np.testing.assert_allclose(dot(10, 3), dot(107, 100), rtol=1e-9)  # depends on m - n only
    np.testing.assert_allclose(dot(5000, 4990), dot(15, 5), rtol=1e-9)


def test_rope_hand_worked():
    """Worked rotations that fix the frequency schedule, the pairing and the direction
    (the decoder's rotary embedding: rotate-half pairs (i, i + D/2), inverse frequency
    theta^(-2i/D), angle = position * inverse frequency).

    D = 4, theta = 100, position 2: inverse frequencies 100^0 = 1 and 100^(-1/2) = 0.1, so
    pair (x0, x2) turns by 2 rad and pair (x1, x3) by 0.2 rad:
        cos 2 = -0.4161468365471424   sin 2 = 0.9092974268256817
        cos .2 = 0.9800665778412416   sin .2 = 0.19866933079506122
    x = (1, 2, 3, 4):
        y0 = 1 cos 2 - 3 sin 2   = -3.1440391170241875
        y2 = 3 cos 2 + 1 sin 2   = -0.33914308281574557
        y1 = 2 cos .2 - 4 sin .2 =  1.1654558325022384
        y3 = 4 cos .2 + 2 sin .2 =  4.317604972955089
    An exponent of -i/D (0.316 for the second pair), interleaved pairs (x0, x1), or the
    opposite rotation (y0 = cos 2 + 3 sin 2) each give different values.

    D = 8, theta = 1e6 (the workloads' base), position 3: inverse frequencies 1,
    10^-1.5, 10^-3, 10^-4.5; angles 3, 0.09486832980505137, 0.003, 9.486832980505139e-05:
        cos = -0.9899924966004454, 0.9955033739876628, 0.999995500003375, 0.9999999955
        sin =  0.1411200080598672, 0.0947260913327461, 0.002999995500002025,
               9.48683296627489e-05
    x = (1, -2, .5, 3, -1.5, 2.5, 4, -.25) rotates pairwise to the values below."""
    y = attention.apply_rope(np.array([[[1.0, 2.0, 3.0, 4.0]]]), [2], 100.0)[0, 0]
    np.testing.assert_allclose(y, [-3.1440391170241875, 1.1654558325022384,
                                   -0.33914308281574557, 4.317604972955089], rtol=0, atol=1e-14)
    x = np.array([[[1.0, -2.0, 0.5, 3.0, -1.5, 2.5, 4.0, -0.25]]])
    y = attention.apply_rope(x, [3], 1e6)[0, 0]
    np.testing.assert_allclose(y, [-0.7783124845106446, -2.2278219763071907, 0.4879977680016794,
                                   3.0000237035824155, 1.6261087529605354, 2.2993062523036647,
                                   4.001481997763501, -0.24971539388601174], rtol=0, atol=1e-14)
    # the angle table itself: position * theta^(-2i/D)
    np.testing.assert_allclose(attention.rope_angles([3], 8, 1e6)[0],
                               [3.0, 0.09486832980505137, 0.003, 9.486832980505139e-05],
                               rtol=1e-15, atol=0)


def test_rmsnorm_hand_worked_eps():
    """The epsilon sits inside the square root, added to the mean square; gains multiply
    element-wise. x = (2, -2, 2, -2): mean square 4; with eps = 5 the scale is 1/sqrt(9) =
    1/3 (eps outside the root would give 1/7, eps added to each square before the mean the
    same 1/3 only because it is added once per element), so with g = (1, 2, 3, 4)
    y = (2/3, -4/3, 2, -8/3). x = (3, 4, 0, 0), eps = 0.25, g = 1: mean square 25/4, scale
    1/sqrt(6.5); y0 = 3/sqrt(6.5) = 1.1766968108291043."""
    y = model.rmsnorm(np.array([[2.0, -2.0, 2.0, -2.0]]), np.array([1.0, 2.0, 3.0, 4.0]), 5.0)
    np.testing.assert_allclose(y[0], [2 / 3, -4 / 3, 2.0, -8 / 3], rtol=0, atol=1e-15)
    y = model.rmsnorm(np.array([[3.0, 4.0, 0.0, 0.0]]), np.ones(4), 0.25)
    np.testing.assert_allclose(y[0], [1.1766968108291043, 1.5689290811054724, 0.0, 0.0],
                               rtol=0, atol=1e-15)


def test_rmsnorm_unit_rms():
    x = np.random.default_rng(6).normal(size=(10, 256)) * 7
    y = model.rmsnorm(x, np.ones(256), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(axis=1)), 1.0, rtol=1e-12)


# -------------------------------------------------------------- whole step

def _tiny(seed=0, batch=2, k=3, ctx=(20, 37), layers=2):
    w = workloads.TINY_FP32.scaled(batch=batch, k=k, ctx_lo=ctx[0], ctx_hi=ctx[1], n_layers=layers)
    cfg = dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=w.n_layers, n_q_heads=w.n_q_heads,
               n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps,
               rope_theta=w.rope_theta, block_size=16)
    layout = workloads.make_kv_layout(w, seed)
    layers_w = [{k_: (None if v is None else v.numpy()) for k_, v in
                 workloads.make_layer_weights(w, seed, l).items()} for l in range(w.n_layers)]
    head = {k_: v.numpy() for k_, v in workloads.make_head_weights(w, seed).items()}
    caches = [tuple(model.widen_cache(c.numpy(), w.dtype) for c in workloads.empty_kv_cache(w, layout))
              for _ in range(w.n_layers)]
    prompts = workloads.make_prompts(w, layout, seed)
    model.prefill(prompts, lambda l: layers_w[l], head, caches, layout.block_tables, cfg)
    return w, cfg, layout, layers_w, head, caches, prompts


def _copy(caches):
    return [(a.copy(), b.copy()) for a, b in caches]


def test_verify_equals_sequential_decode():
    w, cfg, layout, lw, head, caches, _ = _tiny()
    toks = workloads.make_step_tokens(w, 1)
    B, k = w.batch, w.k
    u = np.full((B, k + 1), 0.5, np.float32)
    r = model.verify_step(toks, lambda l: lw[l], head, _copy(caches), layout.block_tables,
                          layout.context_lens, cfg, None, u)
    seq_caches = _copy(caches)
    for j in range(k + 1):
        ctx_j = layout.context_lens + j
        rj = model.verify_step(toks[:, j:j + 1], lambda l: lw[l], head, seq_caches,
                               layout.block_tables, ctx_j, cfg, None, u[:, :1])
        np.testing.assert_allclose(r["logits"][:, j], rj["logits"][:, 0], atol=2e-6, rtol=1e-5)


def test_prefill_writes_same_kv_as_verify():
    w, cfg, layout, lw, head, caches, prompts = _tiny(batch=2, k=2)
    toks = workloads.make_step_tokens(w, 2)
    c1 = _copy(caches)
    model.verify_step(toks, lambda l: lw[l], head, c1, layout.block_tables, layout.context_lens,
                      cfg, None, np.full((w.batch, w.k + 1), 0.5, np.float32))
    c2 = [tuple(np.zeros_like(a) for a in c) for c in caches]
    longer = [np.concatenate([p, t]) for p, t in zip(prompts, toks)]
    model.prefill(longer, lambda l: lw[l], head, c2, layout.block_tables, cfg)
    for b in range(w.batch):
        n = layout.context_lens[b] + w.k + 1
        for l in range(w.n_layers):
            K1, V1 = attention.gather_kv(c1[l][0], c1[l][1], layout.block_tables[b], n, 0)
            K2, V2 = attention.gather_kv(c2[l][0], c2[l][1], layout.block_tables[b], n, 0)
            np.testing.assert_allclose(K1, K2, atol=1e-6, rtol=1e-5)
            np.testing.assert_allclose(V1, V2, atol=1e-6, rtol=1e-5)


def test_route_records_shape():
    w, cfg, layout, lw, head, caches, _ = _tiny(batch=2, k=1, layers=1)
    toks = workloads.make_step_tokens(w, 3)
    r = model.verify_step(toks, lambda l: lw[l], head, _copy(caches), layout.block_tables,
                          layout.context_lens, cfg, None, np.full((2, 2), 0.5, np.float32))
    assert r["routes"].shape == (1, 4, w.top_k)
    assert ((r["routes"] >= 0) & (r["routes"] < w.n_experts)).all()
