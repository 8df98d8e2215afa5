"""Benchmark of the speculative-decoding verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload full_depth_bf16]

A step is one molt_verify_step call: the whole hot path (embedding, 48 decoder layers
with paged attention and top-8 routed MoE, final norm, LM head, fused accept/resample
sampler) over one batch of B = 128 sequences with k = 4 drafts at context 8192, vocab
151936, bf16, random-init weights of that shape and seeded synthetic inputs, all
resident in HBM before the timed region. Drafts follow the method's serving setup:
q_i = softmax(target row i-1 + N(0, 0.5^2)) and x_i ~ q_i, built with untimed passes.

Prints one JSON line: verified tokens/s (= B*(1+k) positions scored per second), the
roofline of the dominant kernel (paged attention, HBM-bound; its average launch time
measured with HIP events on the library's stream during the timed region), and the
CPU oracle timed on a bounded sample of the same workload (cpu_baseline).

The same line carries `configs`: the other seeded workloads measured beside it, each
with its own oracle baseline -- the tiny f32 decoder (the whole step), one bf16 layer
at the 35B-A3B-like shape (B 64, k 4, context 4096), that layer at long agent contexts
(B 16, context U[32768, 65536]) and with fp8 experts under Zipf(1.2) routing (B 256,
k 8, context 2048; plus a one-expert fp8 GEMM at that row count). A layer workload's
step is one molt_decoder_forward call over its B(1+k) positions; `--workload <name>`
measures one of them alone (profiling runs).
"""
import argparse
import json
import os
import sys
import time

import numpy as np
import torch

import workloads

HBM_PEAK_GBS = 8000.0
ATTN_EVERY = 8                 # attention launches bracketed in the timed region: every 8th
BF16_PEAK_TFLOPS = 2500.0


ROOT = os.path.dirname(os.path.abspath(__file__))


def attention_traffic():
    """Measured HBM bytes per attention launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, each
    scaled by a 1 GiB copy's reading), only while the kernel source is the one the counters
    were taken on; None otherwise."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "attention_traffic.json")))
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec["source_sha256"]:
        return None
    return int(1024 * (rec["fetch_kib_per_dispatch"] * rec["fetch_scale"] +
                       rec["write_kib_per_dispatch"] * rec["write_scale"]))


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attention_bytes(w, ctx):
    """Algorithmic bytes of one attention launch: every cached K and V vector of every
    (sequence, kv head) read once, q read once, the output written once."""
    e = 2 if w.dtype == "bf16" else 4
    kv = int(np.sum(ctx.astype(np.int64) + w.k + 1)) * w.n_kv_heads * w.head_dim * e * 2
    T = w.batch * (w.k + 1)
    qo = 2 * T * w.n_q_heads * w.head_dim * e
    return kv + qo


def layer_weight_bytes(w):
    """Weights one layer reads at this batch: every expert (T*K = 5120 pairs over 128
    experts leave none untouched), the attention projections and the router."""
    eb = 1 if w.expert_dtype == "fp8" else 2
    d, D = w.d_model, w.head_dim
    experts = w.n_experts * 3 * w.d_ff * d * eb
    dense = ((w.n_q_heads + 2 * w.n_kv_heads) * D * d + d * w.n_q_heads * D + w.n_experts * d) * 2
    return experts + dense


def step_bytes(w, ctx, samp_bytes):
    """Algorithmic HBM bytes of one whole verify step: every layer's attention (K/V, q, out)
    and weights, the LM head's weights and logits, the sampler's reads."""
    T = w.batch * (w.k + 1)
    return (w.n_layers * (attention_bytes(w, ctx) + layer_weight_bytes(w))
            + w.vocab * w.d_model * 2 + T * w.vocab * 4 + samp_bytes)


def sampler_roofline(w, molt, out, tokens, q, u, reps=20):
    """The standalone sampler (molt_spec_accept) on the step's own logits, drafts, q and
    uniforms, timed with HIP events on the library's stream after the timed region.
    Algorithmic bytes: every logit read once (softmax statistics), then per sequence one
    full row for the final draw and, when that draw is a residual against q (a rejection),
    one q row."""
    import torch
    B, k, V = w.batch, w.k, w.vocab
    logits = out["logits"]
    drafts = tokens[:, 1:].contiguous()
    ws = torch.empty(molt._lib.load().molt_spec_accept_workspace_size(B, k, V), dtype=torch.uint8,
                     device=logits.device)
    res = molt.spec_accept(logits, drafts, u, q, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        molt.spec_accept(logits, drafts, u, q, workspace=ws, out=res)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    rejected = int((res[1] < k).sum().item())
    nbytes = B * (k + 1) * V * 4 + B * V * 4 + rejected * V * 4
    return {"avg_ms": ms, "bytes": nbytes, "rejected": rejected}


def other_rooflines(w, groups, samp):
    """Fractions of roofline of the other headline kernels: the sampler (HBM), the expert
    GEMMs (HBM: every expert's weights read once per layer; also their raw MFMA rate) and the
    LM head (MFMA, bf16 dense peak)."""
    B, k, V, d = w.batch, w.k, w.vocab, w.d_model
    T = B * (k + 1)
    out = {}
    a = samp["bytes"] / (samp["avg_ms"] / 1e3) / 1e9
    out["sampler"] = {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                      "frac": round(a / HBM_PEAK_GBS, 4), "avg_launch_ms": round(samp["avg_ms"], 4),
                      "algorithmic_bytes_per_launch": samp["bytes"],
                      "note": f"molt_spec_accept on the step's logits; {samp['rejected']} of {B} draws residual against q"}
    t, n = groups["expert_gemm"]
    if n:
        pair_ms = 2 * t / n                       # gate_up + down per layer
        eb = 1 if w.expert_dtype == "fp8" else 2
        wbytes = w.n_experts * 3 * w.d_ff * d * eb
        flops = 2.0 * T * w.top_k * 3 * w.d_ff * d
        a = wbytes / (pair_ms / 1e3) / 1e9
        mf = flops / (pair_ms / 1e3) / 1e12
        peak_tf = 5000.0 if eb == 1 else BF16_PEAK_TFLOPS
        out["expert_gemm"] = {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                              "frac": round(a / HBM_PEAK_GBS, 4), "avg_layer_ms": round(pair_ms, 4),
                              "algorithmic_bytes_per_layer": wbytes,
                              "mfma_tflops": round(mf, 1), "mfma_frac": round(mf / peak_tf, 4),
                              "note": "all experts' weights once per layer (gate_up + down); the MFMA "
                                      "fraction is capped by arithmetic intensity at this batch"}
    t, n = groups["lm_head"]
    if n:
        ms = t / n
        tf = 2.0 * T * V * d / (ms / 1e3) / 1e12
        out["lm_head"] = {"bound": "mfma", "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS,
                          "unit": "TFLOP/s", "frac": round(tf / BF16_PEAK_TFLOPS, 4),
                          "avg_launch_ms": round(ms, 4)}
    return out


def mtp_measure(w, seed, molt, model, layout, kv, tokens, u, q, reps=5):
    """The MTP draft step (molt_mtp_draft) after this verify step: one head layer of the
    target's shape with its own cache, sampled drafts with their q. Timed with HIP events on
    the library's stream after the timed region (inputs resident: the verify step's hidden
    rows, accepted counts and emitted tokens). Algorithmic bytes: the head's K/V read once
    per row batch (the catch-up rows, then each drafting row), every expert's weights and
    eh_proj once per row batch, the LM head once per draft, and q written."""
    import torch
    dev = "cuda"
    B, k, V, d = w.batch, w.k, w.vocab, w.d_model
    mt = workloads.make_mtp_weights(w, seed, device=dev)
    mtp = molt.Mtp(mt["enorm"], mt["hnorm"], mt["eh_proj"], mt["layer"], mt["final_norm"],
                   n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                   top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta)
    del mt
    hkc, hvc = workloads.make_kv_cache(w, layout, seed, w.n_layers, device=dev)
    hkv = molt.KVCache([hkc], [hvc], kv.block_tables, kv.context_lens)
    vs = molt.verify_step(model, kv, tokens, u, q, want_logits=False, want_hidden=True)
    n = vs["n_accepted"]
    nxt = vs["tokens"].gather(1, n.long()[:, None])[:, 0].contiguous()
    ud = workloads.make_uniforms(B, k - 1, seed, tag="mtp_u", device=dev)
    ws = torch.empty(molt.mtp_draft_workspace_size(model, mtp, B, k, layout.block_tables.shape[1]),
                     dtype=torch.uint8, device=dev)
    res = molt.mtp_draft(model, mtp, hkv, vs["hidden"], tokens, n, nxt, ud, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        molt.mtp_draft(model, mtp, hkv, vs["hidden"], tokens, n, nxt, ud, workspace=ws, out=res)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    molt.profile_enable(True)
    molt.mtp_draft(model, mtp, hkv, vs["hidden"], tokens, n, nxt, ud, workspace=ws, out=res)
    torch.cuda.synchronize()
    molt.profile_enable(False)
    groups = {g: molt.profile_read(g) for g in molt._lib.PROF_GROUPS}
    e = 1 if w.expert_dtype == "fp8" else 2
    ctx = layout.context_lens.astype(np.int64)
    na = n.cpu().numpy().astype(np.int64)
    kvrow = w.n_kv_heads * w.head_dim * 2 * 2          # K and V bytes per cached position
    abytes = int((ctx + k + 1).sum()) * kvrow + sum(int((ctx + na + i + 1).sum()) * kvrow for i in range(1, k))
    ebytes = k * (w.n_experts * 3 * w.d_ff * d * e + 2 * d * d * 2
                  + ((w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim * d + d * w.n_q_heads * w.head_dim) * 2)
    hbytes = k * V * d * 2 + B * k * V * 4
    nbytes = abytes + ebytes + hbytes
    gbs = nbytes / (ms / 1e3) / 1e9
    drafts = res["drafts"].cpu().numpy()
    assert ((drafts >= 0) & (drafts < V)).all()
    return {"avg_ms": round(ms, 3), "drafts_per_s": round(B * k / (ms / 1e3), 1),
            "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": nbytes,
            "groups_ms": {g: round(t, 3) for g, (t, _) in groups.items()},
            "note": f"one MTP draft step (k = {k} sampled drafts with q, B = {B}) after the verify "
                    "step: catch-up rows + k-1 drafting rows of one head layer, the shared LM head "
                    "and the draws; bytes = head K/V per row batch + weights per row batch + LM "
                    "head per draft + q"}


def replay_measure(molt, model, kv, tokens, u, q, reps=3):
    """The actor's recompute of the step's emitted tokens with routing replay
    (molt_score_tokens with the verify step's tokens, out_tokens and out_routes), timed with
    HIP events after the timed region; also whether it reproduced the recorded behavior
    log-probabilities bit for bit (the consistency diagnostic)."""
    import torch
    v = molt.verify_step(model, kv, tokens, u, q, want_logits=False, want_routes=True)
    r = molt.score_tokens(model, kv, tokens, v["tokens"], replay_routes=v["routes"])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        molt.score_tokens(model, kv, tokens, v["tokens"], replay_routes=v["routes"])
    e1.record()
    torch.cuda.synchronize()
    emitted = v["tokens"] >= 0
    same = bool(torch.equal(r["logprobs"][emitted], v["logprobs"][emitted]))
    return {"avg_ms": round(e0.elapsed_time(e1) / reps, 3), "reproduces_behavior_logprobs": same,
            "note": "molt_score_tokens over the verify step's tokens with its emitted tokens as "
                    "targets and its recorded routes replayed"}


REPREFILL_TOKENS = 256


def reprefill_measure(w, seed, molt, model, layout, kv, reps=3):
    """Cache-hit re-prefill of an agent's growing context: sequence 0's cached 16-token
    blocks below its context (8192 positions) are the hit, and a new turn of
    REPREFILL_TOKENS tokens is prefilled at that context into spare blocks (molt_prefill,
    B = 1). Timed with HIP events after the timed region."""
    import torch
    dev = "cuda"
    ctx = int(layout.context_lens[0]) // 16 * 16
    used = set(int(b) for b in layout.block_tables.ravel() if b >= 0)
    spare = [b for b in range(layout.num_blocks) if b not in used][:REPREFILL_TOKENS // 16]
    row = np.concatenate([layout.block_tables[0][:ctx // 16], np.array(spare, np.int32)]).astype(np.int32)
    kv1 = molt.KVCache(kv.k_caches, kv.v_caches, torch.from_numpy(row[None, :].copy()).to(dev),
                       torch.tensor([ctx], dtype=torch.int32, device=dev))
    g = np.random.Generator(np.random.Philox(workloads._seed(seed, w.name, "reprefill")))
    toks = torch.from_numpy(g.integers(0, w.vocab, (1, REPREFILL_TOKENS)).astype(np.int32)).to(dev)
    lens = torch.tensor([REPREFILL_TOKENS], dtype=torch.int32, device=dev)
    ws = torch.empty(molt.prefill_workspace_size(model, 1, REPREFILL_TOKENS, len(row)), dtype=torch.uint8,
                     device=dev)
    out = molt.prefill(model, kv1, toks, lens, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        molt.prefill(model, kv1, toks, lens, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    assert torch.isfinite(out["logits"]).all()
    ms = e0.elapsed_time(e1) / reps
    # per-group breakdown from one more call with every group bracketed (untimed above)
    molt.profile_enable(True)
    molt.prefill(model, kv1, toks, lens, workspace=ws)
    torch.cuda.synchronize()
    molt.profile_enable(False)
    groups = {gr: molt.profile_read(gr) for gr in molt._lib.PROF_GROUPS}
    kvrow = w.n_kv_heads * w.head_dim * 2 * 2
    nbytes = (w.n_layers * (layer_weight_bytes(w) + (ctx + REPREFILL_TOKENS) * kvrow)
              + w.vocab * w.d_model * 2)
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"avg_ms": round(ms, 3), "cached_tokens": ctx, "new_tokens": REPREFILL_TOKENS,
            "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": int(nbytes),
            "groups_ms": {gr: round(t, 3) for gr, (t, _) in groups.items()},
            "note": "molt_prefill of one session's new turn at context 8192 (its cached prefix read "
                    "from the paged cache, not recomputed): the cache-hit re-prefill latency"}


CPU_SAMPLE_SEQS, CPU_SAMPLE_LAYERS = 8, 12


def host(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


def build(w, seed, molt, keep_host=0):
    """Generates the model on the GPU; GEMM weights are packed into the library's tiled
    layout in place of the row-major ones. Row-major host copies of the head and of the
    first `keep_host` layers are kept for the CPU baseline."""
    dev = "cuda"
    # room for the draft head's rows too (up to k - 1 positions past the verify window), and
    # spare blocks for the re-prefill measurement
    layout = workloads.make_kv_layout(w, seed, spare_blocks=REPREFILL_TOKENS // 16, extra_tokens=w.k)
    layers, kcs, vcs, host_layers = [], [], [], []
    for l in range(w.n_layers):
        lw = workloads.make_layer_weights(w, seed, l, device=dev)
        if l < keep_host:
            host_layers.append({k_: (None if v is None else host(v)) for k_, v in lw.items()})
        for key in molt.Model.PACKED:
            lw[key] = molt.pack_weights(lw[key])
        layers.append(lw)
        kc, vc = workloads.make_kv_cache(w, layout, seed, l, device=dev)
        kcs.append(kc)
        vcs.append(vc)
        if l % 8 == 0 or l == w.n_layers - 1:
            log(f"[bench] layer {l + 1}/{w.n_layers} generated, "
                f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB resident")
    head = workloads.make_head_weights(w, seed, device=dev)
    host_head = {k_: host(v) for k_, v in head.items()}
    head["lm_head"] = molt.pack_weights(head["lm_head"])
    model = molt.Model(layers, head, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                       head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta,
                       packed=True)
    kv = molt.KVCache(kcs, vcs, torch.from_numpy(layout.block_tables).to(dev),
                      torch.from_numpy(layout.context_lens).to(dev))
    return layout, host_layers, host_head, model, kv


def make_drafts(w, seed, molt, model, kv, ws):
    """Autoregressive drafts: q_i = softmax(target row i-1 + N(0, sigma^2)), x_i ~ q_i.
    Row i-1 only depends on tokens 0..i-1 (causal), so pass i fixes draft i."""
    dev = "cuda"
    B, k, V = w.batch, w.k, w.vocab
    g = np.random.Generator(np.random.Philox(workloads._seed(seed, w.name, "last")))
    tokens = torch.from_numpy(g.integers(0, V, (B, k + 1)).astype(np.int32)).to(dev)
    q = torch.empty(B, k, V, dtype=torch.float32, device=dev)
    u = workloads.make_uniforms(B, k, seed, device=dev)
    gen = workloads.rng(seed, w.name, "draft-sample", device=dev)
    for i in range(1, k + 1):
        out = molt.verify_step(model, kv, tokens, u, None, workspace=ws)
        row = out["logits"][:, i - 1]
        noise = torch.randn(B, V, generator=gen, device=dev) * w.draft_sigma
        qi = torch.softmax(row + noise, dim=-1)
        q[:, i - 1] = qi
        tokens[:, i] = torch.multinomial(qi, 1, generator=gen).squeeze(1).int()
        log(f"[bench] draft position {i}/{k} built")
    return tokens, q, u


def cpu_baseline(w, layout, host_layers, head, kv, tokens, q, u, n_seq=CPU_SAMPLE_SEQS,
                 sample_layers=CPU_SAMPLE_LAYERS):
    """Oracle on a bounded sample: `n_seq` sequences ((1+k) positions each) through
    `sample_layers` of the layers (row-major host copies), then the LM head and the
    sampler; the per-layer time is scaled to all layers. Returns (positions/s, seconds
    measured, threads, description)."""
    import oracle.model as omodel
    from oracle import sampler as osamp
    threads = blas_threads()

    sample_layers = min(sample_layers, len(host_layers))
    cfg = dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=sample_layers,
               n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, top_k=w.top_k,
               rms_eps=w.rms_eps, rope_theta=w.rope_theta, block_size=16)
    # the sample's blocks, renumbered densely
    blk_rows = [layout.block_tables[b][layout.block_tables[b] >= 0] for b in range(n_seq)]
    blocks = np.concatenate(blk_rows)
    bt = np.full((n_seq, max(len(r) for r in blk_rows)), -1)
    pos = 0
    for b, r in enumerate(blk_rows):
        bt[b, :len(r)] = np.arange(pos, pos + len(r))
        pos += len(r)
    lw = host_layers
    caches = []
    idx = torch.from_numpy(blocks).long().cuda()
    for l in range(sample_layers):
        kc = omodel.widen_cache(host(kv.k_caches[l][idx]), w.dtype)
        vc = omodel.widen_cache(host(kv.v_caches[l][idx]), w.dtype)
        caches.append((kc, vc))
    ctx = layout.context_lens[:n_seq]
    hh = head
    toks = host(tokens)[:n_seq]
    t0 = time.perf_counter()
    x = omodel.embed(toks, hh, cfg)
    x, _ = omodel.decoder_forward(x, lambda l: lw[l], caches, bt, ctx, w.k, cfg)
    t1 = time.perf_counter()
    logits = omodel.lm_logits(x, hh, cfg).reshape(n_seq, w.k + 1, -1)
    osamp.spec_accept(logits, toks[:, 1:], host(u)[:n_seq], host(q)[:n_seq])
    t2 = time.perf_counter()
    per_step = (t1 - t0) * (w.n_layers / sample_layers) + (t2 - t1)
    value = n_seq * (w.k + 1) / per_step
    desc = (f"{n_seq} of {w.batch} sequences ({n_seq * (w.k + 1)} positions) through {sample_layers} of {w.n_layers} "
            f"layers ({t1 - t0:.2f} s, scaled x{w.n_layers / sample_layers:g}) + LM head + sampler "
            f"({t2 - t1:.2f} s); float64 NumPy oracle")
    return value, t2 - t0, threads, desc


# ------------------------------------------------------------------ host description

def host_info():
    """The host the oracle runs on: core counts, BLAS library and threads, CPU model."""
    info = {"os_cpu_count": os.cpu_count(), "sched_affinity": len(os.sched_getaffinity(0))}
    try:
        from threadpoolctl import threadpool_info
        info["blas"] = [{k_: i.get(k_) for k_ in ("internal_api", "version", "num_threads",
                                                  "threading_layer")} for i in threadpool_info()]
    except Exception as e:                                    # noqa: BLE001
        info["blas"] = f"unknown ({e})"
    try:
        with open("/proc/cpuinfo") as f:
            info["cpu_model"] = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        info["cpu_model"] = None
    return info


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:                                         # noqa: BLE001
        return os.cpu_count() or 1


# ------------------------------------------------------------------ layer workloads

FLUSH_BYTES = 1 << 30          # written between timed iterations: evicts L2 and the MALL
LAYER_ITERS, LAYER_WARMUP = 20, 3
CPU_LAYER_SEQS = {"layer_bf16": 4, "long_ctx_bf16": 2, "fp8_zipf": 4}


def _timed(fn, flush, iters, warmup, prep=None):
    """Median and mean of `iters` calls of fn(), each bracketed by HIP events on torch's
    current stream (the library's stream), with the flush buffer rewritten and prep() run
    before each, outside the events."""
    for _ in range(warmup):
        if prep:
            prep()
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(iters)]
    for e0, e1 in ev:
        flush.zero_()
        if prep:
            prep()
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    t = np.array([e0.elapsed_time(e1) for e0, e1 in ev])
    return float(np.median(t)), float(t.mean())


def _groups(molt, fn, flush, reps=3, prep=None):
    """Per-kernel-group times of `reps` further calls, every group bracketed."""
    molt.profile_enable(True)
    for _ in range(reps):
        flush.zero_()
        if prep:
            prep()
        fn()
    torch.cuda.synchronize()
    molt.profile_enable(False)
    return {g: (t / reps, n // reps) for g, (t, n) in
            ((g, molt.profile_read(g)) for g in molt._lib.PROF_GROUPS)}


def _frac(achieved, peak):
    return round(achieved / peak, 4)


def dense_weight_bytes(w):
    D, d = w.head_dim, w.d_model
    return ((w.n_q_heads + 2 * w.n_kv_heads) * D * d + d * w.n_q_heads * D + w.n_experts * d) * 2


def dense_flops(w, T):
    return 2.0 * T * dense_weight_bytes(w) / 2


def layer_cpu_baseline(w, layout, lh, kc, vc, x0, n_seq):
    """The oracle's attention block and MoE block for the first n_seq sequences of the
    layer workload (their (1+k) positions, their own cache blocks), timed on the host."""
    import oracle.model as omodel
    seqs = list(range(n_seq))
    rows = [layout.block_tables[b][layout.block_tables[b] >= 0] for b in seqs]
    idx = torch.from_numpy(np.concatenate(rows)).long().to(kc.device)
    bt = np.full((n_seq, max(len(r) for r in rows)), -1, dtype=np.int64)
    pos = 0
    for i, r in enumerate(rows):
        bt[i, :len(r)] = np.arange(pos, pos + len(r))
        pos += len(r)
    okc = omodel.widen_cache(host(kc.index_select(0, idx)), w.dtype)
    ovc = omodel.widen_cache(host(vc.index_select(0, idx)), w.dtype)
    kp1 = w.k + 1
    xr = host(x0)[np.concatenate([np.arange(b * kp1, (b + 1) * kp1) for b in seqs])]
    cfg = dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=1, n_q_heads=w.n_q_heads,
               n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps,
               rope_theta=w.rope_theta, block_size=16)
    t0 = time.perf_counter()
    xo = omodel.attention_block(xr, lh, okc, ovc, bt, layout.context_lens[seqs], w.k, cfg)
    omodel.moe_block(xo, lh, cfg)
    secs = time.perf_counter() - t0
    return {"value": round(len(xr) / secs, 2), "unit": "verified tokens/s", "cores": blas_threads(),
            "kind": "oracle",
            "sample": f"{n_seq} of {w.batch} sequences ({len(xr)} positions) through the layer "
                      f"(attention block + MoE block), float64 NumPy oracle",
            "seconds": round(secs, 2)}


def hot_expert_gemm(w, seed, molt, flush, M):
    """One fp8 expert of the layer's shape with every one of M rows routed to it (E = K = 1
    through molt_moe_layer): the dense limit of a Zipf-hot expert. Its two GEMMs are timed
    as the expert-GEMM kernel group."""
    dev = "cuda"
    one = w.scaled(n_experts=1, top_k=1, zipf=None)
    lw = workloads.make_layer_weights(one, seed, 0, device=dev)
    x = workloads.make_hidden(one, seed, T=M, device=dev).to(torch.bfloat16)
    wr, wgu, wd = (molt.pack_weights(lw[k_]) for k_ in ("w_router", "w_gate_up", "w_down"))
    ws = torch.empty(molt._lib.load().molt_moe_layer_workspace_size(M, w.d_model, 1, 1, w.d_ff, 1, 2),
                     dtype=torch.uint8, device=dev)

    def call():
        molt.moe_layer(x, wr, wgu, wd, 1, s_gate_up=lw["s_gate_up"], s_down=lw["s_down"],
                       workspace=ws, packed=True, n_experts=1)

    _timed(call, flush, 5, 3)
    t, n = _groups(molt, call, flush, reps=10)["expert_gemm"]
    flops = 2.0 * M * 3 * w.d_ff * w.d_model
    tf = flops / (t / 1e3) / 1e12
    return {"rows": M, "gemm_ms": round(t, 4), "tflops": round(tf, 1), "peak": 5000.0,
            "unit": "TFLOP/s", "frac": _frac(tf, 5000.0), "flops": flops,
            "note": "gate_up + down of one fp8 expert with every row routed to it "
                    "(arithmetic intensity ~4600 flop/B: MFMA-bound)"}


def layer_measure(w, seed, molt, flush, cpu=True):
    """One decoder layer of a layer workload: the residual stream x [B(1+k), d] N(0,1), the
    layer's weights, and a random paged cache, all resident; median of LAYER_ITERS timed
    molt_decoder_forward calls (x restored before each, outside the events)."""
    dev = "cuda"
    B, k = w.batch, w.k
    T = B * (k + 1)
    layout = workloads.make_kv_layout(w, seed)
    lw = workloads.make_layer_weights(w, seed, 0, device=dev)
    lh = {k_: (None if v is None else host(v)) for k_, v in lw.items()} if cpu else None
    for key in molt.Model.PACKED:
        lw[key] = molt.pack_weights(lw[key])
    model = molt.Model([lw], None, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                       head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps,
                       rope_theta=w.rope_theta, packed=True)
    kc, vc = workloads.make_kv_cache(w, layout, seed, 0, device=dev)
    kv = molt.KVCache([kc], [vc], torch.from_numpy(layout.block_tables).to(dev),
                      torch.from_numpy(layout.context_lens).to(dev))
    x0 = workloads.make_hidden(w, seed, device=dev)
    x = x0.clone()
    ws = torch.empty(molt.decoder_workspace_size(model, B, k, layout.block_tables.shape[1]),
                     dtype=torch.uint8, device=dev)
    routes = molt.decoder_forward(model, kv, B, k, x, want_routes=True, workspace=ws)
    torch.cuda.synchronize()
    counts = np.bincount(routes.cpu().numpy().ravel(), minlength=w.n_experts)

    def call():
        molt.decoder_forward(model, kv, B, k, x, workspace=ws)

    def restore():
        x.copy_(x0)

    log(f"[bench] {w.name}: timing {LAYER_ITERS} layer calls")
    med, mean = _timed(call, flush, LAYER_ITERS, LAYER_WARMUP, prep=restore)
    groups = _groups(molt, call, flush, prep=restore)
    eb = 1 if w.expert_dtype == "fp8" else 2
    touched = int((counts > 0).sum())
    ebytes = touched * 3 * w.d_ff * w.d_model * eb
    abytes = attention_bytes(w, layout.context_lens)
    dbytes = dense_weight_bytes(w)
    nbytes = abytes + ebytes + dbytes
    eflops = 2.0 * T * w.top_k * 3 * w.d_ff * w.d_model
    epeak = 5000.0 if eb == 1 else BF16_PEAK_TFLOPS
    out = {"workload": w.name, "batch": B, "k": k,
           "context": [int(layout.context_lens.min()), int(layout.context_lens.max())],
           "positions": T, "layer_us": round(med * 1e3, 1), "layer_us_mean": round(mean * 1e3, 1),
           "verified_tokens_per_s": round(T / (med / 1e3), 1),
           "roofline": {"bound": "hbm", "algorithmic_bytes": int(nbytes),
                        "roofline_us": round(nbytes / (HBM_PEAK_GBS * 1e9) * 1e6, 1),
                        "achieved": round(nbytes / (med / 1e3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": _frac(nbytes / (med / 1e3) / 1e9, HBM_PEAK_GBS),
                        "note": "attention K/V + q + out, touched experts' weights, attention "
                                "projections and router, each once"}}
    ta, na = groups["attention"]
    if na:
        a = abytes / (ta / na / 1e3) / 1e9
        out["attention"] = {"avg_launch_us": round(ta / na * 1e3, 1), "algorithmic_bytes": int(abytes),
                            "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": _frac(a, HBM_PEAK_GBS)}
    te, ne = groups["expert_gemm"]
    if ne:
        a = ebytes / (te / 1e3) / 1e9
        tf = eflops / (te / 1e3) / 1e12
        ai = eflops / ebytes
        attain = min(epeak, ai * HBM_PEAK_GBS / 1e3)
        out["expert_gemm"] = {"gate_up_plus_down_us": round(te * 1e3, 1), "touched_experts": touched,
                              "weight_bytes": int(ebytes), "achieved": round(a, 1), "peak": HBM_PEAK_GBS,
                              "unit": "GB/s", "frac": _frac(a, HBM_PEAK_GBS),
                              "mfma_tflops": round(tf, 1), "mfma_peak": epeak,
                              "mfma_frac": _frac(tf, epeak),
                              "attainable_tflops": round(attain, 1),
                              "frac_of_attainable": _frac(tf, attain)}
    tp, npj = groups["projections"]
    if npj:
        tf = dense_flops(w, T) / (tp / 1e3) / 1e12
        attain = min(BF16_PEAK_TFLOPS, dense_flops(w, T) / dbytes * HBM_PEAK_GBS / 1e3)
        out["projections"] = {"qkv_o_router_us": round(tp * 1e3, 1), "mfma_tflops": round(tf, 1),
                              "mfma_peak": BF16_PEAK_TFLOPS, "mfma_frac": _frac(tf, BF16_PEAK_TFLOPS),
                              "attainable_tflops": round(attain, 1), "frac_of_attainable": _frac(tf, attain)}
    out["other_kernels_us"] = round((med - ta - te - tp) * 1e3, 1)
    if w.zipf is not None:
        srt = np.sort(counts)[::-1]
        out["expert_load"] = {"max_over_mean": round(float(counts.max() / counts.mean()), 2),
                              "top8_rows": srt[:8].tolist(), "empty_experts": int((counts == 0).sum())}
        out["hot_expert_gemm"] = hot_expert_gemm(w, seed, molt, flush, int(counts.max()))
        out["dense_expert_gemm"] = hot_expert_gemm(w, seed, molt, flush, T)
    if cpu:
        log(f"[bench] {w.name}: timing the CPU oracle")
        out["cpu_baseline"] = layer_cpu_baseline(w, layout, lh, kc, vc, x0, CPU_LAYER_SEQS[w.name])
    del model, kv, kc, vc, lw
    torch.cuda.empty_cache()
    return out


def tiny_measure(w, seed, molt, flush, cpu=True):
    """The tiny f32 decoder's whole verify step (2 layers, B 4, k 3, vocab 2048): the cache is
    filled by molt_prefill of the seeded prompts, then molt_verify_step is timed (a
    latency-bound configuration); the oracle's whole step on all cores and on one thread."""
    dev = "cuda"
    B, k = w.batch, w.k
    layout = workloads.make_kv_layout(w, seed)
    layers = [workloads.make_layer_weights(w, seed, l, device=dev) for l in range(w.n_layers)]
    head = workloads.make_head_weights(w, seed, device=dev)
    lh = [{k_: (None if v is None else host(v)) for k_, v in lw.items()} for lw in layers]
    hh = {k_: host(v) for k_, v in head.items()}
    model = molt.Model(layers, head, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                       head_dim=w.head_dim, top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta)
    caches = [workloads.empty_kv_cache(w, layout, device=dev) for _ in range(w.n_layers)]
    bt = torch.from_numpy(layout.block_tables).to(dev)
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    for b, p in enumerate(workloads.make_prompts(w, layout, seed)):   # one sequence at a time
        kvb = molt.KVCache(kcs, vcs, bt[b:b + 1].contiguous(), torch.zeros(1, dtype=torch.int32, device=dev))
        molt.prefill(model, kvb, torch.from_numpy(p[None, :].copy()).to(dev),
                     torch.tensor([len(p)], dtype=torch.int32, device=dev))
    kv = molt.KVCache(kcs, vcs, bt, torch.from_numpy(layout.context_lens).to(dev))
    toks = torch.from_numpy(workloads.make_step_tokens(w, seed)).to(dev)
    q = workloads.make_softmax_q(B, k, w.vocab, seed, device=dev)
    u = workloads.make_uniforms(B, k, seed, device=dev)
    ws = torch.empty(molt.verify_step_workspace_size(model, B, k, layout.block_tables.shape[1]),
                     dtype=torch.uint8, device=dev)
    res = molt.verify_step(model, kv, toks, u, q, workspace=ws)
    med, mean = _timed(lambda: molt.verify_step(model, kv, toks, u, q, workspace=ws, out=res),
                       flush, LAYER_ITERS, LAYER_WARMUP)
    T = B * (k + 1)
    out = {"workload": w.name, "positions": T, "step_us": round(med * 1e3, 1),
           "verified_tokens_per_s": round(T / (med / 1e3), 1),
           "note": "latency-bound (31 MB of weights): no roofline fraction is claimed"}
    if cpu:
        import oracle.model as omodel
        cfg = dict(dtype=w.dtype, expert_dtype=w.expert_dtype, n_layers=w.n_layers,
                   n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                   top_k=w.top_k, rms_eps=w.rms_eps, rope_theta=w.rope_theta, block_size=16)
        kch = [(omodel.widen_cache(host(a), w.dtype), omodel.widen_cache(host(b), w.dtype))
               for a, b in zip(kv.k_caches, kv.v_caches)]

        def run():
            c = [(a.copy(), b.copy()) for a, b in kch]
            t0 = time.perf_counter()
            omodel.verify_step(host(toks), lambda l: lh[l], hh, c, layout.block_tables,
                               layout.context_lens, cfg, host(q), host(u))
            return time.perf_counter() - t0

        secs = run()
        try:
            from threadpoolctl import threadpool_limits
            with threadpool_limits(limits=1):
                secs1 = run()
            one = {"value": round(T / secs1, 2), "cores": 1, "seconds": round(secs1, 3)}
        except Exception as e:                                # noqa: BLE001
            one = f"unavailable ({e})"
        out["cpu_baseline"] = {"value": round(T / secs, 2), "unit": "verified tokens/s",
                               "cores": blas_threads(), "kind": "oracle",
                               "sample": f"the whole step ({T} positions), float64 NumPy oracle",
                               "seconds": round(secs, 3), "single_thread": one}
    return out


def acceptance_prediction(out, q, k):
    """Closed form of the expected accepted count from the step's own rows: a draft drawn
    from q_i passes with probability alpha_i = sum_t min(p_t, q_t) = 1 - TV(p, q) (p =
    softmax of logits row i-1), so E[n] = sum_i prod_{j<=i} alpha_j per sequence."""
    alpha = torch.stack([torch.minimum(torch.softmax(out["logits"][:, i].double(), dim=-1),
                                       q[:, i].double()).sum(dim=-1) for i in range(k)], dim=1)
    en = torch.cumprod(alpha, dim=1).sum(dim=1)
    return {"predicted_mean_accepted_fraction": round(float(en.mean()) / k, 4),
            "mean_alpha": round(float(alpha.mean()), 4),
            "note": "E[n]/k from alpha_i = 1 - TV(p_{i-1}, q_i) of the step's own logits and q"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="full_depth_bf16", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--verify-only", action="store_true",
                    help="skip the draft-head, replay and re-prefill measurements (profiling runs)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device-to-device copy (HBM counter calibration)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads measured beside the headline")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {a.gpus}): the verify step shards by "
              "sequence with no communication, so each GPU's share is this single-GPU workload.",
              file=sys.stderr)
        sys.exit(2)
    if a.calibrate_copy:
        src = torch.empty(2 ** 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": 2 ** 30, "bytes_written": 2 ** 30,
                          "launches": 5}))
        return
    import paper_2607_21653_amd as molt
    molt.load()
    w = workloads.WORKLOADS[a.workload]
    flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda")
    info = None if a.no_cpu_baseline else host_info()
    if w.name != workloads.FULL_DEPTH_BF16.name:
        # one of the other workloads alone (profiling runs)
        m = (tiny_measure if w.name == workloads.TINY_FP32.name else layer_measure)(
            w, a.seed, molt, flush, cpu=not a.no_cpu_baseline)
        if info is not None:
            m["cpu_baseline"]["host"] = info
        print(json.dumps({"metric": "verified tokens/s per MI355X (verify step) + % HBM/MFMA roofline",
                          "value": m["verified_tokens_per_s"], "unit": "verified tokens/s", "n_gpus": 1,
                          "higher_is_better": True, "dtype": w.dtype, "data": "synthetic",
                          "config": {"workload": w.name}, "measurement": m}))
        return
    other_workloads = {}
    if not a.no_configs:
        for cw in (workloads.TINY_FP32, workloads.LAYER_BF16, workloads.LONG_CTX_BF16, workloads.FP8_ZIPF):
            log(f"[bench] workload {cw.name}")
            other_workloads[cw.name] = (tiny_measure if cw.name == workloads.TINY_FP32.name else layer_measure)(
                cw, a.seed, molt, flush, cpu=not a.no_cpu_baseline)
    del flush
    torch.cuda.empty_cache()
    t_setup = time.time()
    layout, host_layers, head, model, kv = build(
        w, a.seed, molt, keep_host=0 if a.no_cpu_baseline else CPU_SAMPLE_LAYERS)
    B, k, V = w.batch, w.k, w.vocab
    ws = torch.empty(molt.verify_step_workspace_size(model, B, k, layout.block_tables.shape[1]),
                     dtype=torch.uint8, device="cuda")
    if w.draft == "perturbed":
        tokens, q, u = make_drafts(w, a.seed, molt, model, kv, ws)
    else:
        tokens = torch.from_numpy(workloads.make_step_tokens(w, a.seed)).cuda()
        q = workloads.make_softmax_q(B, k, V, a.seed, device="cuda")
        u = workloads.make_uniforms(B, k, a.seed, device="cuda")
    out = {"tokens": torch.empty(B, k + 1, dtype=torch.int32, device="cuda"),
           "n_accepted": torch.empty(B, dtype=torch.int32, device="cuda"),
           "logprobs": torch.empty(B, k + 1, dtype=torch.float32, device="cuda"),
           "logits": torch.empty(B, k + 1, V, dtype=torch.float32, device="cuda")}
    log(f"[bench] setup {time.time() - t_setup:.1f} s; warmup {a.warmup} steps")
    for _ in range(a.warmup):
        molt.verify_step(model, kv, tokens, u, q, workspace=ws, out=out)
    torch.cuda.synchronize()
    log(f"[bench] timing {a.steps} steps")
    # Inside the timed region only the roofline kernel (attention) is bracketed by events,
    # in every 8th layer (6 launches per step, all of one shape): every event pair costs
    # ~2.6 us of stream time (0.25 ms per step with all 48 bracketed).
    molt.profile_enable(["attention"], every=ATTN_EVERY)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        molt.verify_step(model, kv, tokens, u, q, workspace=ws, out=out)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    molt.profile_enable(False)
    ms = (t1 - t0) * 1e3 / a.steps
    attn_ms, attn_n = molt.profile_read("attention")
    # the same steps again with no event inside, for the instrumentation's cost
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(a.steps):
        molt.verify_step(model, kv, tokens, u, q, workspace=ws, out=out)
    torch.cuda.synchronize()
    ms_plain = (time.perf_counter() - t2) * 1e3 / a.steps
    # per-group breakdown from separate, untimed steps with every group bracketed
    log("[bench] kernel-group breakdown (untimed steps)")
    molt.profile_enable(True)
    for _ in range(min(a.steps, 3)):
        molt.verify_step(model, kv, tokens, u, q, workspace=ws, out=out)
    torch.cuda.synchronize()
    molt.profile_enable(False)
    groups = {g: molt.profile_read(g) for g in molt._lib.PROF_GROUPS}
    n_break = min(a.steps, 3)
    samp = sampler_roofline(w, molt, out, tokens, q, u)
    n_acc = out["n_accepted"].cpu().numpy()
    accept = acceptance_prediction(out, q, k) if k > 0 else None
    mtp = rep = rpf = None
    if not a.verify_only:
        log("[bench] MTP draft step")
        mtp = mtp_measure(w, a.seed, molt, model, layout, kv, tokens, u, q) if k > 0 else None
        log("[bench] replay recompute")
        rep = replay_measure(molt, model, kv, tokens, u, q)
        log("[bench] cache-hit re-prefill")
        rpf = reprefill_measure(w, a.seed, molt, model, layout, kv)
    positions = B * (k + 1)
    value = positions / (ms / 1e3)
    emitted = float((n_acc + 1).sum()) / (ms / 1e3)

    attn_avg = attn_ms / max(attn_n, 1)
    abytes = attention_bytes(w, layout.context_lens)
    achieved = abytes / (attn_avg / 1e3) / 1e9
    lm_ms, lm_n = groups["lm_head"]
    lm_flops = 2.0 * positions * V * w.d_model
    per_group = {g: {"avg_ms": (t / n if n else None), "launches": n, "share_of_step":
                     (t / n_break / ms if n else None)} for g, (t, n) in groups.items()}
    res = {
        "metric": "verified tokens/s per MI355X (verify step) + % HBM/MFMA roofline",
        "value": round(value, 1),
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded random-init weights, KV and drafts; no checkpoint or dataset)",
        "config": {"workload": w.name, "layers": w.n_layers, "batch": B, "k": k,
                   "context": int(layout.context_lens.max()), "vocab": V, "d_model": w.d_model,
                   "heads": f"{w.n_q_heads}q/{w.n_kv_heads}kv x {w.head_dim}",
                   "experts": f"{w.n_experts} top-{w.top_k}, ffn {w.d_ff}", "block": 16,
                   "drafts": f"q = softmax(target + N(0, {w.draft_sigma}^2))" if w.draft == "perturbed" else "uniform"},
        "roofline": {"kernel": "paged attention (attn_lds_kernel + split merge), per layer launch",
                     "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": attention_traffic(),
                     "algorithmic_bytes_per_launch": abytes, "avg_launch_ms": round(attn_avg, 4),
                     "timed_launches": attn_n,
                     "note": f"HIP events around every {ATTN_EVERY}th layer's attention launch "
                             "inside the timed region (all layers launch the same shape)"},
        "ms_per_step_without_events": round(ms_plain, 3),
        "emitted_tokens_per_s": round(emitted, 1),
        "mean_accepted_fraction": round(float(n_acc.mean()) / k, 4) if k else None,
        "acceptance_closed_form": accept,
        "kernel_groups": per_group,
        "kernel_groups_note": f"HIP-event times of each group over {n_break} untimed steps after the timed region",
        "lm_head_tflops": round(lm_flops / (lm_ms / max(lm_n, 1) / 1e3) / 1e12, 1) if lm_n else None,
        "other_rooflines": other_rooflines(w, groups, samp),
        "step_roofline": (lambda nb: {"bound": "hbm", "achieved": round(nb / (ms / 1e3) / 1e9, 1),
                                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                      "frac": round(nb / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                                      "algorithmic_bytes": int(nb),
                                      "note": "the whole step: every layer's attention K/V + q + out "
                                              "and weights, LM head weights + logits, sampler reads"})(
            step_bytes(w, layout.context_lens, samp["bytes"])),
        "mtp_draft": mtp,
        "replay_recompute": rep,
        "reprefill": rpf,
        "configs": other_workloads or None,
    }
    if not a.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        v, secs, threads, desc = cpu_baseline(w, layout, host_layers, head, kv, tokens, q, u)
        res["cpu_baseline"] = {"value": round(v, 3), "unit": "verified tokens/s", "cores": threads,
                               "kind": "oracle", "sample": desc, "seconds": round(secs, 2),
                               "host": info}
    print(json.dumps(res))


if __name__ == "__main__":
    main()
