"""Top-K routed mixture-of-experts layer with SwiGLU experts.

The policy is a mixture-of-experts model whose expert choices are recorded for
routing replay (Sec. 4.1; Sec. 5.4 runs a 35B-A3B MoE). Per token t with
normalised input y_t:
    g_t = y_t W_r^T (+ bias)                       float32 router logits
    (e_j, w_j)_{j<K} = top-K(g_t), softmax weights  (routing.topk_route)
    FFN_e(y) = (silu(y W_g,e^T) * (y W_u,e^T)) W_d,e^T
    out_t = sum_{j=0..K-1} w_j FFN_{e_j}(y_t)       summed in slot order
Rounding points (shared reading with the GPU path): the SwiGLU product h is
stored in the activation dtype (bf16, or f32 for the f32 model) before the down
projection; expert outputs and the weighted sum are float32. With fp8 experts the
input row and h are each quantised per row (codecs.fp8_quantize_rows) and the
products are rescaled by s_row * s_channel. With replay ids, the experts are
given and only their weights come from the router (routing replay).

Weight containers are the raw stored arrays: float32 (f32), uint16 bit patterns
(bf16) or uint8 codes (fp8); each expert is widened exactly on use. Per-expert
matrix products use numpy's matmul on the rows routed to that expert (rows are
independent, so this is the per-token definition evaluated in batches).
"""
import numpy as np

from . import codecs, routing


def widen(w, dtype):
    w = np.asarray(w)
    if dtype == "f32":
        return w.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return codecs.bf16_bits_to_f32(w).astype(np.float64)
    if dtype == "fp8":
        return codecs.fp8_decode(w)
    raise ValueError(dtype)


def round_act(x, act_dtype):
    x = np.asarray(x, dtype=np.float64)
    if act_dtype == "bf16":
        return codecs.round_bf16(x)
    return x.astype(np.float32).astype(np.float64)


def silu(x):
    return x / (1.0 + np.exp(-x))


def moe_layer(y, w_router, w_gate_up, w_down, K, act_dtype, expert_dtype,
              s_gate_up=None, s_down=None, router_bias=None, replay_ids=None, tokens=None):
    """y: [T, d] float64 values (already in the activation dtype). w_router: [E, d]
    float64 values. Returns dict with out [len(tokens), d] float32 and routing data."""
    y = np.asarray(y, dtype=np.float64)
    T, d = y.shape
    E = w_router.shape[0]
    F = w_gate_up.shape[1] // 2
    g = routing.router_logits_f32(y, w_router, router_bias)
    if replay_ids is None:
        ids, wts, margin, order_margin = routing.topk_route(g, K)
    else:
        ids = np.asarray(replay_ids, dtype=np.int32).reshape(T, K)
        sel = np.take_along_axis(g.astype(np.float64), ids.astype(np.int64), axis=1)
        ev = np.exp(sel - sel.max(axis=1, keepdims=True))
        wts = (ev / ev.sum(axis=1, keepdims=True)).astype(np.float32)
        margin = np.full(T, np.inf)
        order_margin = np.full(T, np.inf)
    counts, offsets, perm, inv = routing.permute(ids, E)
    tok = np.arange(T) if tokens is None else np.asarray(tokens)
    want = np.zeros(T, dtype=bool)
    want[tok] = True
    o = {}  # (t, j) -> float32 expert output
    fp8 = expert_dtype == "fp8"
    if fp8:
        xq, sx = codecs.fp8_quantize_rows(y.astype(np.float32))
        xval = codecs.fp8_decode(xq)
    for e in range(E):
        pairs = [(t, j) for t in tok for j in range(K) if ids[t, j] == e]
        if not pairs:
            continue
        rows = np.array([t for t, _ in pairs])
        Wgu = widen(w_gate_up[e], expert_dtype)      # [2F, d]
        Wd = widen(w_down[e], expert_dtype)          # [d, F]
        if fp8:
            acc = xval[rows] @ Wgu.T                  # exact products of codes
            a = acc * sx[rows].astype(np.float64)[:, None] * np.asarray(s_gate_up[e], np.float64)[None, :]
        else:
            a = y[rows] @ Wgu.T
        h = round_act(silu(a[:, :F]) * a[:, F:], act_dtype)
        if fp8:
            hq, sh = codecs.fp8_quantize_rows(h.astype(np.float32))
            acc = codecs.fp8_decode(hq) @ Wd.T
            out_e = acc * sh.astype(np.float64)[:, None] * np.asarray(s_down[e], np.float64)[None, :]
        else:
            out_e = h @ Wd.T
        out_e = out_e.astype(np.float32)
        for r, (t, j) in enumerate(pairs):
            o[(t, j)] = out_e[r]
    out = np.zeros((len(tok), d), dtype=np.float32)
    for i, t in enumerate(tok):
        acc = np.zeros(d, dtype=np.float64)
        for j in range(K):
            acc += np.float64(wts[t, j]) * o[(t, j)].astype(np.float64)
        out[i] = acc.astype(np.float32)
    return {"out": out, "ids": ids, "weights": wts, "router_logits": g, "margin": margin, "order_margin": order_margin,
            "counts": counts, "offsets": offsets, "perm": perm, "inv": inv}


def dense_swiglu(y, w_gate_up, w_down, act_dtype):
    """Textbook dense SwiGLU FFN (one expert, no routing), float64 products; h rounded
    to the activation dtype like the MoE path."""
    W = np.asarray(w_gate_up, np.float64)
    F = W.shape[0] // 2
    a = np.asarray(y, np.float64) @ W.T
    h = round_act(silu(a[:, :F]) * a[:, F:], act_dtype)
    return (h @ np.asarray(w_down, np.float64).T).astype(np.float32)
