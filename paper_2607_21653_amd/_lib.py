"""ctypes binding of libmolt.so: argument marshalling only.

Every function takes torch tensors that already live on the GPU, checks dtypes,
shapes and contiguity, allocates outputs and the workspace with torch (device
memory is torch's job), and calls the C entry point of the same name on torch's
current stream. There is no fallback: if the library is missing or no GPU is
present, the call raises."""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmolt.so")

MOLT_F32, MOLT_BF16, MOLT_FP8_E4M3 = 0, 1, 2
NOALLOC_SCRATCH_BYTES = 8 << 20   # MOLT_NOALLOC_SCRATCH_BYTES of include/molt.h
DTYPE_CODE = {torch.float32: MOLT_F32, torch.bfloat16: MOLT_BF16, torch.uint8: MOLT_FP8_E4M3}
NAME_CODE = {"f32": MOLT_F32, "bf16": MOLT_BF16, "fp8": MOLT_FP8_E4M3}

_lib = None

c_int, c_size, c_vp, c_float = ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_float


class MoltModel(ctypes.Structure):
    _fields_ = [(n, c_int) for n in ("n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim",
                                     "n_experts", "top_k", "d_ff", "vocab")] + [
        ("rms_eps", c_float), ("rope_theta", c_float), ("dtype", c_int), ("expert_dtype", c_int),
        ("embed", c_vp), ("final_norm", c_vp), ("lm_head", c_vp),
        ("attn_norm", c_vp), ("w_qkv", c_vp), ("w_o", c_vp), ("moe_norm", c_vp),
        ("w_router", c_vp), ("router_bias", c_vp), ("w_gate_up", c_vp), ("w_down", c_vp),
        ("s_gate_up", c_vp), ("s_down", c_vp)]


class MoltKV(ctypes.Structure):
    _fields_ = [("k_cache", c_vp), ("v_cache", c_vp), ("block_tables", c_vp),
                ("context_lens", c_vp), ("max_blocks_per_seq", c_int), ("num_blocks", c_int),
                ("block_size", c_int)]


class MoltMtp(ctypes.Structure):
    _fields_ = [("enorm", c_vp), ("hnorm", c_vp), ("eh_proj", c_vp),
                ("layer", ctypes.POINTER(MoltModel))]


_SIGS = {
    "molt_last_error": (ctypes.c_char_p, []),
    "molt_version": (c_int, []),
    "molt_spec_accept_workspace_size": (c_size, [c_int, c_int, c_int]),
    "molt_spec_accept": (c_int, [c_vp, c_vp, c_vp, c_vp, c_int, c_int, c_int, c_vp, c_vp, c_vp,
                                 c_vp, c_size, c_vp]),
    "molt_spec_accept_noalloc": (c_int, [c_vp, c_vp, c_vp, c_vp, c_int, c_int, c_int, c_vp, c_vp,
                                         c_vp, c_vp]),
    "molt_moe_layer_workspace_size": (c_size, [c_int] * 5 + [c_int, c_int]),
    "molt_moe_layer": (c_int, [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_int, c_int, c_int,
                               c_int, c_int, c_int, c_int, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                               c_vp, c_vp, c_size, c_vp]),
    "molt_pack_weights": (c_int, [c_vp, c_vp, ctypes.c_longlong, ctypes.c_longlong, c_vp]),
    "molt_dense_gemm_workspace_size": (c_size, [c_int, c_int, c_int, c_int]),
    "molt_dense_gemm": (c_int, [c_vp, c_vp, c_vp, c_int, c_int, c_int, c_int, c_int, c_vp, c_size, c_vp]),
    "molt_paged_attention_workspace_size": (c_size, [c_int] * 6),
    "molt_paged_attention": (c_int, [c_vp, c_vp, c_vp, c_vp, c_vp, c_int, c_int, c_int, c_int,
                                     c_int, c_int, c_int, c_vp, c_vp, c_size, c_vp]),
    "molt_decoder_workspace_size": (c_size, [ctypes.POINTER(MoltModel), c_int, c_int, c_int]),
    "molt_decoder_forward": (c_int, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltKV), c_int,
                                     c_int, c_vp, c_vp, c_vp, c_size, c_vp]),
    "molt_profile_enable": (c_int, [c_int]),
    "molt_profile_every": (c_int, [c_int]),
    "molt_profile_read": (c_int, [c_int, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(c_int)]),
    "molt_verify_step_workspace_size": (c_size, [ctypes.POINTER(MoltModel), c_int, c_int, c_int]),
    "molt_verify_step": (c_int, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltKV), c_int, c_int,
                                 c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                 c_size, c_vp]),
    "molt_prefill_workspace_size": (c_size, [ctypes.POINTER(MoltModel), c_int, c_int, c_int]),
    "molt_prefill": (c_int, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltKV), c_int, c_int, c_vp,
                             c_vp, c_vp, c_vp, c_vp, c_vp, c_size, c_vp]),
    "molt_prefix_cache_create": (c_vp, [c_int]),
    "molt_prefix_cache_destroy": (None, [c_vp]),
    "molt_prefix_cache_acquire": (c_int, [c_vp, c_vp, c_int, c_int, c_vp, c_int,
                                          ctypes.POINTER(c_int)]),
    "molt_prefix_cache_commit": (c_int, [c_vp, c_vp, c_int, c_vp, c_int]),
    "molt_prefix_cache_release": (c_int, [c_vp, c_vp, c_int]),
    "molt_prefix_cache_stats": (c_int, [c_vp, ctypes.POINTER(ctypes.c_longlong)]),
    "molt_score_tokens_workspace_size": (c_size, [ctypes.POINTER(MoltModel), c_int, c_int, c_int]),
    "molt_score_tokens": (c_int, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltKV), c_int, c_int,
                                  c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_size, c_vp]),
    "molt_mtp_draft_workspace_size": (c_size, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltMtp),
                                               c_int, c_int, c_int]),
    "molt_mtp_draft_window_workspace_size": (c_size, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltMtp),
                                                      c_int, c_int, c_int, c_int]),
    "molt_mtp_draft_window": (c_int, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltMtp),
                                      ctypes.POINTER(MoltKV), c_int, c_int, c_int, c_vp, c_vp, c_vp,
                                      c_vp, c_vp, c_vp, c_vp, c_vp, c_size, c_vp]),
    "molt_mtp_draft": (c_int, [ctypes.POINTER(MoltModel), ctypes.POINTER(MoltMtp),
                               ctypes.POINTER(MoltKV), c_int, c_int, c_vp, c_vp, c_vp, c_vp, c_vp,
                               c_vp, c_vp, c_vp, c_size, c_vp]),
}


class MoltError(RuntimeError):
    pass


def load(path=LIB_PATH):
    """Loads the library (once). Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise MoltError(f"{path} is missing: build it with `python -m paper_2607_21653_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def exported_symbols():
    return list(_SIGS)


def _check(status, name):
    if status != 0:
        msg = _lib.molt_last_error().decode()
        raise MoltError(f"{name} returned {status}: {msg}")


def _ptr(t):
    return None if t is None else t.data_ptr()


def _dev(t, dtype, shape=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise MoltError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise MoltError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise MoltError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise MoltError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _workspace(nbytes, device, ws=None):
    if nbytes == 0:
        return None, 0
    if ws is not None and ws.numel() >= nbytes:
        return ws, ws.numel()
    t = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return t, nbytes


# ------------------------------------------------------------------ spec accept

def spec_accept(logits, draft_tokens, uniforms, draft_probs=None, out=None, workspace=None):
    """logits [B, k+1, V] f32; draft_tokens [B, k] i32; uniforms [B, k+1] f32;
    draft_probs [B, k, V] f32 or None (one-hot q). Returns (tokens, n_accepted, logprobs)."""
    lib = load()
    B, kp1, V = logits.shape
    k = kp1 - 1
    _dev(logits, torch.float32, name="logits")
    _dev(uniforms, torch.float32, (B, kp1), "uniforms")
    if k > 0:
        _dev(draft_tokens, torch.int32, (B, k), "draft_tokens")
    _dev(draft_probs, torch.float32, (B, k, V), "draft_probs")
    dev = logits.device
    if out is None:
        out = (torch.empty(B, kp1, dtype=torch.int32, device=dev),
               torch.empty(B, dtype=torch.int32, device=dev),
               torch.empty(B, kp1, dtype=torch.float32, device=dev))
    toks, n, lp = out
    ws, nb = _workspace(lib.molt_spec_accept_workspace_size(B, k, V), dev, workspace)
    st = lib.molt_spec_accept(_ptr(logits), _ptr(draft_probs), _ptr(draft_tokens) if k > 0 else None,
                              _ptr(uniforms), B, k, V, _ptr(toks), _ptr(n), _ptr(lp), _ptr(ws), nb,
                              _stream())
    _check(st, "molt_spec_accept")
    return toks, n, lp


def spec_accept_noalloc(logits, draft_tokens, uniforms, draft_probs=None, out=None):
    """molt_spec_accept_noalloc: spec_accept with the library's fixed per-GPU scratch array
    instead of a workspace (no device allocation inside the call when `out` is given)."""
    lib = load()
    B, kp1, V = logits.shape
    k = kp1 - 1
    _dev(logits, torch.float32, name="logits")
    _dev(uniforms, torch.float32, (B, kp1), "uniforms")
    if k > 0:
        _dev(draft_tokens, torch.int32, (B, k), "draft_tokens")
    _dev(draft_probs, torch.float32, (B, k, V), "draft_probs")
    dev = logits.device
    if out is None:
        out = (torch.empty(B, kp1, dtype=torch.int32, device=dev),
               torch.empty(B, dtype=torch.int32, device=dev),
               torch.empty(B, kp1, dtype=torch.float32, device=dev))
    toks, n, lp = out
    st = lib.molt_spec_accept_noalloc(_ptr(logits), _ptr(draft_probs),
                                      _ptr(draft_tokens) if k > 0 else None, _ptr(uniforms), B, k, V,
                                      _ptr(toks), _ptr(n), _ptr(lp), _stream())
    _check(st, "molt_spec_accept_noalloc")
    return toks, n, lp


# ------------------------------------------------------------------ weight layout

def pack_weights(w):
    """w (row-major, last dim contiguous) in the library's tiled GEMM operand layout
    (molt_pack_weights). Same dtype; shape [R, last] with the rows padded to a multiple
    of 32, except that a matrix whose row count is already such a multiple keeps its shape."""
    lib = load()
    _dev(w, None, name="w")
    rows = w.numel() // w.shape[-1]
    padded = (rows + 31) // 32 * 32
    shape = tuple(w.shape) if padded == rows else (padded, w.shape[-1])
    out = torch.empty(shape, dtype=w.dtype, device=w.device)
    _check(lib.molt_pack_weights(_ptr(w), _ptr(out), rows, w.shape[-1] * w.element_size(), _stream()),
           "molt_pack_weights")
    return out


def _rows(t):
    return t.numel() // t.shape[-1]


# ------------------------------------------------------------------ MoE layer

def moe_layer(x, w_router, w_gate_up, w_down, top_k, router_bias=None, s_gate_up=None,
              s_down=None, replay_ids=None, want_routing=False, workspace=None, packed=False,
              n_experts=None):
    """x [T, d] (f32|bf16); weights as in molt.h (fp8 experts as uint8 codes): router and
    expert weights row-major (packed here, per call), or already tiled with packed=True
    (then give n_experts when the router's row count is not a multiple of 32).
    Returns out [T, d] f32, or (out, ids, weights, counts, offsets, perm) with want_routing."""
    lib = load()
    T, d = x.shape
    E = n_experts if n_experts is not None else w_router.shape[0]
    if not packed:
        _dev(w_router, x.dtype, (E, d), "w_router")
        w_router = pack_weights(w_router)
        w_gate_up, w_down = pack_weights(w_gate_up), pack_weights(w_down)
    F = w_gate_up.shape[1] // 2
    act = DTYPE_CODE[x.dtype]
    wdt = DTYPE_CODE[w_gate_up.dtype]
    _dev(x, None, name="x")
    _dev(w_router, x.dtype, ((E + 31) // 32 * 32 if E % 32 else E, d), "w_router")
    _dev(w_gate_up, None, (E, 2 * F, d), "w_gate_up")
    _dev(w_down, w_gate_up.dtype, (E, d, F), "w_down")
    _dev(router_bias, torch.float32, (E,), "router_bias")
    _dev(s_gate_up, torch.float32, (E, 2 * F), "s_gate_up")
    _dev(s_down, torch.float32, (E, d), "s_down")
    _dev(replay_ids, torch.int32, (T, top_k), "replay_ids")
    dev = x.device
    out = torch.empty(T, d, dtype=torch.float32, device=dev)
    ids = wts = counts = offsets = perm = None
    if want_routing:
        ids = torch.empty(T, top_k, dtype=torch.int32, device=dev)
        wts = torch.empty(T, top_k, dtype=torch.float32, device=dev)
        counts = torch.empty(E, dtype=torch.int32, device=dev)
        offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
        perm = torch.empty(T * top_k, dtype=torch.int32, device=dev)
    ws, nb = _workspace(lib.molt_moe_layer_workspace_size(T, d, E, top_k, F, act, wdt), dev, workspace)
    st = lib.molt_moe_layer(_ptr(x), _ptr(w_router), _ptr(router_bias), _ptr(w_gate_up), _ptr(w_down),
                            _ptr(s_gate_up), _ptr(s_down), T, d, E, top_k, F, act, wdt,
                            _ptr(replay_ids), _ptr(out), _ptr(ids), _ptr(wts), _ptr(counts),
                            _ptr(offsets), _ptr(perm), _ptr(ws), nb, _stream())
    _check(st, "molt_moe_layer")
    if want_routing:
        return out, ids, wts, counts, offsets, perm
    return out


# ------------------------------------------------------------------ dense GEMM

def dense_gemm(A, B, C=None, accumulate=False, workspace=None):
    """C [M, N] f32 = A [M, K] @ B [N, K]^T (+ C when accumulate); A, B f32 or bf16,
    row-major (packed into the tiled operand layout here)."""
    lib = load()
    M, K = A.shape
    N = B.shape[0]
    _dev(A, None, name="A")
    _dev(B, A.dtype, (N, K), "B")
    if C is None:
        C = torch.zeros(M, N, dtype=torch.float32, device=A.device)
    _dev(C, torch.float32, (M, N), "C")
    At, Bt = pack_weights(A), pack_weights(B)
    dt = DTYPE_CODE[A.dtype]
    ws, nb = _workspace(lib.molt_dense_gemm_workspace_size(M, N, K, dt), A.device, workspace)
    _check(lib.molt_dense_gemm(_ptr(At), _ptr(Bt), _ptr(C), M, N, K, dt, 1 if accumulate else 0,
                               _ptr(ws), nb, _stream()), "molt_dense_gemm")
    return C


# ------------------------------------------------------------------ paged attention

def paged_attention(q, k_cache, v_cache, block_tables, context_lens, k, workspace=None):
    """q [B*(1+k), Hq, D]; caches [nb, Hkv, 16, D] / [nb, Hkv, D, 16]; returns [T, Hq*D]."""
    lib = load()
    T, Hq, D = q.shape
    B = context_lens.shape[0]
    Hkv = k_cache.shape[1]
    if T != B * (k + 1):
        raise MoltError(f"q has {T} rows, expected B*(1+k) = {B * (k + 1)}")
    _dev(q, None, name="q")
    _dev(k_cache, q.dtype, name="k_cache")
    _dev(v_cache, q.dtype, name="v_cache")
    _dev(block_tables, torch.int32, name="block_tables")
    _dev(context_lens, torch.int32, (B,), "context_lens")
    maxb = block_tables.shape[1]
    out = torch.empty(T, Hq * D, dtype=q.dtype, device=q.device)
    ws, nb = _workspace(lib.molt_paged_attention_workspace_size(B, k, Hq, Hkv, D, maxb), q.device, workspace)
    st = lib.molt_paged_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_tables),
                                  _ptr(context_lens), B, k, Hq, Hkv, D, maxb, DTYPE_CODE[q.dtype],
                                  _ptr(out), _ptr(ws), nb, _stream())
    _check(st, "molt_paged_attention")
    return out


# ------------------------------------------------------------------ model / decoder / step

class Model:
    """Holds the device weights of a decoder and the molt_model struct that points at them.
    layers: list of dicts with attn_norm, w_qkv, w_o, moe_norm, w_router, w_gate_up, w_down,
    optional router_bias, s_gate_up, s_down. head: dict with embed, final_norm, lm_head
    (optional for the decoder-only entry point). GEMM weights (w_qkv, w_o, w_router,
    w_gate_up, w_down, lm_head) row-major, packed here into tiled copies; or already tiled
    with packed=True (then pass vocab when the head has no embedding)."""

    PACKED = ("w_qkv", "w_o", "w_router", "w_gate_up", "w_down")

    def __init__(self, layers, head=None, n_q_heads=None, n_kv_heads=None, head_dim=None,
                 top_k=None, rms_eps=1e-6, rope_theta=1e6, packed=False, vocab=None):
        head = dict(head or {})
        if not packed:   # keep tiled copies of the GEMM weights (the caller keeps its own)
            layers = [dict(lw, **{k_: pack_weights(lw[k_]) for k_ in self.PACKED}) for lw in layers]
            if "lm_head" in head:
                head["lm_head"] = pack_weights(head["lm_head"])
        self.layers, self.head = layers, head
        l0 = layers[0]
        E, twoF, d = l0["w_gate_up"].shape
        self.dtype = l0["w_qkv"].dtype
        m = MoltModel()
        m.n_layers = len(layers)
        m.d_model, m.n_q_heads, m.n_kv_heads, m.head_dim = d, n_q_heads, n_kv_heads, head_dim
        m.n_experts, m.top_k, m.d_ff = E, top_k, twoF // 2
        m.vocab = vocab if vocab is not None else (self.head["embed"].shape[0] if "embed" in self.head else 0)
        m.rms_eps, m.rope_theta = rms_eps, rope_theta
        m.dtype = DTYPE_CODE[self.dtype]
        m.expert_dtype = DTYPE_CODE[l0["w_gate_up"].dtype]
        self._arrays = []

        def arr(key, optional=False):
            vals = [lw.get(key) for lw in layers]
            if optional and all(v is None for v in vals):
                return None
            a = (c_vp * len(vals))(*[None if v is None else v.data_ptr() for v in vals])
            self._arrays.append(a)
            return ctypes.cast(a, c_vp)

        for key in ("attn_norm", "w_qkv", "w_o", "moe_norm", "w_router", "w_gate_up", "w_down"):
            setattr(m, key, arr(key))
        for key in ("router_bias", "s_gate_up", "s_down"):
            setattr(m, key, arr(key, optional=True))
        for key in ("embed", "final_norm", "lm_head"):
            setattr(m, key, self.head[key].data_ptr() if key in self.head else None)
        self.struct = m


class KVCache:
    """Per-layer paged caches plus the block tables and context lengths (all on the GPU)."""

    def __init__(self, k_caches, v_caches, block_tables, context_lens):
        self.k_caches, self.v_caches = k_caches, v_caches
        self.block_tables, self.context_lens = block_tables, context_lens
        self._k = (c_vp * len(k_caches))(*[t.data_ptr() for t in k_caches])
        self._v = (c_vp * len(v_caches))(*[t.data_ptr() for t in v_caches])
        s = MoltKV()
        s.k_cache = ctypes.cast(self._k, c_vp)
        s.v_cache = ctypes.cast(self._v, c_vp)
        s.block_tables = block_tables.data_ptr()
        s.context_lens = context_lens.data_ptr()
        s.max_blocks_per_seq = block_tables.shape[1]
        s.num_blocks = k_caches[0].shape[0]
        s.block_size = 16
        self.struct = s


def decoder_workspace_size(model, B, k, max_blocks):
    return load().molt_decoder_workspace_size(ctypes.byref(model.struct), B, k, max_blocks)


def decoder_forward(model, kv, B, k, x, want_routes=False, workspace=None):
    """Runs every layer on the residual stream x [B*(1+k), d] f32 in place."""
    lib = load()
    _dev(x, torch.float32, (B * (k + 1), model.struct.d_model), "x")
    routes = None
    if want_routes:
        routes = torch.empty(model.struct.n_layers, B * (k + 1), model.struct.top_k,
                             dtype=torch.int32, device=x.device)
    ws, nb = _workspace(decoder_workspace_size(model, B, k, kv.struct.max_blocks_per_seq), x.device, workspace)
    st = lib.molt_decoder_forward(ctypes.byref(model.struct), ctypes.byref(kv.struct), B, k, _ptr(x),
                                  _ptr(routes), _ptr(ws), nb, _stream())
    _check(st, "molt_decoder_forward")
    return routes


def verify_step_workspace_size(model, B, k, max_blocks):
    return load().molt_verify_step_workspace_size(ctypes.byref(model.struct), B, k, max_blocks)


def verify_step(model, kv, tokens, uniforms, draft_probs=None, want_logits=True, want_routes=False,
                workspace=None, out=None, want_hidden=False):
    """tokens [B, 1+k] i32. Returns dict(tokens, n_accepted, logprobs, logits?, routes?,
    hidden?) (hidden: the final residual stream [B*(1+k), d] f32, the draft head's input)."""
    lib = load()
    B, kp1 = tokens.shape
    k = kp1 - 1
    V = model.struct.vocab
    dev = tokens.device
    _dev(tokens, torch.int32, name="tokens")
    _dev(uniforms, torch.float32, (B, kp1), "uniforms")
    _dev(draft_probs, torch.float32, (B, k, V), "draft_probs")
    if out is None:
        out = {"tokens": torch.empty(B, kp1, dtype=torch.int32, device=dev),
               "n_accepted": torch.empty(B, dtype=torch.int32, device=dev),
               "logprobs": torch.empty(B, kp1, dtype=torch.float32, device=dev)}
        if want_logits:
            out["logits"] = torch.empty(B, kp1, V, dtype=torch.float32, device=dev)
        if want_routes:
            out["routes"] = torch.empty(model.struct.n_layers, B * kp1, model.struct.top_k,
                                        dtype=torch.int32, device=dev)
        if want_hidden:
            out["hidden"] = torch.empty(B * kp1, model.struct.d_model, dtype=torch.float32, device=dev)
    ws, nb = _workspace(verify_step_workspace_size(model, B, k, kv.struct.max_blocks_per_seq), dev, workspace)
    st = lib.molt_verify_step(ctypes.byref(model.struct), ctypes.byref(kv.struct), B, k, _ptr(tokens),
                              _ptr(draft_probs), _ptr(uniforms), _ptr(out.get("logits")),
                              _ptr(out["tokens"]), _ptr(out["n_accepted"]), _ptr(out["logprobs"]),
                              _ptr(out.get("routes")), _ptr(out.get("hidden")), _ptr(ws), nb,
                              _stream())
    _check(st, "molt_verify_step")
    return out


def prefill_workspace_size(model, B, n, max_blocks):
    return load().molt_prefill_workspace_size(ctypes.byref(model.struct), B, n, max_blocks)


def prefill(model, kv, tokens, lens, want_hidden=False, want_routes=False, workspace=None):
    """Paged prefill (molt_prefill): tokens [B, n] i32 at positions context_lens[b] + j,
    lens [B] i32 in [1, n]. Returns dict(logits [B, V] of each last new row, hidden?, routes?)."""
    lib = load()
    B, n = tokens.shape
    m = model.struct
    dev = tokens.device
    _dev(tokens, torch.int32, name="tokens")
    _dev(lens, torch.int32, (B,), "lens")
    out = {"logits": torch.empty(B, m.vocab, dtype=torch.float32, device=dev)}
    if want_hidden:
        out["hidden"] = torch.empty(B * n, m.d_model, dtype=torch.float32, device=dev)
    if want_routes:
        out["routes"] = torch.empty(m.n_layers, B * n, m.top_k, dtype=torch.int32, device=dev)
    ws, nb = _workspace(prefill_workspace_size(model, B, n, kv.struct.max_blocks_per_seq), dev, workspace)
    st = lib.molt_prefill(ctypes.byref(m), ctypes.byref(kv.struct), B, n, _ptr(tokens), _ptr(lens),
                          _ptr(out["logits"]), _ptr(out.get("hidden")), _ptr(out.get("routes")),
                          _ptr(ws), nb, _stream())
    _check(st, "molt_prefill")
    return out


class PrefixCache:
    """The session-consistent prefix cache (host side, molt_prefix_cache_*): block ids of a
    pool of num_blocks blocks for the callers' block tables. Token lists and rows are host
    (numpy / Python) values."""

    def __init__(self, num_blocks):
        self._lib = load()
        self._c = self._lib.molt_prefix_cache_create(num_blocks)
        if not self._c:
            raise MoltError("molt_prefix_cache_create failed")
        self.num_blocks = num_blocks

    def __del__(self):
        if getattr(self, "_c", None):
            self._lib.molt_prefix_cache_destroy(self._c)
            self._c = None

    def acquire(self, tokens, extra_tokens=0, max_blocks=None):
        """-> (row [n_blocks] int32, n_cached), or None when the pool is exhausted or the row
        would need more than max_blocks blocks."""
        import numpy as np
        toks = np.ascontiguousarray(tokens, dtype=np.int32)
        n = len(toks)
        mb = max_blocks if max_blocks is not None else (n + extra_tokens + 15) // 16
        row = np.empty(max(mb, 1), dtype=np.int32)
        hit = c_int(0)
        r = self._lib.molt_prefix_cache_acquire(self._c, toks.ctypes.data, n, extra_tokens,
                                                row.ctypes.data, mb, ctypes.byref(hit))
        if r < 0:
            return None
        return row[:r].copy(), hit.value

    def commit(self, tokens, row):
        import numpy as np
        toks = np.ascontiguousarray(tokens, dtype=np.int32)
        row = np.ascontiguousarray(row, dtype=np.int32)
        _check(self._lib.molt_prefix_cache_commit(self._c, toks.ctypes.data, len(toks), row.ctypes.data,
                                                  len(row)), "molt_prefix_cache_commit")

    def release(self, row):
        import numpy as np
        row = np.ascontiguousarray(row, dtype=np.int32)
        _check(self._lib.molt_prefix_cache_release(self._c, row.ctypes.data, len(row)),
               "molt_prefix_cache_release")

    def stats(self):
        out = (ctypes.c_longlong * 7)()
        _check(self._lib.molt_prefix_cache_stats(self._c, out), "molt_prefix_cache_stats")
        keys = ("free", "cached", "referenced", "evictable", "lookup_tokens", "hit_tokens", "evictions")
        return dict(zip(keys, list(out)))


def score_tokens_workspace_size(model, B, k, max_blocks):
    return load().molt_score_tokens_workspace_size(ctypes.byref(model.struct), B, k, max_blocks)


def score_tokens(model, kv, tokens, targets, replay_routes=None, want_logits=False, want_routes=False,
                 workspace=None):
    """Behavior-log-prob recompute (molt_score_tokens): tokens, targets [B, 1+k] i32,
    replay_routes [L, B*(1+k), K] i32 or None. Returns dict(logprobs, logits?, routes?)."""
    lib = load()
    B, kp1 = tokens.shape
    k = kp1 - 1
    m = model.struct
    dev = tokens.device
    _dev(tokens, torch.int32, name="tokens")
    _dev(targets, torch.int32, (B, kp1), "targets")
    _dev(replay_routes, torch.int32, (m.n_layers, B * kp1, m.top_k), "replay_routes")
    out = {"logprobs": torch.empty(B, kp1, dtype=torch.float32, device=dev)}
    if want_logits:
        out["logits"] = torch.empty(B, kp1, m.vocab, dtype=torch.float32, device=dev)
    if want_routes:
        out["routes"] = torch.empty(m.n_layers, B * kp1, m.top_k, dtype=torch.int32, device=dev)
    ws, nb = _workspace(score_tokens_workspace_size(model, B, k, kv.struct.max_blocks_per_seq), dev,
                        workspace)
    st = lib.molt_score_tokens(ctypes.byref(m), ctypes.byref(kv.struct), B, k, _ptr(tokens),
                               _ptr(targets), _ptr(replay_routes), _ptr(out["logprobs"]),
                               _ptr(out.get("logits")), _ptr(out.get("routes")), _ptr(ws), nb,
                               _stream())
    _check(st, "molt_score_tokens")
    return out


class Mtp:
    """The MTP draft head: enorm, hnorm [d] f32, eh_proj [d, 2d] (row-major; packed here
    into its tiled copy, or already tiled with packed=True), and its decoder layer as a
    one-layer Model whose head holds the output norm (final_norm)."""

    def __init__(self, enorm, hnorm, eh_proj, layer, final_norm, n_q_heads, n_kv_heads, head_dim,
                 top_k, rms_eps=1e-6, rope_theta=1e6, packed=False):
        self.enorm, self.hnorm = enorm, hnorm
        self.eh_proj = eh_proj if packed else pack_weights(eh_proj)
        self.layer = Model([layer], {"final_norm": final_norm}, n_q_heads=n_q_heads,
                           n_kv_heads=n_kv_heads, head_dim=head_dim, top_k=top_k, rms_eps=rms_eps,
                           rope_theta=rope_theta, packed=packed, vocab=0)
        s = MoltMtp()
        s.enorm, s.hnorm, s.eh_proj = enorm.data_ptr(), hnorm.data_ptr(), self.eh_proj.data_ptr()
        s.layer = ctypes.pointer(self.layer.struct)
        self.struct = s


def mtp_draft_workspace_size(target, mtp, B, k, max_blocks, window=None):
    return load().molt_mtp_draft_window_workspace_size(
        ctypes.byref(target.struct), ctypes.byref(mtp.struct), B, k + 1 if window is None else window,
        k, max_blocks)


def mtp_draft(target, mtp, kv, hidden, tokens, n_accepted, next_tokens, uniforms=None,
              greedy=False, k=None, workspace=None, out=None):
    """One draft step (molt_mtp_draft_window): after a verify step (tokens [B, 1+k], the
    default k) or after a prefill (tokens [B, n] = its window, n_accepted = lens - 1, k given).
    hidden [B*W, d] f32, n_accepted [B] i32, next_tokens [B] i32, uniforms [B, k] f32 (unused
    when greedy). Returns dict(drafts [B, k] i32, draft_probs [B, k, V] f32 or None)."""
    lib = load()
    B, W = tokens.shape
    k = W - 1 if k is None else k
    V, d = target.struct.vocab, target.struct.d_model
    dev = tokens.device
    _dev(hidden, torch.float32, (B * W, d), "hidden")
    _dev(tokens, torch.int32, name="tokens")
    _dev(n_accepted, torch.int32, (B,), "n_accepted")
    _dev(next_tokens, torch.int32, (B,), "next_tokens")
    if not greedy:
        _dev(uniforms, torch.float32, (B, k), "uniforms")
    if out is None:
        out = {"drafts": torch.empty(B, k, dtype=torch.int32, device=dev),
               "draft_probs": None if greedy else torch.empty(B, k, V, dtype=torch.float32, device=dev)}
    ws, nb = _workspace(mtp_draft_workspace_size(target, mtp, B, k, kv.struct.max_blocks_per_seq, W), dev,
                        workspace)
    st = lib.molt_mtp_draft_window(ctypes.byref(target.struct), ctypes.byref(mtp.struct),
                                   ctypes.byref(kv.struct), B, W, k, _ptr(hidden), _ptr(tokens),
                                   _ptr(n_accepted), _ptr(next_tokens),
                                   _ptr(None if greedy else uniforms), _ptr(out["drafts"]),
                                   _ptr(out["draft_probs"]), _ptr(ws), nb, _stream())
    _check(st, "molt_mtp_draft")
    return out


# ------------------------------------------------------------------ kernel-group timing

PROF_GROUPS = {"attention": 0, "expert_gemm": 1, "lm_head": 2, "sampler": 3, "projections": 4}


def profile_enable(on=True, every=1):
    """on: True (all groups), False (stop), or an iterable of group names to time; every:
    time only launches 0, every, 2 every, ... of each group."""
    if on is True:
        mask = -1
    elif not on:
        mask = 0
    else:
        mask = 0
        for g in on:
            mask |= 1 << PROF_GROUPS[g]
    _check(load().molt_profile_every(every), "molt_profile_every")
    _check(load().molt_profile_enable(mask), "molt_profile_enable")


def profile_read(group):
    """(total milliseconds, number of timed launches) of a kernel group since enable."""
    ms, n = ctypes.c_double(0), c_int(0)
    _check(load().molt_profile_read(PROF_GROUPS[group], ctypes.byref(ms), ctypes.byref(n)),
           "molt_profile_read")
    return ms.value, n.value
