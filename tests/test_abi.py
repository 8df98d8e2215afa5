"""CPU-side checks of the C-ABI library: it loads, it exports every function that
include/molt.h declares, workspace queries answer, and argument validation rejects bad
calls with the documented status before touching the GPU (no compute call is made)."""
import ctypes
import os
import re

import pytest

import paper_2607_21653_amd as molt
from paper_2607_21653_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, UNSUPPORTED, WORKSPACE = 0, -1, -2, -3


@pytest.fixture(scope="module")
def L():
    return molt.load()


def _declared():
    src = open(os.path.join(ROOT, "include", "molt.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(molt_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert len(names) >= 12
    raw = ctypes.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n
    assert set(names) == set(molt.exported_symbols())


def test_version_and_error_string(L):
    assert L.molt_version() == 103
    assert isinstance(L.molt_last_error(), bytes)


def test_profile_every_validation(L):
    assert L.molt_profile_every(0) == INVALID
    assert L.molt_profile_every(-3) == INVALID
    assert L.molt_profile_every(1) == OK


def test_workspace_queries(L):
    assert L.molt_spec_accept_workspace_size(128, 4, 151936) > 0
    assert L.molt_spec_accept_workspace_size(0, 4, 10) == 0
    assert L.molt_moe_layer_workspace_size(640, 2048, 128, 8, 768, 1, 1) > 640 * 8 * 2048 * 4
    assert L.molt_moe_layer_workspace_size(64, 2048, 128, 8, 768, 0, 1) == 0     # bad pair
    assert L.molt_paged_attention_workspace_size(16, 4, 32, 4, 128, 4097) > 0    # split key range
    assert L.molt_paged_attention_workspace_size(128, 4, 32, 4, 128, 513) == 0    # one split: none


def _accept(L, B=2, k=1, V=10, logits=1, drafts=1, u=1, toks=1, n=1, ws=1, wsb=1 << 20):
    p = lambda f: ctypes.c_void_p(0x1000) if f else None
    return L.molt_spec_accept(p(logits), None, p(drafts), p(u), B, k, V, p(toks), p(n), None,
                              p(ws), wsb, None)


def test_spec_accept_validation(L):
    assert _accept(L, B=0) == INVALID
    assert _accept(L, k=-1) == INVALID
    assert _accept(L, V=0) == INVALID
    assert _accept(L, logits=0) == INVALID
    assert _accept(L, drafts=0) == INVALID
    assert _accept(L, u=0) == INVALID
    assert _accept(L, toks=0) == INVALID
    assert _accept(L, n=0) == INVALID
    assert _accept(L, ws=0) == WORKSPACE
    assert _accept(L, wsb=16) == WORKSPACE
    assert b"workspace" in L.molt_last_error()
    assert _accept(L, B=10 ** 7, k=4, V=151936) == INVALID       # grid limit


def test_moe_validation(L):
    p = ctypes.c_void_p(0x1000)
    args = dict(T=4, d=256, E=8, K=2, F=512, act=1, w=1)

    def call(**kw):
        a = dict(args, **kw)
        return L.molt_moe_layer(p, p, None, p, p, None, None, a["T"], a["d"], a["E"], a["K"], a["F"],
                                a["act"], a["w"], None, p, None, None, None, None, None, p, 1 << 30, None)
    assert call(T=0) == INVALID
    assert call(K=9) == INVALID
    assert call(E=300, K=2) == INVALID
    assert call(d=100) == INVALID
    assert call(act=0, w=1) == INVALID            # f32 activations need f32 experts
    assert call(w=2) == INVALID                   # fp8 without scales
    assert call(w=2, d=192) == INVALID            # fp8 needs d % 128


def test_attention_validation(L):
    p = ctypes.c_void_p(0x1000)

    def call(B=2, k=4, Hq=32, Hkv=4, D=128, mb=10, dt=1, ws=p, wsb=1 << 30):
        return L.molt_paged_attention(p, p, p, p, p, B, k, Hq, Hkv, D, mb, dt, p, ws, wsb, None)
    assert call(D=96) == INVALID
    assert call(Hq=30) == INVALID
    assert call(k=-1) == INVALID
    assert call(Hq=256, Hkv=1, k=0) == INVALID    # 256 query heads per kv head (a tile holds 128 rows)
    assert call(dt=2) == INVALID
    assert call(B=2, mb=2000, ws=None, wsb=0) == WORKSPACE


def test_pack_validation(L):
    p, q = ctypes.c_void_p(0x1000), ctypes.c_void_p(0x2000)
    assert L.molt_pack_weights(None, q, 32, 128, None) == INVALID
    assert L.molt_pack_weights(p, p, 32, 128, None) == INVALID      # in place
    assert L.molt_pack_weights(p, q, 32, 0, None) == INVALID        # row_bytes < 128
    assert L.molt_pack_weights(p, q, 32, 192, None) == INVALID      # row_bytes % 128
    assert L.molt_pack_weights(p, q, 0, 128, None) == INVALID


def test_model_validation(L):
    m = _lib.MoltModel()
    kv = _lib.MoltKV()
    assert L.molt_decoder_forward(None, ctypes.byref(kv), 1, 1, ctypes.c_void_p(1), None, None, 0, None) == INVALID
    m.n_layers = 0
    assert L.molt_decoder_forward(ctypes.byref(m), ctypes.byref(kv), 1, 1, ctypes.c_void_p(1), None,
                                  None, 0, None) == INVALID
    assert L.molt_verify_step(ctypes.byref(m), ctypes.byref(kv), 1, 1, None, None, None, None, None,
                              None, None, None, None, None, 0, None) == INVALID


def test_mtp_validation(L):
    """Host-side checks of molt_mtp_draft: nothing is enqueued for a bad request."""
    t, lay, kv = _lib.MoltModel(), _lib.MoltModel(), _lib.MoltKV()
    t.d_model, t.vocab, t.dtype = 256, 2048, _lib.MOLT_BF16
    t.embed = t.lm_head = ctypes.c_void_p(0x1000)
    lay.n_layers, lay.d_model, lay.dtype = 2, 256, _lib.MOLT_BF16
    mtp = _lib.MoltMtp()
    mtp.enorm = mtp.hnorm = mtp.eh_proj = ctypes.c_void_p(0x2000)
    mtp.layer = ctypes.pointer(lay)
    args = (ctypes.c_void_p(1),) * 4 + (None, ctypes.c_void_p(1), None, None, 0, None)
    assert L.molt_mtp_draft(ctypes.byref(t), None, ctypes.byref(kv), 4, 3, *args) == INVALID
    assert L.molt_mtp_draft(ctypes.byref(t), ctypes.byref(mtp), ctypes.byref(kv), 4, 0, *args) == INVALID
    assert "k = 0" in L.molt_last_error().decode()
    # a two-layer head
    assert L.molt_mtp_draft(ctypes.byref(t), ctypes.byref(mtp), ctypes.byref(kv), 4, 3, *args) == INVALID
    assert "n_layers = 2" in L.molt_last_error().decode()
    lay.n_layers, lay.d_model = 1, 512
    assert L.molt_mtp_draft(ctypes.byref(t), ctypes.byref(mtp), ctypes.byref(kv), 4, 3, *args) == INVALID
    assert "d_model" in L.molt_last_error().decode()
    # sampled drafts without uniforms
    lay.d_model = 256
    probs = ctypes.c_void_p(0x3000)
    a2 = (ctypes.c_void_p(1),) * 4 + (None, ctypes.c_void_p(1), probs, None, 0, None)
    assert L.molt_mtp_draft(ctypes.byref(t), ctypes.byref(mtp), ctypes.byref(kv), 4, 3, *a2) == INVALID
    assert L.molt_mtp_draft_workspace_size(ctypes.byref(t), None, 4, 3, 8) == 0
    assert L.molt_mtp_draft_workspace_size(ctypes.byref(t), ctypes.byref(mtp), 4, 0, 8) == 0


def test_spec_accept_noalloc_validation(L):
    """The allocation-free accept validates like molt_spec_accept and rejects shapes whose
    scratch need exceeds its fixed array, before any GPU call."""
    p = ctypes.c_void_p(0x1000)
    call = lambda B, k, V, logits=p, u=p, toks=p: L.molt_spec_accept_noalloc(
        logits, None, p, u, B, k, V, toks, p, None, None)
    assert call(0, 1, 10) == INVALID
    assert call(2, 1, 10, logits=None) == INVALID
    assert call(2, 1, 10, u=None) == INVALID
    assert call(2, 1, 10, toks=None) == INVALID
    limit = _lib.NOALLOC_SCRATCH_BYTES
    assert L.molt_spec_accept_workspace_size(128, 8, 151936) <= limit
    assert L.molt_spec_accept_workspace_size(4096, 8, 151936) > limit
    assert call(4096, 8, 151936) == INVALID
    assert b"scratch" in L.molt_last_error()
