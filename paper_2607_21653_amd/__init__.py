"""MI355X-native speculative-decoding verify step of a mixture-of-experts policy.

The compute runs in hand-written HIP kernels for gfx950 behind a C ABI
(include/molt.h, libmolt.so); this package is the thin Python binding."""
from ._lib import (MOLT_BF16, MOLT_F32, MOLT_FP8_E4M3, KVCache, Model, MoltError, Mtp,  # noqa: F401
                   decoder_forward, decoder_workspace_size, dense_gemm, exported_symbols, load, moe_layer,
                   mtp_draft, mtp_draft_workspace_size, pack_weights, paged_attention, prefill,
                   prefill_workspace_size, PrefixCache, profile_enable,
                   profile_read, score_tokens, score_tokens_workspace_size, spec_accept, spec_accept_noalloc,
                   verify_step,
                   verify_step_workspace_size)
