/*
 * molt.h -- C ABI of the MI355X (gfx950) speculative-decoding verify step.
 *
 * The method: a mixture-of-experts policy served with speculative decoding. Its
 * serving engine drafts k tokens per sequence and verifies them with the target
 * model; k = 0 disables speculation (paper Sec. 4.1, table of scaling controls:
 * number of speculative tokens). Verification runs one target forward pass over
 * the 1+k positions of every sequence (paged-KV attention, top-K routed expert
 * FFNs, LM head) and then applies the speculative accept rule min(1, p/q) with a
 * residual resample at temperature 1 and no truncation (Sec. 5.3, Sec. 5.4). The
 * engine returns the emitted token IDs and their behavior log-probabilities
 * (Sec. 4.2, Eq. 1) and, for routing replay, the experts each token used
 * (Sec. 4.1; route records travel with every experience, Sec. 4.4).
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless marked "host". Arrays are row-major.
 *  - The caller owns every buffer. The library allocates no device memory: each
 *    call takes a caller-provided workspace of at least *_workspace_size() bytes
 *    (256-byte aligned start recommended; any alignment is accepted). The one
 *    exception, molt_spec_accept_noalloc, uses a fixed array the library holds
 *    per GPU instead.
 *  - Calls are asynchronous on `stream` and never synchronise. Results are valid
 *    after the stream is synchronised. The library keeps no state between calls
 *    (weights and KV cache may be overwritten between calls, e.g. on a weight
 *    refit).
 *  - Arguments are validated on the host BEFORE anything is enqueued; a
 *    validation failure enqueues nothing and returns a negative status, with a
 *    message available from molt_last_error() (thread-local). Values that live
 *    in device memory (token IDs, block IDs, context lengths) cannot be checked
 *    on the host: out-of-range values there give undefined results, except where
 *    a function states otherwise.
 *  - A failed kernel launch returns MOLT_ERR_HIP with the HIP error string.
 *  - Calls that share a workspace must not overlap in time.
 *
 * Cache layout (PagedAttention-style blocks of 16 tokens, block table per
 * sequence; the paper's rollout engines use vLLM's paged cache, Sec. 2):
 *    K cache  [num_blocks, n_kv_heads, 16, head_dim]   one token's head vector contiguous
 *    V cache  [num_blocks, n_kv_heads, head_dim, 16]   the 16 tokens of a dim contiguous
 * Position p of sequence b lives in block block_tables[b * max_blocks_per_seq + p / 16],
 * slot p % 16. context_lens[b] counts tokens already cached; the 1+k new tokens
 * take positions context_lens[b] .. context_lens[b] + k. After a step the caller
 * advances context_lens[b] by n_accepted[b] + 1; slots of rejected drafts are
 * overwritten by the next step.
 */
#ifndef MOLT_H
#define MOLT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* molt_stream_t; /* the same type as hipStream_t */

typedef enum {
  MOLT_OK = 0,
  MOLT_ERR_INVALID_ARG = -1, /* NULL required pointer, bad size, bad combination  */
  MOLT_ERR_UNSUPPORTED = -2, /* valid request this library does not implement     */
  MOLT_ERR_WORKSPACE = -3,   /* workspace missing or smaller than *_workspace_size */
  MOLT_ERR_HIP = -4,         /* a HIP runtime call or kernel launch failed         */
  MOLT_ERR_CAPACITY = -5     /* the block pool has no free or evictable block left  */
} molt_status;

typedef enum {
  MOLT_F32 = 0,     /* IEEE binary32                                            */
  MOLT_BF16 = 1,    /* bfloat16 (upper half of binary32), round-to-nearest-even */
  MOLT_FP8_E4M3 = 2 /* OCP fp8 e4m3fn: bias 7, max +-448, no inf               */
} molt_dtype;

/* Message of the last failed call on this thread ("" if none). Valid until the
 * next call on the same thread. */
const char* molt_last_error(void);

/* ABI version of this header (major * 100 + minor). */
int molt_version(void);

/* ------------------------------------------------------------------------------
 * molt_spec_accept -- speculative accept / residual resample (Sec. 4.1 control
 * table: k speculative tokens; Sec. 4.2: token IDs and behavior log-probs
 * recorded at generation time; Sec. 5.3/5.4: temperature 1, no top-p/top-k).
 * The rule is the published speculative-sampling rule (Leviathan et al. 2023,
 * Chen et al. 2023): draft i (1..k) is judged by logits row i-1 and kept iff
 *       u[b, i-1] * q_i(x_i) * S < exp(l_x - m)      (i.e. u < p/q), strict,
 * with m = max_t l_t and S = sum_t exp(l_t - m) of that row. At the first
 * rejection the final token is drawn from norm(max(0, p - q)); if all k pass, a
 * bonus token is drawn from row k. The draw uses u[b, k] and an integer inverse
 * CDF: R_t = floor(r_t * 2^62), Tot = sum R_t, target = (Tot * floor(u * 2^32)) >> 32,
 * token = first t with prefix(R)_t > target (zero residual mass falls back to p).
 *
 *   logits         [B, k+1, V] f32   target logits (row j scores position j)
 *   draft_probs    [B, k, V]   f32   q of each draft position; NULL = one-hot q at
 *                                    the draft (greedy drafting)
 *   draft_tokens   [B, k]      i32   drafts in [0, V); an out-of-range draft is
 *                                    rejected (never read through); NULL iff k == 0
 *   uniforms       [B, k+1]    f32   in [0, 1): k accept tests, then the final draw
 *   out_tokens     [B, k+1]    i32   emitted tokens: n accepted drafts, then the
 *                                    final token; the rest -1
 *   out_num_accepted [B]       i32   n in [0, k]
 *   out_logprobs   [B, k+1]    f32   log p_j(token_j) of each emitted token at its
 *                                    row; the rest NaN. May be NULL.
 * Errors: INVALID_ARG for NULL required pointers, B < 1, k < 0, V < 1 or
 * B*(k+1)*V >= 2^62; WORKSPACE for a short workspace. Rows whose logits are all
 * -inf or contain NaN give undefined tokens.
 * ---------------------------------------------------------------------------- */
size_t molt_spec_accept_workspace_size(int B, int k, int V);
int molt_spec_accept(const float* logits, const float* draft_probs, const int32_t* draft_tokens,
                     const float* uniforms, int B, int k, int V, int32_t* out_tokens,
                     int32_t* out_num_accepted, float* out_logprobs, void* workspace,
                     size_t workspace_bytes, molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_spec_accept_noalloc -- molt_spec_accept for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. The same rule, kernels and results (bit for bit) as molt_spec_accept, with
 * the workspace replaced by a fixed array of MOLT_NOALLOC_SCRATCH_BYTES (8 MiB) of device
 * memory that the library holds on every GPU it runs on until the process ends. The call
 * allocates nothing (no hipMalloc, no allocating library routine); its first call on a
 * device looks up that device's array, so the current device must be the stream's.
 * Every call on one GPU shares that GPU's array, which keeps the last call's contents
 * (each call writes every entry before reading it, so nothing needs clearing): calls that
 * overlap in time on one GPU (several streams or host threads) race and give undefined
 * results.
 * Arguments as molt_spec_accept, without the workspace.
 * Errors: as molt_spec_accept, and INVALID_ARG when molt_spec_accept_workspace_size(B, k,
 * V) exceeds MOLT_NOALLOC_SCRATCH_BYTES (B = 128, k = 8, V = 151936 needs 0.9 MB; the
 * need grows as B * (k + 1) * ceil(V / 8192) * 12 + B * ceil(V / 8192) * 264 bytes);
 * HIP when the array cannot be looked up.
 * ---------------------------------------------------------------------------- */
#define MOLT_NOALLOC_SCRATCH_BYTES (8u << 20)
int molt_spec_accept_noalloc(const float* logits, const float* draft_probs,
                             const int32_t* draft_tokens, const float* uniforms, int B, int k,
                             int V, int32_t* out_tokens, int32_t* out_num_accepted,
                             float* out_logprobs, molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_moe_layer -- top-K routed SwiGLU mixture-of-experts on normalised input
 * (the MoE policy of Sec. 5.4; expert choices are the route records kept for
 * routing replay, Sec. 4.1):
 *   g = x W_r^T (+ router_bias)                 f32 router logits [T, E]
 *   ids, w = top-K of g (descending, ties to the lower expert ID, -0 == +0),
 *            softmax over the K selected logits
 *   out[t] = sum_{j<K} w[t,j] * FFN_{ids[t,j]}(x[t])   (slot order, f32)
 *   FFN_e(x) = (silu(x W_g,e^T) * (x W_u,e^T)) W_d,e^T, SwiGLU product stored in
 *            act_dtype before the down projection.
 * fp8 experts: x and the SwiGLU product are quantised per row (s = amax/448,
 * codes = e4m3(v / s), saturating, round-to-nearest-even); products are rescaled
 * by s_row * s_channel.
 *
 *   x            [T, d]        act_dtype (F32 or BF16)
 *   w_router     [E, d]        act_dtype, tiled (molt_pack_weights)
 *   router_bias  [E]           f32, or NULL (added to the logits before top-K)
 *   w_gate_up    [E, 2F, d]    w_dtype: rows 0..F-1 gate, F..2F-1 up; TILED layout
 *                              (molt_pack_weights with rows = E*2F, row_bytes = d*size)
 *   w_down       [E, d, F]     w_dtype, TILED layout (rows = E*d, row_bytes = F*size)
 *   s_gate_up    [E, 2F] f32, s_down [E, d] f32: per-output-channel scales, required
 *                iff w_dtype == FP8_E4M3, else ignored
 *   replay_ids   [T, K] i32 or NULL: use these experts (distinct, in [0, E)) and take
 *                only their weights from the router (routing replay)
 *   out          [T, d] f32    the weighted expert sum (no residual)
 *   out_ids, out_weights [T, K] i32 / f32: route records, may be NULL
 *   out_counts [E], out_offsets [E+1], out_perm [T*K] i32: the stable (expert,
 *                token, slot) grouping, may be NULL
 * Supported: (act, w) in {(F32, F32), (BF16, BF16), (BF16, FP8_E4M3)}; d % 64 == 0,
 * F % 64 == 0 (fp8: % 128), 1 <= K <= E <= 256, K <= 64. T >= 1.
 * ---------------------------------------------------------------------------- */
size_t molt_moe_layer_workspace_size(int T, int d, int E, int K, int F, molt_dtype act_dtype,
                                     molt_dtype w_dtype);
int molt_moe_layer(const void* x, const void* w_router, const float* router_bias,
                   const void* w_gate_up, const void* w_down, const float* s_gate_up,
                   const float* s_down, int T, int d, int E, int K, int F, molt_dtype act_dtype,
                   molt_dtype w_dtype, const int32_t* replay_ids, float* out, int32_t* out_ids,
                   float* out_weights, int32_t* out_counts, int32_t* out_offsets,
                   int32_t* out_perm, void* workspace, size_t workspace_bytes,
                   molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_pack_weights -- the GEMM operand layout of this library (a layout choice of the
 * implementation; the paper fixes none). A row-major byte matrix of `rows` rows and
 * `row_bytes` bytes per row, rows padded with zero rows to R = 32 * ceil(rows / 32), is
 * cut into 32-row x 128-byte tiles; tile (rb, kb) takes the 4096 bytes at
 * ((rb * row_bytes / 128) + kb) * 4096, and byte j of row r of the matrix (rb = r / 32,
 * kb = j / 128) sits inside it at
 *     ((j % 64) / 16) * 1024 + (((j % 128) / 64) * 32 + r % 32) * 16 + j % 16.
 * Every weight matrix a GEMM of this library reads ([out, in], K = in contiguous) is in
 * this layout, packed once at load: w_qkv, w_o, w_router, lm_head with rows = out
 * features, row_bytes = in * sizeof(dtype); w_gate_up as rows = E*2F, row_bytes =
 * d * sizeof(w_dtype); w_down as rows = E*d, row_bytes = F * sizeof(w_dtype). Embeddings,
 * norms and fp8 scales stay row-major. dst receives R * row_bytes bytes and must not
 * overlap src.
 * Errors: INVALID_ARG for NULL or equal pointers, rows < 1, row_bytes < 128 or
 * row_bytes % 128 != 0.
 * ---------------------------------------------------------------------------- */
int molt_pack_weights(const void* src, void* dst, long long rows, long long row_bytes,
                      molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_paged_attention -- multi-query paged decode attention of the verify step
 * (PagedAttention cache, Sec. 2). Token t = b*(1+k) + j is query position j of
 * sequence b and attends to positions 0 .. context_lens[b] + j (its own included);
 * query head h reads kv head h / (Hq/Hkv); scores scaled by 1/sqrt(D); softmax in
 * f32. The cache must already hold the 1+k new positions.
 *
 *   q             [T, Hq, D]  dtype           T = B*(1+k)
 *   k_cache, v_cache          dtype, layouts above
 *   block_tables  [B, max_blocks_per_seq] i32;  context_lens [B] i32
 *   out           [T, Hq*D]   dtype
 * Supported: dtype F32 or BF16, D in {64, 128}, Hq % Hkv == 0, Hq/Hkv*(1+k) <= 128.
 * context_lens[b] + k + 1 <= 16 * max_blocks_per_seq is the caller's duty.
 * ---------------------------------------------------------------------------- */
size_t molt_paged_attention_workspace_size(int B, int k, int n_q_heads, int n_kv_heads,
                                           int head_dim, int max_blocks_per_seq);
int molt_paged_attention(const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_tables, const int32_t* context_lens, int B, int k,
                         int n_q_heads, int n_kv_heads, int head_dim, int max_blocks_per_seq,
                         molt_dtype dtype, void* out, void* workspace, size_t workspace_bytes,
                         molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_dense_gemm -- the dense projection of the verify step's decoder (QKV, O, router,
 * LM head): C[M, N] (f32, row-major) = A[M, K] * B[N, K]^T, or C += A * B^T with
 * accumulate != 0 (the O projection adds into the residual stream). A and B in `dtype`
 * (F32 or BF16) and in the tiled layout of molt_pack_weights (rows = M resp. N, row_bytes =
 * K * sizeof(dtype); padding rows are read, their products dropped); f32 accumulation.
 * Supported: M, N, K >= 1, K * sizeof(dtype) % 128 == 0. The workspace holds split-K
 * partial sums for small grids (size from molt_dense_gemm_workspace_size, may be 0);
 * splits are added in a fixed order, so results are deterministic.
 * ---------------------------------------------------------------------------- */
size_t molt_dense_gemm_workspace_size(int M, int N, int K, molt_dtype dtype);
int molt_dense_gemm(const void* A, const void* B, float* C, int M, int N, int K, molt_dtype dtype,
                    int accumulate, void* workspace, size_t workspace_bytes, molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * Model description: a HOST struct holding device pointers; read only during a
 * call. Per-layer members are HOST arrays of n_layers device pointers.
 * Pre-norm decoder (Sec. 5.3/5.4 run MoE decoders):
 *   x += Attn(RMSNorm(x)); x += MoE(RMSNorm(x))    per layer, x f32
 * RMSNorm(x) = x / sqrt(mean(x^2) + rms_eps) * g, rounded to dtype.
 * RoPE: rotate-half pairs (i, i + D/2), inverse frequency rope_theta^(-2i/D),
 * angle = position * inv_freq, evaluated in f64.
 * dtype F32 requires expert_dtype F32; dtype BF16 allows BF16 or FP8_E4M3 experts.
 * ---------------------------------------------------------------------------- */
typedef struct molt_model {
  int n_layers, d_model, n_q_heads, n_kv_heads, head_dim, n_experts, top_k, d_ff, vocab;
  float rms_eps, rope_theta;
  molt_dtype dtype;        /* activations, embeddings, attention/router/LM-head weights, KV */
  molt_dtype expert_dtype; /* expert weights                                              */
  const void* embed;       /* [V, d] dtype (needed by molt_verify_step)                   */
  const float* final_norm; /* [d]                                                         */
  const void* lm_head;     /* [V, d] dtype, tiled (molt_pack_weights)                     */
  const float* const* attn_norm;   /* [L] -> [d]                                          */
  const void* const* w_qkv;        /* [L] -> [(Hq + 2 Hkv) D, d]: q, k, v heads; tiled   */
  const void* const* w_o;          /* [L] -> [d, Hq D], tiled                             */
  const float* const* moe_norm;    /* [L] -> [d]                                          */
  const void* const* w_router;     /* [L] -> [E, d], tiled                                */
  const float* const* router_bias; /* NULL, or [L] -> [E] f32 (entries may be NULL)       */
  const void* const* w_gate_up;    /* [L] -> [E, 2F, d], tiled (molt_pack_weights)        */
  const void* const* w_down;       /* [L] -> [E, d, F], tiled (molt_pack_weights)         */
  const float* const* s_gate_up;   /* [L] -> [E, 2F] f32, fp8 experts only, else NULL     */
  const float* const* s_down;      /* [L] -> [E, d] f32                                   */
} molt_model;

typedef struct molt_kv {
  void* const* k_cache;        /* HOST array [n_layers] of device K caches (layout above) */
  void* const* v_cache;        /* HOST array [n_layers] of device V caches                */
  const int32_t* block_tables; /* [B, max_blocks_per_seq] physical block IDs              */
  const int32_t* context_lens; /* [B] tokens already cached                               */
  int max_blocks_per_seq;
  int num_blocks;
  int block_size; /* must be 16 */
} molt_kv;

/* ------------------------------------------------------------------------------
 * molt_decoder_forward -- all n_layers decoder layers of the verify step on a
 * given residual stream (token t = b*(1+k) + j at position context_lens[b] + j).
 * Writes the new keys/values of every layer into the cache.
 *   x           [B*(1+k), d] f32, in/out (the residual stream)
 *   out_routes  [n_layers, B*(1+k), top_k] i32 expert IDs, or NULL
 * Requirements as for molt_moe_layer and molt_paged_attention.
 * ---------------------------------------------------------------------------- */
size_t molt_decoder_workspace_size(const molt_model* m, int B, int k, int max_blocks_per_seq);
int molt_decoder_forward(const molt_model* m, const molt_kv* kv, int B, int k, float* x,
                         int32_t* out_routes, void* workspace, size_t workspace_bytes,
                         molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_verify_step -- the whole verify step: embed tokens, run the decoder,
 * final RMSNorm, LM head to f32 logits, then molt_spec_accept's rule.
 *   tokens       [B, 1+k] i32: the last emitted token, then the k drafts (in [0, V))
 *   draft_probs, uniforms, out_tokens, out_num_accepted, out_logprobs: as in
 *                molt_spec_accept (drafts are tokens[:, 1:])
 *   out_logits   [B, 1+k, V] f32, or NULL (then kept in the workspace)
 *   out_routes   [n_layers, B*(1+k), top_k] i32, or NULL
 *   out_hidden   [B*(1+k), d] f32 final residual stream (before the final norm), or
 *                NULL: the input of molt_mtp_draft
 * ---------------------------------------------------------------------------- */
size_t molt_verify_step_workspace_size(const molt_model* m, int B, int k, int max_blocks_per_seq);
int molt_verify_step(const molt_model* m, const molt_kv* kv, int B, int k, const int32_t* tokens,
                     const float* draft_probs, const float* uniforms, float* out_logits,
                     int32_t* out_tokens, int32_t* out_num_accepted, float* out_logprobs,
                     int32_t* out_routes, float* out_hidden, void* workspace,
                     size_t workspace_bytes, molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * molt_prefill -- paged prefill of a window of new tokens per sequence: the verify step's
 * forward over tokens[b, 0..n) at positions context_lens[b] + j (cached positions below
 * context_lens[b], e.g. a prefix-cache hit, are read, not recomputed), then the final norm
 * and LM head of each sequence's last new row (row lens[b] - 1). Prefix caching enters the
 * serving engine (Sec. 4.1, Sec. 5.3); a cache-hit re-prefill of an agent's growing context
 * computes only the positions past the hit (Sec. 5.4).
 *   tokens      [B, n] i32; rows j >= lens[b] are padding (computed, their cache slots
 *               written; the caller advances context_lens[b] by lens[b] only)
 *   lens        [B] i32 in [1, n]
 *   out_logits  [B, V] f32: logits of row lens[b] - 1
 *   out_hidden  [B*n, d] f32 final residual stream (before the final norm), or NULL
 *   out_routes  [n_layers, B*n, top_k] i32, or NULL
 * Writes the cache at positions context_lens[b] .. context_lens[b] + n - 1;
 * context_lens[b] + n <= 16 * max_blocks_per_seq is the caller's duty.
 * ---------------------------------------------------------------------------- */
size_t molt_prefill_workspace_size(const molt_model* m, int B, int n, int max_blocks_per_seq);
int molt_prefill(const molt_model* m, const molt_kv* kv, int B, int n, const int32_t* tokens,
                 const int32_t* lens, float* out_logits, float* out_hidden, int32_t* out_routes,
                 void* workspace, size_t workspace_bytes, molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * Session-consistent prefix cache (HOST side: every pointer below is a host pointer; no
 * device memory, no stream). Hands out physical block ids of a pool of num_blocks blocks
 * of 16 positions for the callers' block tables, reusing the blocks of a cached prefix
 * only when its token IDs match exactly (Sec. 4.2: a rewritten history starts anew).
 *  - A full block is identified by its 16 token IDs and its parent (the cached block of
 *    the preceding 16 tokens); cached blocks form a tree, and dropping a block's entry
 *    drops its subtree's.
 *  - acquire: the longest chain of cached full blocks matching tokens[0..n), at most
 *    (n - 1) / 16 blocks (at least one position is left to compute), each gaining a
 *    reference; then ceil((n + extra_tokens) / 16) blocks in all, each missing one the
 *    lowest free block id, or, with none free, after evicting the least recently released
 *    cached block without references. Writes block_table[0..max_blocks) (-1 past the
 *    row), *n_cached = 16 * hits (the caller prefills tokens[n_cached..n) at context
 *    n_cached); returns the row's block count, MOLT_ERR_INVALID_ARG (bad argument, or more
 *    than max_blocks blocks needed) or MOLT_ERR_CAPACITY (pool exhausted; nothing changed
 *    but the hit blocks' recency).
 *  - commit: once the keys/values of tokens[0..n) are in the row's blocks, every full
 *    block whose prefix is not cached yet becomes cached (a prefix cached elsewhere keeps
 *    that block).
 *  - release: the row's blocks lose a reference (last block first); a block left without
 *    references becomes evictable (cached) or free.
 *  - stats: out[7] = free blocks, cached blocks, referenced blocks, evictable blocks,
 *    tokens looked up, tokens hit, evictions.
 * Not thread-safe: one host thread per cache.
 * ---------------------------------------------------------------------------- */
typedef struct molt_prefix_cache molt_prefix_cache;
molt_prefix_cache* molt_prefix_cache_create(int num_blocks);   /* NULL if num_blocks < 1 */
void molt_prefix_cache_destroy(molt_prefix_cache* cache);
int molt_prefix_cache_acquire(molt_prefix_cache* cache, const int32_t* tokens, int n,
                              int extra_tokens, int32_t* block_table, int max_blocks,
                              int* n_cached);
int molt_prefix_cache_commit(molt_prefix_cache* cache, const int32_t* tokens, int n,
                             const int32_t* block_table, int n_blocks);
int molt_prefix_cache_release(molt_prefix_cache* cache, const int32_t* block_table, int n_blocks);
int molt_prefix_cache_stats(const molt_prefix_cache* cache, long long* out);

/* ------------------------------------------------------------------------------
 * molt_score_tokens -- behavior-log-prob recompute with routing replay: the actor's pass
 * over the tokens the engine emitted (Sec. 4.1: rollout routing replay records expert
 * choices during generation and reuses them in the actor, with route alignment and
 * numerical-consistency diagnostics; Sec. 4.2, Eq. 1: recorded token IDs and behavior
 * log-probabilities). The verify step's forward over tokens[b, 0..k] at positions
 * context_lens[b] + j, with each MoE layer's experts taken from replay_routes (their
 * weights still come from the router, a softmax over the router logits of the given
 * experts; replay_routes NULL: the router chooses), then
 *   out_logprobs[b, j] = log softmax(logits[b, j])[targets[b, j]]   (NaN for a target
 *                        outside [0, V)), computed exactly as molt_spec_accept's log-probs.
 * On the weights that generated them, tokens = the verify step's tokens, targets = its
 * out_tokens and replay_routes = its out_routes reproduce its out_logprobs and logits bit
 * for bit. Writes the window's keys/values into the cache like molt_verify_step.
 *   tokens, targets  [B, 1+k] i32;  replay_routes [n_layers, B*(1+k), top_k] i32 or NULL
 *                    (an id outside [0, E) is taken as expert 0)
 *   out_logprobs     [B, 1+k] f32;  out_logits [B, 1+k, V] f32 or NULL;
 *   out_routes       [n_layers, B*(1+k), top_k] i32 or NULL (the routes used)
 * ---------------------------------------------------------------------------- */
size_t molt_score_tokens_workspace_size(const molt_model* m, int B, int k, int max_blocks_per_seq);
int molt_score_tokens(const molt_model* m, const molt_kv* kv, int B, int k, const int32_t* tokens,
                      const int32_t* targets, const int32_t* replay_routes, float* out_logprobs,
                      float* out_logits, int32_t* out_routes, void* workspace,
                      size_t workspace_bytes, molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * MTP draft head: the checkpoint's multi-token-prediction head that drafts the k
 * tokens the next verify step checks (Sec. 4.1 control table: number of
 * speculative tokens; Sec. 5.4: the MTP head shortens generation about five-fold).
 * The paper does not print the head; it is the DeepSeek-V3 MTP module: one decoder
 * layer of the target's structure with its own paged KV cache, sharing the target's
 * embedding and LM head:
 *   x = [RMSNorm(Emb(t); enorm) ; RMSNorm(h; hnorm)] eh_proj^T   (halves rounded to dtype)
 *   x = layer(x);  logits = RMSNorm(x; layer->final_norm) lm_head^T;  q = softmax(logits)
 * A row (h_p, token at p+1) sits at cache position p and predicts the token at p+2.
 * ---------------------------------------------------------------------------- */
typedef struct molt_mtp {
  const float* enorm;       /* [d] gain of the embedding half                            */
  const float* hnorm;       /* [d] gain of the hidden-state half                         */
  const void* eh_proj;      /* [d, 2d] dtype, tiled (molt_pack_weights, row_bytes 2d*es) */
  const molt_model* layer;  /* the head's decoder layer: n_layers = 1, the target's
                               d_model/heads/experts/dtypes; layer->final_norm is the
                               head's output norm; its embed/lm_head/vocab are not used  */
} molt_mtp;

/* ------------------------------------------------------------------------------
 * molt_mtp_draft -- one draft step after a verify step of sequence b (context c_b,
 * tokens x_0..x_k at positions c_b..c_b+k, n_b accepted drafts, emitted token y_b):
 *  * catch-up: rows j = 0..k at positions c_b + j with h = hidden row b*(1+k)+j and
 *    token x_{j+1} (j < n_b) or y_b (j >= n_b); row n_b yields draft 1 (rows past n_b
 *    are computed and ignored; their cache slots are rewritten later);
 *  * drafting: draft i+1 (i = 1..k-1) from one row at position c_b + n_b + i with h =
 *    the head's previous output and token = draft i.
 * Each draft is drawn from q with molt_spec_accept's integer inverse CDF and one
 * uniform; with out_draft_probs == NULL the drafts are greedy (first argmax of the
 * logits; verify them with draft_probs = NULL).
 *   target        the target model (embed, lm_head, vocab, d_model, dtype are used)
 *   mtp, mtp_kv   the head and its one-layer cache; mtp_kv's block tables and
 *                 context_lens are the verify step's (c_b, before the caller advances)
 *   k             >= 1
 *   hidden        [B*(1+k), d] f32: molt_verify_step's out_hidden
 *   tokens        [B, 1+k] i32: the verify step's tokens
 *   n_accepted    [B] i32 in [0, k];  next_tokens [B] i32: out_tokens[b, n_accepted[b]]
 *   uniforms      [B, k] f32 in [0, 1) (draft i+1 uses uniforms[b, i]); NULL if greedy
 *   out_drafts    [B, k] i32: the next verify step's drafts
 *   out_draft_probs [B, k, V] f32: q of each draft (the next verify step's draft_probs),
 *                 or NULL for greedy drafts
 * Writes the head's cache at positions c_b .. c_b + k and c_b + n_b + 1 .. c_b + n_b + k
 * - 1; c_b + max(k, n_b + k - 1) < 16 * max_blocks_per_seq is the caller's duty
 * (positions past the block table are computed and not written).
 * ---------------------------------------------------------------------------- */
/* molt_mtp_draft_window -- the same step with a catch-up window of `window` rows per
 * sequence instead of 1+k: hidden [B*window, d] and tokens [B, window] at positions
 * c_b .. c_b + window - 1, n_accepted[b] in [0, window - 1] the row that yields draft 1.
 * After a prefill (window = its n, n_accepted = lens - 1, next_tokens = the token sampled
 * from its logits, hidden = its out_hidden) it fills the head's cache for the prompt and
 * drafts the first k tokens; molt_mtp_draft is window = k + 1. Positions written:
 * c_b .. c_b + window - 1 and c_b + n_b + 1 .. c_b + n_b + k - 1. */
size_t molt_mtp_draft_window_workspace_size(const molt_model* target, const molt_mtp* mtp, int B,
                                            int window, int k, int max_blocks_per_seq);
int molt_mtp_draft_window(const molt_model* target, const molt_mtp* mtp, const molt_kv* mtp_kv,
                          int B, int window, int k, const float* hidden, const int32_t* tokens,
                          const int32_t* n_accepted, const int32_t* next_tokens,
                          const float* uniforms, int32_t* out_drafts, float* out_draft_probs,
                          void* workspace, size_t workspace_bytes, molt_stream_t stream);
size_t molt_mtp_draft_workspace_size(const molt_model* target, const molt_mtp* mtp, int B, int k,
                                     int max_blocks_per_seq);
int molt_mtp_draft(const molt_model* target, const molt_mtp* mtp, const molt_kv* mtp_kv, int B,
                   int k, const float* hidden, const int32_t* tokens, const int32_t* n_accepted,
                   const int32_t* next_tokens, const float* uniforms, int32_t* out_drafts,
                   float* out_draft_probs, void* workspace, size_t workspace_bytes,
                   molt_stream_t stream);

/* ------------------------------------------------------------------------------
 * Kernel-group timing (a measurement aid, not part of the method). While a group is
 * enabled, every launch of it is bracketed by two HIP events recorded on the call's
 * stream (each pair costs a few microseconds of stream time: enable only the groups
 * being measured); molt_profile_read synchronises on the recorded events and returns the
 * summed elapsed time and the number of bracketed launches of one group. Events come
 * from a pool of 4096 pairs created on the first enable (no device memory);
 * launches beyond the pool are not timed. Process-wide state: enable, run and read
 * from one host thread.
 * Groups: 0 attention (+ split merge), 1 expert GEMMs (gate_up + down), 2 LM head,
 * 3 sampler (all four passes), 4 dense projections (QKV, O, router).
 * ---------------------------------------------------------------------------- */
typedef enum {
  MOLT_PROF_ATTENTION = 0,
  MOLT_PROF_EXPERT_GEMM = 1,
  MOLT_PROF_LM_HEAD = 2,
  MOLT_PROF_SAMPLER = 3,
  MOLT_PROF_PROJECTIONS = 4
} molt_prof_group;
/* group_mask: bit g times group g (-1: all); nonzero starts and clears, 0 stops */
int molt_profile_enable(int group_mask);
/* time only every n-th launch of each enabled group (launches 0, n, 2n, ... counted per
 * group from the last enable; default 1 = every launch). INVALID_ARG for n < 1. */
int molt_profile_every(int n);
int molt_profile_read(int group, double* total_ms, int* launches);

#ifdef __cplusplus
}
#endif
#endif /* MOLT_H */
