// Internal host-side interface between the C-ABI layer and the kernel files.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/molt.h"

namespace molt {

// ------------------------------------------------------------- workspace carving
struct Carver {
  char* base;
  size_t used = 0;
  size_t cap;
  Carver(void* p, size_t c) : base(static_cast<char*>(p)), cap(c) {}
  template <typename T>
  T* take(size_t n) {
    // 256-byte aligned addresses (the sizes reserve 256 bytes for an unaligned base)
    const size_t b = reinterpret_cast<size_t>(base);
    used = ((b + used + 255) & ~size_t(255)) - b;
    T* p = reinterpret_cast<T*>(base ? base + used : nullptr);
    used += n * sizeof(T);
    return p;
  }
};

// ------------------------------------------------------------- sampler
int sampler_chunk_elems();
size_t sampler_ws_bytes(int B, int k, int V);
hipError_t launch_spec_accept(const float* logits, const float* q, const int32_t* drafts,
                              const float* u, int B, int k, int V, int32_t* out_tokens,
                              int32_t* out_n, float* out_lp, void* ws, hipStream_t s,
                              int draft_stride = -1, int draft_offset = 0);

// Scores of given tokens: out[r] = log softmax(logits[r])[targets[r]] with the accept
// decisions' row moments (NaN for a target outside [0, V)).
size_t token_logprob_ws_bytes(long rows, int V);
hipError_t launch_token_logprobs(const float* logits, long rows, int V, const int32_t* targets,
                                 float* out, void* ws, hipStream_t s);

// Draws of the MTP draft head, one per row: token ~ softmax(logits[b]) by the integer
// inverse CDF of launch_spec_accept (a step without drafts, uniform u[b]); with q_out also
// q_out[b * q_stride + t] = softmax(logits[b])_t. u == nullptr: greedy, token = first argmax.
size_t draft_draw_ws_bytes(int B, int V);
hipError_t launch_draft_draw(const float* logits, int B, int V, const float* u, int32_t* out_tok,
                             float* q_out, long q_stride, void* ws, hipStream_t s);

// ------------------------------------------------------------- elementwise
hipError_t launch_embed(const void* table, const int32_t* tokens, int T, int d, int V,
                        molt_dtype dt, float* x, hipStream_t s);
// x[t] += sum of nparts split-K partials (part[s * T * d ..], split order) and, with o, the
// MoE combine sum_j w[t, j] o[t * K + j]; then with g: y = rmsnorm(x) * g in act dtype,
// tiled layout (rows padded to 32 by the caller's allocation), optionally with its fp8
// row codes (tiled) and scales, and row-major copies of y (y_rows, bf16) and of its codes
// (yq_rows)
hipError_t launch_residual_norm(float* x, const float* part, int nparts, const float* o,
                                const float* w, int K, const float* g, int T, int d, float eps,
                                molt_dtype dt, void* y, uint8_t* yq, float* ys, hipStream_t s,
                                void* y_rows = nullptr, uint8_t* yq_rows = nullptr);
// RoPE cos/sin of the step's B*(1+k) positions (f64 pairs, [T, D/2]), shared by all layers;
// with kv_slot also each token's KV-cache slot (block * 16 + position % 16, -1 when the block
// table entry is out of range)
hipError_t launch_rope_table(const int32_t* ctx, int B, int k, int D, float theta, void* table,
                             const int32_t* bt, int max_blocks, int num_blocks, int32_t* kv_slot,
                             hipStream_t s);
hipError_t launch_rope_kv_write(const float* qkv, int B, int k, int Hq, int Hkv, int D,
                                const void* table, const int32_t* ctx, const int32_t* bt,
                                int max_blocks, int num_blocks, molt_dtype dt, void* q_out,
                                void* k_cache, void* v_cache, hipStream_t s);
// fp8 rows of a tiled bf16 matrix: rows = *n_rows when n_rows is given (padded expert
// order, pperm marks padding rows), else max_rows
hipError_t launch_quant_rows_tiled(const uint16_t* h, const int32_t* pperm, const int32_t* n_rows,
                                   long max_rows, int cols, uint8_t* q, float* scale,
                                   hipStream_t s);
// out[t] (+)= sum_j w[t, j] o[t * K + j]
hipError_t launch_combine(const float* o, const float* w, int T, int K, int d, float* out,
                          bool accumulate, hipStream_t s);

// MTP draft head rows. Catch-up row bW+j (W rows per sequence) takes token tokens[b, j+1]
// (j < n_b) or next[b], and u_col[b] = u[b, 0] (u: [B, k], may be null).
hipError_t launch_mtp_catchup(const int32_t* tokens, const int32_t* n_acc, const int32_t* next,
                              const float* u, int B, int W, int k, int32_t* row_tok, float* u_col,
                              hipStream_t s);
// y[t] = [RMSNorm(Emb[tok[t]]; ge) ; RMSNorm(h[t]; gh)] rounded to dt, tiled [T, 2d]
hipError_t launch_mtp_input(const void* embed, const int32_t* tok, const float* h, const float* ge,
                            const float* gh, int T, int d, int V, float eps, molt_dtype dt,
                            void* y, hipStream_t s);
// hsel[b] = x[b(k+1) + n_b + delta] (f32), ysel row b = yf row b(k+1) + n_b + delta (tiled,
// dt); n_b + delta clamped to [0, k]
hipError_t launch_mtp_select(const float* x, const void* yf, const int32_t* n_acc, int B, int k,
                             int d, molt_dtype dt, float* hsel, void* ysel, hipStream_t s,
                             int delta = 0);
// drafts[b, i] = tok[b]; then (i + 1 < k) row_tok[b] = tok[b], ctx_next[b] = ctx[b] + n_b +
// i + 1 (n_b clamped to [0, W - 1]), u_col[b] = u[b, i + 1]
hipError_t launch_mtp_record(const int32_t* tok, int i, int B, int W, int k, const int32_t* ctx,
                             const int32_t* n_acc, const float* u, int32_t* drafts,
                             int32_t* row_tok, int32_t* ctx_next, float* u_col, hipStream_t s);

// ------------------------------------------------------------- routing
// top-K + softmax of router logits (the sum, in order, of nparts split-K partials
// logits[s * T * E ..]; or replay ids); stable permutation perm (position -> pair) and its
// padded copy (pperm: padded row -> pair or -1, n_padded rows); tile table in padded rows
// n_tiles of launch_route is followed by 2 x kTileQueues ints: the per-XCD tile queues of the
// gate_up and down GEMMs, which the permutation zeroes.
constexpr int kTileQueues = 8;
hipError_t launch_route(const float* logits, int nparts, const float* bias, const int32_t* replay,
                        int T, int E, int K, int32_t* ids, float* w, int32_t* counts,
                        int32_t* offsets, int32_t* perm, int32_t* pperm, int32_t* n_padded,
                        int tile_m, int32_t* tiles, int max_tiles, int32_t* n_tiles,
                        hipStream_t s);
int max_expert_tiles(int T, int E, int K, int tile_m);
long max_padded_rows(int T, int E, int K);

// ------------------------------------------------------------- GEMMs
// C[M, N] (f32, row-major) = A[M, K] * B[N, K]^T, A/B in dt (F32 or BF16), both tiled (rows
// padded to 32); epilogue adds into C when accumulate. bf16 may split K when `part` holds
// enough floats for the partial sums (gemm_plan). With splits_out the fixed-order sum of
// the partials is left to the caller: *splits_out = S > 1 means C was not touched and
// part[s * M * N ..] holds split s; S = 1 means C was written as usual.
struct GemmPlan { int bm, splits; };
GemmPlan gemm_plan(int M, int N, int K, long part_elems);
hipError_t launch_gemm(const void* A, const void* Bw, float* C, int M, int N, int K, molt_dtype dt,
                       bool accumulate, float* part, long part_elems, hipStream_t s,
                       int* splits_out = nullptr);
// bf16 QKV projection (A tiled [M, K_in], weights tiled [(Hq + 2 Hkv) * 128, K_in]) with the
// RoPE of launch_rope_kv_write and its q / paged K / paged V writes fused into the epilogue;
// head_dim 128, same arithmetic (f32 sums rotated in f64 with the step's table)
hipError_t launch_qkv_rope(const void* A, const void* Bw, int M, int K_in, int Hq, int Hkv,
                           const void* table, const int32_t* kv_slot, void* q_out, void* k_cache,
                           void* v_cache, hipStream_t s);
// Grouped expert GEMMs over the tile table built by launch_route. bf16/fp8: A and the
// weights in the tiled layout, gate_up writes h tiled; f32: row-major A and h, tiled
// weights. Rows are padded-order; down writes o[pair]. gate_up with a_rows (the token
// rows in the expert dtype, row-major [T, K]) reads each padded row's token row through
// pperm instead of the gathered copy a.
hipError_t launch_moe_gate_up(const void* a, const void* a_rows, const float* a_scale,
                              const int32_t* pperm, int K_top, const void* w_gu, const float* s_gu,
                              int d, int F, molt_dtype wdt, const int32_t* tiles,
                              const int32_t* n_tiles, int max_tiles, int tile_m, void* h,
                              hipStream_t s);
hipError_t launch_moe_down(const void* a, const float* a_scale, const int32_t* pperm,
                           const void* w_d, const float* s_d, int d, int F, molt_dtype wdt,
                           const int32_t* tiles, const int32_t* n_tiles, int max_tiles,
                           int tile_m, float* o, hipStream_t s);
// row-major [rows, row_bytes] -> tiled layout (row_bytes % 128 == 0), rows padded to a
// multiple of 32 with zeros
hipError_t launch_pack_tiled(const void* src, void* dst, long rows, long row_bytes, hipStream_t s);
// tiled rows in padded expert order from tiled token rows: row = src[pperm[row] / K_top];
// padding rows are left unwritten
hipError_t launch_gather_tiled(const void* src, const int32_t* pperm, int K_top,
                               const int32_t* n_rows, long max_rows, long row_bytes, void* dst,
                               hipStream_t s);
int moe_tile_m(molt_dtype wdt, int T, int K, int E);

// ------------------------------------------------------------- attention
size_t attention_ws_bytes(int B, int k, int Hq, int Hkv, int D, int max_blocks);
// out [T, Hq*D] row-major, or tiled (rows padded to 32 by the caller) with out_tiled
hipError_t launch_paged_attention(const void* q, const void* kc, const void* vc, const int32_t* bt,
                                  const int32_t* ctx, int B, int k, int Hq, int Hkv, int D,
                                  int max_blocks, molt_dtype dt, void* out, bool out_tiled,
                                  void* ws, hipStream_t s);

}  // namespace molt
