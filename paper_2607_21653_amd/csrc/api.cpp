// C-ABI layer: host-side validation (before anything is enqueued), workspace
// carving and launch sequencing for the verify step. No device allocation, no
// synchronisation, no state kept between calls.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return MOLT_OK;
}

int hip_status(hipError_t e, const char* where) {
  if (e != hipSuccess) return fail(MOLT_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}

// ---- kernel-group timing with HIP events (opt-in, process-wide)
struct Profiler {
  static constexpr int kPairs = 4096;
  int mask = 0;                 // bit g: group g is timed
  int every = 1;                // time launches 0, every, 2 every, ... of each group
  int seen[8] = {};             // launches of each group since the last enable
  bool ready = false;
  hipEvent_t ev[2 * kPairs];
  int used = 0;
  int group[kPairs];
};
Profiler g_prof;

struct ProfScope {
  int slot = -1;
  hipStream_t s;
  ProfScope(int grp, hipStream_t st) : s(st) {
    if (!((g_prof.mask >> grp) & 1) || g_prof.used >= Profiler::kPairs) return;
    if (g_prof.seen[grp]++ % g_prof.every != 0) return;
    slot = g_prof.used++;
    g_prof.group[slot] = grp;
    hipEventRecord(g_prof.ev[2 * slot], s);
  }
  ~ProfScope() {
    if (slot >= 0) hipEventRecord(g_prof.ev[2 * slot + 1], s);
  }
};

#define REQUIRE(cond, ...)                                   \
  do {                                                       \
    if (!(cond)) return fail(MOLT_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)

int check_ws(void* ws, size_t have, size_t need) {
  if (need > 0 && (ws == nullptr || have < need))
    return fail(MOLT_ERR_WORKSPACE, "workspace of %zu bytes at %p is smaller than the %zu required",
                have, ws, need);
  return MOLT_OK;
}

}  // namespace

extern "C" {

const char* molt_last_error(void) { return g_err.c_str(); }

int molt_version(void) { return 103; }

// ------------------------------------------------------------------ profiling

int molt_profile_enable(int group_mask) {
  const bool enable = group_mask != 0;
  if (enable && !g_prof.ready) {
    for (int i = 0; i < 2 * Profiler::kPairs; ++i) {
      hipError_t e = hipEventCreate(&g_prof.ev[i]);
      if (e != hipSuccess) return hip_status(e, "molt_profile_enable");
    }
    g_prof.ready = true;
  }
  if (enable) {
    g_prof.used = 0;
    for (int& n : g_prof.seen) n = 0;
  }
  g_prof.mask = group_mask;
  return ok();
}

int molt_profile_every(int n) {
  REQUIRE(n >= 1, "n = %d must be >= 1", n);
  g_prof.every = n;
  return ok();
}

int molt_profile_read(int group, double* total_ms, int* launches) {
  REQUIRE(total_ms && launches, "NULL output pointer");
  double tot = 0.0;
  int n = 0;
  for (int i = 0; i < g_prof.used; ++i) {
    if (g_prof.group[i] != group) continue;
    hipError_t e = hipEventSynchronize(g_prof.ev[2 * i + 1]);
    if (e != hipSuccess) return hip_status(e, "molt_profile_read");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]);
    if (e != hipSuccess) return hip_status(e, "molt_profile_read");
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return ok();
}

// ------------------------------------------------------------------ spec accept

static int spec_accept_shape_ok(int B, int k, int V) {
  REQUIRE(B >= 1, "B = %d must be >= 1", B);
  REQUIRE(k >= 0, "k = %d must be >= 0", k);
  REQUIRE(V >= 1, "V = %d must be >= 1", V);
  const double rows = double(B) * (k + 1);
  REQUIRE(rows * V < 4.0e18, "B*(k+1)*V too large");
  const double nch = std::ceil(double(V) / molt::sampler_chunk_elems());
  REQUIRE(rows * nch < 16777216.0, "B*(k+1)*ceil(V/%d) = %.0f exceeds 2^24 workgroups",
          molt::sampler_chunk_elems(), rows * nch);
  return MOLT_OK;
}

size_t molt_spec_accept_workspace_size(int B, int k, int V) {
  if (B < 1 || k < 0 || V < 1) return 0;
  return molt::sampler_ws_bytes(B, k, V);
}

int molt_spec_accept(const float* logits, const float* draft_probs, const int32_t* draft_tokens,
                     const float* uniforms, int B, int k, int V, int32_t* out_tokens,
                     int32_t* out_num_accepted, float* out_logprobs, void* workspace,
                     size_t workspace_bytes, molt_stream_t stream) {
  if (int r = spec_accept_shape_ok(B, k, V)) return r;
  REQUIRE(logits, "logits is NULL");
  REQUIRE(uniforms, "uniforms is NULL");
  REQUIRE(k == 0 || draft_tokens, "draft_tokens is NULL with k = %d", k);
  REQUIRE(out_tokens, "out_tokens is NULL");
  REQUIRE(out_num_accepted, "out_num_accepted is NULL");
  if (int r = check_ws(workspace, workspace_bytes, molt_spec_accept_workspace_size(B, k, V)))
    return r;
  hipError_t e;
  {
    ProfScope ps(MOLT_PROF_SAMPLER, reinterpret_cast<hipStream_t>(stream));
    e = molt::launch_spec_accept(logits, draft_probs, draft_tokens, uniforms, B, k, V, out_tokens,
                                 out_num_accepted, out_logprobs, workspace,
                                 reinterpret_cast<hipStream_t>(stream));
  }
  return hip_status(e, "molt_spec_accept");
}

// ------------------------------------------------------------------ spec accept, no allocation

// The fixed scratch array of the allocation-free accept: one copy per GPU, held until the
// process ends. In host code `scratch` names a host-side stand-in, not device memory: host
// code reaches the array only through the address hipGetSymbolAddress returns for the
// current device.
static __device__ __align__(256) unsigned char scratch[MOLT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;

struct ScratchSlot {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[kMaxDevices];

// Device address of the current device's scratch array, looked up on the first call on
// that device (with it current) and kept.
hipError_t scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  ScratchSlot& slot = g_scratch[dev];
  std::call_once(slot.once, [&slot] {
    slot.err = hipGetSymbolAddress(&slot.ptr, HIP_SYMBOL(scratch));
  });
  *out = slot.ptr;
  return slot.err;
}

}  // namespace

int molt_spec_accept_noalloc(const float* logits, const float* draft_probs,
                             const int32_t* draft_tokens, const float* uniforms, int B, int k,
                             int V, int32_t* out_tokens, int32_t* out_num_accepted,
                             float* out_logprobs, molt_stream_t stream) {
  if (int r = spec_accept_shape_ok(B, k, V)) return r;
  REQUIRE(logits, "logits is NULL");
  REQUIRE(uniforms, "uniforms is NULL");
  REQUIRE(k == 0 || draft_tokens, "draft_tokens is NULL with k = %d", k);
  REQUIRE(out_tokens, "out_tokens is NULL");
  REQUIRE(out_num_accepted, "out_num_accepted is NULL");
  const size_t need = molt_spec_accept_workspace_size(B, k, V);
  REQUIRE(need <= size_t(MOLT_NOALLOC_SCRATCH_BYTES),
          "B = %d, k = %d, V = %d need %zu bytes of scratch; the allocation-free entry point "
          "holds %zu (use molt_spec_accept with a workspace)",
          B, k, V, need, size_t(MOLT_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  hipError_t e = scratch_on_current_device(&ws);
  if (e != hipSuccess) return hip_status(e, "molt_spec_accept_noalloc: scratch lookup");
  {
    ProfScope ps(MOLT_PROF_SAMPLER, reinterpret_cast<hipStream_t>(stream));
    e = molt::launch_spec_accept(logits, draft_probs, draft_tokens, uniforms, B, k, V, out_tokens,
                                 out_num_accepted, out_logprobs, ws,
                                 reinterpret_cast<hipStream_t>(stream));
  }
  return hip_status(e, "molt_spec_accept_noalloc");
}

// ------------------------------------------------------------------ helpers

static size_t dt_size(molt_dtype t) { return t == MOLT_F32 ? 4 : t == MOLT_BF16 ? 2 : 1; }

static bool act_ok(molt_dtype a) { return a == MOLT_F32 || a == MOLT_BF16; }

static bool pair_ok(molt_dtype act, molt_dtype w) {
  return (act == MOLT_F32 && w == MOLT_F32) || (act == MOLT_BF16 && (w == MOLT_BF16 || w == MOLT_FP8_E4M3));
}

namespace {

long pad32(long n) { return (n + 31) / 32 * 32; }

// floats of split-K partial sums a dense GEMM of this shape would use (0: no split)
long gemm_part_elems(int M, int N, int K, molt_dtype dt) {
  if (dt != MOLT_BF16) return 0;
  const molt::GemmPlan g = molt::gemm_plan(M, N, K, 1L << 62);
  return g.splits > 1 ? long(g.splits) * M * N : 0;
}

struct MoeWs {
  float* g; int32_t* ids; float* w; int32_t* counts; int32_t* offsets; int32_t* perm;
  int32_t* pperm; int32_t* n_padded; int32_t* tiles; int32_t* n_tiles;
  uint8_t* xq; float* xs; void* xt; void* h; uint8_t* hq; float* hs; float* o;
  float* part; long part_elems;   // split-K partial sums of the router GEMM
  long max_rows; int max_tiles; int tile_m;
};

// Intermediates of the grouped GEMMs live in padded expert order (each expert's rows start
// at a multiple of 32), tiled: the gathered activations xt (expert dtype), the SwiGLU
// product h (act dtype) and its fp8 codes hq/hs. xq/xs: fp8 codes of the input when the
// caller has none. The per-pair expert outputs o are row-major in pair order (token * K +
// slot).
MoeWs carve_moe(molt::Carver& c, int T, int d, int E, int K, int F, molt_dtype act, molt_dtype w) {
  MoeWs m{};
  const long P = long(T) * K;
  const int tm = molt::moe_tile_m(w, T, K, E);
  m.tile_m = tm;
  m.max_tiles = molt::max_expert_tiles(T, E, K, tm);
  m.max_rows = molt::max_padded_rows(T, E, K);
  const long R = m.max_rows;
  m.g = c.take<float>(long(T) * E);
  m.ids = c.take<int32_t>(P);
  m.w = c.take<float>(P);
  m.counts = c.take<int32_t>(E);
  m.offsets = c.take<int32_t>(E + 1);
  m.perm = c.take<int32_t>(P);
  m.pperm = c.take<int32_t>(R);
  m.n_padded = c.take<int32_t>(1);
  m.tiles = c.take<int32_t>(long(m.max_tiles) * 4);
  m.n_tiles = c.take<int32_t>(1 + 2 * molt::kTileQueues);   // + the GEMMs' tile queues
  if (w == MOLT_FP8_E4M3) {
    m.xq = c.take<uint8_t>(pad32(T) * d);
    m.xs = c.take<float>(pad32(T));
    m.hq = c.take<uint8_t>(R * F);
    m.hs = c.take<float>(R);
  }
  m.xt = c.take<uint8_t>(R * d * dt_size(w));
  m.h = c.take<uint8_t>(R * F * dt_size(act));
  m.o = c.take<float>(P * d);
  m.part_elems = gemm_part_elems(T, E, d, act);
  m.part = c.take<float>(m.part_elems);
  return m;
}

int moe_shape_ok(int T, int d, int E, int K, int F, molt_dtype act, molt_dtype w) {
  REQUIRE(T >= 1, "T = %d must be >= 1", T);
  REQUIRE(E >= 1 && E <= 256, "E = %d must be in [1, 256]", E);
  REQUIRE(K >= 1 && K <= E && K <= 64, "K = %d must be in [1, min(E, 64)]", K);
  REQUIRE(pair_ok(act, w), "unsupported (activation, expert) dtype pair (%d, %d)", int(act), int(w));
  const int mult = w == MOLT_FP8_E4M3 ? 128 : 64;
  REQUIRE(d >= mult && d % mult == 0, "d = %d must be a positive multiple of %d", d, mult);
  REQUIRE(F >= mult && F % mult == 0, "F = %d must be a positive multiple of %d", F, mult);
  REQUIRE(double(T) * K * (F > d ? F : d) < 2.0e9, "T*K*max(F, d) too large");
  return MOLT_OK;
}

// Enqueues the MoE layer on normalised input x (act dtype, tiled, rows padded to 32; xq/xs =
// its tiled fp8 codes when the caller already quantised them). Router and expert weights
// tiled. With out: out = sum (accumulate: out += sum); without, the per-pair expert outputs
// m.o and route weights m.w are left for the caller to combine.
hipError_t run_moe(const MoeWs& m, const void* x, const uint8_t* xq, const float* xs,
                   const void* w_router, const float* bias, const void* w_gu, const void* w_d,
                   const float* s_gu, const float* s_d, int T, int d, int E, int K, int F,
                   molt_dtype act, molt_dtype wdt, const int32_t* replay, float* out,
                   bool accumulate, hipStream_t s, const void* x_rows = nullptr) {
  hipError_t e;
  int nparts = 1;
  {
    ProfScope ps(MOLT_PROF_PROJECTIONS, s);
    if ((e = molt::launch_gemm(x, w_router, m.g, T, E, d, act, false, m.part, m.part_elems, s,
                               &nparts)) != hipSuccess)
      return e;
  }
  if ((e = molt::launch_route(nparts > 1 ? m.part : m.g, nparts, bias, replay, T, E, K, m.ids, m.w,
                              m.counts, m.offsets, m.perm, m.pperm, m.n_padded, m.tile_m,
                              m.tiles, m.max_tiles, m.n_tiles, s)) != hipSuccess)
    return e;
  const bool fp8 = wdt == MOLT_FP8_E4M3;
  const bool xq_given = xq != nullptr;
  if (fp8 && xq == nullptr) {
    if ((e = molt::launch_quant_rows_tiled(static_cast<const uint16_t*>(x), nullptr, nullptr, T, d,
                                           m.xq, m.xs, s)) != hipSuccess)
      return e;
    xq = m.xq;
    xs = m.xs;
  }
  // row-major token rows at hand (bf16 rows of x for bf16 experts, the caller's fp8 codes
  // for fp8 experts): gate_up reads them through the permutation, no gathered copy
  const bool rows = x_rows != nullptr &&
                    (wdt == MOLT_BF16 ? act == MOLT_BF16 : wdt == MOLT_FP8_E4M3 && xq_given);
  const void* src = fp8 ? static_cast<const void*>(xq) : x;
  if (!rows && (e = molt::launch_gather_tiled(src, m.pperm, K, m.n_padded, m.max_rows,
                                              long(d) * dt_size(wdt), m.xt, s)) != hipSuccess)
    return e;
  {
    ProfScope ps(MOLT_PROF_EXPERT_GEMM, s);
    if ((e = molt::launch_moe_gate_up(m.xt, rows ? x_rows : nullptr, xs, m.pperm, K, w_gu, s_gu, d,
                                      F, wdt, m.tiles, m.n_tiles, m.max_tiles, m.tile_m, m.h,
                                      s)) != hipSuccess)
      return e;
  }
  if (fp8) {
    if ((e = molt::launch_quant_rows_tiled(static_cast<const uint16_t*>(m.h), m.pperm, m.n_padded,
                                           m.max_rows, F, m.hq, m.hs, s)) != hipSuccess)
      return e;
  }
  {
    ProfScope ps(MOLT_PROF_EXPERT_GEMM, s);
    if ((e = molt::launch_moe_down(fp8 ? static_cast<const void*>(m.hq) : m.h, m.hs, m.pperm, w_d,
                                   s_d, d, F, wdt, m.tiles, m.n_tiles, m.max_tiles, m.tile_m, m.o,
                                   s)) !=
        hipSuccess)
      return e;
  }
  if (out == nullptr) return hipSuccess;
  return molt::launch_combine(m.o, m.w, T, K, d, out, accumulate, s);
}

hipError_t copy_out(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (dst == nullptr || bytes == 0) return hipSuccess;
  return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, s);
}

}  // namespace

// ------------------------------------------------------------------ MoE layer

size_t molt_moe_layer_workspace_size(int T, int d, int E, int K, int F, molt_dtype act,
                                     molt_dtype w) {
  if (T < 1 || E < 1 || K < 1 || d < 1 || F < 1 || !pair_ok(act, w)) return 0;
  molt::Carver c(nullptr, 0);
  c.take<uint8_t>(pad32(T) * d * dt_size(act));   // tiled copy of x
  carve_moe(c, T, d, E, K, F, act, w);
  return c.used + 256;
}

int molt_moe_layer(const void* x, const void* w_router, const float* router_bias,
                   const void* w_gate_up, const void* w_down, const float* s_gate_up,
                   const float* s_down, int T, int d, int E, int K, int F, molt_dtype act_dtype,
                   molt_dtype w_dtype, const int32_t* replay_ids, float* out, int32_t* out_ids,
                   float* out_weights, int32_t* out_counts, int32_t* out_offsets,
                   int32_t* out_perm, void* workspace, size_t workspace_bytes,
                   molt_stream_t stream) {
  if (int r = moe_shape_ok(T, d, E, K, F, act_dtype, w_dtype)) return r;
  REQUIRE(x && w_router && w_gate_up && w_down && out, "a required pointer is NULL");
  REQUIRE(w_dtype != MOLT_FP8_E4M3 || (s_gate_up && s_down), "fp8 experts need s_gate_up and s_down");
  if (int r = check_ws(workspace, workspace_bytes,
                       molt_moe_layer_workspace_size(T, d, E, K, F, act_dtype, w_dtype)))
    return r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  molt::Carver c(workspace, workspace_bytes);
  void* xt = c.take<uint8_t>(pad32(T) * d * dt_size(act_dtype));
  MoeWs m = carve_moe(c, T, d, E, K, F, act_dtype, w_dtype);
  hipError_t e = molt::launch_pack_tiled(x, xt, T, long(d) * dt_size(act_dtype), s);
  if (e == hipSuccess)
    e = run_moe(m, xt, nullptr, nullptr, w_router, router_bias, w_gate_up, w_down, s_gate_up,
                s_down, T, d, E, K, F, act_dtype, w_dtype, replay_ids, out, false, s, x);
  const size_t P = size_t(T) * K;
  if (e == hipSuccess) e = copy_out(out_ids, m.ids, P * 4, s);
  if (e == hipSuccess) e = copy_out(out_weights, m.w, P * 4, s);
  if (e == hipSuccess) e = copy_out(out_counts, m.counts, size_t(E) * 4, s);
  if (e == hipSuccess) e = copy_out(out_offsets, m.offsets, size_t(E + 1) * 4, s);
  if (e == hipSuccess) e = copy_out(out_perm, m.perm, P * 4, s);
  return hip_status(e, "molt_moe_layer");
}

// ------------------------------------------------------------------ weight layout

int molt_pack_weights(const void* src, void* dst, long long rows, long long row_bytes,
                      molt_stream_t stream) {
  REQUIRE(src && dst, "a required pointer is NULL");
  REQUIRE(src != dst, "packing in place is not supported");
  REQUIRE(rows >= 1, "rows = %lld must be >= 1", rows);
  REQUIRE(row_bytes >= 128 && row_bytes % 128 == 0,
          "row_bytes = %lld must be a positive multiple of 128", row_bytes);
  return hip_status(molt::launch_pack_tiled(src, dst, rows, row_bytes,
                                            reinterpret_cast<hipStream_t>(stream)),
                    "molt_pack_weights");
}

// ------------------------------------------------------------------ dense GEMM

size_t molt_dense_gemm_workspace_size(int M, int N, int K, molt_dtype dtype) {
  if (M < 1 || N < 1 || K < 1 || !act_ok(dtype)) return 0;
  const long e = gemm_part_elems(M, N, K, dtype);
  return e ? size_t(e) * 4 + 256 : 0;
}

int molt_dense_gemm(const void* A, const void* B, float* C, int M, int N, int K, molt_dtype dtype,
                    int accumulate, void* workspace, size_t workspace_bytes, molt_stream_t stream) {
  REQUIRE(A && B && C, "a required pointer is NULL");
  REQUIRE(M >= 1 && N >= 1 && K >= 1, "M, N, K must be >= 1 (got %d, %d, %d)", M, N, K);
  REQUIRE(act_ok(dtype), "dtype must be F32 or BF16");
  REQUIRE(long(K) * dt_size(dtype) % 128 == 0, "K * sizeof(dtype) must be a multiple of 128 (K = %d)", K);
  if (int r = check_ws(workspace, workspace_bytes, molt_dense_gemm_workspace_size(M, N, K, dtype)))
    return r;
  hipError_t e;
  {
    ProfScope ps(MOLT_PROF_PROJECTIONS, reinterpret_cast<hipStream_t>(stream));
    e = molt::launch_gemm(A, B, C, M, N, K, dtype, accumulate != 0, static_cast<float*>(workspace),
                          long(workspace_bytes / 4), reinterpret_cast<hipStream_t>(stream));
  }
  return hip_status(e, "molt_dense_gemm");
}

// ------------------------------------------------------------------ paged attention

static int attn_shape_ok(int B, int k, int Hq, int Hkv, int D, int max_blocks, molt_dtype dt) {
  REQUIRE(B >= 1, "B = %d must be >= 1", B);
  REQUIRE(k >= 0, "k = %d must be >= 0", k);
  REQUIRE(act_ok(dt), "attention dtype must be F32 or BF16");
  REQUIRE(D == 64 || D == 128, "head_dim = %d must be 64 or 128", D);
  REQUIRE(Hkv >= 1 && Hq >= Hkv && Hq % Hkv == 0, "n_q_heads %d must be a multiple of n_kv_heads %d", Hq, Hkv);
  REQUIRE(dt == MOLT_F32 || Hq / Hkv <= 128, "Hq/Hkv = %d exceeds 128", Hq / Hkv);
  REQUIRE(double(B) * (k + 1) * Hq < 2.0e9, "B * (1+k) * Hq too large");
  REQUIRE(max_blocks >= 1, "max_blocks_per_seq = %d must be >= 1", max_blocks);
  REQUIRE(double(B) * Hkv * ((max_blocks + 63) / 64) < 2.0e9, "grid too large");
  return MOLT_OK;
}

size_t molt_paged_attention_workspace_size(int B, int k, int Hq, int Hkv, int D, int max_blocks) {
  if (B < 1 || k < 0 || Hq < 1 || Hkv < 1 || D < 1 || max_blocks < 1) return 0;
  return molt::attention_ws_bytes(B, k, Hq, Hkv, D, max_blocks);
}

int molt_paged_attention(const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_tables, const int32_t* context_lens, int B, int k,
                         int Hq, int Hkv, int D, int max_blocks, molt_dtype dtype, void* out,
                         void* workspace, size_t workspace_bytes, molt_stream_t stream) {
  if (int r = attn_shape_ok(B, k, Hq, Hkv, D, max_blocks, dtype)) return r;
  REQUIRE(q && k_cache && v_cache && block_tables && context_lens && out, "a required pointer is NULL");
  const size_t need = molt_paged_attention_workspace_size(B, k, Hq, Hkv, D, max_blocks);
  if (int r = check_ws(workspace, workspace_bytes, dtype == MOLT_F32 ? 0 : need)) return r;
  hipError_t e;
  {
    ProfScope ps(MOLT_PROF_ATTENTION, reinterpret_cast<hipStream_t>(stream));
    e = molt::launch_paged_attention(q, k_cache, v_cache, block_tables, context_lens, B, k, Hq, Hkv,
                                     D, max_blocks, dtype, out, false, workspace,
                                     reinterpret_cast<hipStream_t>(stream));
  }
  return hip_status(e, "molt_paged_attention");
}

// ------------------------------------------------------------------ decoder / verify step

namespace {

int model_ok(const molt_model* m, const molt_kv* kv, int B, int k, bool need_head) {
  REQUIRE(m != nullptr, "model is NULL");
  REQUIRE(m->n_layers >= 1, "n_layers = %d must be >= 1", m->n_layers);
  REQUIRE(act_ok(m->dtype), "model dtype must be F32 or BF16");
  if (int r = moe_shape_ok(B * (k + 1), m->d_model, m->n_experts, m->top_k, m->d_ff, m->dtype,
                           m->expert_dtype))
    return r;
  REQUIRE(m->d_model <= 16384, "d_model = %d must be <= 16384", m->d_model);
  REQUIRE(m->rms_eps >= 0.f, "rms_eps must be >= 0");
  REQUIRE(m->rope_theta > 0.f, "rope_theta must be > 0");
  REQUIRE(m->attn_norm && m->w_qkv && m->w_o && m->moe_norm && m->w_router && m->w_gate_up &&
              m->w_down,
          "a per-layer weight array is NULL");
  for (int l = 0; l < m->n_layers; ++l) {
    REQUIRE(m->attn_norm[l] && m->w_qkv[l] && m->w_o[l] && m->moe_norm[l] && m->w_router[l] &&
                m->w_gate_up[l] && m->w_down[l],
            "layer %d: a weight pointer is NULL", l);
    if (m->expert_dtype == MOLT_FP8_E4M3)
      REQUIRE(m->s_gate_up && m->s_down && m->s_gate_up[l] && m->s_down[l],
              "layer %d: fp8 experts need s_gate_up and s_down", l);
  }
  if (need_head) {
    REQUIRE(m->vocab >= 1, "vocab = %d must be >= 1", m->vocab);
    REQUIRE(m->embed && m->lm_head && m->final_norm, "embed, final_norm and lm_head are required");
  }
  REQUIRE(kv != nullptr, "kv is NULL");
  REQUIRE(kv->block_size == 16, "block_size = %d must be 16", kv->block_size);
  REQUIRE(kv->k_cache && kv->v_cache && kv->block_tables && kv->context_lens, "a kv pointer is NULL");
  for (int l = 0; l < m->n_layers; ++l)
    REQUIRE(kv->k_cache[l] && kv->v_cache[l], "layer %d: cache pointer is NULL", l);
  REQUIRE(kv->num_blocks >= 1, "num_blocks = %d must be >= 1", kv->num_blocks);
  return attn_shape_ok(B, k, m->n_q_heads, m->n_kv_heads, m->head_dim, kv->max_blocks_per_seq,
                       m->dtype);
}

struct DecWs {
  void* y; uint8_t* yq; float* ys; float* qkv; void* q; void* attn; void* attn_ws; MoeWs moe;
  void* y_rows;                   // the pre-MoE y row-major (bf16 experts) or its fp8 codes
                                  // row-major (fp8 experts): the expert GEMM's input
  float* part; long part_elems;   // split-K partial sums of the QKV and O projections
  void* rope;                     // RoPE cos/sin of the step's positions, [T, D/2] f64 pairs
  int32_t* kv_slot;               // KV-cache slot of each token of the step (or -1)
};

DecWs carve_dec(molt::Carver& c, const molt_model* m, int B, int k, int max_blocks) {
  DecWs w{};
  const long T = long(B) * (k + 1);
  const int d = m->d_model, D = m->head_dim, Hq = m->n_q_heads, Hkv = m->n_kv_heads;
  const size_t es = dt_size(m->dtype);
  const long Tp = pad32(T);                 // GEMM operands: tiled, rows padded to 32
  w.y = c.take<uint8_t>(Tp * d * es);
  if (m->expert_dtype == MOLT_FP8_E4M3) {
    w.yq = c.take<uint8_t>(Tp * d);
    w.ys = c.take<float>(Tp);
  }
  if (m->dtype == MOLT_BF16 && m->expert_dtype == MOLT_BF16) w.y_rows = c.take<uint8_t>(T * d * es);
  if (m->expert_dtype == MOLT_FP8_E4M3) w.y_rows = c.take<uint8_t>(T * d);
  if (!(m->dtype == MOLT_BF16 && D == 128))   // else RoPE is fused into the QKV epilogue
    w.qkv = c.take<float>(T * (Hq + 2 * Hkv) * D);
  w.q = c.take<uint8_t>(T * Hq * D * es);
  w.attn = c.take<uint8_t>(Tp * Hq * D * es);
  const size_t aws = m->dtype == MOLT_F32 ? 0 : molt::attention_ws_bytes(B, k, Hq, Hkv, D, max_blocks);
  w.attn_ws = c.take<uint8_t>(aws);
  w.moe = carve_moe(c, int(T), d, m->n_experts, m->top_k, m->d_ff, m->dtype, m->expert_dtype);
  const long pq = gemm_part_elems(int(T), (Hq + 2 * Hkv) * D, d, m->dtype);
  const long po = gemm_part_elems(int(T), d, Hq * D, m->dtype);
  w.part_elems = pq > po ? pq : po;
  w.part = c.take<float>(w.part_elems);
  w.rope = c.take<double>(T * D);
  w.kv_slot = c.take<int32_t>(T);
  return w;
}

// All layers on the residual stream x. With final_g, the last layer's MoE combine is fused
// with the final RMSNorm, whose tiled output goes to final_y. With replay ([L, T, K] expert
// ids), every MoE layer takes its experts from it (routing replay).
hipError_t run_decoder(const DecWs& w, const molt_model* m, const molt_kv* kv, int B, int k,
                       float* x, int32_t* routes, const float* final_g, void* final_y,
                       hipStream_t s, const int32_t* replay = nullptr) {
  const int T = B * (k + 1);
  const int d = m->d_model, D = m->head_dim, Hq = m->n_q_heads, Hkv = m->n_kv_heads;
  const int K = m->top_k, L = m->n_layers;
  const bool fp8 = m->expert_dtype == MOLT_FP8_E4M3;
  hipError_t e = hipSuccess;
#define RUN(call) do { if ((e = (call)) != hipSuccess) return e; } while (0)
  RUN(molt::launch_rope_table(kv->context_lens, B, k, D, m->rope_theta, w.rope, kv->block_tables,
                              kv->max_blocks_per_seq, kv->num_blocks, w.kv_slot, s));
  RUN(molt::launch_residual_norm(x, nullptr, 0, nullptr, nullptr, 0, m->attn_norm[0], T, d,
                                 m->rms_eps, m->dtype, w.y, nullptr, nullptr, s));
  for (int l = 0; l < L; ++l) {
    if (m->dtype == MOLT_BF16 && D == 128) {
      // one 128-column tile per head: RoPE and the KV-cache write in the GEMM epilogue
      ProfScope ps(MOLT_PROF_PROJECTIONS, s);
      RUN(molt::launch_qkv_rope(w.y, m->w_qkv[l], T, d, Hq, Hkv, w.rope, w.kv_slot, w.q,
                                kv->k_cache[l], kv->v_cache[l], s));
    } else {
      {
        ProfScope ps(MOLT_PROF_PROJECTIONS, s);
        RUN(molt::launch_gemm(w.y, m->w_qkv[l], w.qkv, T, (Hq + 2 * Hkv) * D, d, m->dtype, false,
                              w.part, w.part_elems, s));
      }
      RUN(molt::launch_rope_kv_write(w.qkv, B, k, Hq, Hkv, D, w.rope, kv->context_lens,
                                     kv->block_tables, kv->max_blocks_per_seq, kv->num_blocks,
                                     m->dtype, w.q, kv->k_cache[l], kv->v_cache[l], s));
    }
    {
      ProfScope ps(MOLT_PROF_ATTENTION, s);
      RUN(molt::launch_paged_attention(w.q, kv->k_cache[l], kv->v_cache[l], kv->block_tables,
                                       kv->context_lens, B, k, Hq, Hkv, D, kv->max_blocks_per_seq,
                                       m->dtype, w.attn, true, w.attn_ws, s));
    }
    int np = 1;   // O projection: accumulate into x, or leave split-K partials
    {
      ProfScope ps(MOLT_PROF_PROJECTIONS, s);
      RUN(molt::launch_gemm(w.attn, m->w_o[l], x, T, d, Hq * D, m->dtype, true, w.part,
                            w.part_elems, s, &np));
    }
    // x += O partials; y = RMSNorm(x) * moe_norm (+ fp8 codes)
    RUN(molt::launch_residual_norm(x, np > 1 ? w.part : nullptr, np > 1 ? np : 0, nullptr, nullptr,
                                   0, m->moe_norm[l], T, d, m->rms_eps, m->dtype, w.y,
                                   fp8 ? w.yq : nullptr, fp8 ? w.ys : nullptr, s,
                                   fp8 ? nullptr : w.y_rows,
                                   fp8 ? static_cast<uint8_t*>(w.y_rows) : nullptr));
    RUN(run_moe(w.moe, w.y, fp8 ? w.yq : nullptr, fp8 ? w.ys : nullptr, m->w_router[l],
                m->router_bias ? m->router_bias[l] : nullptr, m->w_gate_up[l], m->w_down[l],
                fp8 ? m->s_gate_up[l] : nullptr, fp8 ? m->s_down[l] : nullptr, T, d,
                m->n_experts, K, m->d_ff, m->dtype, m->expert_dtype,
                replay ? replay + size_t(l) * T * K : nullptr, nullptr, false, s, w.y_rows));
    if (routes) RUN(copy_out(routes + size_t(l) * T * K, w.moe.ids, size_t(T) * K * 4, s));
    // x += MoE combine; then the next layer's attention norm (or the final norm)
    const bool last = l + 1 == L;
    RUN(molt::launch_residual_norm(x, nullptr, 0, w.moe.o, w.moe.w, K,
                                   last ? final_g : m->attn_norm[l + 1], T, d, m->rms_eps,
                                   m->dtype, last ? final_y : w.y, nullptr, nullptr, s));
  }
#undef RUN
  return e;
}

}  // namespace

size_t molt_decoder_workspace_size(const molt_model* m, int B, int k, int max_blocks) {
  if (!m || B < 1 || k < 0 || max_blocks < 1 || !pair_ok(m->dtype, m->expert_dtype)) return 0;
  molt::Carver c(nullptr, 0);
  carve_dec(c, m, B, k, max_blocks);
  return c.used + 256;
}

int molt_decoder_forward(const molt_model* m, const molt_kv* kv, int B, int k, float* x,
                         int32_t* out_routes, void* workspace, size_t workspace_bytes,
                         molt_stream_t stream) {
  if (int r = model_ok(m, kv, B, k, false)) return r;
  REQUIRE(x, "x is NULL");
  if (int r = check_ws(workspace, workspace_bytes,
                       molt_decoder_workspace_size(m, B, k, kv->max_blocks_per_seq)))
    return r;
  molt::Carver c(workspace, workspace_bytes);
  DecWs w = carve_dec(c, m, B, k, kv->max_blocks_per_seq);
  return hip_status(run_decoder(w, m, kv, B, k, x, out_routes, nullptr, nullptr,
                                reinterpret_cast<hipStream_t>(stream)),
                    "molt_decoder_forward");
}

namespace {
struct StepWs { float* x; void* yf; float* logits; void* samp; DecWs dec; };
StepWs carve_step(molt::Carver& c, const molt_model* m, int B, int k, int max_blocks, bool own_logits) {
  StepWs w{};
  const long T = long(B) * (k + 1);
  w.x = c.take<float>(T * m->d_model);
  w.yf = c.take<uint8_t>(pad32(T) * m->d_model * dt_size(m->dtype));
  w.logits = own_logits ? c.take<float>(T * long(m->vocab)) : nullptr;
  w.samp = c.take<uint8_t>(molt::sampler_ws_bytes(B, k, m->vocab));
  w.dec = carve_dec(c, m, B, k, max_blocks);
  return w;
}
}  // namespace

size_t molt_verify_step_workspace_size(const molt_model* m, int B, int k, int max_blocks) {
  if (!m || B < 1 || k < 0 || max_blocks < 1 || m->vocab < 1 || !pair_ok(m->dtype, m->expert_dtype))
    return 0;
  molt::Carver c(nullptr, 0);
  carve_step(c, m, B, k, max_blocks, true);
  return c.used + 256;
}

int molt_verify_step(const molt_model* m, const molt_kv* kv, int B, int k, const int32_t* tokens,
                     const float* draft_probs, const float* uniforms, float* out_logits,
                     int32_t* out_tokens, int32_t* out_num_accepted, float* out_logprobs,
                     int32_t* out_routes, float* out_hidden, void* workspace,
                     size_t workspace_bytes, molt_stream_t stream) {
  if (int r = model_ok(m, kv, B, k, true)) return r;
  if (int r = spec_accept_shape_ok(B, k, m->vocab)) return r;
  REQUIRE(tokens && uniforms && out_tokens && out_num_accepted, "a required pointer is NULL");
  if (int r = check_ws(workspace, workspace_bytes,
                       molt_verify_step_workspace_size(m, B, k, kv->max_blocks_per_seq)))
    return r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  molt::Carver c(workspace, workspace_bytes);
  StepWs w = carve_step(c, m, B, k, kv->max_blocks_per_seq, true);
  float* logits = out_logits ? out_logits : w.logits;
  float* x = out_hidden ? out_hidden : w.x;   // the residual stream
  const int T = B * (k + 1);
  hipError_t e = molt::launch_embed(m->embed, tokens, T, m->d_model, m->vocab, m->dtype, x, s);
  if (e == hipSuccess) e = run_decoder(w.dec, m, kv, B, k, x, out_routes, m->final_norm, w.yf, s);
  if (e == hipSuccess) {
    ProfScope ps(MOLT_PROF_LM_HEAD, s);
    e = molt::launch_gemm(w.yf, m->lm_head, logits, T, m->vocab, m->d_model, m->dtype, false,
                          nullptr, 0, s);
  }
  // drafts are tokens[:, 1:]: the sampler reads them with row stride k+1
  if (e == hipSuccess) {
    ProfScope ps(MOLT_PROF_SAMPLER, s);
    e = molt::launch_spec_accept(logits, draft_probs, tokens, uniforms, B, k, m->vocab, out_tokens,
                                 out_num_accepted, out_logprobs, w.samp, s, k + 1, 1);
  }
  return hip_status(e, "molt_verify_step");
}

// ------------------------------------------------------------------ prefill

namespace {
struct PrefillWs { float* x; void* yf; float* hsel; void* ysel; DecWs dec; };
PrefillWs carve_prefill(molt::Carver& c, const molt_model* m, int B, int n, int max_blocks,
                        bool own_x) {
  PrefillWs w{};
  const long T = long(B) * n;
  const size_t es = dt_size(m->dtype);
  w.x = own_x ? c.take<float>(T * m->d_model) : nullptr;
  w.yf = c.take<uint8_t>(pad32(T) * m->d_model * es);
  w.hsel = c.take<float>(long(B) * m->d_model);
  w.ysel = c.take<uint8_t>(pad32(B) * m->d_model * es);
  w.dec = carve_dec(c, m, B, n - 1, max_blocks);
  return w;
}
}  // namespace

size_t molt_prefill_workspace_size(const molt_model* m, int B, int n, int max_blocks) {
  if (!m || B < 1 || n < 1 || max_blocks < 1 || m->vocab < 1 || !pair_ok(m->dtype, m->expert_dtype))
    return 0;
  molt::Carver c(nullptr, 0);
  carve_prefill(c, m, B, n, max_blocks, true);
  return c.used + 256;
}

int molt_prefill(const molt_model* m, const molt_kv* kv, int B, int n, const int32_t* tokens,
                 const int32_t* lens, float* out_logits, float* out_hidden, int32_t* out_routes,
                 void* workspace, size_t workspace_bytes, molt_stream_t stream) {
  REQUIRE(n >= 1, "n = %d must be >= 1", n);
  if (int r = model_ok(m, kv, B, n - 1, true)) return r;
  REQUIRE(tokens && lens && out_logits, "a required pointer is NULL");
  if (int r = check_ws(workspace, workspace_bytes,
                       molt_prefill_workspace_size(m, B, n, kv->max_blocks_per_seq)))
    return r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  molt::Carver c(workspace, workspace_bytes);
  PrefillWs w = carve_prefill(c, m, B, n, kv->max_blocks_per_seq, true);
  float* x = out_hidden ? out_hidden : w.x;
  const int T = B * n;
  hipError_t e = molt::launch_embed(m->embed, tokens, T, m->d_model, m->vocab, m->dtype, x, s);
  if (e == hipSuccess) e = run_decoder(w.dec, m, kv, B, n - 1, x, out_routes, m->final_norm, w.yf, s);
  if (e == hipSuccess)   // each sequence's last new row: row b n + lens[b] - 1
    e = molt::launch_mtp_select(x, w.yf, lens, B, n - 1, m->d_model, m->dtype, w.hsel, w.ysel, s, -1);
  if (e == hipSuccess) {
    ProfScope ps(MOLT_PROF_LM_HEAD, s);
    e = molt::launch_gemm(w.ysel, m->lm_head, out_logits, B, m->vocab, m->d_model, m->dtype, false,
                          nullptr, 0, s);
  }
  return hip_status(e, "molt_prefill");
}

// ------------------------------------------------------------------ replay recompute

namespace {
struct ScoreWs { float* x; void* yf; float* logits; void* lp; DecWs dec; };
ScoreWs carve_score(molt::Carver& c, const molt_model* m, int B, int k, int max_blocks) {
  ScoreWs w{};
  const long T = long(B) * (k + 1);
  w.x = c.take<float>(T * m->d_model);
  w.yf = c.take<uint8_t>(pad32(T) * m->d_model * dt_size(m->dtype));
  w.logits = c.take<float>(T * long(m->vocab));
  w.lp = c.take<uint8_t>(molt::token_logprob_ws_bytes(T, m->vocab));
  w.dec = carve_dec(c, m, B, k, max_blocks);
  return w;
}
}  // namespace

size_t molt_score_tokens_workspace_size(const molt_model* m, int B, int k, int max_blocks) {
  if (!m || B < 1 || k < 0 || max_blocks < 1 || m->vocab < 1 || !pair_ok(m->dtype, m->expert_dtype))
    return 0;
  molt::Carver c(nullptr, 0);
  carve_score(c, m, B, k, max_blocks);
  return c.used + 256;
}

int molt_score_tokens(const molt_model* m, const molt_kv* kv, int B, int k, const int32_t* tokens,
                      const int32_t* targets, const int32_t* replay_routes, float* out_logprobs,
                      float* out_logits, int32_t* out_routes, void* workspace,
                      size_t workspace_bytes, molt_stream_t stream) {
  if (int r = model_ok(m, kv, B, k, true)) return r;
  if (int r = spec_accept_shape_ok(B, k, m->vocab)) return r;
  REQUIRE(tokens && targets && out_logprobs, "a required pointer is NULL");
  if (int r = check_ws(workspace, workspace_bytes,
                       molt_score_tokens_workspace_size(m, B, k, kv->max_blocks_per_seq)))
    return r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  molt::Carver c(workspace, workspace_bytes);
  ScoreWs w = carve_score(c, m, B, k, kv->max_blocks_per_seq);
  float* logits = out_logits ? out_logits : w.logits;
  const int T = B * (k + 1);
  hipError_t e = molt::launch_embed(m->embed, tokens, T, m->d_model, m->vocab, m->dtype, w.x, s);
  if (e == hipSuccess)
    e = run_decoder(w.dec, m, kv, B, k, w.x, out_routes, m->final_norm, w.yf, s, replay_routes);
  if (e == hipSuccess) {
    ProfScope ps(MOLT_PROF_LM_HEAD, s);
    e = molt::launch_gemm(w.yf, m->lm_head, logits, T, m->vocab, m->d_model, m->dtype, false,
                          nullptr, 0, s);
  }
  if (e == hipSuccess) {
    ProfScope ps(MOLT_PROF_SAMPLER, s);
    e = molt::launch_token_logprobs(logits, T, m->vocab, targets, out_logprobs, w.lp, s);
  }
  return hip_status(e, "molt_score_tokens");
}

// ------------------------------------------------------------------ MTP draft head

namespace {

struct MtpWs {
  int32_t* row_tok; float* u_col; int32_t* ctx_next; int32_t* tok;
  void* y2; float* part; long part_elems;
  float* x; void* yf; float* hsel; void* ysel; float* logits; void* draw;
  DecWs cat, one;   // decoder workspaces of the catch-up rows (B, W) and a drafting row (B, 1)
};

MtpWs carve_mtp(molt::Carver& c, const molt_model* t, const molt_model* L, int B, int W,
                int max_blocks) {
  MtpWs w{};
  const long T = long(B) * W;
  const int d = t->d_model;
  const size_t es = dt_size(t->dtype);
  w.row_tok = c.take<int32_t>(T);
  w.u_col = c.take<float>(B);
  w.ctx_next = c.take<int32_t>(B);
  w.tok = c.take<int32_t>(B);
  w.y2 = c.take<uint8_t>(pad32(T) * 2 * d * es);
  w.part_elems = gemm_part_elems(int(T), d, 2 * d, t->dtype);
  w.part = c.take<float>(w.part_elems);
  w.x = c.take<float>(T * d);
  w.yf = c.take<uint8_t>(pad32(T) * d * es);
  w.hsel = c.take<float>(long(B) * d);
  w.ysel = c.take<uint8_t>(pad32(B) * d * es);
  w.logits = c.take<float>(long(B) * t->vocab);
  w.draw = c.take<uint8_t>(molt::draft_draw_ws_bytes(B, t->vocab));
  w.cat = carve_dec(c, L, B, W - 1, max_blocks);
  w.one = carve_dec(c, L, B, 0, max_blocks);
  return w;
}

int mtp_ok(const molt_model* t, const molt_mtp* mtp, const molt_kv* kv, int B, int W, int k) {
  REQUIRE(t && mtp && kv, "target, mtp and mtp_kv are required");
  REQUIRE(mtp->layer, "mtp->layer is NULL");
  const molt_model* L = mtp->layer;
  REQUIRE(k >= 1, "k = %d must be >= 1 to draft", k);
  REQUIRE(W >= 1, "window = %d must be >= 1", W);
  REQUIRE(act_ok(t->dtype), "target dtype must be F32 or BF16");
  REQUIRE(t->vocab >= 1 && t->embed && t->lm_head, "the target's embed, lm_head and vocab are required");
  REQUIRE(L->n_layers == 1, "the head has n_layers = %d, must be 1", L->n_layers);
  REQUIRE(L->d_model == t->d_model && L->dtype == t->dtype,
          "the head's d_model/dtype (%d, %d) differ from the target's (%d, %d)", L->d_model,
          int(L->dtype), t->d_model, int(t->dtype));
  REQUIRE(mtp->enorm && mtp->hnorm && mtp->eh_proj && L->final_norm,
          "enorm, hnorm, eh_proj and layer->final_norm are required");
  REQUIRE(2L * t->d_model * long(dt_size(t->dtype)) % 128 == 0, "2 d * sizeof(dtype) must be a multiple of 128");
  if (int r = spec_accept_shape_ok(B, 0, t->vocab)) return r;
  return model_ok(L, kv, B, W - 1, false);
}

}  // namespace

size_t molt_mtp_draft_window_workspace_size(const molt_model* target, const molt_mtp* mtp, int B,
                                            int window, int k, int max_blocks) {
  if (!target || !mtp || !mtp->layer || B < 1 || window < 1 || k < 1 || max_blocks < 1 ||
      target->vocab < 1 || !pair_ok(mtp->layer->dtype, mtp->layer->expert_dtype))
    return 0;
  molt::Carver c(nullptr, 0);
  carve_mtp(c, target, mtp->layer, B, window, max_blocks);
  return c.used + 256;
}

size_t molt_mtp_draft_workspace_size(const molt_model* target, const molt_mtp* mtp, int B, int k,
                                     int max_blocks) {
  return molt_mtp_draft_window_workspace_size(target, mtp, B, k + 1, k, max_blocks);
}

int molt_mtp_draft_window(const molt_model* target, const molt_mtp* mtp, const molt_kv* mtp_kv,
                          int B, int window, int k, const float* hidden, const int32_t* tokens,
                          const int32_t* n_accepted, const int32_t* next_tokens,
                          const float* uniforms, int32_t* out_drafts, float* out_draft_probs,
                          void* workspace, size_t workspace_bytes, molt_stream_t stream) {
  const int W = window;
  if (int r = mtp_ok(target, mtp, mtp_kv, B, W, k)) return r;
  REQUIRE(hidden && tokens && n_accepted && next_tokens && out_drafts, "a required pointer is NULL");
  REQUIRE(out_draft_probs == nullptr || uniforms, "sampled drafts (out_draft_probs) need uniforms");
  if (int r = check_ws(workspace, workspace_bytes,
                       molt_mtp_draft_window_workspace_size(target, mtp, B, W, k,
                                                            mtp_kv->max_blocks_per_seq)))
    return r;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  molt::Carver c(workspace, workspace_bytes);
  MtpWs w = carve_mtp(c, target, mtp->layer, B, W, mtp_kv->max_blocks_per_seq);
  const molt_model* L = mtp->layer;
  const int d = target->d_model, V = target->vocab, T = B * W;
  const molt_dtype dt = target->dtype;
  const float* u = out_draft_probs ? uniforms : nullptr;   // greedy drafts draw nothing
  molt_kv one = *mtp_kv;        // drafting rows: context c_b + n_b + i per sequence
  one.context_lens = w.ctx_next;
  hipError_t e = hipSuccess;
#define RUN(call) do { if ((e = (call)) != hipSuccess) return hip_status(e, "molt_mtp_draft"); } while (0)
  // catch-up rows
  RUN(molt::launch_mtp_catchup(tokens, n_accepted, next_tokens, u, B, W, k, w.row_tok, w.u_col, s));
  RUN(molt::launch_mtp_input(target->embed, w.row_tok, hidden, mtp->enorm, mtp->hnorm, T, d, V,
                             L->rms_eps, dt, w.y2, s));
  {
    ProfScope ps(MOLT_PROF_PROJECTIONS, s);
    RUN(molt::launch_gemm(w.y2, mtp->eh_proj, w.x, T, d, 2 * d, dt, false, w.part, w.part_elems, s));
  }
  RUN(run_decoder(w.cat, L, mtp_kv, B, W - 1, w.x, nullptr, L->final_norm, w.yf, s));
  RUN(molt::launch_mtp_select(w.x, w.yf, n_accepted, B, W - 1, d, dt, w.hsel, w.ysel, s));
  for (int i = 0; i < k; ++i) {
    {
      ProfScope ps(MOLT_PROF_LM_HEAD, s);
      RUN(molt::launch_gemm(i == 0 ? w.ysel : w.yf, target->lm_head, w.logits, B, V, d, dt, false,
                            nullptr, 0, s));
    }
    {
      ProfScope ps(MOLT_PROF_SAMPLER, s);
      RUN(molt::launch_draft_draw(w.logits, B, V, u ? w.u_col : nullptr, w.tok,
                                  out_draft_probs ? out_draft_probs + long(i) * V : nullptr,
                                  long(k) * V, w.draw, s));
    }
    RUN(molt::launch_mtp_record(w.tok, i, B, W, k, mtp_kv->context_lens, n_accepted, u, out_drafts,
                                w.row_tok, w.ctx_next, w.u_col, s));
    if (i + 1 == k) break;
    // drafting row: the head's previous output and draft i + 1 (the input kernel has read
    // x before the projection overwrites it)
    RUN(molt::launch_mtp_input(target->embed, w.row_tok, i == 0 ? w.hsel : w.x, mtp->enorm,
                               mtp->hnorm, B, d, V, L->rms_eps, dt, w.y2, s));
    {
      ProfScope ps(MOLT_PROF_PROJECTIONS, s);
      RUN(molt::launch_gemm(w.y2, mtp->eh_proj, w.x, B, d, 2 * d, dt, false, w.part, w.part_elems, s));
    }
    RUN(run_decoder(w.one, L, &one, B, 0, w.x, nullptr, L->final_norm, w.yf, s));
  }
#undef RUN
  return ok();
}

int molt_mtp_draft(const molt_model* target, const molt_mtp* mtp, const molt_kv* mtp_kv, int B,
                   int k, const float* hidden, const int32_t* tokens, const int32_t* n_accepted,
                   const int32_t* next_tokens, const float* uniforms, int32_t* out_drafts,
                   float* out_draft_probs, void* workspace, size_t workspace_bytes,
                   molt_stream_t stream) {
  return molt_mtp_draft_window(target, mtp, mtp_kv, B, k + 1, k, hidden, tokens, n_accepted,
                               next_tokens, uniforms, out_drafts, out_draft_probs, workspace,
                               workspace_bytes, stream);
}

}  // extern "C"
