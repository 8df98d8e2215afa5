// Row-wise kernels of the verify step: token embedding, RMSNorm (+ per-row fp8
// quantisation), fp8 quantisation of tiled rows, RoPE with the paged-KV write of the 1+k
// new positions, and the weighted expert combine; and the MTP draft head's row
// bookkeeping and input normalisation. All are HBM-bound with a few bytes per element; one
// workgroup per token row.
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr int kThreads = 256;

MOLT_DEV float load_act(const void* p, long i, molt_dtype dt) {
  return dt == MOLT_BF16 ? bf16_to_f32(static_cast<const uint16_t*>(p)[i])
                         : static_cast<const float*>(p)[i];
}
MOLT_DEV void store_act(void* p, long i, float v, molt_dtype dt) {
  if (dt == MOLT_BF16) static_cast<uint16_t*>(p)[i] = f32_to_bf16(v);
  else static_cast<float*>(p)[i] = v;
}

// x[t, :] = Emb[tokens[t], :] widened to f32 (an out-of-range token gives a zero row)
__global__ __launch_bounds__(kThreads) void embed_kernel(const void* __restrict__ table,
                                                         const int32_t* __restrict__ tokens, int d,
                                                         int V, molt_dtype dt,
                                                         float* __restrict__ x) {
  const int t = blockIdx.x;
  const int tok = tokens[t];
  const bool ok = tok >= 0 && tok < V;
  for (int i = threadIdx.x; i < d; i += kThreads)
    x[long(t) * d + i] = ok ? load_act(table, long(tok) * d + i, dt) : 0.f;
}

// Residual update and RMSNorm of token row t, fused:
//   x[t] += part[0][t] + part[1][t] + ...   (split-K partial sums of the O projection, in
//                                            split order; nparts = 0: none)
//   x[t] += sum_j w[t, j] * o[t * K + j]     (MoE combine, slot order; o = NULL: none)
//   y = x[t] / sqrt(mean(x[t]^2) + eps) * g  rounded to dt, tiled (g = NULL: no norm)
// With yq, also the per-row fp8 code of y (s = amax|y| / 448, code = e4m3(y / s)); with
// y_rows (bf16) and yq_rows, also y and its codes in row-major order (read by the expert
// GEMM through the permutation).
// Each thread owns runs of 8 consecutive elements (d % 8 == 0, d <= 8 * 256 * kNormRuns),
// kept in registers from the residual update to the stores: one 16-byte store of y per run
// (8 bf16 are contiguous in the tiled layout).
constexpr int kNormRuns = 8;

template <typename T>
MOLT_DEV void add8(float (&v)[8], const T* src, float wgt) {
  const float4 a = *reinterpret_cast<const float4*>(src);
  const float4 b = *reinterpret_cast<const float4*>(src + 4);
  v[0] += wgt * a.x; v[1] += wgt * a.y; v[2] += wgt * a.z; v[3] += wgt * a.w;
  v[4] += wgt * b.x; v[5] += wgt * b.y; v[6] += wgt * b.z; v[7] += wgt * b.w;
}

__global__ __launch_bounds__(kThreads) void residual_norm_kernel(
    float* __restrict__ x, const float* __restrict__ part, int nparts, long part_stride,
    const float* __restrict__ o, const float* __restrict__ w, int K, const float* __restrict__ g,
    int d, float eps, molt_dtype dt, void* __restrict__ y, uint8_t* __restrict__ yq,
    float* __restrict__ ys, void* __restrict__ y_rows, uint8_t* __restrict__ yq_rows) {
  __shared__ float red[kThreads / kWave];
  const int t = blockIdx.x;
  float* xr = x + long(t) * d;
  float v[kNormRuns][8];
  // the gains are loaded with x: loaded after the x stores, they would wait for those
  float gv[kNormRuns][8];
  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < kNormRuns; ++r) {
    const int i = (threadIdx.x + r * kThreads) * 8;
    if (i >= d) break;
    if (g) {
      const float4 ga = *reinterpret_cast<const float4*>(g + i);
      const float4 gb = *reinterpret_cast<const float4*>(g + i + 4);
      gv[r][0] = ga.x; gv[r][1] = ga.y; gv[r][2] = ga.z; gv[r][3] = ga.w;
      gv[r][4] = gb.x; gv[r][5] = gb.y; gv[r][6] = gb.z; gv[r][7] = gb.w;
    }
    const float4 a = *reinterpret_cast<const float4*>(xr + i);
    const float4 b = *reinterpret_cast<const float4*>(xr + i + 4);
    v[r][0] = a.x; v[r][1] = a.y; v[r][2] = a.z; v[r][3] = a.w;
    v[r][4] = b.x; v[r][5] = b.y; v[r][6] = b.z; v[r][7] = b.w;
    if (nparts > 0 || o) {
      // each addend is summed exactly as v += p (splits) and v += (sum_j w_j o_j) (slots)
#pragma unroll 4
      for (int s = 0; s < nparts; ++s) add8(v[r], part + s * part_stride + long(t) * d + i, 1.0f);
      if (o) {
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
        for (int j = 0; j < K; ++j) add8(acc, o + (long(t) * K + j) * d + i, w[long(t) * K + j]);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[r][e] += acc[e];
      }
      *reinterpret_cast<float4*>(xr + i) = make_float4(v[r][0], v[r][1], v[r][2], v[r][3]);
      *reinterpret_cast<float4*>(xr + i + 4) = make_float4(v[r][4], v[r][5], v[r][6], v[r][7]);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[r][e] * v[r][e];
  }
  if (g == nullptr) return;
  ss = block_sum_dpp<kThreads / kWave>(ss, red);
  const float rs = 1.0f / sqrtf(ss / float(d) + eps);
  float amax = 0.f;
#pragma unroll
  for (int r = 0; r < kNormRuns; ++r) {
    const int i = (threadIdx.x + r * kThreads) * 8;
    if (i >= d) break;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float u = v[r][e] * rs * gv[r][e];
      if (dt == MOLT_BF16) u = round_to_bf16(u);
      v[r][e] = u;
      amax = fmaxf(amax, fabsf(u));
    }
    if (dt == MOLT_BF16) {
      uint32_t pk[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        pk[e] = uint32_t(f32_to_bf16(v[r][2 * e])) | (uint32_t(f32_to_bf16(v[r][2 * e + 1])) << 16);
      *reinterpret_cast<uint4*>(static_cast<uint8_t*>(y) + tiled_offset(t, 2L * i, 2L * d)) =
          make_uint4(pk[0], pk[1], pk[2], pk[3]);
      if (y_rows)
        *reinterpret_cast<uint4*>(static_cast<uint8_t*>(y_rows) + 2L * (long(t) * d + i)) =
            make_uint4(pk[0], pk[1], pk[2], pk[3]);
    } else {
      uint8_t* yb = static_cast<uint8_t*>(y);
      *reinterpret_cast<float4*>(yb + tiled_offset(t, 4L * i, 4L * d)) =
          make_float4(v[r][0], v[r][1], v[r][2], v[r][3]);
      *reinterpret_cast<float4*>(yb + tiled_offset(t, 4L * (i + 4), 4L * d)) =
          make_float4(v[r][4], v[r][5], v[r][6], v[r][7]);
    }
  }
  if (yq == nullptr) return;
  amax = block_max_dpp<kThreads / kWave>(amax, red);
  const float sc = amax / 448.0f;
  // v / sc: IEEE for tiny scales, else the reciprocal with one fma correction (same codes;
  // the values are the bf16-rounded y, |v| <= amax)
  const float rsc = 1.0f / sc;
  auto codes = [&](auto div) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < kNormRuns; ++r) {
      const int i = (threadIdx.x + r * kThreads) * 8;
      if (i >= d) break;
      uint32_t c[2] = {0u, 0u};
      if (sc > 0.f) {
#pragma unroll
        for (int e = 0; e < 8; e += 2) c[e / 4] |= f32x2_to_fp8e4m3(div(v[r][e]), div(v[r][e + 1])) << (8 * (e % 4));
      }
      *reinterpret_cast<uint2*>(yq + tiled_offset(t, i, d)) = make_uint2(c[0], c[1]);
      if (yq_rows) *reinterpret_cast<uint2*>(yq_rows + long(t) * d + i) = make_uint2(c[0], c[1]);
    }
  };
  if (sc > kFastDivMinScale) codes([&](float x) { return div_by_scale(x, sc, rsc); });
  else codes([&](float x) { return x / sc; });
  if (threadIdx.x == 0) ys[t] = sc;
}

// Per-row fp8 quantisation of tiled bf16 rows into tiled e4m3 codes (s = amax / 448,
// code = e4m3(v / s), zero row -> s = 0): the SwiGLU product of the grouped GEMMs (rows in
// padded expert order, count on the device, padding rows with pair -1 get zero codes and
// scale 0) or an input activation (all `rows` rows). One wavefront per row; lane l holds
// the 4-column chunks l, l + 64, ... in registers from the amax to the codes (the row is
// read once; rows past 64 * kQuantRegChunks * 4 columns re-read the rest).
constexpr int kQuantRegChunks = 16;
__global__ __launch_bounds__(kThreads) void quant_rows_tiled_kernel(
    const uint16_t* __restrict__ h, const int32_t* __restrict__ pperm,
    const int32_t* __restrict__ n_rows, long rows, int cols, uint8_t* __restrict__ q,
    float* __restrict__ scale) {
  const long r = long(blockIdx.x) * (kThreads / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (r >= (n_rows ? long(*n_rows) : rows)) return;
  const bool pad = pperm && pperm[r] < 0;
  const long rb_in = 2L * cols, rb_out = cols;
  const uint8_t* hb = reinterpret_cast<const uint8_t*>(h);
  const int nch = cols / 4;                  // 4-column chunks of the row
  auto load = [&](int ch) __attribute__((always_inline)) {
    return *reinterpret_cast<const uint2*>(hb + tiled_offset(r, 8L * ch, rb_in));
  };
  uint2 reg[kQuantRegChunks];
  float amax = 0.f;
#pragma unroll
  for (int k = 0; k < kQuantRegChunks; ++k) {
    const int ch = lane + kWave * k;
    reg[k] = ch < nch ? load(ch) : make_uint2(0u, 0u);
  }
  auto absmax = [&](uint2 v) __attribute__((always_inline)) {
    return fmaxf(fmaxf(fabsf(bf16_to_f32(uint16_t(v.x))), fabsf(bf16_to_f32(uint16_t(v.x >> 16)))),
                 fmaxf(fabsf(bf16_to_f32(uint16_t(v.y))), fabsf(bf16_to_f32(uint16_t(v.y >> 16)))));
  };
#pragma unroll
  for (int k = 0; k < kQuantRegChunks; ++k) amax = fmaxf(amax, absmax(reg[k]));
  for (int ch = lane + kWave * kQuantRegChunks; ch < nch; ch += kWave) amax = fmaxf(amax, absmax(load(ch)));
  amax = pad ? 0.f : wave_max(amax);
  const float s = amax / 448.0f;
  // v / s: IEEE for tiny scales, else the reciprocal with one fma correction (same codes)
  const float rs = 1.0f / s;
  auto encode = [&](int ch, uint2 v, auto div) __attribute__((always_inline)) {
    uint32_t code = 0u;
    if (s > 0.f)
      code = f32x2_to_fp8e4m3(div(bf16_to_f32(uint16_t(v.x))), div(bf16_to_f32(uint16_t(v.x >> 16)))) |
             (f32x2_to_fp8e4m3(div(bf16_to_f32(uint16_t(v.y))), div(bf16_to_f32(uint16_t(v.y >> 16)))) << 16);
    *reinterpret_cast<uint32_t*>(q + tiled_offset(r, 4L * ch, rb_out)) = code;
  };
  auto encode_all = [&](auto div) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kQuantRegChunks; ++k) {
      const int ch = lane + kWave * k;
      if (ch < nch) encode(ch, reg[k], div);
    }
    for (int ch = lane + kWave * kQuantRegChunks; ch < nch; ch += kWave) encode(ch, load(ch), div);
  };
  if (s > kFastDivMinScale) encode_all([&](float x) { return div_by_scale(x, s, rs); });
  else encode_all([&](float x) { return x / s; });
  if (lane == 0) scale[r] = s;
}

// RoPE angle table of the step: token t = b*(1+k)+j sits at position ctx[b]+j; pair i
// (i, i+D/2) turns by position * theta^(-2i/D); cos and sin evaluated in f64, once per step
// for all layers. table[t][i] = {cos, sin}.
__global__ __launch_bounds__(kThreads) void rope_table_kernel(
    const int32_t* __restrict__ ctx, int k, int D, float theta, double2* __restrict__ table,
    const int32_t* __restrict__ bt, int max_blocks, int num_blocks, int32_t* __restrict__ kv_slot) {
  const int t = blockIdx.x;
  const int b = t / (k + 1);
  const long pos = long(ctx[b]) + t % (k + 1);
  if (kv_slot && threadIdx.x == 0) {
    const int blk = bt[long(b) * max_blocks + pos / 16];
    kv_slot[t] = blk >= 0 && blk < num_blocks ? blk * 16 + int(pos % 16) : -1;
  }
  for (int i = threadIdx.x; i < D / 2; i += kThreads) {
    const double inv_freq = pow(double(theta), -2.0 * double(i) / double(D));
    const double ang = double(pos) * inv_freq;
    table[long(t) * (D / 2) + i] = make_double2(cos(ang), sin(ang));
  }
}

// RoPE on q and k of token t (rotation in f64 with the step's table), then
// q -> q_out[t, Hq, D]; k -> K cache slot; v -> V cache slot (transposed layout).
__global__ __launch_bounds__(kThreads) void rope_kv_kernel(
    const float* __restrict__ qkv, int k, int Hq, int Hkv, int D, const double2* __restrict__ table,
    const int32_t* __restrict__ ctx, const int32_t* __restrict__ bt, int max_blocks, int num_blocks,
    molt_dtype dt, void* __restrict__ q_out, void* __restrict__ kc, void* __restrict__ vc) {
  const int t = blockIdx.x;
  const int b = t / (k + 1), j = t % (k + 1);
  const long pos = long(ctx[b]) + j;
  const int half = D / 2;
  const double2* cs = table + long(t) * half;
  const int width = (Hq + 2 * Hkv) * D;
  const float* row = qkv + long(t) * width;
  const int blk = bt[long(b) * max_blocks + pos / 16];
  const int slot = int(pos % 16);
  const bool blk_ok = blk >= 0 && blk < num_blocks;
  // rotations: (Hq + Hkv) heads x half pairs
  for (int w = threadIdx.x; w < (Hq + Hkv) * half; w += kThreads) {
    const int h = w / half, i = w % half;
    const double a = row[h * D + i], c = row[h * D + i + half];
    const double2 r = cs[i];
    const float lo = float(a * r.x - c * r.y);
    const float hi = float(c * r.x + a * r.y);
    if (h < Hq) {
      store_act(q_out, (long(t) * Hq + h) * D + i, lo, dt);
      store_act(q_out, (long(t) * Hq + h) * D + i + half, hi, dt);
    } else if (blk_ok) {
      const int hk = h - Hq;
      const long base = ((long(blk) * Hkv + hk) * 16 + slot) * D;
      store_act(kc, base + i, lo, dt);
      store_act(kc, base + i + half, hi, dt);
    }
  }
  if (!blk_ok) return;
  for (int w = threadIdx.x; w < Hkv * D; w += kThreads) {
    const int hk = w / D, i = w % D;
    const float v = row[(Hq + Hkv + hk) * D + i];
    store_act(vc, ((long(blk) * Hkv + hk) * D + i) * 16 + slot, v, dt);
  }
}

// out[t] (+)= sum_{j<K} w[t,j] * o[t*K+j], slot order, f32
__global__ __launch_bounds__(kThreads) void combine_kernel(const float* __restrict__ o,
                                                           const float* __restrict__ w, int K,
                                                           int d, float* __restrict__ out,
                                                           bool accumulate) {
  const int t = blockIdx.x;
  for (int i = threadIdx.x * 4; i < d; i += kThreads * 4) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < K; ++j) {
      const float wj = w[long(t) * K + j];
      const float4 v = *reinterpret_cast<const float4*>(o + (long(t) * K + j) * d + i);
      acc.x += wj * v.x; acc.y += wj * v.y; acc.z += wj * v.z; acc.w += wj * v.w;
    }
    float4* dst = reinterpret_cast<float4*>(out + long(t) * d + i);
    if (accumulate) {
      float4 x = *dst;
      acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
    }
    *dst = acc;
  }
}


// ---------------------------------------------------------------- MTP draft head rows
// (the head's input halves and the row bookkeeping of its catch-up and drafting rows)

MOLT_DEV int clamp_n(int n, int k) { return n < 0 ? 0 : n > k ? k : n; }

// catch-up row r = b W + j (W rows per sequence) takes token x_{j+1} (j < n_b) or y_b;
// u_col[b] = u[b, 0] (u: [B, k] draft uniforms)
__global__ void mtp_catchup_kernel(const int32_t* __restrict__ tokens,
                                   const int32_t* __restrict__ n_acc,
                                   const int32_t* __restrict__ next, const float* __restrict__ u,
                                   int B, int W, int k, int32_t* __restrict__ row_tok,
                                   float* __restrict__ u_col) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= B * W) return;
  const int b = r / W, j = r % W;
  const int nb = clamp_n(n_acc[b], W - 1);
  row_tok[r] = j < nb ? tokens[r + 1] : next[b];
  if (j == 0 && u) u_col[b] = u[long(b) * k];
}

// One normalised half of a head input row: v (8 consecutive elements per run) scaled by
// 1 / sqrt(mean(v^2) + eps) and g, rounded to dt, stored at columns [col0, col0 + d) of the
// tiled [rows, 2d] matrix y.
MOLT_DEV void norm_half_store(float (&v)[kNormRuns][8], const float* __restrict__ g, int d,
                              float eps, molt_dtype dt, void* __restrict__ y, int t, int col0,
                              float* red) {
  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < kNormRuns; ++r) {
    const int i = (threadIdx.x + r * kThreads) * 8;
    if (i >= d) break;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[r][e] * v[r][e];
  }
  ss = block_sum_dpp<kThreads / kWave>(ss, red);
  const float rs = 1.0f / sqrtf(ss / float(d) + eps);
  const long es = dt == MOLT_BF16 ? 2 : 4, rb = 2L * d * es;
#pragma unroll
  for (int r = 0; r < kNormRuns; ++r) {
    const int i = (threadIdx.x + r * kThreads) * 8;
    if (i >= d) break;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      o[e] = v[r][e] * rs * g[i + e];
      if (dt == MOLT_BF16) o[e] = round_to_bf16(o[e]);
    }
    uint8_t* yb = static_cast<uint8_t*>(y);
    if (dt == MOLT_BF16) {
      uint32_t pk[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        pk[e] = uint32_t(f32_to_bf16(o[2 * e])) | (uint32_t(f32_to_bf16(o[2 * e + 1])) << 16);
      *reinterpret_cast<uint4*>(yb + tiled_offset(t, 2L * (col0 + i), rb)) =
          make_uint4(pk[0], pk[1], pk[2], pk[3]);
    } else {
      *reinterpret_cast<float4*>(yb + tiled_offset(t, 4L * (col0 + i), rb)) =
          make_float4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<float4*>(yb + tiled_offset(t, 4L * (col0 + i + 4), rb)) =
          make_float4(o[4], o[5], o[6], o[7]);
    }
  }
}

// y[t] = [RMSNorm(Emb[tok[t]]; ge) ; RMSNorm(h[t]; gh)], each half rounded to dt, tiled
// [rows padded to 32, 2d] (an out-of-range token gives a zero embedding half)
__global__ __launch_bounds__(kThreads) void mtp_input_kernel(
    const void* __restrict__ embed, const int32_t* __restrict__ tok, const float* __restrict__ h,
    const float* __restrict__ ge, const float* __restrict__ gh, int d, int V, float eps,
    molt_dtype dt, void* __restrict__ y) {
  __shared__ float red[kThreads / kWave];
  const int t = blockIdx.x;
  const int id = tok[t];
  const bool ok = id >= 0 && id < V;
  float v[kNormRuns][8];
#pragma unroll
  for (int r = 0; r < kNormRuns; ++r) {
    const int i = (threadIdx.x + r * kThreads) * 8;
    if (i >= d) break;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[r][e] = ok ? load_act(embed, long(id) * d + i + e, dt) : 0.f;
  }
  norm_half_store(v, ge, d, eps, dt, y, t, 0, red);
  const float* hr = h + long(t) * d;
#pragma unroll
  for (int r = 0; r < kNormRuns; ++r) {
    const int i = (threadIdx.x + r * kThreads) * 8;
    if (i >= d) break;
    const float4 a = *reinterpret_cast<const float4*>(hr + i);
    const float4 b = *reinterpret_cast<const float4*>(hr + i + 4);
    v[r][0] = a.x; v[r][1] = a.y; v[r][2] = a.z; v[r][3] = a.w;
    v[r][4] = b.x; v[r][5] = b.y; v[r][6] = b.z; v[r][7] = b.w;
  }
  norm_half_store(v, gh, d, eps, dt, y, t, d, red);
}

// row b of hsel / ysel = row b(k+1) + clamp(n_b + delta) of x (f32 [T, d]) / yf (tiled
// [T, d] dt): the draft head's catch-up row n_b (delta 0), a prefill's last row (delta -1)
__global__ __launch_bounds__(kThreads) void mtp_select_kernel(
    const float* __restrict__ x, const uint8_t* __restrict__ yf, const int32_t* __restrict__ n_acc,
    int delta, int k, int d, int es, float* __restrict__ hsel, uint8_t* __restrict__ ysel) {
  const int b = blockIdx.x;
  const long src = long(b) * (k + 1) + clamp_n(n_acc[b] + delta, k);
  for (int i = threadIdx.x * 4; i < d; i += kThreads * 4)
    *reinterpret_cast<float4*>(hsel + long(b) * d + i) = *reinterpret_cast<const float4*>(x + src * d + i);
  const long rb = long(d) * es;
  for (long c = threadIdx.x; c < rb / 16; c += kThreads)   // 16 bytes of a row are contiguous
    *reinterpret_cast<uint4*>(ysel + tiled_offset(b, 16 * c, rb)) =
        *reinterpret_cast<const uint4*>(yf + tiled_offset(src, 16 * c, rb));
}

// after draft i + 1 is drawn (tok): drafts[b, i] = tok[b]; for the next drafting row its
// token, its context (position c_b + n_b + i + 1 is the row's own) and its uniform
__global__ void mtp_record_kernel(const int32_t* __restrict__ tok, int i, int B, int W, int k,
                                  const int32_t* __restrict__ ctx, const int32_t* __restrict__ n_acc,
                                  const float* __restrict__ u, int32_t* __restrict__ drafts,
                                  int32_t* __restrict__ row_tok, int32_t* __restrict__ ctx_next,
                                  float* __restrict__ u_col) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int t = tok[b];
  drafts[long(b) * k + i] = t;
  if (i + 1 < k) {
    row_tok[b] = t;
    ctx_next[b] = ctx[b] + clamp_n(n_acc[b], W - 1) + i + 1;
    if (u) u_col[b] = u[long(b) * k + i + 1];
  }
}

}  // namespace

hipError_t launch_embed(const void* table, const int32_t* tokens, int T, int d, int V,
                        molt_dtype dt, float* x, hipStream_t s) {
  embed_kernel<<<T, kThreads, 0, s>>>(table, tokens, d, V, dt, x);
  return hipGetLastError();
}

hipError_t launch_residual_norm(float* x, const float* part, int nparts, const float* o,
                                const float* w, int K, const float* g, int T, int d, float eps,
                                molt_dtype dt, void* y, uint8_t* yq, float* ys, hipStream_t s,
                                void* y_rows, uint8_t* yq_rows) {
  residual_norm_kernel<<<T, kThreads, 0, s>>>(x, part, nparts, long(T) * d, o, w, K, g, d, eps, dt,
                                              y, yq, ys, dt == MOLT_BF16 ? y_rows : nullptr,
                                              yq ? yq_rows : nullptr);
  return hipGetLastError();
}

hipError_t launch_rope_table(const int32_t* ctx, int B, int k, int D, float theta, void* table,
                             const int32_t* bt, int max_blocks, int num_blocks, int32_t* kv_slot,
                             hipStream_t s) {
  rope_table_kernel<<<B * (k + 1), kThreads, 0, s>>>(ctx, k, D, theta, static_cast<double2*>(table),
                                                     bt, max_blocks, num_blocks, kv_slot);
  return hipGetLastError();
}

hipError_t launch_rope_kv_write(const float* qkv, int B, int k, int Hq, int Hkv, int D,
                                const void* table, const int32_t* ctx, const int32_t* bt,
                                int max_blocks, int num_blocks, molt_dtype dt, void* q_out,
                                void* k_cache, void* v_cache, hipStream_t s) {
  rope_kv_kernel<<<B * (k + 1), kThreads, 0, s>>>(qkv, k, Hq, Hkv, D,
                                                   static_cast<const double2*>(table), ctx, bt,
                                                   max_blocks, num_blocks, dt, q_out, k_cache,
                                                   v_cache);
  return hipGetLastError();
}

hipError_t launch_quant_rows_tiled(const uint16_t* h, const int32_t* pperm, const int32_t* n_rows,
                                   long max_rows, int cols, uint8_t* q, float* scale,
                                   hipStream_t s) {
  constexpr int rows_per_block = kThreads / kWave;
  const long grid = (max_rows + rows_per_block - 1) / rows_per_block;
  if (grid == 0) return hipSuccess;
  quant_rows_tiled_kernel<<<grid, kThreads, 0, s>>>(h, pperm, n_rows, max_rows, cols, q, scale);
  return hipGetLastError();
}

hipError_t launch_combine(const float* o, const float* w, int T, int K, int d, float* out,
                          bool accumulate, hipStream_t s) {
  combine_kernel<<<T, kThreads, 0, s>>>(o, w, K, d, out, accumulate);
  return hipGetLastError();
}

hipError_t launch_mtp_catchup(const int32_t* tokens, const int32_t* n_acc, const int32_t* next,
                              const float* u, int B, int W, int k, int32_t* row_tok, float* u_col,
                              hipStream_t s) {
  const int T = B * W;
  mtp_catchup_kernel<<<(T + kThreads - 1) / kThreads, kThreads, 0, s>>>(tokens, n_acc, next, u, B, W,
                                                                       k, row_tok, u_col);
  return hipGetLastError();
}

hipError_t launch_mtp_input(const void* embed, const int32_t* tok, const float* h, const float* ge,
                            const float* gh, int T, int d, int V, float eps, molt_dtype dt,
                            void* y, hipStream_t s) {
  mtp_input_kernel<<<T, kThreads, 0, s>>>(embed, tok, h, ge, gh, d, V, eps, dt, y);
  return hipGetLastError();
}

hipError_t launch_mtp_select(const float* x, const void* yf, const int32_t* n_acc, int B, int k,
                             int d, molt_dtype dt, float* hsel, void* ysel, hipStream_t s,
                             int delta) {
  mtp_select_kernel<<<B, kThreads, 0, s>>>(x, static_cast<const uint8_t*>(yf), n_acc, delta, k, d,
                                           dt == MOLT_BF16 ? 2 : 4, hsel,
                                           static_cast<uint8_t*>(ysel));
  return hipGetLastError();
}

hipError_t launch_mtp_record(const int32_t* tok, int i, int B, int W, int k, const int32_t* ctx,
                             const int32_t* n_acc, const float* u, int32_t* drafts,
                             int32_t* row_tok, int32_t* ctx_next, float* u_col, hipStream_t s) {
  mtp_record_kernel<<<(B + kThreads - 1) / kThreads, kThreads, 0, s>>>(tok, i, B, W, k, ctx, n_acc, u,
                                                                      drafts, row_tok, ctx_next, u_col);
  return hipGetLastError();
}

}  // namespace molt
