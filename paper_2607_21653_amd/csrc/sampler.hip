// Fused vocab-wide softmax statistics, speculative accept, residual resample and
// behavior log-probs (the serving engine's speculative-decoding accept rule with
// temperature 1 and no truncation; paper Sec. 4.1 control table, Sec. 4.2, Sec. 5.3/5.4;
// rule of Leviathan et al. 2023 / Chen et al. 2023).
//
// Four launches, all HBM-streaming and deterministic (fixed reduction orders, integer
// prefix sums, no atomics):
//   1. chunk_stats  grid = rows * chunks: per 8192-logit chunk its max and
//                   sum exp(l - chunk max) (f32 exp of the exactly compensated
//                   difference, f64 accumulation across threads).
//   2. accept       one thread per sequence: combines the chunk statistics of the rows
//                   it needs into (m, S), runs the k accept tests u*q*S < exp(l_x - m)
//                   in f64, writes accepted drafts and their log-probs, and the
//                   descriptor of the final draw (row, residual mode).
//   3. draw_mass    grid = B * chunks: per chunk, the integer mass sum floor(r_t 2^62)
//                   of the residual max(0, p - q) (or p for a bonus draw), p_t from an
//                   f64 exp so that the only rounding left in the draw is that of S.
//   4. draw_pick    one workgroup per sequence: Tot, target = (Tot * floor(u 2^32)) >> 32,
//                   the chunk holding the target, then an in-chunk integer scan.
// Bytes: pass 1 reads B(1+k)V logits once; passes 3-4 read one row (+ one q row on a
// rejection) per sequence, plus one chunk again.
#include "device_common.h"
#include "internal.h"

// The draw recomputes each grid mass in two kernels; both must round identically, so no
// floating-point contraction in this file.
#pragma clang fp contract(off)

namespace molt {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 32;
constexpr int kChunk = kThreads * kPerThread;  // 8192 logits per chunk

struct FinalDraw {
  double m;      // row max
  double S;      // row sum exp(l - m)
  int row;       // row index inside the sequence (0..k)
  int mode;      // 0: draw from p, 1: residual with q row, 2: residual with one-hot q
  int draft;     // the rejected draft (mode 2)
  int pad;
};

// ---- pass 1 ---------------------------------------------------------------------------
template <bool kVec>
__global__ __launch_bounds__(kThreads) void chunk_stats_kernel(const float* __restrict__ logits,
                                                               long rows, int V, int nch,
                                                               float* __restrict__ cmax,
                                                               double* __restrict__ csum) {
  __shared__ float redf[kThreads / kWave];
  __shared__ double redd[kThreads / kWave];
  const long id = blockIdx.x;
  const long row = id / nch;
  const int c = int(id % nch);
  const float* src = logits + row * long(V) + long(c) * kChunk;
  const int n = min(kChunk, V - c * kChunk);
  float v[kPerThread];
  if (kVec) {
    // 16-byte loads: element 4*(tid + 256 i) + e
#pragma unroll
    for (int i = 0; i < kPerThread / 4; ++i) {
      int e0 = 4 * (threadIdx.x + kThreads * i);
      float4 t = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      if (e0 < n) t = *reinterpret_cast<const float4*>(src + e0);  // n % 4 == 0 here
      v[4 * i + 0] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      int e = threadIdx.x + kThreads * i;
      v[i] = e < n ? src[e] : -INFINITY;
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) mx = fmaxf(mx, v[i]);
  mx = block_max<kThreads / kWave>(mx, redf);
  float s = 0.f;
  if (mx != -INFINITY) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      // exp(l - mx) with the rounding of l - mx compensated: d + err == l - mx exactly
      // (TwoSum), exp(d + err) ~ expf(d) * (1 + err)
      const float d = v[i] - mx;
      const float bb = d - v[i];
      const float err = (v[i] - (d - bb)) + (-mx - bb);
      const float e = expf(d);
      s += (d == -INFINITY) ? 0.f : e + e * err;  // padding: exp(-inf) = 0
    }
  }
  double sd = block_sum<kThreads / kWave, double>(double(s), redd);
  if (threadIdx.x == 0) {
    cmax[id] = mx;
    csum[id] = sd;
  }
}

__device__ void row_moments(const float* cmax, const double* csum, long row, int nch, double& m,
                            double& S) {
  float mx = -INFINITY;
  for (int c = 0; c < nch; ++c) mx = fmaxf(mx, cmax[row * nch + c]);
  double acc = 0.0;
  for (int c = 0; c < nch; ++c) {
    float cm = cmax[row * nch + c];
    if (cm != -INFINITY) acc += csum[row * nch + c] * exp(double(cm) - double(mx));
  }
  m = double(mx);
  S = acc;
}

// ---- pass 2 ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void accept_kernel(
    const float* __restrict__ logits, const float* __restrict__ q, const int32_t* __restrict__ drafts,
    const float* __restrict__ u, int B, int k, int V, int nch, const float* __restrict__ cmax,
    const double* __restrict__ csum, int32_t* __restrict__ out_tokens, int32_t* __restrict__ out_n,
    float* __restrict__ out_lp, FinalDraw* __restrict__ fin, int dstride, int doff) {
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b >= B) return;
  const long r0 = long(b) * (k + 1);
  int n = k;
  int mode = 0, rej_draft = 0;
  double m = 0.0, S = 1.0;
  for (int i = 1; i <= k; ++i) {
    const int row = i - 1;
    row_moments(cmax, csum, r0 + row, nch, m, S);
    const int x = drafts[long(b) * dstride + doff + row];
    bool accept = false;
    double lx = 0.0;
    if (x >= 0 && x < V) {
      lx = double(logits[(r0 + row) * V + x]);
      const double ex = exp(lx - m);
      const double qx = q ? double(q[(long(b) * k + row) * V + x]) : 1.0;
      const double lhs = double(u[r0 + row]) * qx * S;
      accept = lhs < ex;
    }
    if (accept) {
      out_tokens[r0 + row] = x;
      if (out_lp) out_lp[r0 + row] = float((lx - m) - log(S));
    } else {
      n = row;
      mode = q ? 1 : 2;
      rej_draft = x;
      break;
    }
  }
  if (mode == 0) row_moments(cmax, csum, r0 + k, nch, m, S);  // bonus row k (also k == 0)
  for (int j = n + 1; j <= k; ++j) {
    out_tokens[r0 + j] = -1;
    if (out_lp) out_lp[r0 + j] = __builtin_nanf("");
  }
  out_n[b] = n;
  FinalDraw f;
  f.m = m;
  f.S = S;
  f.row = n;
  f.mode = mode;
  f.draft = rej_draft;
  f.pad = 0;
  fin[b] = f;
}

// residual mass of one logit on the 2^62 grid
__device__ __forceinline__ unsigned long long grid_mass(float l, double m, double invS, int mode,
                                                        float qv, bool is_draft) {
  const double p = exp(double(l) - m) * invS;   // f64: only the rounding of S remains
  double r = p;
  if (mode == 1) r = p - double(qv);
  else if (mode == 2 && is_draft) r = p - 1.0;
  if (!(r > 0.0)) return 0ull;
  return (unsigned long long)(r * 4611686018427387904.0);  // 2^62; truncation == floor
}

// ---- pass 3 ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void draw_mass_kernel(
    const float* __restrict__ logits, const float* __restrict__ q, int k, int V, int nch,
    const FinalDraw* __restrict__ fin, unsigned long long* __restrict__ chunk_tot) {
  __shared__ unsigned long long red[kThreads / kWave];
  const long id = blockIdx.x;
  const int b = int(id / nch);
  const int c = int(id % nch);
  const FinalDraw f = fin[b];
  const float* lrow = logits + (long(b) * (k + 1) + f.row) * V;
  const float* qrow = (f.mode == 1) ? q + (long(b) * k + f.row) * V : nullptr;
    const double invS = 1.0 / f.S;
  const int base = c * kChunk;
  const int n = min(kChunk, V - base);
  unsigned long long acc = 0;
  for (int i = threadIdx.x; i < n; i += kThreads) {
    const int t = base + i;
    acc += grid_mass(lrow[t], f.m, invS, f.mode, qrow ? qrow[t] : 0.f, t == f.draft);
  }
  acc = block_sum<kThreads / kWave, unsigned long long>(acc, red);
  if (threadIdx.x == 0) chunk_tot[id] = acc;
}

// ---- pass 4 ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void draw_pick_kernel(
    const float* __restrict__ logits, const float* __restrict__ q, const float* __restrict__ u,
    int k, int V, int nch, const FinalDraw* __restrict__ fin,
    unsigned long long* __restrict__ chunk_tot, int32_t* __restrict__ out_tokens,
    float* __restrict__ out_lp) {
  __shared__ unsigned long long scan[kThreads];
  __shared__ unsigned long long s_target;
  __shared__ int s_chunk, s_mode, s_token;
  __shared__ unsigned long long red[kThreads / kWave];
  const int b = blockIdx.x;
  FinalDraw f = fin[b];
  const float* lrow = logits + (long(b) * (k + 1) + f.row) * V;
  const float* qrow = (f.mode == 1) ? q + (long(b) * k + f.row) * V : nullptr;
    const double invS = 1.0 / f.S;
  const unsigned long long* tots = chunk_tot + long(b) * nch;

  if (threadIdx.x == 0) {
    unsigned long long tot = 0;
    for (int c = 0; c < nch; ++c) tot += tots[c];
    s_mode = (tot == 0) ? 0 : f.mode;       // vanished residual: fall back to p
    scan[0] = tot;
  }
  __syncthreads();
  const int mode = s_mode;
  if (mode != f.mode) {
    // recompute the per-chunk masses of p (rare degenerate path)
    for (int c = 0; c < nch; ++c) {
      unsigned long long acc = 0;
      const int base = c * kChunk, n = min(kChunk, V - base);
      for (int i = threadIdx.x; i < n; i += kThreads)
        acc += grid_mass(lrow[base + i], f.m, invS, 0, 0.f, false);
      acc = block_sum<kThreads / kWave, unsigned long long>(acc, red);
      if (threadIdx.x == 0) chunk_tot[long(b) * nch + c] = acc;
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) {
    unsigned long long tot = 0;
    for (int c = 0; c < nch; ++c) tot += tots[c];
    const float ub = u[long(b) * (k + 1) + k];
    const unsigned long long u32 = (unsigned long long)(double(ub) * 4294967296.0);
    const unsigned long long target = (tot >> 32) * u32 + (((tot & 0xffffffffull) * u32) >> 32);
    unsigned long long pre = 0;
    int c = 0;
    for (; c < nch - 1; ++c) {
      if (pre + tots[c] > target) break;
      pre += tots[c];
    }
    s_chunk = c;
    s_target = target - pre;  // offset inside chunk c
    s_token = -1;
  }
  __syncthreads();
  const int c = s_chunk;
  const unsigned long long tgt = s_target;
  // each thread owns kPerThread consecutive logits of the chunk
  const int base = c * kChunk;
  const int n = min(kChunk, V - base);
  const int e0 = threadIdx.x * kPerThread;
  unsigned long long mass[kPerThread];
  unsigned long long local = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int e = e0 + i;
    unsigned long long g = 0;
    if (e < n) {
      const int t = base + e;
      g = grid_mass(lrow[t], f.m, invS, mode, qrow ? qrow[t] : 0.f, t == f.draft);
    }
    mass[i] = g;
    local += g;
  }
  // inclusive block scan of the per-thread totals (Hillis-Steele, integers: exact)
  scan[threadIdx.x] = local;
  __syncthreads();
  for (int off = 1; off < kThreads; off <<= 1) {
    unsigned long long add = threadIdx.x >= off ? scan[threadIdx.x - off] : 0ull;
    __syncthreads();
    scan[threadIdx.x] += add;
    __syncthreads();
  }
  const unsigned long long incl = scan[threadIdx.x];
  const unsigned long long excl = incl - local;
  if (local > 0 && excl <= tgt && tgt < incl) {
    unsigned long long run = excl;
    for (int i = 0; i < kPerThread; ++i) {
      run += mass[i];
      if (run > tgt) {
        s_token = base + e0 + i;
        break;
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int tok = s_token;
    out_tokens[long(b) * (k + 1) + f.row] = tok;
    if (out_lp)
      out_lp[long(b) * (k + 1) + f.row] =
          tok >= 0 ? float((double(lrow[tok]) - f.m) - log(f.S)) : __builtin_nanf("");
  }
}

}  // namespace

int sampler_chunk_elems() { return kChunk; }

size_t sampler_ws_bytes(int B, int k, int V) {
  const long nch = (V + kChunk - 1) / kChunk;
  const long rows = long(B) * (k + 1);
  Carver c(nullptr, 0);
  c.take<float>(rows * nch);
  c.take<double>(rows * nch);
  c.take<FinalDraw>(B);
  c.take<unsigned long long>(long(B) * nch);
  return c.used + 256;
}

hipError_t launch_spec_accept(const float* logits, const float* q, const int32_t* drafts,
                              const float* u, int B, int k, int V, int32_t* out_tokens,
                              int32_t* out_n, float* out_lp, void* ws, hipStream_t s,
                              int draft_stride, int draft_offset) {
  const int nch = (V + kChunk - 1) / kChunk;
  const long rows = long(B) * (k + 1);
  Carver c(ws, 0);
  float* cmax = c.take<float>(rows * nch);
  double* csum = c.take<double>(rows * nch);
  FinalDraw* fin = c.take<FinalDraw>(B);
  unsigned long long* ctot = c.take<unsigned long long>(long(B) * nch);
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
  if (vec)
    chunk_stats_kernel<true><<<dim3(unsigned(rows * nch)), kThreads, 0, s>>>(logits, rows, V, nch,
                                                                              cmax, csum);
  else
    chunk_stats_kernel<false><<<dim3(unsigned(rows * nch)), kThreads, 0, s>>>(logits, rows, V, nch,
                                                                               cmax, csum);
  accept_kernel<<<dim3((B + kThreads - 1) / kThreads), kThreads, 0, s>>>(
      logits, q, drafts, u, B, k, V, nch, cmax, csum, out_tokens, out_n, out_lp, fin,
      draft_stride < 0 ? k : draft_stride, draft_offset);
  draw_mass_kernel<<<dim3(unsigned(long(B) * nch)), kThreads, 0, s>>>(logits, q, k, V, nch, fin,
                                                                       ctot);
  draw_pick_kernel<<<dim3(B), kThreads, 0, s>>>(logits, q, u, k, V, nch, fin, ctot, out_tokens,
                                                out_lp);
  return hipGetLastError();
}

}  // namespace molt
