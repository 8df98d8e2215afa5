// Fused vocab-wide softmax statistics, speculative accept, residual resample and
// behavior log-probs (the serving engine's speculative-decoding accept rule with
// temperature 1 and no truncation; paper Sec. 4.1 control table, Sec. 4.2, Sec. 5.3/5.4;
// rule of Leviathan et al. 2023 / Chen et al. 2023).
//
// Four launches, all deterministic (fixed reduction orders, integer prefix sums, no
// atomics):
//   1. chunk_stats  grid = rows * chunks: per 8192-logit chunk its max and
//                   sum exp(l - chunk max) (f32 exp2 with the roundings of the difference and
//                   of the base change compensated, f64 accumulation across threads).
//   2. decide       one workgroup per sequence: row moments (m, S) from the chunk
//                   statistics, the k tests u*q*S < exp(l_x - m) in f64, the accepted drafts
//                   with their log-probs, n, and the descriptor of the final draw.
//   3. mass         grid = B * chunks: the integer mass floor(r_t 2^62) of each logit of the
//                   final draw's row (residual max(0, p - q), or p for a bonus draw; p_t to
//                   ~1e-10 relative, so that the only rounding that matters in the draw is
//                   that of S, which scales every mass alike), summed per 256-logit
//                   sub-block and per chunk.
//   4. draw_pick    one wavefront per sequence: Tot, target = (Tot * floor(u 2^32)) >> 32,
//                   then three integer prefix searches (chunk, sub-block, 4 logits per lane)
//                   that recompute only the one sub-block's masses.
// Bytes: pass 1 reads the B(1+k)V logits once; pass 3 reads one row (+ one q row on a
// rejection) per sequence; pass 4 reads 1 KB (+ 1 KB) per sequence. Pass 1 and 3 are VALU
// bound as much as HBM bound (without packed math a wave64 instruction takes 4 cycles), so
// their per-logit instruction counts are kept small.
#include "device_common.h"
#include "internal.h"

// The draw recomputes masses in two kernels; both must round identically, so no
// floating-point contraction in this file.
#pragma clang fp contract(off)

namespace molt {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 32;
constexpr int kChunk = kThreads * kPerThread;  // 8192 logits per chunk
constexpr int kSub = 4 * kWave;                // 256 logits per draw sub-block
constexpr int kSubs = kChunk / kSub;           // 32 sub-blocks per chunk
constexpr int kRowsPerBatch = 16;              // accept rows examined per batch (4 per wave)
constexpr float kL2e = 0x1.715476p+0f;         // log2(e) rounded to f32
constexpr float kL2eLo = 0x1.4ae0c0p-26f;      // log2(e) - kL2e
constexpr float kLn2 = 0x1.62e430p-1f;         // ln 2

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
    // 16-byte nontemporal loads (each logit is read once here), element 4*(tid + 256 i) + e,
    // from clamped addresses so that no branch separates them (n % 4 == 0 here)
#pragma unroll
    for (int i = 0; i < kPerThread / 4; ++i) {
      const int e0 = 4 * (threadIdx.x + kThreads * i);
      const floatx4_t t = __builtin_nontemporal_load(reinterpret_cast<const floatx4_t*>(src + min(e0, n - 4)));
      const bool in = e0 < n;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * i + e] = in ? t[e] : -INFINITY;
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
    // exp(l - mx) to ~1 ulp with every rounding compensated: logits below mx - 200 (and the
    // padding's -inf) are raised to it, where exp underflows to 0 in f32; d + err == l - mx
    // exactly (TwoSum); d log2(e) = t + terr (FMA split, log2(e) = kL2e + kL2eLo); then
    // exp(l - mx) = 2^t * exp(terr ln2 + err) ~ 2^t (1 + terr ln2 + err), with 2^t from the
    // hardware exp2 (1 ulp)
    const float lo = mx - 200.0f, nmx = -mx;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const float vc = fmaxf(v[i], lo);
      const float d = vc + nmx;
      const float bb = d - vc;
      const float err = (vc - (d - bb)) + (nmx - bb);
      const float t = d * kL2e;
      const float terr = fmaf(d, kL2eLo, fmaf(d, kL2e, -t));
      const float e = __builtin_amdgcn_exp2f(t);
      s += fmaf(e, fmaf(terr, kLn2, err), e);
    }
  }
  double sd = block_sum<kThreads / kWave, double>(double(s), redd);
  if (threadIdx.x == 0) {
    cmax[id] = mx;
    csum[id] = sd;
  }
}

// inclusive prefix sum over the wavefront (integers: exact)
MOLT_DEV unsigned long long wave_incl_scan(unsigned long long v, int lane) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const unsigned long long u = __shfl_up(v, o, kWave);
    if (lane >= o) v += u;
  }
  return v;
}

// exp(x) for x <= 0 by the table-driven method of P. T. P. Tang (ACM TOMS 15(2), 1989):
// x = (256 m + j) ln2/256 + r with |r| <= ln2/512 (reduction in f64, exact), exp(x) =
// 2^m * 2^(j/256) * (1 + p(r)), tab[j] = 2^(j/256) in f64 (built in LDS by exp_table_init)
// and p(r) = r + r^2/2 + r^3/6 evaluated in f32: |p| < 1.4e-3, so its f32 rounding and the
// truncation (r^4/24 < 1.4e-13) leave a relative error below 3e-10, far inside the 2e-8 of
// the integer total within which a draw counts as a near-tie. About a third of the
// instructions of a library f64 exp; the draw evaluates it for every logit of B rows.
constexpr double kExpInvL = 0x1.71547652b82fep+8;   // 256 / ln2
constexpr double kExpLhi = 0x1.62e42fef80000p-9;    // ln2 / 256, 34 significant bits
constexpr double kExpLlo = 0x1.1cf79abc9e3b4p-44;   // ln2 / 256 - kExpLhi

MOLT_DEV double exp_nonpos(double x, const double* tab) {
  // below -746 the result underflows to 0 (2^-1077); -inf and NaN land there too
  x = fmax(x, -746.0);
  const double n = rint(x * kExpInvL);
  const int N = int(n);
  double r = fma(-n, kExpLhi, x);                    // exact: n * kExpLhi has <= 53 bits
  r = fma(-n, kExpLlo, r);
  const float rf = float(r);
  const float pf = rf * fmaf(rf, fmaf(rf, 1.0f / 6.0f, 0.5f), 1.0f);
  const double t = tab[N & 255];
  return ldexp(fma(t, double(pf), t), N >> 8);       // N >> 8 == floor(N / 256)
}

// tab[j] = 2^(j / 256), j < 256, by nthreads threads; the caller synchronises
MOLT_DEV void exp_table_init(double* tab, int tid, int nthreads) {
  for (int j = tid; j < 256; j += nthreads) tab[j] = exp2(double(j) / 256.0);
}

// floor(r * 2^62) for 0 <= r <= 1 + 2^-52: r 2^30 = hi + f exactly (hi = its integer part,
// f its exact fraction), floor(f 2^32) = lo; r 2^62 = hi 2^32 + f 2^32
MOLT_DEV unsigned long long grid_floor(double r) {
  const double s = r * 1073741824.0;                  // 2^30
  const uint32_t hi = uint32_t(s);
  const uint32_t lo = uint32_t((s - double(hi)) * 4294967296.0);
  return (static_cast<unsigned long long>(hi) << 32) | lo;
}

// residual mass of one logit on the 2^62 grid
MOLT_DEV unsigned long long grid_mass(float l, double m, double invS, int mode, float qv,
                                      bool is_draft, const double* tab) {
  const double p = exp_nonpos(double(l) - m, tab) * invS;   // only S's rounding remains
  double r = p;
  if (mode == 1) r = p - double(qv);
  else if (mode == 2 && is_draft) r = p - 1.0;
  return r > 0.0 ? grid_floor(r) : 0ull;
}

// The 4 consecutive logits [t0, t0 + 4) of a draw row and, for a residual draw against a
// q row, their q values (0 past V). Loads are issued separately from the arithmetic so that
// a thread's loads are all in flight before the first exp waits on one.
struct Quad {
  float l[4], q[4];
};

template <bool kVec>
MOLT_DEV void quad_load(const float* lrow, const float* qrow, int t0, int V, int mode, Quad& d) {
  // Unconditional loads from clamped addresses (values past V are masked by quad_mass; a
  // non-residual draw reads its logits row again in place of q): no branch separates a
  // load from the next one, so none waits for an earlier one to return.
  const float* qsrc = mode == 1 ? qrow : lrow;
  if (kVec) {
    const int a = min(t0, V - 4);       // V % 4 == 0, V >= 4: the quad is all in or all out
    const float4 x = *reinterpret_cast<const float4*>(lrow + a);
    const float4 y = *reinterpret_cast<const float4*>(qsrc + a);
    d.l[0] = x.x; d.l[1] = x.y; d.l[2] = x.z; d.l[3] = x.w;
    d.q[0] = y.x; d.q[1] = y.y; d.q[2] = y.z; d.q[3] = y.w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int a = min(t0 + e, V - 1);
      d.l[e] = lrow[a];
      d.q[e] = qsrc[a];
    }
  }
}

// masses of a loaded quad (0 past V), and their sum
MOLT_DEV unsigned long long quad_mass(const Quad& d, int t0, int V, const FinalDraw& f, double invS,
                                      int mode, const double* tab, unsigned long long (&g)[4]) {
  unsigned long long sum = 0;
  const int dr = f.draft - t0;                       // the draft's place in the quad, if any
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    g[e] = t0 + e < V ? grid_mass(d.l[e], f.m, invS, mode, d.q[e], dr == e, tab) : 0ull;
    sum += g[e];
  }
  return sum;
}

// ---- pass 2 ---------------------------------------------------------------------------
// One workgroup per sequence: its accept decisions, batches of 16 rows (row r on wavefront
// r % 4): row moments (m, S) from the chunk statistics, the tests u*q*S < exp(l_x - m) in
// f64, the accepted drafts and their log-probs, n, and the descriptor of the final draw.
__global__ __launch_bounds__(kThreads) void decide_kernel(
    const float* __restrict__ logits, const float* __restrict__ q, const int32_t* __restrict__ drafts,
    const float* __restrict__ u, int k, int V, int nch, const float* __restrict__ cmax,
    const double* __restrict__ csum, int dstride, int doff, int32_t* __restrict__ out_tokens,
    int32_t* __restrict__ out_n, float* __restrict__ out_lp, FinalDraw* __restrict__ fin) {
  __shared__ double s_m[kRowsPerBatch], s_S[kRowsPerBatch], s_lx[kRowsPerBatch];
  __shared__ int s_ok[kRowsPerBatch], s_x[kRowsPerBatch];
  __shared__ int s_n;
  __shared__ FinalDraw s_fin;
  const int b = blockIdx.x;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const long r0 = long(b) * (k + 1);
  if (threadIdx.x == 0) s_n = -1;
  // ---- the sequence's decisions, batches of 16 rows (row r on wavefront r % 4)
  for (int base = 0; base <= k; base += kRowsPerBatch) {
    constexpr int kPer = kRowsPerBatch / 4;
    float cm[kPer];
    double cs[kPer];
    int xv[kPer];
    float uv[kPer];
    // issue every load of the batch first: chunk statistics (lane = chunk) and, on lane 0,
    // the draft id and its uniform
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int r = base + wave + 4 * j;
      cm[j] = -INFINITY;
      cs[j] = 0.0;
      xv[j] = -1;
      uv[j] = 0.f;
      if (r <= k && lane < nch) {
        cm[j] = cmax[(r0 + r) * nch + lane];
        cs[j] = csum[(r0 + r) * nch + lane];
      }
      if (r < k && lane == 0) {
        xv[j] = drafts[long(b) * dstride + doff + r];
        uv[j] = u[r0 + r];
      }
    }
    float lxv[kPer];
    float qxv[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int r = base + wave + 4 * j;
      lxv[j] = 0.f;
      qxv[j] = 1.f;
      const int x = xv[j];
      if (r < k && lane == 0 && x >= 0 && x < V) {
        lxv[j] = logits[(r0 + r) * V + x];
        if (q) qxv[j] = q[(long(b) * k + r) * V + x];
      }
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int r = base + wave + 4 * j;
      if (r > k) break;
      // row moments: m = max of the chunk maxima, S = sum csum * exp(cmax - m) (f64)
      float mx = -INFINITY;
      for (int cc = lane; cc < nch; cc += kWave) {
        const float v = cc == lane ? cm[j] : cmax[(r0 + r) * nch + cc];
        mx = fmaxf(mx, v);
      }
      mx = wave_max(mx);
      double acc = 0.0;
      for (int cc = lane; cc < nch; cc += kWave) {
        const float v = cc == lane ? cm[j] : cmax[(r0 + r) * nch + cc];
        const double sv = cc == lane ? cs[j] : csum[(r0 + r) * nch + cc];
        if (v != -INFINITY) acc += sv * exp(double(v) - double(mx));
      }
      acc = wave_sum(acc);
      if (lane == 0) {
        const int i = r - base;
        const double m = double(mx);
        s_m[i] = m;
        s_S[i] = acc;
        s_x[i] = xv[j];
        s_ok[i] = 0;
        if (r < k) {
          const int x = xv[j];
          bool accept = false;
          double lx = 0.0;
          if (x >= 0 && x < V) {
            lx = double(lxv[j]);
            const double ex = exp(lx - m);
            const double qx = q ? double(qxv[j]) : 1.0;
            accept = double(uv[j]) * qx * acc < ex;
          }
          s_ok[i] = accept;
          s_lx[i] = lx;
        }
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      // first rejection in this batch decides n; accepted rows before it are emitted
      const int last = min(k, base + kRowsPerBatch - 1);
      for (int r = base; r <= last; ++r) {
        const int i = r - base;
        if (r == k || !s_ok[i]) {
          s_n = r;
          FinalDraw f;
          f.m = s_m[i];
          f.S = s_S[i];
          f.row = r;
          f.mode = r == k ? 0 : (q ? 1 : 2);
          f.draft = r == k ? -1 : s_x[i];
          f.pad = 0;
          s_fin = f;
          break;
        }
        out_tokens[r0 + r] = s_x[i];
        if (out_lp) out_lp[r0 + r] = float((s_lx[i] - s_m[i]) - log(s_S[i]));
      }
    }
    __syncthreads();
    if (s_n >= 0) break;
  }
  const int n = s_n;
  for (int j = n + 1 + int(threadIdx.x); j <= k; j += kThreads) {
    out_tokens[r0 + j] = -1;
    if (out_lp) out_lp[r0 + j] = __builtin_nanf("");
  }
  if (threadIdx.x == 0) {
    out_n[b] = n;
    fin[b] = s_fin;
  }
}

// ---- pass 3 ---------------------------------------------------------------------------
// Integer mass of chunk c of sequence b's final-draw row. Logit t of the chunk sits at
// c*8192 + 2048 w + 256 i + 4 l + e for wavefront w, step i < 8, lane l, e < 4; sub-block
// 8 w + i is [256 (8 w + i), +256) of the chunk.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void mass_kernel(
    const float* __restrict__ logits, const float* __restrict__ q, int k, int V, int nch,
    const FinalDraw* __restrict__ fin, unsigned long long* __restrict__ chunk_tot,
    unsigned long long* __restrict__ sub_tot) {
  __shared__ unsigned long long s_sub[kSubs];
  __shared__ double s_tab[256];
  exp_table_init(s_tab, threadIdx.x, kThreads);
  const int b = blockIdx.x / nch;
  const int c = blockIdx.x % nch;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const long r0 = long(b) * (k + 1);
  const FinalDraw f = fin[b];
  __syncthreads();
  const float* lrow = logits + (r0 + f.row) * V;
  const float* qrow = f.mode == 1 ? q + (long(b) * k + f.row) * V : nullptr;
  const double invS = 1.0 / f.S;
  const int t_base = c * kChunk + 2048 * wave + 4 * lane;
  Quad qd[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) quad_load<kVec>(lrow, qrow, t_base + kSub * i, V, f.mode, qd[i]);
  unsigned long long part[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    unsigned long long g[4];
    part[i] = quad_mass(qd[i], t_base + kSub * i, V, f, invS, f.mode, s_tab, g);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const unsigned long long sb = wave_sum(part[i]);
    if (lane == 0) s_sub[8 * wave + i] = sb;
  }
  __syncthreads();
  if (threadIdx.x < kSubs) sub_tot[(long(b) * nch + c) * kSubs + threadIdx.x] = s_sub[threadIdx.x];
  if (threadIdx.x == 0) {
    unsigned long long tot = 0;
    for (int j = 0; j < kSubs; ++j) tot += s_sub[j];
    chunk_tot[long(b) * nch + c] = tot;
  }
}

// ---- pass 4 ---------------------------------------------------------------------------
// One wavefront per sequence. Zero residual mass (p <= q everywhere after rounding) falls
// back to p: the chunk and sub-block masses of p are then recomputed here (rare path).
template <bool kVec>
__global__ __launch_bounds__(kWave) void draw_pick_kernel(
    const float* __restrict__ logits, const float* __restrict__ q, const float* __restrict__ u,
    int k, int V, int nch, const FinalDraw* __restrict__ fin,
    const unsigned long long* __restrict__ chunk_tot, const unsigned long long* __restrict__ sub_tot,
    int32_t* __restrict__ out_tokens, float* __restrict__ out_lp) {
  __shared__ double s_tab[256];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  exp_table_init(s_tab, lane, kWave);
  __syncthreads();
  const FinalDraw f = fin[b];
  const float* lrow = logits + (long(b) * (k + 1) + f.row) * V;
  const float* qrow = f.mode == 1 ? q + (long(b) * k + f.row) * V : nullptr;
  const double invS = 1.0 / f.S;
  const unsigned long long* tots = chunk_tot + long(b) * nch;
  const float ub = u[long(b) * (k + 1) + k];
  unsigned long long tot = 0;
  for (int c = lane; c < nch; c += kWave) tot += tots[c];
  tot = wave_sum(tot);
  int mode = f.mode;
  // sum of the masses of sub-block j of chunk c under `mode`, recomputed by the wavefront
  auto sub_mass = [&](int c, int j, int md) {
    unsigned long long g[4];
    const int t0 = c * kChunk + kSub * j + 4 * lane;
    Quad d;
    quad_load<kVec>(lrow, qrow, t0, V, md, d);
    return wave_sum(quad_mass(d, t0, V, f, invS, md, s_tab, g));
  };
  if (tot == 0 && mode != 0) {
    mode = 0;
    tot = 0;
    for (int c = 0; c < nch; ++c)
      for (int j = 0; j < kSubs; ++j) tot += sub_mass(c, j, 0);
  }
  const unsigned long long u32 = (unsigned long long)(double(ub) * 4294967296.0);
  // target = (tot * u32) >> 32 without a 128-bit type
  const unsigned long long target = (tot >> 32) * u32 + (((tot & 0xffffffffull) * u32) >> 32);
  // 1. the chunk holding the target
  unsigned long long pre = 0;   // mass before the current window
  int chunk = -1;
  for (int c0 = 0; c0 < nch && chunk < 0; c0 += kWave) {
    const int c = c0 + lane;
    unsigned long long v = 0;
    if (mode == f.mode) {
      if (c < nch) v = tots[c];
    } else {
      // fallback: chunk masses of p, one chunk at a time (wavefront-wide sums)
      for (int cc = c0; cc < min(nch, c0 + kWave); ++cc) {
        unsigned long long sm = 0;
        for (int j = 0; j < kSubs; ++j) sm += sub_mass(cc, j, 0);
        if (lane == cc - c0) v = sm;
      }
    }
    const unsigned long long incl = wave_incl_scan(v, lane);
    const unsigned long long hit = __ballot(c < nch && pre + incl > target);
    if (hit) {
      const int l = __builtin_ctzll(hit);
      chunk = c0 + l;
      pre += __shfl(incl - v, l, kWave);
    } else {
      pre += __shfl(incl, kWave - 1, kWave);
    }
  }
  int token = -1;
  if (chunk >= 0) {
    // 2. the sub-block inside the chunk (lanes 0..31 hold the 32 sub-block masses)
    unsigned long long v = 0;
    if (mode == f.mode) {
      if (lane < kSubs) v = sub_tot[(long(b) * nch + chunk) * kSubs + lane];
    } else {
      for (int j = 0; j < kSubs; ++j) {
        const unsigned long long s = sub_mass(chunk, j, 0);
        if (lane == j) v = s;
      }
    }
    unsigned long long incl = wave_incl_scan(v, lane);
    unsigned long long hit = __ballot(lane < kSubs && pre + incl > target);
    if (hit) {
      const int j = __builtin_ctzll(hit);
      pre += __shfl(incl - v, j, kWave);
      // 3. four logits per lane inside the sub-block
      unsigned long long g[4];
      const int t0 = chunk * kChunk + kSub * j + 4 * lane;
      Quad d;
      quad_load<kVec>(lrow, qrow, t0, V, mode, d);
      const unsigned long long mine = quad_mass(d, t0, V, f, invS, mode, s_tab, g);
      incl = wave_incl_scan(mine, lane);
      hit = __ballot(pre + incl > target);
      if (hit) {
        const int l = __builtin_ctzll(hit);
        if (lane == l) {
          unsigned long long run = pre + incl - mine;
          for (int e = 0; e < 4; ++e) {
            run += g[e];
            if (run > target) {
              token = t0 + e;
              break;
            }
          }
        }
        token = __shfl(token, l, kWave);
      }
    }
  }
  if (lane == 0) {
    out_tokens[long(b) * (k + 1) + f.row] = token;
    if (out_lp)
      out_lp[long(b) * (k + 1) + f.row] =
          token >= 0 ? float((double(lrow[token]) - f.m) - log(f.S)) : __builtin_nanf("");
  }
}


// ---- MTP draft draws --------------------------------------------------------------------
// q[b * q_stride + t] = softmax(logits[b])_t in f32: (m, S) combined from the chunk
// statistics exactly as the accept decisions combine them, exp(l - m) by the table exp.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void softmax_write_kernel(const float* __restrict__ logits,
                                                                 int V, int nch,
                                                                 const float* __restrict__ cmax,
                                                                 const double* __restrict__ csum,
                                                                 float* __restrict__ q, long q_stride) {
  __shared__ double tab[256];
  __shared__ double s_m, s_inv;
  const long row = blockIdx.x / nch;
  const int c = int(blockIdx.x % nch);
  exp_table_init(tab, threadIdx.x, kThreads);
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    float mx = -INFINITY;
    for (int cc = lane; cc < nch; cc += kWave) mx = fmaxf(mx, cmax[row * nch + cc]);
    mx = wave_max(mx);
    double acc = 0.0;
    for (int cc = lane; cc < nch; cc += kWave) {
      const float v = cmax[row * nch + cc];
      if (v != -INFINITY) acc += csum[row * nch + cc] * exp(double(v) - double(mx));
    }
    acc = wave_sum(acc);
    if (lane == 0) {
      s_m = double(mx);
      s_inv = 1.0 / acc;
    }
  }
  __syncthreads();
  const double m = s_m, inv = s_inv;
  const float* src = logits + row * long(V) + long(c) * kChunk;
  float* dst = q + row * q_stride + long(c) * kChunk;
  const int n = min(kChunk, V - c * kChunk);
  if (kVec) {
#pragma unroll 2
    for (int i = 0; i < kPerThread / 4; ++i) {
      const int e0 = 4 * (threadIdx.x + kThreads * i);
      if (e0 >= n) break;
      const floatx4_t l = __builtin_nontemporal_load(reinterpret_cast<const floatx4_t*>(src + e0));
      floatx4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = float(exp_nonpos(double(l[e]) - m, tab) * inv);
      *reinterpret_cast<floatx4_t*>(dst + e0) = o;
    }
  } else {
    for (int e = threadIdx.x; e < n; e += kThreads)
      dst[e] = float(exp_nonpos(double(src[e]) - m, tab) * inv);
  }
}

// out[b] = the first index of the largest logit of row b (0 for a row with no finite max)
__global__ __launch_bounds__(kThreads) void argmax_kernel(const float* __restrict__ logits, int V,
                                                          int32_t* __restrict__ out) {
  __shared__ float s_v[kThreads / kWave];
  __shared__ int s_i[kThreads / kWave];
  const long row = blockIdx.x;
  const float* src = logits + row * long(V);
  float best = -INFINITY;
  int bi = V;
  for (int t = threadIdx.x; t < V; t += kThreads) {   // a thread's indices increase
    const float v = src[t];
    if (v > best) { best = v; bi = t; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(best, o, kWave);
    const int oi = __shfl_xor(bi, o, kWave);
    if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
  }
  const int w = threadIdx.x / kWave;
  if (threadIdx.x % kWave == 0) { s_v[w] = best; s_i[w] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int j = 1; j < kThreads / kWave; ++j)
      if (s_v[j] > best || (s_v[j] == best && s_i[j] < bi)) { best = s_v[j]; bi = s_i[j]; }
    out[row] = bi < V ? bi : 0;
  }
}


// ---- scores of given tokens -------------------------------------------------------------
// lp[r] = (l[r, y] - m) - ln S for y = targets[r] in [0, V), else NaN: one wavefront per row,
// (m, S) combined from the chunk statistics exactly as the accept decisions combine them,
// so that a recompute of emitted tokens reproduces the recorded log-probs bit for bit.
__global__ __launch_bounds__(kWave) void token_logprob_kernel(const float* __restrict__ logits,
                                                              int V, int nch,
                                                              const float* __restrict__ cmax,
                                                              const double* __restrict__ csum,
                                                              const int32_t* __restrict__ targets,
                                                              float* __restrict__ out) {
  const long row = blockIdx.x;
  const int lane = threadIdx.x;
  float mx = -INFINITY;
  for (int cc = lane; cc < nch; cc += kWave) mx = fmaxf(mx, cmax[row * nch + cc]);
  mx = wave_max(mx);
  double acc = 0.0;
  for (int cc = lane; cc < nch; cc += kWave) {
    const float v = cmax[row * nch + cc];
    if (v != -INFINITY) acc += csum[row * nch + cc] * exp(double(v) - double(mx));
  }
  acc = wave_sum(acc);
  if (lane == 0) {
    const int y = targets[row];
    out[row] = (y >= 0 && y < V)
                   ? float((double(logits[row * long(V) + y]) - double(mx)) - log(acc))
                   : __builtin_nanf("");
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
  c.take<unsigned long long>(long(B) * nch * kSubs);
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
  unsigned long long* stot = c.take<unsigned long long>(long(B) * nch * kSubs);
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0) &&
                   (q == nullptr || (reinterpret_cast<uintptr_t>(q) & 15) == 0);
  const int ds = draft_stride < 0 ? k : draft_stride;
  const dim3 g1{unsigned(rows * nch)}, g2{unsigned(long(B) * nch)}, g3{unsigned(B)};
  if (vec) {
    chunk_stats_kernel<true><<<g1, kThreads, 0, s>>>(logits, rows, V, nch, cmax, csum);
    decide_kernel<<<g3, kThreads, 0, s>>>(logits, q, drafts, u, k, V, nch, cmax, csum, ds,
                                          draft_offset, out_tokens, out_n, out_lp, fin);
    mass_kernel<true><<<g2, kThreads, 0, s>>>(logits, q, k, V, nch, fin, ctot, stot);
    draw_pick_kernel<true><<<g3, kWave, 0, s>>>(logits, q, u, k, V, nch, fin, ctot, stot,
                                                out_tokens, out_lp);
  } else {
    chunk_stats_kernel<false><<<g1, kThreads, 0, s>>>(logits, rows, V, nch, cmax, csum);
    decide_kernel<<<g3, kThreads, 0, s>>>(logits, q, drafts, u, k, V, nch, cmax, csum, ds,
                                          draft_offset, out_tokens, out_n, out_lp, fin);
    mass_kernel<false><<<g2, kThreads, 0, s>>>(logits, q, k, V, nch, fin, ctot, stot);
    draw_pick_kernel<false><<<g3, kWave, 0, s>>>(logits, q, u, k, V, nch, fin, ctot, stot,
                                                 out_tokens, out_lp);
  }
  return hipGetLastError();
}

size_t draft_draw_ws_bytes(int B, int V) {
  Carver c(nullptr, 0);
  c.take<uint8_t>(sampler_ws_bytes(B, 0, V));
  c.take<int32_t>(B);
  c.take<float>(B);
  return c.used + 256;
}

hipError_t launch_draft_draw(const float* logits, int B, int V, const float* u, int32_t* out_tok,
                             float* q_out, long q_stride, void* ws, hipStream_t s) {
  if (u == nullptr) {
    argmax_kernel<<<B, kThreads, 0, s>>>(logits, V, out_tok);
    return hipGetLastError();
  }
  Carver c(ws, 0);
  void* samp = c.take<uint8_t>(sampler_ws_bytes(B, 0, V));
  int32_t* n = c.take<int32_t>(B);
  float* lp = c.take<float>(B);
  // a draw from p is the bonus draw of a step without drafts (k = 0, one uniform per row)
  hipError_t e = launch_spec_accept(logits, nullptr, out_tok, u, B, 0, V, out_tok, n, lp, samp, s);
  if (e != hipSuccess || q_out == nullptr) return e;
  // the row statistics of pass 1 sit at the start of the sampler's workspace
  const int nch = (V + kChunk - 1) / kChunk;
  Carver cs(samp, 0);
  const float* cmax = cs.take<float>(long(B) * nch);
  const double* csum = cs.take<double>(long(B) * nch);
  const bool vec = (V % 4 == 0) && (q_stride % 4 == 0) &&
                   ((reinterpret_cast<uintptr_t>(logits) & 15) == 0) &&
                   ((reinterpret_cast<uintptr_t>(q_out) & 15) == 0);
  const dim3 g{unsigned(long(B) * nch)};
  if (vec) softmax_write_kernel<true><<<g, kThreads, 0, s>>>(logits, V, nch, cmax, csum, q_out, q_stride);
  else softmax_write_kernel<false><<<g, kThreads, 0, s>>>(logits, V, nch, cmax, csum, q_out, q_stride);
  return hipGetLastError();
}

size_t token_logprob_ws_bytes(long rows, int V) {
  const long nch = (V + kChunk - 1) / kChunk;
  Carver c(nullptr, 0);
  c.take<float>(rows * nch);
  c.take<double>(rows * nch);
  return c.used + 256;
}

hipError_t launch_token_logprobs(const float* logits, long rows, int V, const int32_t* targets,
                                 float* out, void* ws, hipStream_t s) {
  const int nch = (V + kChunk - 1) / kChunk;
  Carver c(ws, 0);
  float* cmax = c.take<float>(rows * nch);
  double* csum = c.take<double>(rows * nch);
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
  const dim3 g1{unsigned(rows * nch)}, g2{unsigned(rows)};
  if (vec) chunk_stats_kernel<true><<<g1, kThreads, 0, s>>>(logits, rows, V, nch, cmax, csum);
  else chunk_stats_kernel<false><<<g1, kThreads, 0, s>>>(logits, rows, V, nch, cmax, csum);
  token_logprob_kernel<<<g2, kWave, 0, s>>>(logits, V, nch, cmax, csum, targets, out);
  return hipGetLastError();
}

}  // namespace molt
