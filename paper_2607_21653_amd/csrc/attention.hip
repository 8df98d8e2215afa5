// Multi-query paged decode attention of the verify step (PagedAttention cache, paper
// Sec. 2; k speculative tokens per sequence, Sec. 4.1). For sequence b and kv head h the
// R = G*(1+k) query rows (G = Hq/Hkv query heads, 1+k positions) share every key/value
// block, so each K/V byte is read once per (b, h) and reused by all R rows on MFMA.
//
// Work split: workgroup = (b, h, split of the key range), 4 wavefronts; the number of
// splits is chosen so the grid holds ~512 workgroups (at B*Hkv >= 512 there is no split and
// no merge pass). Each wavefront takes block pairs (32 keys) round-robin and keeps its own
// online softmax; the next pair's fragments are loaded into a second register set while
// the current pair computes (software pipelining through registers). Per pair, on
// v_mfma_f32_16x16x32_bf16:
//   S^T[32 keys x R] = K Q^T   (A = K rows straight from the cache: [16 keys x 32 dims]
//                               per operand, 16 B per lane; B = Q^T held in registers)
//   O^T[D x R]      += V^T P^T (A = V^T: the V cache stores a block as [D][16 tokens], so
//                               a lane's 4 consecutive keys of one dim are 8 contiguous
//                               bytes; B = P^T is exactly the S^T accumulator layout
//                               rounded to bf16: no cross-lane shuffles)
// The MFMA k-index is a free permutation as long as A and B agree: slot s of lane group g
// is key 4g+s of the first block (s < 4) or of the second block (s >= 4).
// Causality: row r = j*G + g (position j) sees keys <= ctx_b + j; only pairs reaching past
// ctx_b need masks. Softmax in f32 with exp2 of log2(e)-scaled scores; the output is
// rescaled lazily, only when a row maximum grows by more than 8 (in log2 units) over the
// reference it was accumulated with. The four wavefronts merge through LDS in a fixed order;
// splits are merged by a log-sum-exp pass (a single split writes the output directly).
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" for running maxima
constexpr float kRescaleSlack = 8.0f; // probabilities may grow to 2^8 before O is rescaled

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

struct AttnParams {
  const uint16_t* q;       // [T, Hq, D]
  const uint16_t* kc;      // [nb, Hkv, 16, D]
  const uint16_t* vc;      // [nb, Hkv, D, 16]
  const int32_t* bt;       // [B, max_blocks]
  const int32_t* ctx;      // [B]
  uint16_t* out;           // [T, Hq * D], row-major or tiled (out_tiled)
  float* part_o;           // [B, Hkv, S, R, D]
  float* part_ml;          // [B, Hkv, S, R, 2]
  int k, Hq, Hkv, max_blocks, splits, blocks_per_split;
  float scale_log2;        // log2(e) / sqrt(D)
  int out_tiled;           // output in the GEMM operand layout (input of the O projection)
};

// element index of output (token t, column c) of `cols` columns
MOLT_DEV long out_index(const AttnParams& p, long t, long c, long cols, int esize) {
  return p.out_tiled ? tiled_index(t, c, cols, esize) : t * cols + c;
}

// K and V^T fragments of one 32-key block pair for one wavefront
template <int D>
struct PairFrags {
  bf16x8_t k[2][D / 32];
  bf16x8_t v[D / 16];
};

template <int D, int RT>
__global__ __launch_bounds__(kThreads) void attn_mfma_kernel(AttnParams p) {
  constexpr int DS = D / 32;      // 32-dim k-steps for S
  constexpr int DT = D / 16;      // 16-dim tiles of O^T
  constexpr int RP = RT * 16;     // padded rows
  __shared__ float s_m[kWaves][RP];
  __shared__ float s_l[kWaves][RP];
  __shared__ float s_o[RP * D];

  const int split = blockIdx.x % p.splits;
  const int bh = blockIdx.x / p.splits;
  const int b = bh / p.Hkv, h = bh % p.Hkv;
  const int G = p.Hq / p.Hkv;
  const int kp1 = p.k + 1;
  const int R = G * kp1;
  const int ctx = p.ctx[b];
  const int nkeys = ctx + kp1;
  const int nblk = (nkeys + 15) / 16;
  const int blk0 = split * p.blocks_per_split;
  const int blk1 = min(blk0 + p.blocks_per_split, nblk);
  // wave-uniform in a scalar register, so block-table reads become scalar loads that do not
  // share the vector memory counter with the K/V prefetch
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int l16 = lane % 16, g4 = lane / 16;
  const float c = p.scale_log2;

  // Q^T fragments: row r = l16 + 16 * rt; dims [32 s + 8 g4, +8)
  bf16x8_t qf[RT][DS];
  int lim[RT];   // last visible key position of the lane's row (-1: padding row)
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = rt * 16 + l16;
    const int j = r / G, gi = r % G;
    lim[rt] = r < R ? ctx + j : -1;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      if (r < R) {
        const uint16_t* src = p.q + ((long(b) * kp1 + j) * p.Hq + h * G + gi) * D + s * 32 + g4 * 8;
        qf[rt][s] = *reinterpret_cast<const bf16x8_t*>(src);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[rt][s][e] = __bf16(0.f);
      }
    }
  }

  floatx4_t o[DT][RT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) o[dt][rt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[RT], l_run[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) { m_run[rt] = kNegBig; l_run[rt] = 0.f; }

  const int* btab = p.bt + long(b) * p.max_blocks;
  const long kv_blk_stride = long(p.Hkv) * 16 * D;
  const uint16_t* kbase = p.kc + long(h) * 16 * D + l16 * D + g4 * 8;
  const uint16_t* vbase = p.vc + long(h) * D * 16 + l16 * 16 + g4 * 4;

  // K/V are read once per step: nontemporal loads (they stream at ~7.1 TB/s on MI355X
  // against ~6.3 TB/s for ordinary loads)
  auto load_pair = [&](PairFrags<D>& f, int pb) {
    const long phys0 = btab[pb];
    const long phys1 = (pb + 1 < blk1) ? btab[pb + 1] : phys0;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      f.k[0][s] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(kbase + phys0 * kv_blk_stride + s * 32));
      f.k[1][s] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(kbase + phys1 * kv_blk_stride + s * 32));
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const bf16x4_t a = __builtin_nontemporal_load(reinterpret_cast<const bf16x4_t*>(vbase + phys0 * kv_blk_stride + dt * 256));
      const bf16x4_t e = __builtin_nontemporal_load(reinterpret_cast<const bf16x4_t*>(vbase + phys1 * kv_blk_stride + dt * 256));
      f.v[dt] = bf16x8_t{a[0], a[1], a[2], a[3], e[0], e[1], e[2], e[3]};
    }
  };

  auto compute_pair = [&](const PairFrags<D>& f, int pb) {
    // S^T tiles: lane holds keys 4 g4 + e of block pb (t = 0) and pb + 1 (t = 1)
    floatx4_t st[2][RT];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < DS; ++s)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.k[t][s], qf[rt][s], acc, 0, 0, 0);
        st[t][rt] = acc;
      }
    // keys at or past pb*16 + 31 <= ctx are visible to every row: no mask needed
    const bool full = pb * 16 + 31 <= ctx;
    if (!full) {
      const bool has2 = pb + 1 < blk1;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int kpos = (pb + t) * 16 + g4 * 4 + e;
            if (!((t == 0 || has2) && kpos <= lim[rt])) st[t][rt][e] = -INFINITY;
          }
    }
    // row maxima (raw scores; the scale is positive) across the lane's 8 keys and 4 groups
    float mx[RT];
    bool grow = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float v = fmaxf(fmaxf(fmaxf(st[0][rt][0], st[0][rt][1]), fmaxf(st[0][rt][2], st[0][rt][3])),
                      fmaxf(fmaxf(st[1][rt][0], st[1][rt][1]), fmaxf(st[1][rt][2], st[1][rt][3])));
      v = fmaxf(v, __shfl_xor(v, 16, kWave));
      v = fmaxf(v, __shfl_xor(v, 32, kWave));
      mx[rt] = v * c;
      grow |= mx[rt] > m_run[rt] + kRescaleSlack;
    }
    // lazy rescale, uniform over the wavefront: only when some row's maximum has grown by
    // more than the slack (the result is the same softmax for any reference maximum)
    if (__builtin_amdgcn_read_exec() & __ballot(grow)) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const float m_new = fmaxf(m_run[rt], mx[rt]);
        const float alpha = exp2f(m_run[rt] - m_new);
        l_run[rt] *= alpha;
        m_run[rt] = m_new;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt][rt] *= alpha;
      }
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const float nm = -m_run[rt];
      float ps = 0.f;
      bf16x8_t pf;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const __bf16 pb16 = __bf16(exp2f(fmaf(st[t][rt][e], c, nm)));
          pf[t * 4 + e] = pb16;
          ps += float(pb16);   // the normaliser sums the same rounded weights the MFMA uses
        }
      l_run[rt] += ps;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        o[dt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.v[dt], pf, o[dt][rt], 0, 0, 0);
    }
  };

  // software pipeline: the next block pair's fragments load while the current one computes
  int pb = blk0 + 2 * wave;
  if (pb < blk1) {
    PairFrags<D> fa, fb;
    load_pair(fa, pb);
    while (true) {
      if (pb + 2 * kWaves < blk1) load_pair(fb, pb + 2 * kWaves);
      compute_pair(fa, pb);
      pb += 2 * kWaves;
      if (pb >= blk1) break;
      if (pb + 2 * kWaves < blk1) load_pair(fa, pb + 2 * kWaves);
      compute_pair(fb, pb);
      pb += 2 * kWaves;
      if (pb >= blk1) break;
    }
  }

  // ---- merge the four wavefronts (fixed order), then write
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float lt = l_run[rt];
    lt += __shfl_xor(lt, 16, kWave);
    lt += __shfl_xor(lt, 32, kWave);
    if (g4 == 0) {
      s_m[wave][rt * 16 + l16] = m_run[rt];
      s_l[wave][rt * 16 + l16] = lt;
    }
  }
  __syncthreads();
  float fac[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = rt * 16 + l16;
    float M = kNegBig;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][r]);
    fac[rt] = exp2f(s_m[wave][r] - M);
  }
  // O^T accumulator element e of lane: dim 16 dt + 4 g4 + e, row 16 rt + l16
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int idx = (rt * 16 + l16) * D + dt * 16 + g4 * 4 + e;
            const float v = o[dt][rt][e] * fac[rt];
            s_o[idx] = (w == 0) ? v : s_o[idx] + v;
          }
    }
    __syncthreads();
  }
  // final row statistics and output
  for (int idx = threadIdx.x; idx < R * D; idx += kThreads) {
    const int r = idx / D, dd = idx % D;
    float M = kNegBig;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][r]);
    float Lsum = 0.f;
    for (int w = 0; w < kWaves; ++w) Lsum += s_l[w][r] * exp2f(s_m[w][r] - M);
    const int j = r / G, gi = r % G;
    if (p.splits == 1) {
      const float v = Lsum > 0.f ? s_o[idx] / Lsum : 0.f;
      p.out[out_index(p, long(b) * kp1 + j, (h * G + gi) * D + dd, long(p.Hq) * D, 2)] = f32_to_bf16(v);
    } else {
      const long pr = (long(bh) * p.splits + split) * R + r;
      p.part_o[pr * D + dd] = s_o[idx];
      if (dd == 0) {
        p.part_ml[pr * 2 + 0] = M;
        p.part_ml[pr * 2 + 1] = Lsum;
      }
    }
  }
}

// log-sum-exp merge over splits: one workgroup per (b, h, row), threads over dims
template <int D>
__global__ __launch_bounds__(D) void attn_merge_kernel(AttnParams p, int out_f32) {
  const int G = p.Hq / p.Hkv;
  const int kp1 = p.k + 1;
  const int R = G * kp1;
  const int r = blockIdx.x % R;
  const int bh = blockIdx.x / R;
  const int b = bh / p.Hkv, h = bh % p.Hkv;
  const int nblk = (p.ctx[b] + kp1 + 15) / 16;
  const int ns = min(p.splits, (nblk + p.blocks_per_split - 1) / p.blocks_per_split);
  float M = kNegBig;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, p.part_ml[((long(bh) * p.splits + s) * R + r) * 2]);
  float L = 0.f, acc = 0.f;
  for (int s = 0; s < ns; ++s) {
    const long pr = (long(bh) * p.splits + s) * R + r;
    const float m = p.part_ml[pr * 2];
    const float f = exp2f(m - M);
    L += p.part_ml[pr * 2 + 1] * f;
    acc += p.part_o[pr * D + threadIdx.x] * f;
  }
  const int j = r / G, gi = r % G;
  const float v = L > 0.f ? acc / L : 0.f;
  const long t = long(b) * kp1 + j, c = (h * G + gi) * D + threadIdx.x;
  if (out_f32) reinterpret_cast<float*>(p.out)[out_index(p, t, c, long(p.Hq) * D, 4)] = v;
  else p.out[out_index(p, t, c, long(p.Hq) * D, 2)] = f32_to_bf16(v);
}

// ---------------------------------------------------------------- f32 VALU path
// One wavefront per (token, query head); 64 keys per step, one key per lane for the
// scores, one dim per lane for the output. Writes per-split partials like the MFMA path.
__global__ __launch_bounds__(kWave) void attn_f32_kernel(const float* __restrict__ q,
                                                         const float* __restrict__ kc,
                                                         const float* __restrict__ vc,
                                                         AttnParams p, int D) {
  const int t = blockIdx.x / p.Hq, hq = blockIdx.x % p.Hq;
  const int kp1 = p.k + 1;
  const int b = t / kp1, j = t % kp1;
  const int G = p.Hq / p.Hkv, h = hq / G;
  const int lim = p.ctx[b] + j;   // last visible key
  const float* qr = q + (long(t) * p.Hq + hq) * D;
  const int* btab = p.bt + long(b) * p.max_blocks;
  const long bs = long(p.Hkv) * 16 * D;
  const int lane = threadIdx.x;
  float m = -INFINITY, l = 0.f;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};   // dims lane, lane+64, ... (D <= 256)
  const float scale = 1.0f / sqrtf(float(D));
  for (int k0 = 0; k0 <= lim; k0 += kWave) {
    const int kp = k0 + lane;
    float s = -INFINITY;
    if (kp <= lim) {
      const float* kr = kc + btab[kp / 16] * bs + long(h) * 16 * D + (kp % 16) * D;
      float d = 0.f;
      for (int i = 0; i < D; ++i) d += qr[i] * kr[i];
      s = d * scale;
    }
    const float mx = wave_max(s);
    const float mn = fmaxf(m, mx);
    const float alpha = m == -INFINITY ? 0.f : expf(m - mn);
    const float pe = s == -INFINITY ? 0.f : expf(s - mn);
    l = l * alpha + wave_sum(pe);
    for (int c = 0; c < 4; ++c) acc[c] *= alpha;
    const int nk = min(kWave, lim + 1 - k0);
    for (int key = 0; key < nk; ++key) {
      const float pk = __shfl(pe, key, kWave);
      const int kk = k0 + key;
      const float* vr = vc + btab[kk / 16] * bs + long(h) * D * 16 + (kk % 16);
      for (int c = 0; c < 4; ++c) {
        const int dd = lane + kWave * c;
        if (dd < D) acc[c] += pk * vr[dd * 16];
      }
    }
    m = mn;
  }
  float* out = reinterpret_cast<float*>(p.out);
  for (int c = 0; c < 4; ++c) {
    const int dd = lane + kWave * c;
    if (dd < D) out[out_index(p, t, long(hq) * D + dd, long(p.Hq) * D, 4)] = acc[c] / l;
  }
}

// Splits of the key range: enough workgroups to fill the chip twice over (512), each split a
// multiple of 8 blocks (4 wavefronts x one 32-key pair) and at least 32 blocks long.
void split_plan(int B, int Hkv, int max_blocks, int& splits, int& bps) {
  const int pairs = B * Hkv;
  int s = (512 + pairs - 1) / pairs;
  const int cap = (max_blocks + 31) / 32;
  if (s > cap) s = cap;
  if (s < 1) s = 1;
  bps = (max_blocks + s - 1) / s;
  bps = (bps + 7) / 8 * 8;
  splits = (max_blocks + bps - 1) / bps;
}

template <int D, int RT>
void launch_mfma(const AttnParams& p, int B, hipStream_t s) {
  attn_mfma_kernel<D, RT><<<B * p.Hkv * p.splits, kThreads, 0, s>>>(p);
}

template <int D>
hipError_t launch_d(const AttnParams& p, int B, int R, hipStream_t s) {
  const int rt = (R + 15) / 16;
  switch (rt) {
    case 1: launch_mfma<D, 1>(p, B, s); break;
    case 2: launch_mfma<D, 2>(p, B, s); break;
    case 3: launch_mfma<D, 3>(p, B, s); break;
    case 4: launch_mfma<D, 4>(p, B, s); break;
    case 5: launch_mfma<D, 5>(p, B, s); break;
    case 6: launch_mfma<D, 6>(p, B, s); break;
    case 7: launch_mfma<D, 7>(p, B, s); break;
    case 8: launch_mfma<D, 8>(p, B, s); break;
    default: return hipErrorInvalidValue;
  }
  if (p.splits > 1) attn_merge_kernel<D><<<B * p.Hkv * R, D, 0, s>>>(p, 0);
  return hipGetLastError();
}

}  // namespace

size_t attention_ws_bytes(int B, int k, int Hq, int Hkv, int D, int max_blocks) {
  int S, bps;
  split_plan(B, Hkv, max_blocks, S, bps);
  if (S <= 1) return 0;
  const long rows = long(B) * (k + 1) * Hq;   // = B * Hkv * R
  Carver c(nullptr, 0);
  c.take<float>(rows * S * D);
  c.take<float>(rows * S * 2);
  return c.used + 256;
}

hipError_t launch_paged_attention(const void* q, const void* kc, const void* vc, const int32_t* bt,
                                  const int32_t* ctx, int B, int k, int Hq, int Hkv, int D,
                                  int max_blocks, molt_dtype dt, void* out, bool out_tiled,
                                  void* ws, hipStream_t s) {
  AttnParams p{};
  p.out_tiled = out_tiled;
  p.q = static_cast<const uint16_t*>(q);
  p.kc = static_cast<const uint16_t*>(kc);
  p.vc = static_cast<const uint16_t*>(vc);
  p.bt = bt;
  p.ctx = ctx;
  p.out = static_cast<uint16_t*>(out);
  p.k = k; p.Hq = Hq; p.Hkv = Hkv; p.max_blocks = max_blocks;
  p.scale_log2 = kLog2e / sqrtf(float(D));
  const int R = (Hq / Hkv) * (k + 1);
  if (dt == MOLT_F32) {
    attn_f32_kernel<<<B * (k + 1) * Hq, kWave, 0, s>>>(static_cast<const float*>(q),
                                                        static_cast<const float*>(kc),
                                                        static_cast<const float*>(vc), p, D);
    return hipGetLastError();
  }
  split_plan(B, Hkv, max_blocks, p.splits, p.blocks_per_split);
  if (p.splits > 1) {
    const long rows = long(B) * (k + 1) * Hq;
    Carver c(ws, 0);
    p.part_o = c.take<float>(rows * p.splits * D);
    p.part_ml = c.take<float>(rows * p.splits * 2);
  }
  if (D == 128) return launch_d<128>(p, B, R, s);
  if (D == 64) return launch_d<64>(p, B, R, s);
  return hipErrorInvalidValue;
}

}  // namespace molt
