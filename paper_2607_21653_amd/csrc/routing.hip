// Router top-K with softmax weights, and the stable token -> expert permutation
// built from wavefront ballots and LDS prefix sums (the expert choices are the route
// records of rollout routing replay, paper Sec. 4.1 and Sec. 4.4).
//
// topk_kernel: one wavefront per token. Each lane holds up to 4 router logits
// (E <= 256) as 64-bit keys: order-preserving f32 bits (with -0 folded into +0) in
// the high word, 0xFFFFFFFF - expert id in the low word, so the maximum key is the
// largest logit with ties resolved to the lower expert id. K rounds of a wavefront
// max-reduction (DPP: with LDS-crossbar shuffles the K rounds were one long chain of
// permute round trips) select the experts in descending order.
//
// permute_kernel: workgroups of 256 threads, each owning a contiguous range of the T*K
// pairs (in (token, slot) order; 64 pairs per workgroup up to 512 workgroups). Each counts
// every pair per expert and the pairs before its range (LDS integer atomics) and scans the
// counts over the experts (offsets, padded offsets, grouped-GEMM tile table); inside the
// range, lanes holding the same expert find each other with 8 ballots over the expert id
// bits, a popcount of the lower lanes gives the rank inside a 64-pair step and a running
// LDS count per (wavefront, expert) adds the earlier steps. Position = offset[e] + pairs of
// e before the range + before the wavefront's part + rank: the stable (expert, token,
// slot) order, bit-exact, with no global atomics. (One 1024-thread workgroup over all
// pairs took 11.5 us at 5120 pairs, this launch ~6.)
// The grouped GEMMs work on a padded copy of that order: every expert's rows start at a
// multiple of 32 (padded offset poff[e] = sum of the earlier counts rounded up to 32), so
// each 32-row block of a GEMM tile belongs to one expert; padded slots hold pair -1. The
// tile table lists (expert, first row, end row) in padded rows.
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr int kMaxE = 256;
constexpr int kPermThreads = 256;
constexpr int kPermWaves = kPermThreads / kWave;
constexpr int kRankSteps = 8;                               // 64-pair steps per wavefront
constexpr int kMaxRange = kPermWaves * kRankSteps * kWave;  // pairs per workgroup, at most
constexpr int kHistBatch = 8;                               // 16-byte id loads in flight
constexpr int kPermRange = 64;                              // pairs per workgroup, at least
constexpr int kPermGrid = 512;                              // workgroups, at most (while the
                                                            // range stays <= kMaxRange)

MOLT_DEV unsigned long long route_key(float v, int e) {
  const float c = v + 0.0f;                  // -0.0 -> +0.0
  const uint32_t u = __float_as_uint(c);
  const uint32_t ord = (u >> 31) ? ~u : (u | 0x80000000u);
  return (static_cast<unsigned long long>(ord) << 32) | (0xFFFFFFFFu - uint32_t(e));
}

// inverse of route_key's high word (-0.0 comes back as +0.0, equal for the softmax)
MOLT_DEV float key_value(unsigned long long key) {
  const uint32_t ord = uint32_t(key >> 32);
  return __uint_as_float((ord >> 31) ? (ord & 0x7fffffffu) : ~ord);
}

__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ logits, int nparts,
                                                   const float* __restrict__ bias,
                                                   const int32_t* __restrict__ replay, int T, int E,
                                                   int K, int32_t* __restrict__ ids,
                                                   float* __restrict__ w) {
  const int t = blockIdx.x * 4 + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (t >= T) return;
  // router logit: the split-K partial sums of the router GEMM added in split order
  const float* gt = logits + long(t) * E;
  const long stride = long(T) * E;
  auto gval = [&](int e) {
    float v = gt[e];
#pragma unroll 8
    for (int s = 1; s < nparts; ++s) v += gt[s * stride + e];
    return v;
  };
  float sel_v = -INFINITY;
  int sel_e = 0;
  if (replay) {
    if (lane < K) {
      int e = replay[long(t) * K + lane];
      if (e < 0 || e >= E) e = 0;              // out-of-range replay id: expert 0
      sel_e = e;
      sel_v = gval(e) + (bias ? bias[e] : 0.f);
    }
  } else {
    unsigned long long key[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane + kWave * i;
      key[i] = e < E ? route_key(gval(e) + (bias ? bias[e] : 0.f), e) : 0ull;
    }
    for (int j = 0; j < K; ++j) {
      unsigned long long mine = key[0];
      int which = 0;
#pragma unroll
      for (int i = 1; i < 4; ++i)
        if (key[i] > mine) { mine = key[i]; which = i; }
      const unsigned long long best = wave_max_dpp(mine);
      if (mine == best && best != 0ull) key[which] = 0ull;   // the unique owner drops it
      if (lane == j) {
        // the key holds the logit's order-preserving bits: decode instead of re-reading
        sel_e = int(0xFFFFFFFFu - uint32_t(best & 0xFFFFFFFFull));
        sel_v = key_value(best);
      }
    }
  }
  // softmax over the K selected logits
  const float m = wave_max_dpp(lane < K ? sel_v : -INFINITY);
  const float ex = lane < K ? expf(sel_v - m) : 0.f;
  const float sum = wave_sum_dpp(ex);
  if (lane < K) {
    ids[long(t) * K + lane] = sel_e;
    w[long(t) * K + lane] = ex / sum;
  }
}

struct PermuteParams {
  const int32_t* ids;      // [P] expert of pair p = t * K + slot
  int P, E, K, tile_m;
  int range;               // pairs per workgroup (<= kMaxRange)
  int32_t* counts;         // [E]
  int32_t* offsets;        // [E + 1]
  int32_t* perm;           // [P] position -> pair
  int32_t* pperm;          // [padded rows] padded row -> pair, -1 for padding
  int32_t* n_padded;
  int4* tiles;             // [max_tiles] (expert, first row, end row, 0) in padded rows
  int max_tiles;
  int32_t* n_tiles;
};

__global__ __launch_bounds__(kPermThreads) void permute_kernel(PermuteParams p) {
  static_assert(kPermThreads == kMaxE, "one thread per expert in the scans");
  __shared__ int tot[kMaxE];               // pairs per expert
  __shared__ int bef[kMaxE];               // pairs per expert before the range
  __shared__ int wc[kPermWaves][kMaxE];    // per (wavefront, expert): its pairs, then the
                                           // expert's pairs before the wavefront's part
  __shared__ int off[kMaxE + 1];
  __shared__ int poff[kMaxE + 1];
  __shared__ int wsum[3][kPermWaves];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int p0 = blockIdx.x * p.range, p1 = min(p0 + p.range, p.P);
  tot[tid] = 0;
  bef[tid] = 0;
  for (int e = lane; e < kMaxE; e += kWave) wc[wave][e] = 0;
  // rank of each pair of the range among the earlier pairs of its expert in its wavefront
  // (wc rows are per wavefront: no barrier needed). Wavefront w owns the contiguous pairs
  // [q0, q0 + per), 64 per step; lanes with the same expert find each other with 8 ballots
  // over the id bits and a popcount of the lower lanes gives the rank inside the step.
  const int per = (p1 - p0 + kPermWaves * kWave - 1) / (kPermWaves * kWave) * kWave;
  const int steps = per / kWave;
  const int q0 = p0 + wave * per;
  const unsigned long long lt = (1ull << lane) - 1ull;
  int ev[kRankSteps], rk[kRankSteps];
#pragma unroll
  for (int u = 0; u < kRankSteps; ++u) {
    const int q = q0 + u * kWave + lane;
    ev[u] = (u < steps && q < p1) ? p.ids[q] : -1;
    rk[u] = 0;
  }
#pragma unroll
  for (int u = 0; u < kRankSteps; ++u) {
    if (u >= steps) break;
    const int e = ev[u];
    const bool valid = e >= 0;
    unsigned long long mask = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (e >> bit) & 1;
      const unsigned long long b = __ballot(valid && on);
      mask &= on ? b : ~b;
    }
    const int below = __popcll(mask & lt);
    int before = 0;
    if (valid) before = wc[wave][e];
    if (valid && below == 0) wc[wave][e] = before + __popcll(mask);
    rk[u] = before + below;
  }
  __syncthreads();
  // every workgroup counts all pairs per expert and those before its range (LDS atomics on
  // integers: exact in any order)
  // (ids read 4 at a time; the allocation holds P ids, so the last group of 4 reads
  // element-wise)
  const int P4 = p.P / 4;
  for (int i0 = 0; i0 < P4; i0 += kPermThreads * kHistBatch) {
    int32x4_t hv[kHistBatch];
#pragma unroll
    for (int u = 0; u < kHistBatch; ++u) {
      const int i = i0 + kPermThreads * u + tid;
      hv[u] = i < P4 ? reinterpret_cast<const int32x4_t*>(p.ids)[i] : int32x4_t{-1, -1, -1, -1};
    }
#pragma unroll
    for (int u = 0; u < kHistBatch; ++u) {
      const int i = 4 * (i0 + kPermThreads * u + tid);
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) {
        if (hv[u][c4] >= 0) {
          atomicAdd(&tot[hv[u][c4]], 1);
          if (i + c4 < p0) atomicAdd(&bef[hv[u][c4]], 1);
        }
      }
    }
  }
  if (tid < p.P - 4 * P4) {
    const int i = 4 * P4 + tid;
    const int e = p.ids[i];
    atomicAdd(&tot[e], 1);
    if (i < p0) atomicAdd(&bef[e], 1);
  }
  __syncthreads();
  // thread e: its expert's pairs before each wavefront's part of the range (all rows read
  // before any write), and the inclusive scans over experts of the count, the count padded
  // to 32 rows and the tile count
  const int c = tid < p.E ? tot[tid] : 0;
  const int tn = (c + p.tile_m - 1) / p.tile_m;
  {
    int cw[kPermWaves];
#pragma unroll
    for (int w2 = 0; w2 < kPermWaves; ++w2) cw[w2] = wc[w2][tid];
    int run = bef[tid];
#pragma unroll
    for (int w2 = 0; w2 < kPermWaves; ++w2) {
      wc[w2][tid] = run;
      run += cw[w2];
    }
  }
  int v[3] = {c, (c + 31) / 32 * 32, tn};
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    v[q] = wave_scan_dpp(v[q]);
    if (lane == kWave - 1) wsum[q][wave] = v[q];
  }
  __syncthreads();
  int nt = 0;
  {
    int add[3] = {0, 0, 0};
#pragma unroll
    for (int w2 = 0; w2 < kPermWaves; ++w2) {
#pragma unroll
      for (int q = 0; q < 3; ++q) add[q] += w2 < wave ? wsum[q][w2] : 0;
      nt += wsum[2][w2];
    }
    off[tid + 1] = v[0] + add[0];
    poff[tid + 1] = v[1] + add[1];
    v[2] += add[2] - tn;                   // this expert's first tile
    if (tid == 0) { off[0] = 0; poff[0] = 0; }
  }
  nt = min(nt, p.max_tiles);
  __syncthreads();
  // workgroup 0: counts, offsets, tile table, padding slots
  if (blockIdx.x == 0) {
    if (tid < p.E) {
      p.counts[tid] = c;
      p.offsets[tid] = off[tid];
      for (int m0 = 0, i = v[2]; m0 < c && i < p.max_tiles; m0 += p.tile_m, ++i)
        p.tiles[i] = make_int4(tid, poff[tid] + m0, poff[tid] + min(m0 + p.tile_m, c), 0);
      for (int r = poff[tid] + c; r < poff[tid + 1]; ++r) p.pperm[r] = -1;
    }
    if (tid == 0) {
      p.offsets[p.E] = off[p.E];
      *p.n_padded = poff[p.E];
      *p.n_tiles = nt;
    }
    // the grouped GEMMs' per-XCD tile queues (gate_up, down) that follow n_tiles
    if (tid < 2 * kTileQueues) p.n_tiles[1 + tid] = 0;
    for (int i = nt + tid; i < p.max_tiles; i += kPermThreads) p.tiles[i] = make_int4(-1, 0, 0, 0);
  }
  // the range's pairs: position = offset + earlier pairs of the expert + rank
#pragma unroll
  for (int u = 0; u < kRankSteps; ++u) {
    if (u >= steps) break;
    const int e = ev[u];
    if (e < 0) continue;
    const int q = q0 + u * kWave + lane;
    const int r = wc[wave][e] + rk[u];
    p.perm[off[e] + r] = q;
    p.pperm[poff[e] + r] = q;
  }
}

}  // namespace

int max_expert_tiles(int T, int E, int K, int tile_m) {
  return (T * K + tile_m - 1) / tile_m + E;
}

long max_padded_rows(int T, int E, int K) {
  const long P = long(T) * K;
  const long worst = P + 31L * (E < P ? E : P);   // every non-empty expert pads < 32 rows
  return (worst + 31) / 32 * 32;
}

hipError_t launch_route(const float* logits, int nparts, const float* bias, const int32_t* replay,
                        int T, int E, int K, int32_t* ids, float* w, int32_t* counts,
                        int32_t* offsets, int32_t* perm, int32_t* pperm, int32_t* n_padded,
                        int tile_m, int32_t* tiles, int max_tiles, int32_t* n_tiles,
                        hipStream_t s) {
  topk_kernel<<<(T + 3) / 4, 256, 0, s>>>(logits, nparts, bias, replay, T, E, K, ids, w);
  PermuteParams p;
  p.ids = ids;
  p.P = T * K;
  p.E = E;
  p.K = K;
  p.tile_m = tile_m;
  p.range = max(kPermRange, (p.P + kPermGrid - 1) / kPermGrid);
  if (p.range > kMaxRange) p.range = kMaxRange;
  p.counts = counts;
  p.offsets = offsets;
  p.perm = perm;
  p.pperm = pperm;
  p.n_padded = n_padded;
  p.tiles = reinterpret_cast<int4*>(tiles);
  p.max_tiles = max_tiles;
  p.n_tiles = n_tiles;
  permute_kernel<<<(p.P + p.range - 1) / p.range, kPermThreads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace molt
