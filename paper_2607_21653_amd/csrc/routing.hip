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
// permute_kernel: one 1024-thread workgroup, one pass over the ids. Wavefront w owns a
// contiguous range of the T*K pairs (in (token, slot) order) and visits it 64 pairs at a
// time: lanes holding the same expert find each other with 8 ballots over the expert id
// bits, a popcount of the lower lanes gives the rank inside the step, and a running LDS
// count per (wavefront, expert) adds the earlier steps. An exclusive prefix of those counts
// over the wavefronts, and wavefront prefix sums over the experts (offsets, padded offsets,
// grouped-GEMM tile table), then give position = offset[e] + earlier wavefronts + rank:
// the stable (expert, token, slot) order, bit-exact, with no atomics.
// The grouped GEMMs work on a padded copy of that order: every expert's rows start at a
// multiple of 32 (padded offset poff[e] = sum of the earlier counts rounded up to 32), so
// each 32-row block of a GEMM tile belongs to one expert; padded slots hold pair -1. The
// tile table lists (expert, first row, end row) in padded rows.
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr int kMaxE = 256;
constexpr int kPermThreads = 1024;
constexpr int kPermWaves = kPermThreads / kWave;

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

__global__ __launch_bounds__(kPermThreads) void permute_kernel(
    const int32_t* __restrict__ ids, int P, int E, int tile_m, int32_t* __restrict__ counts_out,
    int32_t* __restrict__ offsets_out, int32_t* __restrict__ perm, int32_t* __restrict__ inv,
    int32_t* __restrict__ pperm, int32_t* __restrict__ n_padded, int4* __restrict__ tiles,
    int max_tiles, int32_t* __restrict__ n_tiles) {
  __shared__ int wc[kPermWaves][kMaxE];    // pass 1: count per (wavefront, expert); then its
                                           // exclusive prefix over the wavefronts
  __shared__ int cnt[kMaxE];
  __shared__ int off[kMaxE + 1];
  __shared__ int poff[kMaxE + 1];
  __shared__ int wsum[3][kMaxE / kWave];
  __shared__ int wtmp[3][kMaxE];
  __shared__ int s_nt;
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  // Wavefront w owns the contiguous pair range [w * per, (w + 1) * per), visited 64 at a
  // time, so pair order = (wavefront, step, lane) order.
  const int steps = (P + kPermThreads - 1) / kPermThreads;
  const int per = steps * kWave;
  const int p0 = wave * per;
  for (int e = lane; e < kMaxE; e += kWave) wc[wave][e] = 0;   // own row only: no barrier
  const unsigned long long lt = (1ull << lane) - 1ull;
  // pass 1: the rank of each pair among the earlier pairs of its expert in this wavefront
  // (earlier steps: the running count in wc; this step: popcount of the lower lanes with the
  // same expert, found with 8 ballots over the id bits). The rank is parked in inv[p] (each
  // thread reads back only what it wrote).
  constexpr int kBatch = 8;                // loads of a batch issue together
  // with one batch (P <= 8 * kPermThreads) pass 2 reuses the ids and ranks held here
  // instead of reading them back from global memory
  const bool one_batch = steps <= kBatch;
  int ev1[kBatch], rk1[kBatch];
#pragma unroll
  for (int u = 0; u < kBatch; ++u) { ev1[u] = -1; rk1[u] = 0; }
  for (int s0 = 0; s0 < steps; s0 += kBatch) {
    int ev[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int p = p0 + (s0 + u) * kWave + lane;
      ev[u] = (s0 + u < steps && p < P) ? ids[p] : -1;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (s0 + u >= steps) break;
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
      if (s0 == 0) {
        ev1[u] = e;
        rk1[u] = before + below;
      }
      if (valid && !one_batch) inv[p0 + (s0 + u) * kWave + lane] = before + below;
    }
  }
  __syncthreads();
  // per expert: exclusive prefix of the wavefront counts (all 16 read before any write),
  // and the total
  if (tid < kMaxE) {
    int c[kPermWaves];
#pragma unroll
    for (int w2 = 0; w2 < kPermWaves; ++w2) c[w2] = wc[w2][tid];
    int run = 0;
#pragma unroll
    for (int w2 = 0; w2 < kPermWaves; ++w2) {
      wc[w2][tid] = run;
      run += c[w2];
    }
    cnt[tid] = tid < E ? run : 0;
  }
  __syncthreads();
  // exclusive prefix sums over experts (threads 0..255, one expert each) of the count, the
  // padded count and the tile count: offsets, padded offsets, first tile of each expert
  int tile0 = 0;
  if (tid < kMaxE) {
    const int c = cnt[tid];
    int v[3] = {c, (c + 31) / 32 * 32, (c + tile_m - 1) / tile_m};
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      v[q] = wave_scan_dpp(v[q]);
      if (lane == kWave - 1) wsum[q][wave] = v[q];
    }
    wtmp[0][tid] = v[0];
    wtmp[1][tid] = v[1];
    wtmp[2][tid] = v[2];
  }
  __syncthreads();
  if (tid < kMaxE) {
    int add[3] = {0, 0, 0};
    for (int w2 = 0; w2 < wave; ++w2)
#pragma unroll
      for (int q = 0; q < 3; ++q) add[q] += wsum[q][w2];
    const int c = cnt[tid];
    const int tn = (c + tile_m - 1) / tile_m;
    off[tid + 1] = wtmp[0][tid] + add[0];
    poff[tid + 1] = wtmp[1][tid] + add[1];
    tile0 = wtmp[2][tid] + add[2] - tn;
    if (tid == 0) { off[0] = 0; poff[0] = 0; }
    if (tid == E - 1) {
      s_nt = min(tile0 + tn, max_tiles);
      *n_tiles = s_nt;
      *n_padded = poff[E];
    }
  }
  __syncthreads();
  if (tid < E) {                                       // this expert's tiles
    const int c = cnt[tid];
    for (int m0 = 0, i = tile0; m0 < c && i < max_tiles; m0 += tile_m, ++i)
      tiles[i] = make_int4(tid, poff[tid] + m0, poff[tid] + min(m0 + tile_m, c), 0);
  }
  for (int i = tid; i < E * 32; i += kPermThreads) {   // padding slots of each expert
    const int e = i / 32, r = cnt[e] + i % 32;
    if (r < poff[e + 1] - poff[e]) pperm[poff[e] + r] = -1;
  }
  for (int i = s_nt + tid; i < max_tiles; i += kPermThreads) tiles[i] = make_int4(-1, 0, 0, 0);
  for (int e = tid; e < E; e += kPermThreads) {
    counts_out[e] = cnt[e];
    offsets_out[e] = off[e];
  }
  if (tid == 0) offsets_out[E] = off[E];
  // pass 2: position = offset of the expert + earlier wavefronts' pairs of it + rank
  if (one_batch) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int e = ev1[u];
      if (e < 0) continue;
      const int p = p0 + u * kWave + lane;
      const int pos = off[e] + wc[wave][e] + rk1[u];
      perm[pos] = p;
      inv[p] = pos;
      pperm[pos - off[e] + poff[e]] = p;
    }
    return;
  }
  for (int s0 = 0; s0 < steps; s0 += kBatch) {
    int ev[kBatch], rk[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int p = p0 + (s0 + u) * kWave + lane;
      const bool ok = s0 + u < steps && p < P;
      ev[u] = ok ? ids[p] : -1;
      rk[u] = ok ? inv[p] : 0;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int e = ev[u];
      if (e < 0) continue;
      const int p = p0 + (s0 + u) * kWave + lane;
      const int pos = off[e] + wc[wave][e] + rk[u];
      perm[pos] = p;
      inv[p] = pos;
      pperm[pos - off[e] + poff[e]] = p;
    }
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
                        int32_t* offsets, int32_t* perm, int32_t* inv, int32_t* pperm,
                        int32_t* n_padded, int tile_m, int32_t* tiles, int max_tiles,
                        int32_t* n_tiles, hipStream_t s) {
  topk_kernel<<<(T + 3) / 4, 256, 0, s>>>(logits, nparts, bias, replay, T, E, K, ids, w);
  permute_kernel<<<1, kPermThreads, 0, s>>>(ids, T * K, E, tile_m, counts, offsets, perm, inv,
                                            pperm, n_padded, reinterpret_cast<int4*>(tiles),
                                            max_tiles, n_tiles);
  return hipGetLastError();
}

}  // namespace molt
