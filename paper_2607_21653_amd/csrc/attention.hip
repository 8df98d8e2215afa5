// Multi-query paged decode attention of the verify step (PagedAttention cache, paper
// Sec. 2; k speculative tokens per sequence, Sec. 4.1). For sequence b and kv head h the
// R = G*(1+k) query rows (G = Hq/Hkv query heads, 1+k positions) share every key/value
// block, so each K/V byte is read once per (b, h) and reused by all R rows on MFMA.
//
// Work split: workgroup = (b, h, query tile, split of the key range), 8 wavefronts (one
// 16-row tile each; those without rows only load). A query tile holds all R rows when
// R <= 128 (the verify step); longer windows (prefill) are cut into tiles of floor(128 / G)
// positions, each reading the keys its last position sees.
// The number of splits is chosen so the grid holds ~512 workgroups (at B*Hkv*tiles >= 512
// there is no split and no merge pass) and no split exceeds 2048 blocks. The wavefronts split the R query rows and
// share every 32-key block pair through a double-buffered LDS ring (details at the kernel).
// Per pair, on v_mfma_f32_16x16x32_bf16:
//   S^T[32 keys x 16 rows] = K Q^T   (A = K rows from LDS, B = Q^T held in registers)
//   O^T[D x 16 rows]      += V^T P^T (A = V^T: the V cache stores a block as [D][16 tokens],
//                                    so 8 consecutive keys of one dim are 16 contiguous
//                                    bytes; B = P^T is the S^T accumulator layout: no
//                                    cross-lane shuffles)
// P is split into two bf16 parts, hi = bf16(p) and lo = bf16(p - hi) (16 significant bits),
// and V^T P^T takes one MFMA per part, so the output is the f32 softmax product up to
// accumulation order. With P rounded to bf16 alone (one MFMA) the end-to-end logits of a
// 2-layer bf16 step moved by up to 1.7e-2 against the exact product (the final RMSNorm
// scales up the residual differences that bf16 flips of the attention output leave).
// Causality: row r = j*G + g (position j) sees keys <= ctx_b + j; only pairs reaching past
// ctx_b need masks. Softmax in f32 with exp2 of log2(e)-scaled scores; the output is
// rescaled lazily, only when a row maximum grows by more than 8 (in log2 units) over the
// reference it was accumulated with. Splits are merged by a log-sum-exp pass (a single
// split writes the output directly). Deterministic.
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" for running maxima
constexpr float kRescaleSlack = 8.0f; // probabilities may grow to 2^8 before O is rescaled
constexpr int kMaxSplitBlocks = 2048; // KV blocks of one split (its block table sits in LDS)


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
  int qtiles, tq;          // query tiles per (b, h) and positions per tile (tq * G <= 128)
  float scale_log2;        // log2(e) / sqrt(D)
  int out_tiled;           // output in the GEMM operand layout (input of the O projection)
};

// element index of output (token t, column c) of `cols` columns
MOLT_DEV long out_index(const AttnParams& p, long t, long c, long cols, int esize) {
  return p.out_tiled ? tiled_index(t, c, cols, esize) : t * cols + c;
}

// ---------------------------------------------------------------- MFMA kernel
// Workgroup = (b, h, query tile, split), NW wavefronts that split the query rows (wavefront
// w owns the 16-row tile w) and share every 32-key block pair through LDS: per pair the
// 64 NW threads copy its K and V blocks (4 x 16 D bytes) with coalesced 16-byte loads,
// kept kDepth pairs ahead in registers, into a double-buffered ring; one LDS-only barrier
// per pair. Each wavefront keeps only its own rows' Q fragments and O accumulator; with 3
// pairs in flight the 8-wavefront kernel takes 122 registers, so two workgroups (16
// wavefronts, 6 pairs in flight) share a CU; no cross-wavefront merge at the end. The
// kernel is bound by the latency of each wavefront's per-pair chain (counters: LDS active
// ~25%, MFMA busy ~17% of cycles), so wavefronts per CU set its pace: at 72 rows and
// context 2048 two row tiles per wavefront of 4 (334 registers, one wavefront per SIMD)
// reached 36% of HBM bandwidth, one 8-wavefront workgroup per CU (6 pairs in flight)
// 45%, two per CU 62%; at 40 rows two 4-wavefront workgroups per CU (6 pairs each) reached
// 56-59% at contexts 4096-65536, two 8-wavefront ones 60-61%.
// Key order inside a pair for the MFMA k-index: lane group g (of 4) holds keys
// 8 (g % 2) .. +7 of block g / 2. S^T MFMA t (t = 0, 1) computes rows m = 4 g + i for keys
// 8 (g % 2) + 4 t + i of block g / 2, so the 8 scores of a lane are those 8 contiguous keys
// and the V^T operand is one 16-byte read of the [D][16] V block.
// LDS swizzles keep every ds_read_b128 conflict-free: K row k (key) of block j stores its
// 16-byte chunk c at chunk c ^ f(k, j); V row d (dim) stores chunk c at c ^ v(d).
template <int D>
MOLT_DEV int kswz(int key, int blk) {
  const int f = (key & 3) | ((key >> 1) & 4);
  return D == 128 ? (f | (blk << 3)) : f;
}
MOLT_DEV int vswz(int dim) { return ((dim >> 2) ^ (dim >> 3)) & 1; }

template <int D, int NW, int KS>
__global__ __launch_bounds__(64 * NW, NW == 8 ? 2 : 1) void attn_lds_kernel(AttnParams p) {
  constexpr int kThreads = 64 * NW;
  constexpr int RTW = 1;                // 16-row tiles per wavefront
  constexpr int NRT = NW / KS;          // row tiles per key group
  constexpr int DS = D / 32;            // 32-dim k-steps for S
  constexpr int DT = D / 16;            // 16-dim tiles of O^T
  constexpr int KB = 16 * D * 2;        // bytes of one K (or V) block
  constexpr int PAIR = 4 * KB;          // K0, K1, V0, V1
  constexpr int CPT = PAIR / 16 / kThreads;   // 16-byte chunks per thread per pair
  static_assert(CPT >= 1 && CPT * 16 * kThreads == PAIR, "chunks per thread");
  // steps (KS pairs each) loaded ahead into registers: 8-wavefront workgroups hold 3 pairs
  // with one key group, which keeps them at 122 registers, so two fit per CU; with two key
  // groups one step (2 pairs) ahead
  constexpr int kDepth = KS == 2 ? 1 : NW == 8 ? 3 : 6;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * KS][PAIR];

  // Workgroup i runs on XCD i % 8. With the work item equal to i and 8 splits, XCD x would
  // take split x of every (b, h): the XCDs of the late splits, empty where a context is
  // shorter than the longest, idled while the others set the kernel's time. With 4 or more
  // splits the work item's low 3 bits are XORed with the group number j = i / 8 (a full
  // group of 8 stays a permutation of itself), so every XCD takes every split index
  // (long-context layer 318 -> 284 us; a hash that also mixed j's higher bits in: 306 us;
  // with 1-2 splits, whose ranges are nearly equal, the mix measured 1-3% slower). Several
  // query tiles of one (b, h) (prefill windows) keep the plain order: there an XCD takes
  // one split's keys for many tiles, which then hit its L2.
  int wi = blockIdx.x;
  if (p.splits >= 4 && p.qtiles == 1 && (wi | 7) < int(gridDim.x)) wi = (wi & ~7) | ((wi ^ (wi >> 3)) & 7);
  const int split = wi % p.splits;
  const int qt = (wi / p.splits) % p.qtiles;
  const int bh = wi / p.splits / p.qtiles;
  const int b = bh / p.Hkv, h = bh % p.Hkv;
  const int G = p.Hq / p.Hkv;
  const int kp1 = p.k + 1;
  const int R = G * kp1;                   // rows of (b, h); this tile holds rows r0 .. r0 + Rt
  const int j0 = qt * p.tq;                // the tile's first position
  const int Rt = G * min(p.tq, kp1 - j0);
  const int r0 = G * j0;
  const int ctx = p.ctx[b];
  const int nkeys = ctx + j0 + Rt / G;     // keys the tile's last position sees
  const int nblk = (nkeys + 15) / 16;
  const int blk0 = split * p.blocks_per_split;
  const int blk1 = min(blk0 + p.blocks_per_split, nblk);
  const int npairs = (blk1 - blk0 + 1) / 2;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int l16 = lane % 16, g4 = lane / 16;
  const float c = p.scale_log2;
  // key group kg takes pairs kg, kg + KS, ...; its wavefront rt holds 16-row tile rt
  const int kg = wave / NRT, rtile = wave % NRT;

  // Q^T fragments of the wavefront's rows r = 16 (rtile + NRT i) + l16, dims [32 s + 8 g4, +8)
  bf16x8_t qf[RTW][DS];
  int lim[RTW];
#pragma unroll
  for (int i = 0; i < RTW; ++i) {
    const int r = 16 * (rtile + NRT * i) + l16;  // row of the tile
    const int j = j0 + r / G, gi = r % G;
    lim[i] = r < Rt ? ctx + j : -1;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      if (r < Rt) {
        qf[i][s] = *reinterpret_cast<const bf16x8_t*>(
            p.q + ((long(b) * kp1 + j) * p.Hq + h * G + gi) * D + s * 32 + g4 * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[i][s][e] = __bf16(0.f);
      }
    }
  }
  floatx4_t o[DT][RTW];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < RTW; ++i) o[dt][i] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[RTW], l_run[RTW];
#pragma unroll
  for (int i = 0; i < RTW; ++i) { m_run[i] = kNegBig; l_run[i] = 0.f; }
  const bool active = 16 * rtile < Rt;  // wavefronts without rows only help with the loads
  const int lim_lo = ctx + j0;          // keys up to here are visible to every row of the tile

  __shared__ int s_bt[kMaxSplitBlocks];
  const int* btab = p.bt + long(b) * p.max_blocks;
  for (int i = threadIdx.x; i < blk1 - blk0; i += kThreads) s_bt[i] = btab[blk0 + i];
  __syncthreads();
  const long kv_blk_stride = long(p.Hkv) * 16 * D;    // elements per physical block
  // staging: the pair's 4 KB / 16 chunks per block (K0, K1, V0, V1 in that order) are
  // numbered c = 0 .. PAIR / 16 - 1; thread t copies chunks t + kThreads u, u < CPT, each from
  // its block (q = c / (KB / 16)) to its swizzled LDS place
  int src_off[CPT], dst_off[CPT];
  bool from_v[CPT], second[CPT];
#pragma unroll
  for (int u = 0; u < CPT; ++u) {
    const int c = threadIdx.x + kThreads * u;
    const int q = c / (KB / 16), ch = c % (KB / 16);
    from_v[u] = q >= 2;
    second[u] = q & 1;
    if (!from_v[u]) {
      const int key = ch / (D / 8), kc = ch % (D / 8);
      src_off[u] = (h * 16 + key) * D + kc * 8;
      dst_off[u] = q * KB + key * (2 * D) + ((kc ^ kswz<D>(key, q & 1)) * 16);
    } else {
      const int dim = ch / 2, vc = ch % 2;
      src_off[u] = (h * D + dim) * 16 + vc * 8;
      dst_off[u] = q * KB + dim * 32 + ((vc ^ vswz(dim)) * 16);
    }
  }
  int32x4_t st[kDepth][KS][CPT];
  // The split's block-table entries are read from LDS: a global load of them, issued behind
  // the K/V prefetches, would have its wait drain every load in flight (the vector memory
  // counter retires in order).
  auto gload_pair = [&](int32x4_t (&dst)[CPT], int pi) __attribute__((always_inline)) {
    const int rel = 2 * min(pi, npairs - 1);
    const long phys0 = s_bt[rel];
    const long phys1r = s_bt[min(rel + 1, blk1 - blk0 - 1)];
    const long phys1 = blk0 + rel + 1 < blk1 ? phys1r : phys0;
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const uint16_t* base = from_v[u] ? p.vc : p.kc;
      dst[u] = __builtin_nontemporal_load(reinterpret_cast<const int32x4_t*>(
          base + (second[u] ? phys1 : phys0) * kv_blk_stride + src_off[u]));
    }
  };
  // step si covers pairs KS si .. KS si + KS - 1; LDS half hf holds a step's pairs in
  // buffers KS hf .. KS hf + KS - 1
  auto gload = [&](int32x4_t (&dst)[KS][CPT], int si) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < KS; ++g) gload_pair(dst[g], KS * si + g);
  };
  auto sstore = [&](const int32x4_t (&src)[KS][CPT], int hf) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < KS; ++g)
#pragma unroll
      for (int u = 0; u < CPT; ++u) *reinterpret_cast<int32x4_t*>(lds[KS * hf + g] + dst_off[u]) = src[g][u];
  };

  // K fragment: block j = l16 / 8, key 8 ((l16 / 4) % 2) + 4 t + l16 % 4 (the swizzle is the
  // same for t = 0 and 1, so t only adds 4 rows), chunk 4 s + g4 (dims 32 s + 8 g4).
  // V fragment: block g4 / 2, dim 16 dt + l16 (the swizzle does not change with dt), chunk g4 % 2
  int koff[DS];
  {
    const int j = l16 / 8, key = 8 * ((l16 / 4) % 2) + l16 % 4;
#pragma unroll
    for (int s = 0; s < DS; ++s) koff[s] = j * KB + key * (2 * D) + (((4 * s + g4) ^ kswz<D>(key, j)) * 16);
  }
  const int voff = (2 + g4 / 2) * KB + l16 * 32 + (((g4 % 2) ^ vswz(l16)) * 16);

  auto compute = [&](int buf, int pi) __attribute__((always_inline)) {
    if (!active) return;
    const int pb = blk0 + 2 * pi;
    const uint8_t* base = lds[buf];
    floatx4_t sv[2][RTW];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8_t kf[DS];
#pragma unroll
      for (int s = 0; s < DS; ++s) kf[s] = *reinterpret_cast<const bf16x8_t*>(base + koff[s] + t * 4 * (2 * D));
#pragma unroll
      for (int i = 0; i < RTW; ++i) {
        floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < DS; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], qf[i][s], acc, 0, 0, 0);
        sv[t][i] = acc;
      }
    }
    // lane's 8 keys: block pb + g4 / 2, keys 8 (g4 % 2) + 4 t + e
    if (!(pb * 16 + 31 <= lim_lo)) {
      const bool blk_ok = (g4 / 2 == 0) || (pb + 1 < blk1);
#pragma unroll
      for (int i = 0; i < RTW; ++i)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int kpos = (pb + g4 / 2) * 16 + 8 * (g4 % 2) + 4 * t + e;
            if (!(blk_ok && kpos <= lim[i])) sv[t][i][e] = -INFINITY;
          }
    }
    float mx[RTW];
    bool grow = false;
#pragma unroll
    for (int i = 0; i < RTW; ++i) {
      float v = fmaxf(fmaxf(fmaxf(sv[0][i][0], sv[0][i][1]), fmaxf(sv[0][i][2], sv[0][i][3])),
                      fmaxf(fmaxf(sv[1][i][0], sv[1][i][1]), fmaxf(sv[1][i][2], sv[1][i][3])));
      v = rows_max4(v);
      mx[i] = v * c;
      grow |= mx[i] > m_run[i] + kRescaleSlack;
    }
    if (__builtin_amdgcn_read_exec() & __ballot(grow)) {
#pragma unroll
      for (int i = 0; i < RTW; ++i) {
        const float m_new = fmaxf(m_run[i], mx[i]);
        const float alpha = exp2f(m_run[i] - m_new);
        l_run[i] *= alpha;
        m_run[i] = m_new;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt][i] *= alpha;
      }
    }
    bf16x8_t pf[RTW], pl[RTW];   // P = hi + lo
#pragma unroll
    for (int i = 0; i < RTW; ++i) {
      const float nm = -m_run[i];
      float ps = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float w = exp2f(fmaf(sv[t][i][e], c, nm));
          const __bf16 hi = __bf16(w);
          pf[i][t * 4 + e] = hi;
          pl[i][t * 4 + e] = __bf16(w - float(hi));   // w - hi is exact in f32
          ps += w;
        }
      l_run[i] += ps;
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const bf16x8_t vf = *reinterpret_cast<const bf16x8_t*>(base + voff + dt * 16 * 32);
#pragma unroll
      for (int i = 0; i < RTW; ++i) {
        o[dt][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[i], o[dt][i], 0, 0, 0);
        o[dt][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl[i], o[dt][i], 0, 0, 0);
      }
    }
  };

  // pipeline: step si sits in LDS half si % 2; register slot (si + 1) % kDepth holds step
  // si + 1 (slots hold si + 1 .. si + kDepth). Step si first stores step si + 1 into the
  // other half (last read before the previous barrier) and refills its slot with step
  // si + 1 + kDepth, so the new loads are in flight during the compute; then each key group
  // computes its pair of step si. Loads past the last pair re-read it.
  const int nsteps = (npairs + KS - 1) / KS;
  auto step = [&](int hf, int si) __attribute__((always_inline)) {
    if (KS * si + kg < npairs) compute(KS * hf + kg, KS * si + kg);
  };
  if (nsteps > 0) {
    gload(st[0], 0);
    sstore(st[0], 0);
#pragma unroll
    for (int u = 1; u <= kDepth; ++u) gload(st[u % kDepth], u);
    lds_barrier();
    // step s sits in LDS half s % 2 (kDepth may be odd, so the parity comes from si)
    int si = 0;
    for (; si + kDepth - 1 < nsteps; si += kDepth) {
      const int par = si & 1;
#pragma unroll
      for (int u = 0; u < kDepth; ++u) {
        sstore(st[(u + 1) % kDepth], 1 - (par ^ (u & 1)));
        gload(st[(u + 1) % kDepth], si + u + 1 + kDepth);
        step(par ^ (u & 1), si + u);
        lds_barrier();
      }
    }
    const int par = si & 1;
#pragma unroll
    for (int u = 0; u < kDepth - 1; ++u) {
      if (si + u < nsteps) {
        sstore(st[(u + 1) % kDepth], 1 - (par ^ (u & 1)));
        step(par ^ (u & 1), si + u);
        lds_barrier();
      }
    }
  }
  if constexpr (KS == 2) {
    // merge the key groups: group 1 leaves its running max, partial sums and O^T in LDS
    // (free after the last barrier), group 0 combines them with its own
    constexpr int kMergeF = DT * 4 + 2;    // floats per lane
    static_assert(NRT * kMergeF * 64 * 4 <= 2 * KS * PAIR, "merge state fits the ring");
    float* mg = reinterpret_cast<float*>(&lds[0][0]) + rtile * kMergeF * 64 + lane;
    if (kg == 1 && active) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int e = 0; e < 4; ++e) mg[(dt * 4 + e) * 64] = o[dt][0][e];
      mg[DT * 4 * 64] = m_run[0];
      mg[(DT * 4 + 1) * 64] = l_run[0];
    }
    lds_barrier();
    if (kg == 1) return;
    if (active) {
      const float m1 = mg[DT * 4 * 64], l1 = mg[(DT * 4 + 1) * 64];
      const float mm = fmaxf(m_run[0], m1);
      const float a0 = exp2f(m_run[0] - mm), a1 = exp2f(m1 - mm);
      m_run[0] = mm;
      l_run[0] = l_run[0] * a0 + l1 * a1;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int e = 0; e < 4; ++e) o[dt][0][e] = o[dt][0][e] * a0 + mg[(dt * 4 + e) * 64] * a1;
    }
  }
  if (!active) return;

  // row totals across the 4 lane groups, then the output (or this split's partials)
#pragma unroll
  for (int i = 0; i < RTW; ++i) {
    float lt = l_run[i];
    lt = rows_sum4(lt);
    const int r = 16 * (rtile + NRT * i) + l16;
    if (r >= Rt) continue;
    const int j = j0 + r / G, gi = r % G;
    // O^T element e of tile dt: dim 16 dt + 4 g4 + e
    if (p.splits == 1) {
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        // the 4 consecutive columns of the lane's rows: one 8-byte store in either layout
        uint16_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = f32_to_bf16(o[dt][i][e] * inv);
        *reinterpret_cast<uint2*>(p.out + out_index(p, long(b) * kp1 + j, (h * G + gi) * D + 16 * dt + 4 * g4,
                                                     long(p.Hq) * D, 2)) =
            make_uint2(uint32_t(v[0]) | (uint32_t(v[1]) << 16), uint32_t(v[2]) | (uint32_t(v[3]) << 16));
      }
    } else {
      const long pr = (long(bh) * p.splits + split) * R + r0 + r;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) *reinterpret_cast<floatx4_t*>(p.part_o + pr * D + 16 * dt + 4 * g4) = o[dt][i];
      if (g4 == 0) {
        p.part_ml[pr * 2 + 0] = m_run[i];
        p.part_ml[pr * 2 + 1] = lt;
      }
    }
  }
}

// log-sum-exp merge over splits: one workgroup per (b, h, group of 1024 / D rows), each
// thread finishing 4 consecutive dims of one row (16-byte partial loads, one 8-byte store;
// one workgroup per row with a thread per dim had taken 12 us for the single layer's 10 MB
// of partials)
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  constexpr int TPR = D / 4;                 // threads per row
  constexpr int RPW = 256 / TPR;             // rows per workgroup
  const int G = p.Hq / p.Hkv;
  const int kp1 = p.k + 1;
  const int R = G * kp1;
  const int groups = (R + RPW - 1) / RPW;
  const int bh = blockIdx.x / groups;
  const int r = (blockIdx.x % groups) * RPW + int(threadIdx.x) / TPR;
  if (r >= R) return;
  const int d4 = (int(threadIdx.x) % TPR) * 4;
  const int b = bh / p.Hkv, h = bh % p.Hkv;
  const int j_end = min(kp1, (r / G / p.tq + 1) * p.tq);      // end of the row's query tile
  const int nblk = (p.ctx[b] + j_end + 15) / 16;
  const int ns = min(p.splits, (nblk + p.blocks_per_split - 1) / p.blocks_per_split);
  const long pr0 = long(bh) * p.splits * R + r;              // split s: pr0 + s R
  float M = kNegBig;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, p.part_ml[(pr0 + long(s) * R) * 2]);
  float L = 0.f;
  floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < ns; ++s) {
    const long pr = pr0 + long(s) * R;
    const float f = exp2f(p.part_ml[pr * 2] - M);
    L += p.part_ml[pr * 2 + 1] * f;
    const floatx4_t o = *reinterpret_cast<const floatx4_t*>(p.part_o + pr * D + d4);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] += o[e] * f;
  }
  const int j = r / G, gi = r % G;
  uint16_t v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = f32_to_bf16(L > 0.f ? acc[e] / L : 0.f);
  const long t = long(b) * kp1 + j, c = (h * G + gi) * D + d4;   // 4 consecutive columns
  *reinterpret_cast<uint2*>(p.out + out_index(p, t, c, long(p.Hq) * D, 2)) =
      make_uint2(uint32_t(v[0]) | (uint32_t(v[1]) << 16), uint32_t(v[2]) | (uint32_t(v[3]) << 16));
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
// multiple of 8 blocks and at least 32 blocks long.
void split_plan(long units, int max_blocks, int& splits, int& bps) {
  const long pairs = units;
  int s = int((512 + pairs - 1) / pairs);
  const int cap = (max_blocks + 31) / 32;
  if (s > cap) s = cap;
  if (s < 1) s = 1;
  if (s < (max_blocks + kMaxSplitBlocks - 1) / kMaxSplitBlocks)
    s = (max_blocks + kMaxSplitBlocks - 1) / kMaxSplitBlocks;
  bps = (max_blocks + s - 1) / s;
  bps = (bps + 7) / 8 * 8;
  splits = (max_blocks + bps - 1) / bps;
}

template <int D>
hipError_t launch_d(const AttnParams& p, int B, int R, hipStream_t s) {
  const int Rt = (p.Hq / p.Hkv) * p.tq;     // rows of a query tile
  const long grid = long(B) * p.Hkv * p.qtiles * p.splits;
  // two key groups when a query tile's row tiles fit half the wavefronts
  if ((Rt + 15) / 16 <= 4) attn_lds_kernel<D, 8, 2><<<grid, 512, 0, s>>>(p);
  else attn_lds_kernel<D, 8, 1><<<grid, 512, 0, s>>>(p);
  if (p.splits > 1) attn_merge_kernel<D><<<B * p.Hkv * ((R + 1024 / D - 1) / (1024 / D)), 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

// Query tiles of (b, h): all G(1+k) rows in one tile when they fit in 128 (every key and
// value read once), else tiles of floor(128 / G) positions (at least one), each read by an
// 8-wavefront workgroup.
static void qtile_plan(int G, int kp1, int& qtiles, int& tq) {
  tq = G * kp1 <= 128 ? kp1 : (G <= 128 ? 128 / G : 1);
  qtiles = (kp1 + tq - 1) / tq;
}

size_t attention_ws_bytes(int B, int k, int Hq, int Hkv, int D, int max_blocks) {
  int S, bps, qtiles, tq;
  qtile_plan(Hq / Hkv, k + 1, qtiles, tq);
  split_plan(long(B) * Hkv * qtiles, max_blocks, S, bps);
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
  qtile_plan(Hq / Hkv, k + 1, p.qtiles, p.tq);
  split_plan(long(B) * Hkv * p.qtiles, max_blocks, p.splits, p.blocks_per_split);
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
