// GEMMs of the verify step on gfx950 MFMA: dense projections (QKV, O, router, LM head)
// and the grouped expert GEMMs of the top-K routed MoE (gate_up with a fused SwiGLU
// epilogue, down), in bf16 (v_mfma_f32_32x32x16_bf16) or fp8 e4m3 with f32 per-row x
// per-channel scales (v_mfma_f32_32x32x64_f8f6f4), f32 accumulation.
//
// Every operand is in the tiled layout of device_common.h (weights packed once at load;
// activations written tiled by their producers, rows padded to a multiple of 32). One
// kernel template streams the weights per wavefront (see below). Grouped launches run over
// a device-side tile table (expert, first row, end row) in padded expert order built by
// the permutation kernel, so the host never reads expert counts.
//
// The f32 model (tiny test model) takes a plain VALU path over the same layouts.
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr int kThreads = 256;
constexpr int kBN = 128;         // output columns per tile (gate_up: 64 gate + 64 up)
constexpr int kRowBytes = 128;   // K-slice, bytes

enum Mode { kDense = 0, kGateUp = 1, kDown = 2 };

// s_waitcnt immediate: vmcnt(0), expcnt(7) and lgkmcnt(15) (no wait on those two)
constexpr int kWaitVmcnt0 = (7 << 4) | (15 << 8);

struct GemmParams {
  const void* A;           // tiled. dense: [M, K]; gate_up: gathered rows [R, K]; down: h [R, K]
  const void* B;           // tiled. dense: [N, K]; gate_up: [E, 2F, K]; down: [E, N, K]
  void* C;                 // dense: f32 [M, ldc]; gate_up: h tiled [R, F]; down: f32 [P, ldc]
  int M, N, K;             // N: output columns (gate_up: F)
  int ldc;
  const int4* tiles;       // grouped: {expert, row0, row1, -}
  const int32_t* n_tiles_live;   // grouped (device): entries of `tiles` in use; null: n_mtiles
  int n_mtiles, n_ntiles;
  const int32_t* perm;     // grouped: padded row -> pair (token * ktop + slot), -1 = padding;
                           // null (dense down mode): row r -> output row r
  int ktop;
  const float* a_scale;    // fp8: per A row (token for gate_up, padded row for down)
  const float* b_scale;    // fp8: [E, b_scale_ld]
  int b_scale_ld;
  int accumulate;          // dense: C += result
  int* queue;              // grouped fp8: per-XCD tile queues (zero at launch)
};

MOLT_DEV floatx16_t mfma(const bf16x8_t& a, const bf16x8_t& b, const floatx16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
MOLT_DEV floatx16_t mfma(const int32x8_t& a, const int32x8_t& b, const floatx16_t& c) {
  // cbsz = blgp = 0: both operands fp8 e4m3; zero scale operands select the unscaled op
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// ---------------------------------------------------------------- grouped expert GEMM
// Expert GEMMs are HBM-bound at the verify step's row counts (tens of rows per expert):
// the weights must stream at full bandwidth and be read once. Workgroup = BM rows of one
// expert x 128 output columns; each of the 4 wavefronts owns 32 output columns (32 weight
// rows) and loads its weight fragments straight from global memory into MFMA operand
// registers, 4 K slices (128 bytes each) ahead; a weight element is used by exactly one
// wavefront, so weights never touch LDS. The BM activation rows, shared by the 4
// wavefronts, go through a double-buffered LDS ring: per slice each thread copies one
// 16-byte chunk of each 4 KB activation block, loaded two slices ahead into registers; one
// LDS-only barrier per slice (it does not wait for the weight loads in flight).
// Both operands are in the tiled layout, so every global load instruction reads 1 KB of
// one page (with row-major operands each instruction touched 32 rows, and the address
// translation requests, not HBM, set the pace) and every LDS fragment read is a
// contiguous 1 KB. Tiles start at multiples of 32 rows (padded expert order), so each
// 32-row block of A is one tile column of the tiled activation buffer.
// The grid is persistent (see stream_gemm_kernel) and, for the bf16 down GEMM when the K
// slices come in multiples of 4, chained: the last steps of a tile issue the first weight and activation
// loads of the workgroup's next tile into the slots where its prologue would put them, so
// a tile starts with its first 4 slices in flight or landed instead of waiting out a fresh
// HBM latency (an unchained tile carried a fixed cost of about a fifth of its time).
// Nothing after those loads waits for them before the next tile's first step: the
// epilogues use LDS-only barriers, and down reads its output rows' pair indices from LDS,
// copied there early in the tile.
struct Slice16 { int32x4_t c[4]; };   // one lane's 64 bytes of a 32-row x 128-byte tile

// Where one (m-tile, n-tile) pair of a grouped launch reads (all wavefront-uniform).
struct StreamTile {
  const uint8_t* b;     // the wavefront's 32 weight rows (gate_up: waves 0-1 gate, 2-3 up)
  const uint8_t* a;     // the tile's first 32-row activation block
  int a_last;           // its last 32-row block that holds rows (0 .. BM / 32 - 1)
  int rot;              // first K slice visited
  int expert, row0, row1, n0;
};

template <int MODE>
MOLT_DEV StreamTile stream_geometry(const GemmParams& p, int id, int nk, int wave) {
  StreamTile g;
  const int mt = id / p.n_ntiles, nt = id % p.n_ntiles;
  // through the constant address space: a scalar load (the table is read-only here), which
  // does not wait behind the vector stores of an epilogue
  typedef const __attribute__((address_space(4))) int32x4_t* ConstTile;
  int4 t = make_int4(0, 0, p.M, 0);                   // no table: one dense row tile
  if (p.tiles != nullptr) {
    const int32x4_t tv = *(ConstTile)(p.tiles + mt);
    t = make_int4(tv[0], tv[1], tv[2], tv[3]);
  }
  g.expert = t.x;
  g.row0 = t.y;                                       // a multiple of 32
  g.row1 = t.z;
  const long RB = long(nk) * kRowBytes;               // bytes per operand row
  long wrow;
  if (MODE == kGateUp) {
    g.n0 = nt * (kBN / 2);
    wrow = long(g.expert) * 2 * p.N + (wave < 2 ? g.n0 + 32 * wave : p.N + g.n0 + 32 * (wave - 2));
  } else {
    g.n0 = nt * kBN;
    wrow = long(g.expert) * p.N + g.n0 + 32 * wave;
  }
  g.b = static_cast<const uint8_t*>(p.B) + wrow * RB;
  g.a = static_cast<const uint8_t*>(p.A) + long(g.row0) * RB;
  g.a_last = (((g.row1 - 1) & ~31) - g.row0) / 32;
  // K slices are visited in an order rotated by the column tile, so the workgroups of one
  // row tile (running side by side on one XCD) read different activation blocks at any
  // moment instead of all hitting the same L2 lines
  g.rot = int((long(nt) * nk) / p.n_ntiles);
  return g;
}

// Persistent grouped GEMM: the grid is what the chip holds at once (a multiple of 8, see
// run_stream). Workgroup b runs on XCD b % 8 and walks that XCD's contiguous eighth of the
// live (m-tile, n-tile) pairs, m-tile major, with the XCD's workgroup count as stride: the
// n-tiles of one row tile run side by side on one XCD, so its activation tile is read from
// HBM once and then hits that XCD's L2. Launching one workgroup per pair left the chip
// at 50-80% of its resident workgroups on average (dispatch gaps between short tiles).
// CHAIN requires K slices in multiples of 4 (the slot pattern then lines up across tiles).
// fp8 launches take each workgroup's later tiles from its XCD's queue instead (see below).
template <int BM, bool FP8, int MODE, bool CHAIN, bool ROWS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(BM <= 64 ? 3 : 2)))
void stream_gemm_kernel(GemmParams p) {
  static_assert(MODE == kGateUp || MODE == kDown, "grouped modes");
  static_assert(!ROWS || (MODE == kGateUp && !CHAIN), "row gather: gate_up");
  constexpr int MS = BM / 32;                        // 32-row MFMA tiles per wavefront
  constexpr int kElem = FP8 ? 1 : 2;
  // weight slices in flight per wavefront (each 4 KB slice of a wavefront's 32 weight rows
  // is 16 registers; 8 in flight measured slower than 4)
  constexpr int WD = 4;
  // activation staging: 2 buffers of MS 4 KB blocks; gate_up's epilogue reuses them, with
  // the space after them, as a BM x 128 f32 tile (2 * BM * 256 bytes)
  __shared__ __attribute__((aligned(16))) uint8_t smem[(MODE == kGateUp ? 4 : 2) * MS * 4096];
  uint8_t (*alds)[MS * 4096] = reinterpret_cast<uint8_t (*)[MS * 4096]>(smem);
  __shared__ int prow[MODE == kDown ? BM : 1];       // down: pair index of each tile row
  // down epilogue: the tile's outputs (BM x 128 f32; 128-row tiles in two 64-column passes)
  constexpr int kEpCols = BM == 128 ? 64 : 128;
  __shared__ __attribute__((aligned(16))) float dep[MODE == kDown ? BM * kEpCols : 1];
  const int total = (p.n_tiles_live != nullptr ? *p.n_tiles_live : p.n_mtiles) * p.n_ntiles;
  const int chunk = (total + 7) / 8;
  const int stride = gridDim.x / 8;
  const int first = (blockIdx.x % 8) * chunk;
  int k8 = blockIdx.x / 8;
  if (k8 >= chunk || first + k8 >= total) return;
  const int nk = int(long(p.K) * kElem / kRowBytes);  // 128-byte K slices
  const long RB = long(nk) * kRowBytes;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const unsigned boff = lane * 16u, aoff = threadIdx.x * 16u;
  auto slice = [&](const StreamTile& t, int kb) __attribute__((always_inline)) {
    const int k = min(kb, nk - 1) + t.rot;
    return long(k >= nk ? k - nk : k) * 4096;
  };
  // weights are read once per step: nontemporal loads
  auto wld = [&](Slice16& f, const StreamTile& t, int kb) __attribute__((always_inline)) {
    const uint8_t* src = t.b + slice(t, kb) + boff;
#pragma unroll
    for (int c = 0; c < 4; ++c) f.c[c] = __builtin_nontemporal_load(reinterpret_cast<const int32x4_t*>(src + 1024 * c));
  };
  // ROWS: thread t copies piece t % 8 (16 bytes) of row t / 8 of each 32-row block from the
  // token's row-major row (roff: its byte offset, set per tile), so each load instruction
  // reads 8 whole 128-byte row slices; in LDS the row's 8 pieces sit at piece ^ swz(row)
  // (conflict-free fragment reads and stores)
  long roff[ROWS ? MS : 1];
  const unsigned rsto = ROWS ? (threadIdx.x / 8) * 128 + ((threadIdx.x % 8) ^ ((threadIdx.x / 16) % 8)) * 16
                             : threadIdx.x * 16;
#define MOLT_GLOAD(ST, T, KB)                                                         \
  {                                                                                   \
    const long off_ = slice(T, KB);                                                   \
    if (ROWS) {                                                                       \
      _Pragma("unroll") for (int b_ = 0; b_ < MS; ++b_)                               \
          ST[b_] = *reinterpret_cast<const int32x4_t*>(static_cast<const uint8_t*>(p.A) + roff[b_ % (ROWS ? MS : 1)] + (off_ >> 5) + (threadIdx.x % 8) * 16); \
    } else {                                                                          \
      _Pragma("unroll") for (int b_ = 0; b_ < MS; ++b_)                               \
          ST[b_] = *reinterpret_cast<const int32x4_t*>((T).a + long(min(b_, (T).a_last)) * 32 * RB + off_ + aoff); \
    }                                                                                 \
  }
#define MOLT_SSTORE(ST, BUF)                                                          \
  {                                                                                   \
    _Pragma("unroll") for (int b_ = 0; b_ < MS; ++b_)                                 \
        *reinterpret_cast<int32x4_t*>(&alds[BUF][b_ * 4096 + rsto]) = ST[b_];         \
  }
  // ROWS fragment reads: lane l takes row l % 32, piece 4 (l / 32) + c for k-step c
  const unsigned rsw = (4 * (lane / 32)) ^ ((lane % 32 / 2) % 8);
  int32x4_t st0[MS], st1[MS];
  Slice16 wb[WD];
  floatx16_t acc[MS];
  StreamTile g = stream_geometry<MODE>(p, first + k8, nk, wave);
  StreamTile gn = g;
  bool more = false;
  bool primed = false;                               // g's first slices already loaded
  // fp8 launches take tiles from their XCD's queue: a workgroup's first tile is k8 as in the
  // static walk, each later one the next of the pool [stride, chunk), taken by thread 0 when
  // the tile enters its last K steps and passed on through LDS in the epilogue, so
  // workgroups that run faster take more tiles (the static walk left an XCD's workgroups
  // ending anywhere between half and all of the kernel's time). Their Zipf-hot tiles are
  // bound by the MFMAs and differ in cost; the bf16 launches are bound by HBM, where the
  // late workgroups still share the full bandwidth and the queue measured 0-5% slower.
  constexpr bool kDyn = FP8 && !CHAIN;
  const bool dyn = kDyn && p.queue != nullptr;
  __shared__ int s_grab;
  int grab = chunk;                                  // thread 0: the next tile (dyn)
  for (;;) {
    // down: the pair index of each of the tile's rows, loaded before the tile's own loads
    int pv = -1;
    if (MODE == kDown && threadIdx.x < BM && g.row0 + int(threadIdx.x) < g.row1)
      pv = p.perm != nullptr ? p.perm[g.row0 + threadIdx.x] : g.row0 + int(threadIdx.x);
    auto put_prow = [&]() __attribute__((always_inline)) {
      if (MODE == kDown && threadIdx.x < BM) prow[threadIdx.x] = pv;
    };
    if (!dyn) {
      const int kn = k8 + stride;
      more = kn < chunk && first + kn < total;
      // the next tile's table entry is read here, not after the epilogue
      if (more) gn = stream_geometry<MODE>(p, first + kn, nk, wave);
    }
    if (ROWS) {
      // rows past the tile's end (and padding rows) read token 0: their outputs are not stored
#pragma unroll
      for (int b_ = 0; b_ < MS; ++b_) {
        const int r = g.row0 + 32 * b_ + int(threadIdx.x / 8);
        const int pr = r < g.row1 ? p.perm[r] : -1;
        roff[b_ % (ROWS ? MS : 1)] = pr < 0 ? 0 : long(pr / p.ktop) * RB;
      }
    }
    if (!primed) {
      MOLT_GLOAD(st0, g, 0);
      MOLT_GLOAD(st1, g, 1);
#pragma unroll
      for (int s = 0; s < WD; ++s) wld(wb[s], g, s);
      // gate_up: every wavefront is done reading the last tile's epilogue tile from LDS
      if (MODE == kGateUp && k8 != int(blockIdx.x / 8)) lds_barrier();
      MOLT_SSTORE(st0, 0);
      MOLT_GLOAD(st0, g, 2);
      lds_barrier();
    }

#pragma unroll
    for (int i = 0; i < MS; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;
    // Step over slice k: LDS buffer U holds its activations, weight slot W its weights,
    // register slot ST_NEXT slice k + 1 (the other slot k + 2). It computes, refills W with
    // slice k + WD, stores slice k + 1 into buffer 1 - U (last read before the previous
    // barrier) and refills ST_NEXT with slice k + 3. In the last WD + 3 steps (TAIL = 1) a
    // refill past the end loads the next tile's slice (chained) or nothing: re-reading the
    // last slice instead cost the 12-slice down GEMM a third more weight loads. fp8: the
    // refills and the activation copy run at raised wave priority, so they issue ahead of
    // the other wavefronts' MFMAs (fp8 Zipf MoE layer 380 -> 370 us; bf16 unchanged).
#define MOLT_STEP(U, ST_NEXT, W, K, TAIL)                                                           \
  {                                                                                                  \
    const uint8_t* base_ = alds[U] + (ROWS ? (lane % 32) * 128 : lane * 16);                         \
    if (!FP8) {                                                                                      \
      _Pragma("unroll") for (int c = 0; c < 4; ++c) {                                                \
        const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(&wb[W].c[c]);                         \
        const unsigned fo_ = ROWS ? ((rsw ^ c) * 16) : c * 1024;                                     \
        _Pragma("unroll") for (int i = 0; i < MS; ++i) acc[i] =                                      \
            mfma(*reinterpret_cast<const bf16x8_t*>(base_ + i * 4096 + fo_), bv, acc[i]);            \
      }                                                                                              \
    } else {                                                                                         \
      _Pragma("unroll") for (int c = 0; c < 2; ++c) {                                                \
        const int32x4_t w0 = wb[W].c[2 * c], w1 = wb[W].c[2 * c + 1];                                \
        const int32x8_t bv = int32x8_t{w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};     \
        const unsigned lo_ = ROWS ? ((rsw ^ (2 * c)) * 16) : 2 * c * 1024;                          \
        const unsigned hi_ = ROWS ? ((rsw ^ (2 * c + 1)) * 16) : (2 * c + 1) * 1024;                \
        _Pragma("unroll") for (int i = 0; i < MS; ++i) {                                             \
          const int32x4_t lo = *reinterpret_cast<const int32x4_t*>(base_ + i * 4096 + lo_);          \
          const int32x4_t hi = *reinterpret_cast<const int32x4_t*>(base_ + i * 4096 + hi_);          \
          acc[i] = mfma(int32x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]}, bv, acc[i]); \
        }                                                                                            \
      }                                                                                              \
    }                                                                                                \
    if (FP8) __builtin_amdgcn_s_setprio(3);                                                          \
    if (!(TAIL) || (K) + WD < nk) wld(wb[W], g, (K) + WD);                                           \
    else if (CHAIN && more) wld(wb[W], gn, (K) + WD - nk);                                           \
    MOLT_SSTORE(ST_NEXT, 1 - (U));                                                                   \
    if (!(TAIL) || (K) + 3 < nk) MOLT_GLOAD(ST_NEXT, g, (K) + 3)                                     \
    else if (CHAIN && more) MOLT_GLOAD(ST_NEXT, gn, (K) + 3 - nk)                                    \
    if (FP8) __builtin_amdgcn_s_setprio(0);                                                          \
    lds_barrier();                                                                                   \
  }
    static_assert(WD == 4, "the step sequence cycles through 4 weight slots");
    int kb = 0;
    for (; kb + WD + 3 < nk; kb += 4) {    // every refill of these 4 steps is in this tile
      MOLT_STEP(0, st1, 0, kb, 0);
      if (kb == 0) put_prow();             // waits for the row load, not for the step's own
      MOLT_STEP(1, st0, 1, kb + 1, 0);
      MOLT_STEP(0, st1, 2, kb + 2, 0);
      MOLT_STEP(1, st0, 3, kb + 3, 0);
    }
    if (kb == 0) {                         // no full 4 steps: a chained tile has had no
      if (primed) lds_barrier();           // barrier since the last tile's epilogue read prow
      put_prow();
    }
    if (dyn && threadIdx.x == 0) grab = stride + atomicAdd(p.queue + blockIdx.x % 8, 1);
    // the last 1..7 slices (kb % 4 == 0, so the slot pattern continues)
    if (kb < nk) MOLT_STEP(0, st1, 0, kb, 1);
    if (kb + 1 < nk) MOLT_STEP(1, st0, 1, kb + 1, 1);
    if (kb + 2 < nk) MOLT_STEP(0, st1, 2, kb + 2, 1);
    if (kb + 3 < nk) MOLT_STEP(1, st0, 3, kb + 3, 1);
    if (kb + 4 < nk) MOLT_STEP(0, st1, 0, kb + 4, 1);
    if (kb + 5 < nk) MOLT_STEP(1, st0, 1, kb + 5, 1);
    if (kb + 6 < nk) MOLT_STEP(0, st1, 2, kb + 6, 1);
#undef MOLT_STEP
    // published by the epilogue's first barrier, read after the tile
    if (dyn && threadIdx.x == 0) s_grab = grab;
    // accumulator element e of lane (lcol, lgrp) in tile i: row 32 i + 8 (e / 4) + 4 lgrp + e % 4
    int lcol = lane % 32, lgrp = lane / 32;
    // opaque per tile: the epilogue's address arithmetic stays here instead of being hoisted
    // out of the tile loop into registers held across the K steps (gate_up spilled them)
    asm volatile("" : "+v"(lcol), "+v"(lgrp));
    if (MODE == kGateUp) {
      // h = silu(gate) * up, bf16, tiled layout over padded rows. The accumulators go to LDS
      // as a BM x 128 tile (gate columns 0-63 from wavefronts 0-1, up columns 64-127 from
      // 2-3; the last step's barrier freed the staging buffers); then each thread finishes
      // 8 consecutive columns of a row per pass and writes them with one 16-byte store.
      float* ep = reinterpret_cast<float*>(smem);
#pragma unroll
      for (int i = 0; i < MS; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) ep[(32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4)) * 128 + 32 * wave + lcol] = acc[i][e];
      // fp8 scales of the thread's units (its 8 columns are the same in every unit) are all
      // loaded before the first store: a load issued after a store has to wait for it
      float sxv[MS];
      float4 swv[4];
      if (FP8) {
        const float* sw = p.b_scale + long(g.expert) * p.b_scale_ld + g.n0 + (threadIdx.x & 7) * 8;
        swv[0] = *reinterpret_cast<const float4*>(sw);
        swv[1] = *reinterpret_cast<const float4*>(sw + 4);
        swv[2] = *reinterpret_cast<const float4*>(sw + p.N);
        swv[3] = *reinterpret_cast<const float4*>(sw + p.N + 4);
        int pr[MS];
#pragma unroll
        for (int j = 0; j < MS; ++j) {
          const int grow = g.row0 + int((threadIdx.x + kThreads * j) >> 3);
          pr[j] = grow < g.row1 ? p.perm[grow] : 0;
        }
#pragma unroll
        for (int j = 0; j < MS; ++j) sxv[j] = p.a_scale[pr[j] / p.ktop];
      }
      lds_barrier();
      // the scales are in before the first store: with the stores behind per-unit branches the
      // compiler would otherwise wait for every earlier store before each unit's scale use
      // (s_waitcnt vmcnt(0), expcnt and lgkmcnt left open)
      if (FP8) __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
      const long hrb = 2L * p.N;
#pragma unroll
      for (int j = 0; j < MS; ++j) {
        const int u = int(threadIdx.x) + kThreads * j;   // BM * 8 units of 8 columns
        const int r = u >> 3, cb = (u & 7) * 8;
        const int grow = g.row0 + r;
        if (grow >= g.row1) continue;
        const float4* gp = reinterpret_cast<const float4*>(ep + r * 128 + cb);
        const float4* up = reinterpret_cast<const float4*>(ep + r * 128 + 64 + cb);
        const float4 g0 = gp[0], g1 = gp[1], u0 = up[0], u1 = up[1];
        float gv[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        float uv[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
        if (FP8) {
          const float sx = sxv[j];
          const float swg[8] = {swv[0].x, swv[0].y, swv[0].z, swv[0].w, swv[1].x, swv[1].y, swv[1].z, swv[1].w};
          const float swu[8] = {swv[2].x, swv[2].y, swv[2].z, swv[2].w, swv[3].x, swv[3].y, swv[3].z, swv[3].w};
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            gv[q] *= sx * swg[q];
            uv[q] *= sx * swu[q];
          }
        }
        uint32_t packed[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          packed[q] = uint32_t(f32_to_bf16(silu(gv[2 * q]) * uv[2 * q])) |
                      (uint32_t(f32_to_bf16(silu(gv[2 * q + 1]) * uv[2 * q + 1])) << 16);
        *reinterpret_cast<int32x4_t*>(static_cast<uint8_t*>(p.C) + tiled_offset(grow, 2L * (g.n0 + cb), hrb)) =
            int32x4_t{int(packed[0]), int(packed[1]), int(packed[2]), int(packed[3])};
      }
    } else {
      // per-pair expert output, f32, row = pair index (token * K + slot). Through LDS, so
      // that each thread writes 4 consecutive columns of a row with one 16-byte store.
      constexpr int kUnits = BM * kEpCols / 4;         // 4-column units per pass
      static_assert(kThreads % (kEpCols / 4) == 0, "a thread's columns are fixed per pass");
      // fp8: the thread's row and channel scales, all loaded before the first store
      float sxd[kUnits / kThreads];
      float4 swd[128 / kEpCols];
      if (FP8) {
        const int c4 = int(threadIdx.x % (kEpCols / 4)) * 4;
#pragma unroll
        for (int q = 0; q < 128 / kEpCols; ++q)
          swd[q] = *reinterpret_cast<const float4*>(p.b_scale + long(g.expert) * p.b_scale_ld + g.n0 + q * kEpCols + c4);
#pragma unroll
        for (int j = 0; j < kUnits / kThreads; ++j) {
          const int grow = g.row0 + int((threadIdx.x + kThreads * j) / (kEpCols / 4));
          sxd[j] = grow < g.row1 ? p.a_scale[grow] : 0.f;
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);   // in before the first store (see gate_up)
      }
#pragma unroll
      for (int pass = 0; pass < 128 / kEpCols; ++pass) {
        const int c0 = pass * kEpCols;                 // first column of this pass
        if (32 * wave >= c0 && 32 * wave < c0 + kEpCols) {
#pragma unroll
          for (int i = 0; i < MS; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              dep[(32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4)) * kEpCols + 32 * wave - c0 + lcol] = acc[i][e];
        }
        lds_barrier();
        auto unit = [&](int j) __attribute__((always_inline)) {
          const int u = int(threadIdx.x) + kThreads * j;
          const int r = u / (kEpCols / 4), c4 = (u % (kEpCols / 4)) * 4;
          const int grow = g.row0 + r;
          if (grow >= g.row1) return;
          float4 v = *reinterpret_cast<const float4*>(dep + r * kEpCols + c4);
          const int c = g.n0 + c0 + c4;
          if (FP8) {
            const float sx = sxd[j];
            const float4 sw = swd[pass];
            v.x *= sx * sw.x;
            v.y *= sx * sw.y;
            v.z *= sx * sw.z;
            v.w *= sx * sw.w;
          }
          *reinterpret_cast<float4*>(static_cast<float*>(p.C) + long(prow[r]) * p.ldc + c) = v;
        };
        if constexpr (FP8) {
#pragma unroll
          for (int j = 0; j < kUnits / kThreads; ++j) unit(j);
        } else {
#pragma unroll 4
          for (int j = 0; j < kUnits / kThreads; ++j) unit(j);
        }
        if (pass + 1 < 128 / kEpCols) lds_barrier();
      }
    }
    if (dyn) {
      k8 = s_grab;
      if (k8 >= chunk || first + k8 >= total) break;
      g = stream_geometry<MODE>(p, first + k8, nk, wave);
      continue;
    }
    if (!more) break;
    k8 += stride;
    g = gn;
    primed = CHAIN;
  }
#undef MOLT_SSTORE
#undef MOLT_GLOAD
}

// Workgroups of `kernel` (kThreads each) resident on the whole device at once, rounded
// down to a multiple of 8 (>= 8).
template <typename K>
int resident_grid(K kernel) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess)
    return 8;
  return (cus * per_cu) / 8 * 8 > 8 ? (cus * per_cu) / 8 * 8 : 8;
}

template <bool FP8, int MODE, bool CHAIN, bool ROWS = false>
hipError_t run_stream_k(GemmParams p, int tile_m, hipStream_t s) {
  // resident workgroups per kernel, queried once per process (one device model)
  static const int r32 = resident_grid(stream_gemm_kernel<32, FP8, MODE, CHAIN, ROWS>);
  static const int r64 = resident_grid(stream_gemm_kernel<64, FP8, MODE, CHAIN, ROWS>);
  static const int r128 = resident_grid(stream_gemm_kernel<128, FP8, MODE, CHAIN, ROWS>);
  const int pairs = (p.n_mtiles * p.n_ntiles + 7) / 8 * 8;   // upper bound of the live pairs
  const int cap = tile_m == 32 ? r32 : tile_m == 64 ? r64 : r128;
  const int grid = pairs < cap ? pairs : cap;
  if (tile_m == 32) stream_gemm_kernel<32, FP8, MODE, CHAIN, ROWS><<<grid, kThreads, 0, s>>>(p);
  else if (tile_m == 64) stream_gemm_kernel<64, FP8, MODE, CHAIN, ROWS><<<grid, kThreads, 0, s>>>(p);
  else stream_gemm_kernel<128, FP8, MODE, CHAIN, ROWS><<<grid, kThreads, 0, s>>>(p);
  return hipGetLastError();
}

template <bool FP8, int MODE>
hipError_t run_stream(GemmParams p, int tile_m, hipStream_t s, bool rows = false) {
  const long nk = long(p.K) * (FP8 ? 1 : 2) / kRowBytes;
  // chained in bf16 for down only: its 12-slice tiles gained (85 -> 82 us per launch at
  // T*K = 5120), gate_up's 32-slice tiles did not (159 -> 161 us)
  if constexpr (!FP8 && MODE == kDown)
    if (nk % 4 == 0) return run_stream_k<false, MODE, true>(p, tile_m, s);
  if constexpr (MODE == kGateUp)
    if (rows) return run_stream_k<FP8, MODE, false, true>(p, tile_m, s);
  return run_stream_k<FP8, MODE, false>(p, tile_m, s);
}

// ---------------------------------------------------------------- LDS-tiled dense GEMM
// Dense projections and the LM head have a few hundred rows: every weight tile feeds
// several row tiles and every activation tile many column tiles, so both operands are
// shared through LDS. Workgroup = BM x 128 outputs, 4 wavefronts in a 2 x 2 grid. Per
// 128-byte K slice the workgroup copies (BM/32 + 4) tiled 4 KB blocks (one 16-byte chunk
// per thread per block: coalesced 4 KB loads from one page) into a double-buffered LDS
// ring, loaded two slices ahead into registers; the tiled layout makes each wavefront's
// MFMA fragment a contiguous 1 KB LDS read (conflict-free, no padding). One barrier per
// slice. Split-K: split s covers slices [s * nk / S, (s + 1) * nk / S) and writes its
// partial sums to `part[s]`; a fixed-order reduction adds them (deterministic).
// Epilogue of the QKV projection with RoPE and the paged-KV write fused in (head_dim 128:
// output column tile nt is head nt; q heads, then k heads, then v heads).
struct RopeKv {
  const double2* table;     // [T][64] {cos, sin} of each token's position
  const int32_t* slot;      // [T] KV-cache slot of token t: block * 16 + position % 16, or -1
  int Hq, Hkv;
  uint16_t* q;              // [T, Hq, 128] bf16
  uint16_t* kc;             // [num_blocks, Hkv, 16, 128]
  uint16_t* vc;             // [num_blocks, Hkv, 128, 16]
};

template <int BM, bool ROPE, int WN, int DEPTH>
__global__ __launch_bounds__(128 * WN) void lds_gemm_kernel(GemmParams p, float* part, int splits,
                                                            RopeKv rk) {
  constexpr int NT = 128 * WN;                // 2 x WN wavefronts
  constexpr int AB = BM / 32;                 // activation row blocks
  constexpr int NB = AB + 4;                  // 4 KB blocks per slice (A then B)
  constexpr int CPT = NB * 256 / NT;          // 16-byte chunks per thread per slice
  constexpr int TM = BM / 64 > 0 ? BM / 64 : 1;   // 32-row MFMA tiles per wavefront
  constexpr int WROWS = 32 * TM;              // rows per wavefront
  constexpr int NJ = 4 / WN;                  // 32-column MFMA tiles per wavefront
  static_assert(BM == 64 || BM == 128, "BM");
  static_assert((NB * 256) % NT == 0, "chunks per thread");
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][NB * 4096];

  const int total = p.n_mtiles * p.n_ntiles * splits;
  const int chunk = (total + 7) / 8;
  const int k8 = blockIdx.x / 8;
  const int id = (blockIdx.x % 8) * chunk + k8;   // XCD-contiguous; split, n-tile, m-tile
  if (k8 >= chunk || id >= total) return;
  const int mt = id % p.n_mtiles;
  const int nt = (id / p.n_mtiles) % p.n_ntiles;
  const int split = id / (p.n_mtiles * p.n_ntiles);
  const int row0 = mt * BM, n0 = nt * kBN;
  const long RB = long(p.K) * 2;
  const int nk = int(RB / kRowBytes);
  const int kb0 = int(long(nk) * split / splits), kb1 = int(long(nk) * (split + 1) / splits);
  // RoPE epilogue: this thread's row's KV-cache slot, read before the K loop (loaded at the
  // epilogue it would wait behind the table loads there)
  int my_slot = -1;
  if constexpr (ROPE) my_slot = rk.slot[min(row0 + int(threadIdx.x % BM), p.M - 1)];

  // chunk q = tid + NT u of a slice is 16-byte chunk q % 256 of block q / 256 (A blocks,
  // then B blocks; each a 4 KB tile, clamped into the padded operands); it lands at byte
  // 16 q of the slice's LDS buffer
  const uint8_t* src[CPT];
#pragma unroll
  for (int u = 0; u < CPT; ++u) {
    const int q = int(threadIdx.x) + NT * u, b = q / 256;
    const int last_a = (p.M - 1) & ~31, last_b = (p.N - 1) & ~31;
    const long r = b < AB ? min(row0 + 32 * b, last_a) : min(n0 + 32 * (b - AB), last_b);
    src[u] = static_cast<const uint8_t*>(b < AB ? p.A : p.B) + r * RB + (q % 256) * 16;
  }
  // register slots of DEPTH slices in flight (native vector type: HIP's int4 struct copied
  // into LDS made the compiler keep these arrays in scratch memory)
  int32x4_t st[DEPTH][CPT];
#define MOLT_GLOAD(ST, KB)                                                            \
  {                                                                                   \
    const long off_ = long(min((KB), kb1 - 1)) * 4096;                                \
    _Pragma("unroll") for (int b_ = 0; b_ < CPT; ++b_)                                \
        ST[b_] = *reinterpret_cast<const int32x4_t*>(src[b_] + off_);                 \
  }
#define MOLT_SSTORE(ST, BUF)                                                          \
  {                                                                                   \
    _Pragma("unroll") for (int b_ = 0; b_ < CPT; ++b_)                                \
        *reinterpret_cast<int32x4_t*>(&lds[BUF][(threadIdx.x + NT * b_) * 16]) = ST[b_]; \
  }
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int wm = wave / WN, wn = wave % WN;     // wavefront rows wm*WROWS.., cols wn*32*NJ..
  floatx16_t acc[TM][NJ];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

#pragma unroll
  for (int j = 0; j < DEPTH; ++j) MOLT_GLOAD(st[j], kb0 + j);
  MOLT_SSTORE(st[0], 0);
  MOLT_GLOAD(st[0], kb0 + DEPTH);
  lds_barrier();
  // Step J (mod DEPTH) over slice k: LDS buffer k % 2 holds slice k, register slot
  // (J + 1) % DEPTH slice k + 1 (loaded DEPTH steps earlier). It computes, stores slice
  // k + 1 into the other buffer (last read before the previous barrier) and refills that
  // slot with slice k + 1 + DEPTH. Loads past the end re-read the last slice.
#define MOLT_STEP(J, K)                                                                           \
  {                                                                                                \
    const uint8_t* base_ = lds[(J) & 1];                                                           \
    _Pragma("unroll") for (int c = 0; c < 4; ++c) {                                                \
      bf16x8_t af[TM], bfr[NJ];                                                                    \
      _Pragma("unroll") for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const bf16x8_t*>(   \
          base_ + ((wm * WROWS) / 32 + i) * 4096 + c * 1024 + lane * 16);                          \
      _Pragma("unroll") for (int j = 0; j < NJ; ++j) bfr[j] = *reinterpret_cast<const bf16x8_t*>(  \
          base_ + (AB + wn * NJ + j) * 4096 + c * 1024 + lane * 16);                               \
      _Pragma("unroll") for (int i = 0; i < TM; ++i)                                               \
          _Pragma("unroll") for (int j = 0; j < NJ; ++j) acc[i][j] = mfma(af[i], bfr[j], acc[i][j]); \
    }                                                                                              \
    MOLT_SSTORE(st[((J) + 1) % DEPTH], 1 - ((J) & 1));                                             \
    MOLT_GLOAD(st[((J) + 1) % DEPTH], (K) + 1 + DEPTH);                                            \
    lds_barrier();                                                                                 \
  }
  static_assert(DEPTH % 2 == 0, "LDS buffer parity follows the slot index");
  int kb = kb0;
  for (; kb + DEPTH - 1 < kb1; kb += DEPTH) {   // loads are clamped, never behind a branch
#pragma unroll
    for (int J = 0; J < DEPTH; ++J) MOLT_STEP(J, kb + J);
  }
#pragma unroll
  for (int J = 0; J < DEPTH - 1; ++J)
    if (kb + J < kb1) MOLT_STEP(J, kb + J);
#undef MOLT_STEP
#undef MOLT_SSTORE
#undef MOLT_GLOAD

  // acc[i][j][e]: row wm*WROWS + 32 i + 8 (e / 4) + 4 (lane / 32) + e % 4,
  // col wn*32*NJ + 32 j + lane % 32
  const int lcol = lane % 32, lgrp = lane / 32;
  if constexpr (ROPE) {
    // The f32 tile goes through the (now idle) LDS ring so that each rotation pair (i, i + 64)
    // meets in one thread; the rotation is done in f64 with the step's cos/sin table. The
    // table entries and cache slots are fetched first, so their latency overlaps the exchange.
    // thread (pr, pi) rotates pair pi of rows pr + PR n, n < BM / PR, in groups of RG rows
    constexpr int PR = NT / 64;
    constexpr int RG = BM / PR < 16 ? BM / PR : 16;
    constexpr int NG = BM / (PR * RG);
    const int h = nt, pi = threadIdx.x % 64, pr = threadIdx.x / 64;
    const bool rotate = h < rk.Hq + rk.Hkv;
    double2 cs[RG];
    auto fetch = [&](int g) __attribute__((always_inline)) {
#pragma unroll
      for (int n = 0; n < RG; ++n)
        cs[n] = rk.table[long(min(row0 + pr + PR * (RG * g + n), p.M - 1)) * 64 + pi];
    };
    __shared__ int s_slot[BM];
    if (rotate) fetch(0);
    if (threadIdx.x < BM) s_slot[threadIdx.x] = row0 + int(threadIdx.x) < p.M ? my_slot : -1;
    __syncthreads();
    float* ob = reinterpret_cast<float*>(&lds[0][0]);     // [BM][128]
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          ob[(wm * WROWS + 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4)) * 128 + wn * 32 * NJ + 32 * j + lcol] =
              acc[i][j][e];
    __syncthreads();
    if (rotate) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        if (g > 0) fetch(g);
        // all of the group's table entries in before its first store: with the stores behind
        // branches the compiler would otherwise wait for every earlier store at each row
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
#pragma unroll
        for (int n = 0; n < RG; ++n) {
          const int r = pr + PR * (RG * g + n), t = row0 + r;
          if (t >= p.M) break;
          const double a = ob[r * 128 + pi], c = ob[r * 128 + pi + 64];
          const uint16_t lo = f32_to_bf16(float(a * cs[n].x - c * cs[n].y));
          const uint16_t hi = f32_to_bf16(float(c * cs[n].x + a * cs[n].y));
          uint16_t* dst;
          if (h < rk.Hq) {
            dst = rk.q + (long(t) * rk.Hq + h) * 128;
          } else {
            const int sl = s_slot[r];
            if (sl < 0) continue;
            dst = rk.kc + ((long(sl >> 4) * rk.Hkv + (h - rk.Hq)) * 16 + (sl & 15)) * 128;
          }
          dst[pi] = lo;
          dst[pi + 64] = hi;
        }
      }
    } else {
      const int hk = h - rk.Hq - rk.Hkv;
      for (int w = threadIdx.x; w < BM * 128; w += NT) {
        const int r = w % BM, i = w / BM, sl = s_slot[r];
        if (sl < 0) continue;
        rk.vc[((long(sl >> 4) * rk.Hkv + hk) * 128 + i) * 16 + (sl & 15)] = f32_to_bf16(ob[r * 128 + i]);
      }
    }
    return;
  }
  float* out = splits > 1 ? part + long(split) * p.M * p.ldc : static_cast<float*>(p.C);
  if (!(splits == 1 && p.accumulate) && row0 + BM <= p.M && n0 + kBN <= p.N) {
    // whole tile: no bounds checks between the stores
    float* base = out + long(row0 + wm * WROWS + 4 * lgrp) * p.ldc + n0 + wn * 32 * NJ + lcol;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) base[long(32 * i + 8 * (e / 4) + (e % 4)) * p.ldc + 32 * j] = acc[i][j][e];
    return;
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = n0 + wn * 32 * NJ + 32 * j + lcol;
    if (c >= p.N) continue;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int grow = row0 + wm * WROWS + 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
        if (grow >= p.M) continue;
        float* dst = out + long(grow) * p.ldc + c;
        *dst = (splits == 1 && p.accumulate) ? *dst + acc[i][j][e] : acc[i][j][e];
      }
  }
}

// ---------------------------------------------------------------- big-tile dense GEMM
// The LM head (640 x 151936 x 2048) is bound by what the memory pipeline can hand the
// MFMAs, so its tile is sized for flops per loaded byte: 160 rows x 256 columns per
// workgroup, 101 flops per byte (the 128 x 128 LDS-tiled kernel reaches 64). Wavefront w
// computes all 160 rows x columns 64 w .. 64 w + 63, so the activation tile is shared by the
// four wavefronts and each weight column block belongs to one of them:
// * the 5 activation blocks (tiled, 4 KB per K slice) go through a 4-stage LDS ring, copied
//   by the LDS-DMA form of the buffer load three slices ahead (each wavefront a quarter of
//   every block; it waits for its own copies and one barrier per slice publishes them);
// * the wavefront's 2 weight blocks are loaded straight into MFMA operand registers (the
//   tiled layout is the fragment layout) kBigDepth slices ahead: they never touch LDS.
// Per 16-wide k step 5 LDS fragments and 2 register fragments feed 10 MFMAs. The barrier
// sits before the last k step of a slice, so the next slice's first fragments are read
// behind that step's MFMAs. The row tiles of one column tile are consecutive on one XCD, so
// its weights come from HBM once.
constexpr int kBigBM = 160, kBigBN = 256;
constexpr int kBigAB = kBigBM / 32;            // activation blocks per K slice
constexpr int kBigAStages = 4;
constexpr int kBigAStage = kBigAB * 4096;
constexpr int kBigDepth = 3;                   // weight slices in flight per wavefront
constexpr int kBigBLoads = 8;                  // weight loads per wavefront per slice

// Buffer resource word 3 for raw byte-addressed loads (32-bit data format, no swizzle).
constexpr int kRawRsrcWord3 = 0x00020000;

MOLT_DEV __amdgpu_buffer_rsrc_t raw_rsrc(const void* base, long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kRawRsrcWord3);
}

// Each lane copies the 16 bytes at voff + soff of the buffer into LDS at l + 16 * lane
// (l wave-uniform). The buffer form is a plain vector-memory instruction for the compiler's
// wait counting (the flat/global form makes it wait for every LDS read in flight).
MOLT_DEV void lds_dma16(__amdgpu_buffer_rsrc_t r, int voff, int soff, uint8_t* l) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)l, 16, voff, soff, 0, 0);
}

__global__ __launch_bounds__(kThreads) void bigtile_gemm_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t ring[kBigAStages * kBigAStage];
  const int total = p.n_mtiles * p.n_ntiles;
  const int chunk = (total + 7) / 8;
  const int k8 = blockIdx.x / 8;
  const int id = (blockIdx.x % 8) * chunk + k8;
  if (k8 >= chunk || id >= total) return;
  const int mt = id % p.n_mtiles, nt = id / p.n_mtiles;
  const int row0 = mt * kBigBM, n0 = nt * kBigBN;
  const long RB = long(p.K) * 2;
  const int nk = int(RB / kRowBytes);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int last_a = (p.M - 1) & ~31, last_b = (p.N - 1) & ~31;
  // byte offsets relative to the activation matrix and to this tile's first weight row; row
  // blocks past the end re-read the last one (their results are never stored)
  const __amdgpu_buffer_rsrc_t ra = raw_rsrc(p.A, long(last_a + 32) * RB);
  const __amdgpu_buffer_rsrc_t rb = raw_rsrc(static_cast<const uint8_t*>(p.B) + long(n0) * RB,
                                             long(min(n0 + kBigBN, last_b + 32) - n0) * RB);
  int avoff[kBigAB], bvoff[2];
#pragma unroll
  for (int j = 0; j < kBigAB; ++j) avoff[j] = int(min(row0 + 32 * j, last_a) * RB) + wave * 1024 + lane * 16;
#pragma unroll
  for (int j = 0; j < 2; ++j) bvoff[j] = int((min(n0 + 64 * wave + 32 * j, last_b) - n0) * RB) + lane * 16;
  // slices past the end re-copy the last one
  auto issue_a = [&](int kb) __attribute__((always_inline)) {
    const int soff = min(kb, nk - 1) * 4096;
    uint8_t* dst = ring + (kb % kBigAStages) * kBigAStage + wave * 1024;
#pragma unroll
    for (int j = 0; j < kBigAB; ++j) lds_dma16(ra, avoff[j], soff, dst + j * 4096);
  };
  typedef bf16x8_t BSlice[4][2];   // [k step][column block]
  auto load_b = [&](int kb, BSlice& b) __attribute__((always_inline)) {
    const int soff = min(kb, nk - 1) * 4096;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[c][j] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rb, bvoff[j] + c * 1024, soff, 0));
  };
  floatx16_t acc[kBigAB][2];
#pragma unroll
  for (int i = 0; i < kBigAB; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  // activation fragments of one k step, two register sets
  bf16x8_t af[2][kBigAB];
  auto frag = [&](const uint8_t* base, int c, int set) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kBigAB; ++i) af[set][i] = *reinterpret_cast<const bf16x8_t*>(base + i * 4096 + c * 1024);
  };
  auto step = [&](int set, const bf16x8_t (&b)[2]) __attribute__((always_inline)) {
    // the scheduler would otherwise sink the next step's reads below these MFMAs
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kBigAB; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma(af[set][i], b[j], acc[i][j]);
    __builtin_amdgcn_sched_barrier(0);
  };
  BSlice bs[kBigDepth];
  issue_a(0);
  issue_a(1);
  issue_a(2);
#pragma unroll
  for (int J = 0; J < kBigDepth; ++J) load_b(J, bs[J]);
  // slice 0's activations are in (what follows them in the queue may be in flight)
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(2 * kBigAB + kBigBLoads * kBigDepth) : "memory");
  frag(ring + lane * 16, 0, 0);
  // Per slice kb the vector-memory queue gets: activations kb + 3 (after the barrier), then
  // weights kb + depth (after the last MFMAs). The barrier of slice kb needs activations
  // kb + 1, issued in slice kb - 2; what may still be in flight behind them is at least
  // weights kb - 2 + depth, activations kb + 2 and weights kb - 1 + depth (exactly that from
  // slice 2 on, more before), so waiting for that many leaves it complete.
  constexpr int kAWait = 2 * kBigBLoads + kBigAB;
  auto body = [&](int kb, BSlice& b) __attribute__((always_inline)) {
    const uint8_t* base = ring + (kb % kBigAStages) * kBigAStage + lane * 16;
    frag(base, 1, 1);
    step(0, b[0]);
    frag(base, 2, 0);
    step(1, b[1]);
    frag(base, 3, 1);
    step(0, b[2]);
    // this wavefront's copies of slice kb + 1 are done and all its reads of slice kb - 1's
    // stage have returned: after the barrier slice kb + 1 is complete for everyone and that
    // stage takes slice kb + 3
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kAWait) : "memory");
    issue_a(kb + 3);
    frag(ring + ((kb + 1) % kBigAStages) * kBigAStage + lane * 16, 0, 0);
    step(1, b[3]);
    load_b(kb + kBigDepth, b);
  };
  int kb = 0;
  for (; kb + kBigDepth - 1 < nk; kb += kBigDepth) {   // register sets are indexed statically
#pragma unroll
    for (int J = 0; J < kBigDepth; ++J) body(kb + J, bs[J]);
  }
#pragma unroll
  for (int J = 0; J < kBigDepth - 1; ++J)
    if (kb + J < nk) body(kb + J, bs[J]);
  // no copy may still be writing into LDS when the workgroup ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // acc[i][j][e]: row 32 i + 8 (e / 4) + 4 lgrp + e % 4, column 64 wave + 32 j + lcol
  const int lcol = lane % 32, lgrp = lane / 32;
  float* C = static_cast<float*>(p.C);
  if (!p.accumulate && row0 + kBigBM <= p.M && n0 + kBigBN <= p.N) {
    // whole tile (all but the last column tile): no bounds checks between the stores (the
    // LM head: 451 -> 411 us; nontemporal stores measured 420 us; without any stores 370 us:
    // the tiles of a round end together and their 40 MB of logits go out in one burst)
    float* base = C + long(row0 + 4 * lgrp) * p.ldc + n0 + 64 * wave + lcol;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < kBigAB; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) base[long(32 * i + 8 * (e / 4) + (e % 4)) * p.ldc + 32 * j] = acc[i][j][e];
    return;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = n0 + 64 * wave + 32 * j + lcol;
    if (col >= p.N) continue;
#pragma unroll
    for (int i = 0; i < kBigAB; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int grow = row0 + 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
        if (grow >= p.M) continue;
        float* dst = C + long(grow) * p.ldc + col;
        *dst = p.accumulate ? *dst + acc[i][j][e] : acc[i][j][e];
      }
  }
}

// C (+)= sum over s of part[s], in split order
__global__ __launch_bounds__(kThreads) void splitk_reduce_kernel(const float* __restrict__ part,
                                                                 int splits, long n, float* __restrict__ C,
                                                                 int accumulate) {
  const long i = long(blockIdx.x) * kThreads + threadIdx.x;
  if (i >= n) return;
  float v = accumulate ? C[i] : 0.f;
  for (int s = 0; s < splits; ++s) v += part[s * n + i];
  C[i] = v;
}

// ---------------------------------------------------------------- tiled-layout kernels
// pack: row-major [rows, RB bytes] -> tiled with rows padded to a multiple of 32 (padding
// rows zero); one thread per 16-byte chunk of the destination
__global__ __launch_bounds__(kThreads) void pack_tiled_kernel(const uint8_t* __restrict__ src,
                                                              uint8_t* __restrict__ dst, long rows,
                                                              long RB) {
  const long q = long(blockIdx.x) * kThreads + threadIdx.x;
  const long per_row = RB / 16;
  const long padded = (rows + 31) / 32 * 32;
  if (q >= padded * per_row) return;
  const long r = q / per_row, j = (q % per_row) * 16;
  int4 v = make_int4(0, 0, 0, 0);
  if (r < rows) v = *reinterpret_cast<const int4*>(src + r * RB + j);
  *reinterpret_cast<int4*>(dst + tiled_offset(r, j, RB)) = v;
}

// gather: tiled activation rows in padded expert order from tiled token rows,
// row = src[pperm[row] / ktop]; one workgroup per 4 KB tile of the destination, thread =
// 16-byte chunk of it. Padding rows are left unwritten: a GEMM output row depends on its
// own operand row only, and the rows computed from padding are never stored. (Workgroups
// over 8 slices of a 32-row block, each thread with 8 loads in flight, took twice as long.)
__global__ __launch_bounds__(kThreads) void gather_tiled_kernel(
    const uint8_t* __restrict__ src, const int32_t* __restrict__ pperm, int ktop,
    const int32_t* __restrict__ n_rows, long RB, uint8_t* __restrict__ dst) {
  const long tile = blockIdx.x;
  const long nk = RB / 128;
  const long rb = tile / nk, kb = tile % nk;
  if (rb * 32 >= *n_rows) return;
  const int quarter = threadIdx.x / 64, l = threadIdx.x % 64;
  const long row = rb * 32 + (l % 32);
  const long j = kb * 128 + (l / 32) * 64 + quarter * 16;
  const int pair = pperm[row];
  if (pair < 0) return;
  *reinterpret_cast<int4*>(dst + tile * 4096 + threadIdx.x * 16) =
      *reinterpret_cast<const int4*>(src + tiled_offset(pair / ktop, j, RB));
}

// ---------------------------------------------------------------- f32 VALU path
// One workgroup per (row tile of 16, column tile of 64); each thread owns 4 outputs.
// Operands tiled as in the MFMA path (f32 element k of row n at byte 4k).
template <int MODE>
__global__ __launch_bounds__(kThreads) void f32_gemm_kernel(GemmParams p) {
  const int id = blockIdx.x;
  const int mt = id % p.n_mtiles, nt = id / p.n_mtiles;
  int expert = 0, row0, row1;
  if (MODE == kDense) {
    row0 = mt * 16;
    row1 = min(row0 + 16, p.M);
  } else {
    const int4 t = p.tiles[mt];
    if (t.x < 0) return;
    expert = t.x;
    row0 = t.y;
    row1 = t.z;
  }
  const int K = p.K;
  const float* A = static_cast<const float*>(p.A);
  const float* B = static_cast<const float*>(p.B);
  for (int o = threadIdx.x; o < 16 * 64; o += kThreads) {
    const int r = o / 64, c = o % 64;
    const int grow = row0 + r;
    const int col = nt * 64 + c;
    if (grow >= row1 || col >= p.N) continue;
    auto a = [&](int kk) { return A[tiled_index(grow, kk, K, 4)]; };
    if (MODE == kGateUp) {
      const long ng = long(expert) * 2 * p.N + col, nu = ng + p.N;
      float g = 0.f, u = 0.f;
      for (int kk = 0; kk < K; ++kk) {
        g += a(kk) * B[tiled_index(ng, kk, K, 4)];
        u += a(kk) * B[tiled_index(nu, kk, K, 4)];
      }
      static_cast<float*>(p.C)[tiled_index(grow, col, p.N, 4)] = silu(g) * u;
    } else {
      const long n = (MODE == kDown ? long(expert) * p.N : 0) + col;
      float s = 0.f;
      for (int kk = 0; kk < K; ++kk) s += a(kk) * B[tiled_index(n, kk, K, 4)];
      const long crow = MODE == kDown ? long(p.perm[grow]) : long(grow);
      float* dst = static_cast<float*>(p.C) + crow * p.ldc + col;
      if (MODE == kDense && p.accumulate) s += *dst;
      *dst = s;
    }
  }
}

}  // namespace

// Row-tile height of the grouped expert GEMMs: large enough that an expert of average load
// fits one tile (its weights are then streamed once), as small as that allows.
int moe_tile_m(molt_dtype wdt, int T, int K, int E) {
  if (wdt == MOLT_F32) return 16;
  const long avg = (long(T) * K + E - 1) / E;
  return avg <= 24 ? 32 : avg <= 56 ? 64 : 128;
}

// Tile height and split-K count of a dense bf16 GEMM: 128-row tiles when there are plenty
// of them, else 64; then the K range is halved while the grid is under one workgroup per
// CU, each split keeps >= 4 slices and the partial sums fit `part_elems` floats.
GemmPlan gemm_plan(int M, int N, int K, long part_elems) {
  GemmPlan g{128, 1};
  const long nt = (N + kBN - 1) / kBN;
  if ((M + 127) / 128 * nt < 512) g.bm = 64;
  const long wg = (M + g.bm - 1) / g.bm * nt;
  const int nk = int(2L * K / kRowBytes);
  while (wg * g.splits < 256 && nk / (2 * g.splits) >= 4 && 2L * g.splits * M * N <= part_elems)
    g.splits *= 2;
  return g;
}

hipError_t launch_gemm(const void* A, const void* Bw, float* C, int M, int N, int K, molt_dtype dt,
                       bool accumulate, float* part, long part_elems, hipStream_t s,
                       int* splits_out) {
  if (splits_out) *splits_out = 1;
  GemmParams p{};
  p.A = A; p.B = Bw; p.C = C; p.M = M; p.N = N; p.K = K; p.ldc = N;
  p.accumulate = accumulate;
  if (dt == MOLT_F32) {
    p.n_mtiles = (M + 15) / 16;
    p.n_ntiles = (N + 63) / 64;
    f32_gemm_kernel<kDense><<<p.n_mtiles * p.n_ntiles, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  if (dt == MOLT_BF16 && !accumulate && M <= 128 && N >= 8192 && N % kBN == 0) {
    // few rows and many columns (the draft head's LM head, one row per sequence): every
    // weight element is used by one row tile only, so the grouped GEMM's weight-streaming
    // kernel in down mode takes it as one "expert" holding all rows (no tile table: one row
    // tile, output row = input row); the 128 x 128 LDS kernel read the weights at about
    // half of HBM bandwidth
    p.tiles = nullptr; p.n_tiles_live = nullptr; p.perm = nullptr;
    p.n_mtiles = 1;
    p.n_ntiles = N / kBN;
    return run_stream<false, kDown>(p, M <= 32 ? 32 : M <= 64 ? 64 : 128, s);
  }
  if (M >= kBigBM && N >= 8192 && long((M + kBigBM - 1) / kBigBM) * ((N + kBigBN - 1) / kBigBN) >= 512 &&
      long(M + 31) * 2 * K < (1L << 31) && long(kBigBN) * 2 * K < (1L << 31)) {
    // many more columns than rows (the LM head): big tiles fed by LDS-DMA (32-bit buffer
    // offsets: the activations and one tile's weights under 2 GB). Below 160 rows (the
    // draft head's LM head: 128) the 128 x 128 LDS kernel measured 5% faster.
    p.n_mtiles = (M + kBigBM - 1) / kBigBM;
    p.n_ntiles = (N + kBigBN - 1) / kBigBN;
    const int grid = (p.n_mtiles * p.n_ntiles + 7) / 8 * 8;
    bigtile_gemm_kernel<<<grid, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  const GemmPlan g = gemm_plan(M, N, K, part_elems);
  p.n_mtiles = (M + g.bm - 1) / g.bm;
  p.n_ntiles = (N + kBN - 1) / kBN;
  const int grid = (p.n_mtiles * p.n_ntiles * g.splits + 7) / 8 * 8;
  // small grids (under two workgroups per CU): 8 wavefronts of 32 x 32 per tile, two per SIMD
  if (g.bm == 64) lds_gemm_kernel<64, false, 4, 2><<<grid, 512, 0, s>>>(p, part, g.splits, RopeKv{});
  else lds_gemm_kernel<128, false, 2, 2><<<grid, kThreads, 0, s>>>(p, part, g.splits, RopeKv{});
  if (g.splits > 1 && splits_out) {
    *splits_out = g.splits;         // the caller adds part[0 .. splits) (in order) into C
  } else if (g.splits > 1) {
    const long n = long(M) * N;
    splitk_reduce_kernel<<<(n + kThreads - 1) / kThreads, kThreads, 0, s>>>(part, g.splits, n, C,
                                                                             accumulate);
  }
  return hipGetLastError();
}

hipError_t launch_qkv_rope(const void* A, const void* Bw, int M, int K_in, int Hq, int Hkv,
                           const void* table, const int32_t* kv_slot, void* q_out, void* k_cache,
                           void* v_cache, hipStream_t s) {
  GemmParams p{};
  p.A = A; p.B = Bw; p.M = M; p.N = (Hq + 2 * Hkv) * 128; p.K = K_in; p.ldc = p.N;
  RopeKv rk{static_cast<const double2*>(table), kv_slot, Hq, Hkv, static_cast<uint16_t*>(q_out),
            static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache)};
  const GemmPlan g = gemm_plan(M, p.N, K_in, 0);     // no split: the epilogue needs whole sums
  p.n_mtiles = (M + g.bm - 1) / g.bm;
  p.n_ntiles = Hq + 2 * Hkv;
  const int grid = (p.n_mtiles * p.n_ntiles + 7) / 8 * 8;
  if (g.bm == 64) lds_gemm_kernel<64, true, 4, 2><<<grid, 512, 0, s>>>(p, nullptr, 1, rk);
  else lds_gemm_kernel<128, true, 2, 2><<<grid, kThreads, 0, s>>>(p, nullptr, 1, rk);
  return hipGetLastError();
}

hipError_t launch_moe_gate_up(const void* a, const void* a_rows, const float* a_scale,
                              const int32_t* pperm, int K_top, const void* w_gu, const float* s_gu,
                              int d, int F, molt_dtype wdt, const int32_t* tiles,
                              const int32_t* n_tiles, int max_tiles, int tile_m, void* h,
                              hipStream_t s) {
  GemmParams p{};
  p.n_tiles_live = n_tiles;
  p.A = a_rows != nullptr && wdt != MOLT_F32 ? a_rows : a;
  p.B = w_gu; p.C = h; p.N = F; p.K = d; p.ldc = F;
  p.tiles = reinterpret_cast<const int4*>(tiles);
  p.n_mtiles = max_tiles;
  p.perm = pperm; p.ktop = K_top;
  p.a_scale = a_scale; p.b_scale = s_gu; p.b_scale_ld = 2 * F;
  if (wdt == MOLT_F32) {
    p.n_ntiles = (F + 63) / 64;
    f32_gemm_kernel<kGateUp><<<max_tiles * p.n_ntiles, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  p.n_ntiles = F / (kBN / 2);
  p.queue = const_cast<int32_t*>(n_tiles) + 1;
  if (wdt == MOLT_FP8_E4M3) return run_stream<true, kGateUp>(p, tile_m, s, a_rows != nullptr);
  return run_stream<false, kGateUp>(p, tile_m, s, a_rows != nullptr);
}

hipError_t launch_moe_down(const void* a, const float* a_scale, const int32_t* pperm,
                           const void* w_d, const float* s_d, int d, int F, molt_dtype wdt,
                           const int32_t* tiles, const int32_t* n_tiles, int max_tiles,
                           int tile_m, float* o, hipStream_t s) {
  GemmParams p{};
  p.n_tiles_live = n_tiles;
  p.A = a; p.B = w_d; p.C = o; p.N = d; p.K = F; p.ldc = d;
  p.tiles = reinterpret_cast<const int4*>(tiles);
  p.n_mtiles = max_tiles;
  p.perm = pperm;
  p.a_scale = a_scale; p.b_scale = s_d; p.b_scale_ld = d;
  if (wdt == MOLT_F32) {
    p.n_ntiles = (d + 63) / 64;
    f32_gemm_kernel<kDown><<<max_tiles * p.n_ntiles, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  p.n_ntiles = d / kBN;
  p.queue = const_cast<int32_t*>(n_tiles) + 1 + kTileQueues;
  if (wdt == MOLT_FP8_E4M3) return run_stream<true, kDown>(p, tile_m, s);
  return run_stream<false, kDown>(p, tile_m, s);
}

hipError_t launch_pack_tiled(const void* src, void* dst, long rows, long row_bytes, hipStream_t s) {
  const long chunks = (rows + 31) / 32 * 32 * (row_bytes / 16);
  if (chunks == 0) return hipSuccess;
  pack_tiled_kernel<<<(chunks + kThreads - 1) / kThreads, kThreads, 0, s>>>(
      static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), rows, row_bytes);
  return hipGetLastError();
}

hipError_t launch_gather_tiled(const void* src, const int32_t* pperm, int K_top,
                               const int32_t* n_rows, long max_rows, long row_bytes, void* dst,
                               hipStream_t s) {
  const long tiles = max_rows / 32 * (row_bytes / 128);
  if (tiles == 0) return hipSuccess;
  gather_tiled_kernel<<<tiles, kThreads, 0, s>>>(static_cast<const uint8_t*>(src), pperm, K_top,
                                                 n_rows, row_bytes, static_cast<uint8_t*>(dst));
  return hipGetLastError();
}

}  // namespace molt
