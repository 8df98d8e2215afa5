// GEMMs of the verify step on gfx950 MFMA: dense projections (QKV, O, router, LM head)
// and the grouped expert GEMMs of the top-K routed MoE (gate_up with a fused SwiGLU
// epilogue, down), in bf16 (v_mfma_f32_32x32x16_bf16) or fp8 e4m3 with f32 per-row x
// per-channel scales (v_mfma_f32_32x32x64_f8f6f4), f32 accumulation.
//
// One kernel template: a workgroup of 4 wavefronts computes a BM x 128 output tile,
// staging 128-byte K-slices of A (BM rows) and B (128 weight rows) through LDS with
// double buffering (rows padded to 144 B so the 16-lane phases of ds_read_b128 hit 16
// distinct bank groups). A rows are gathered: dense rows, token rows via the expert
// permutation (gate_up), or the expert's contiguous rows (down). Grouped launches run
// over a device-side tile table (expert, first row, end row) built by the permutation
// kernel, so the host never reads expert counts; unused table slots exit at once.
// All matrices are row-major with K contiguous (weights [out, in]).
//
// The f32 model (tiny test model) takes a plain VALU path with the same epilogues.
#include "device_common.h"
#include "internal.h"

namespace molt {
namespace {

constexpr int kThreads = 256;
constexpr int kBN = 128;         // output columns per tile (gate_up: 64 gate + 64 up)
constexpr int kRowBytes = 128;   // K-slice per stage, bytes
constexpr int kLdsStride = 144;  // padded LDS row

enum Mode { kDense = 0, kGateUp = 1, kDown = 2 };

struct GemmParams {
  const void* A;           // dense: [M, K]; gate_up: tokens [T, K] (x or fp8 codes); down: h [P, K]
  const void* B;           // dense: [N, K]; gate_up: [E, 2F, K]; down: [E, N, K]
  void* C;                 // dense/down: f32 [.., ldc]; gate_up: h [P, F] (act dtype)
  int M, N, K;             // N: output columns (gate_up: F)
  int ldc;
  const int4* tiles;       // grouped: {expert, row0, row1, -}
  const int32_t* n_tiles_live;   // grouped (device): entries of `tiles` in use
  int n_mtiles, n_ntiles;
  const int32_t* perm;     // gate_up: permuted pair -> token * ktop + slot
  int ktop;
  const float* a_scale;    // fp8: per A row (token for gate_up, permuted row for down)
  const float* b_scale;    // fp8: [E, b_scale_ld]
  int b_scale_ld;
  int accumulate;          // dense: C += result
  int xcd_remap;
};

// MFMA operand fragment types
template <bool FP8> struct Frag;
template <> struct Frag<false> { typedef bf16x8_t T; };
template <> struct Frag<true> { typedef int32x8_t T; };

MOLT_DEV floatx16_t mfma(const bf16x8_t& a, const bf16x8_t& b, const floatx16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
MOLT_DEV floatx16_t mfma(const int32x8_t& a, const int32x8_t& b, const floatx16_t& c) {
  // cbsz = blgp = 0: both operands fp8 e4m3; zero scale operands select the unscaled op
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

template <int BM>
struct WaveLayout {
  static constexpr int WM = BM >= 128 ? 2 : 1;   // wavefronts along M
  static constexpr int WN = 4 / WM;              // wavefronts along N
  static constexpr int TM = BM / WM / 32;        // 32x32 MFMA tiles per wave along M
  static constexpr int TN = kBN / WN / 32;       // ... along N
};

template <int BM, bool FP8, int MODE>
__global__ __launch_bounds__(kThreads) void mfma_gemm_kernel(GemmParams p) {
  typedef WaveLayout<BM> L;
  constexpr int kElem = FP8 ? 1 : 2;
  constexpr int kBK = kRowBytes / kElem;              // K elements per stage
  constexpr int kARows = BM / 32, kBRows = kBN / 32;  // 16-byte loads per thread
  constexpr int kStage = (BM + kBN) * kLdsStride;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kStage];

  // ---- which tile
  int id = blockIdx.x;
  const int G = gridDim.x;
  if (p.xcd_remap && (G % 8) == 0) id = (id % 8) * (G / 8) + id / 8;  // same XCD: neighbours
  const int mt = id % p.n_mtiles;
  const int nt = id / p.n_mtiles;
  int expert = 0, row0, row1;
  if (MODE == kDense) {
    row0 = mt * BM;
    row1 = min(row0 + BM, p.M);
  } else {
    const int4 tinfo = p.tiles[mt];
    if (tinfo.x < 0) return;
    expert = tinfo.x;
    row0 = tinfo.y;
    row1 = tinfo.z;
  }
  const int n0 = (MODE == kGateUp) ? nt * (kBN / 2) : nt * kBN;
  const long K = p.K;

  // ---- per-thread global row pointers (16-byte chunk c of rows r = tid/8 + 32 i)
  const int chunk = threadIdx.x % 8;
  const uint8_t* a_src[kARows];
  const uint8_t* b_src[kBRows];
#pragma unroll
  for (int i = 0; i < kARows; ++i) {
    const int r = threadIdx.x / 8 + 32 * i;
    const int grow = row0 + r;
    a_src[i] = nullptr;
    if (grow < row1) {
      long arow = grow;
      if (MODE == kGateUp) arow = p.perm[grow] / p.ktop;
      a_src[i] = static_cast<const uint8_t*>(p.A) + (arow * K) * kElem + chunk * 16;
    }
  }
#pragma unroll
  for (int i = 0; i < kBRows; ++i) {
    const int r = threadIdx.x / 8 + 32 * i;
    long brow;
    bool ok = true;
    if (MODE == kGateUp) {
      brow = long(expert) * 2 * p.N + (r < kBN / 2 ? n0 + r : p.N + n0 + r - kBN / 2);
    } else if (MODE == kDown) {
      brow = long(expert) * p.N + n0 + r;
    } else {
      brow = n0 + r;
      ok = n0 + r < p.N;
    }
    b_src[i] = ok ? static_cast<const uint8_t*>(p.B) + (brow * K) * kElem + chunk * 16 : nullptr;
  }

  int4 ra[kARows], rb[kBRows];
  auto gload = [&](int kb) {
    const long off = long(kb) * kRowBytes;
#pragma unroll
    for (int i = 0; i < kARows; ++i)
      ra[i] = a_src[i] ? *reinterpret_cast<const int4*>(a_src[i] + off) : make_int4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < kBRows; ++i)
      rb[i] = b_src[i] ? *reinterpret_cast<const int4*>(b_src[i] + off) : make_int4(0, 0, 0, 0);
  };
  auto sstore = [&](int buf) {
    uint8_t* base = lds + buf * kStage;
#pragma unroll
    for (int i = 0; i < kARows; ++i)
      *reinterpret_cast<int4*>(base + (threadIdx.x / 8 + 32 * i) * kLdsStride + chunk * 16) = ra[i];
#pragma unroll
    for (int i = 0; i < kBRows; ++i)
      *reinterpret_cast<int4*>(base + (BM + threadIdx.x / 8 + 32 * i) * kLdsStride + chunk * 16) = rb[i];
  };

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int wm = wave / L::WN, wn = wave % L::WN;
  const int wrow = wm * (BM / L::WM), wcol = wn * (kBN / L::WN);
  floatx16_t acc[L::TM][L::TN];
#pragma unroll
  for (int i = 0; i < L::TM; ++i)
#pragma unroll
    for (int j = 0; j < L::TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int nk = int(K / kBK);
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kb = 0; kb < nk; ++kb) {
    if (kb + 1 < nk) gload(kb + 1);
    const uint8_t* base = lds + (kb & 1) * kStage;
    const int lrow = lane % 32, lhalf = lane / 32;
    if (!FP8) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {  // 4 k-steps of 16
        bf16x8_t af[L::TM], bfr[L::TN];
#pragma unroll
        for (int i = 0; i < L::TM; ++i)
          af[i] = *reinterpret_cast<const bf16x8_t*>(base + (wrow + i * 32 + lrow) * kLdsStride + s * 32 + lhalf * 16);
#pragma unroll
        for (int j = 0; j < L::TN; ++j)
          bfr[j] = *reinterpret_cast<const bf16x8_t*>(base + (BM + wcol + j * 32 + lrow) * kLdsStride + s * 32 + lhalf * 16);
#pragma unroll
        for (int i = 0; i < L::TM; ++i)
#pragma unroll
          for (int j = 0; j < L::TN; ++j) acc[i][j] = mfma(af[i], bfr[j], acc[i][j]);
      }
    } else {
#pragma unroll
      for (int s = 0; s < 2; ++s) {  // 2 k-steps of 64
        int32x8_t af[L::TM], bfr[L::TN];
#pragma unroll
        for (int i = 0; i < L::TM; ++i) {
          const uint8_t* q = base + (wrow + i * 32 + lrow) * kLdsStride + s * 64 + lhalf * 32;
          int32x4_t lo = *reinterpret_cast<const int32x4_t*>(q);
          int32x4_t hi = *reinterpret_cast<const int32x4_t*>(q + 16);
          af[i] = int32x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
#pragma unroll
        for (int j = 0; j < L::TN; ++j) {
          const uint8_t* q = base + (BM + wcol + j * 32 + lrow) * kLdsStride + s * 64 + lhalf * 32;
          int32x4_t lo = *reinterpret_cast<const int32x4_t*>(q);
          int32x4_t hi = *reinterpret_cast<const int32x4_t*>(q + 16);
          bfr[j] = int32x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
#pragma unroll
        for (int i = 0; i < L::TM; ++i)
#pragma unroll
          for (int j = 0; j < L::TN; ++j) acc[i][j] = mfma(af[i], bfr[j], acc[i][j]);
      }
    }
    if (kb + 1 < nk) sstore((kb + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue. acc[i][j][e] holds row wrow+32i+8(e/4)+4(lane/32)+e%4, col wcol+32j+lane%32
  const int lcol = lane % 32, lgrp = lane / 32;
  if (MODE == kGateUp) {
    // waves holding "up" columns (tile cols 64..127) park them in LDS; the "gate" waves
    // finish h = silu(gate) * up for their columns
    float* upbuf = reinterpret_cast<float*>(lds);   // [BM][64]
    const bool is_up = wcol >= kBN / 2;
    if (is_up) {
#pragma unroll
      for (int i = 0; i < L::TM; ++i)
#pragma unroll
        for (int j = 0; j < L::TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int r = wrow + 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
            const int c = wcol - kBN / 2 + 32 * j + lcol;
            upbuf[r * 64 + c] = acc[i][j][e];
          }
    }
    __syncthreads();
    if (!is_up) {
#pragma unroll
      for (int i = 0; i < L::TM; ++i)
#pragma unroll
        for (int j = 0; j < L::TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int r = wrow + 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
            const int c = wcol + 32 * j + lcol;
            const int grow = row0 + r;
            if (grow >= row1) continue;
            float g = acc[i][j][e], u = upbuf[r * 64 + c];
            if (FP8) {
              const float sx = p.a_scale[p.perm[grow] / p.ktop];
              const float* sw = p.b_scale + long(expert) * p.b_scale_ld;
              g = g * sx * sw[n0 + c];
              u = u * sx * sw[p.N + n0 + c];
            }
            const float h = silu(g) * u;
            static_cast<uint16_t*>(p.C)[long(grow) * p.ldc + n0 + c] = f32_to_bf16(h);
          }
    }
  } else {
#pragma unroll
    for (int i = 0; i < L::TM; ++i)
#pragma unroll
      for (int j = 0; j < L::TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = wrow + 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
          const int c = n0 + wcol + 32 * j + lcol;
          const int grow = row0 + r;
          if (grow >= row1 || c >= p.N) continue;
          float v = acc[i][j][e];
          if (FP8) v = v * p.a_scale[grow] * p.b_scale[long(expert) * p.b_scale_ld + c];
          float* dst = static_cast<float*>(p.C) + long(grow) * p.ldc + c;
          if (MODE == kDense && p.accumulate) v += *dst;
          *dst = v;
        }
  }
}

// ---------------------------------------------------------------- weight-streaming grouped GEMM
// Expert GEMMs are HBM-bound at the verify step's row counts (tens of rows per expert),
// so the weights must stream at full bandwidth and be read once. Workgroup = BM rows of
// one expert x 128 output columns; each of the 4 wavefronts owns 32 output columns (32
// weight rows) and loads its weight fragments straight from global memory into MFMA
// operand registers, kPD 128-byte K slices ahead; a weight element is used by exactly one
// wavefront, so no LDS and no barrier is needed in the main loop. The activation rows
// (shared by the 4 wavefronts, served from L2) are loaded per wavefront kPA slices ahead.
// Both operands are in the tiled layout, so every load instruction reads 1 KB of one page:
// with row-major operands each instruction touched 32 rows, and the address translation
// requests, not HBM, set the pace. Tiles start at multiples of 32 rows (padded expert
// order), so each 32-row block of A is one tile column of the tiled activation buffer.
struct Slice16 { int4 c[4]; };   // one lane's 64 bytes of a 32-row x 128-byte tile

template <int BM, bool FP8, int MODE>
__global__ __launch_bounds__(kThreads) void moe_stream_kernel(GemmParams p) {
  static_assert(MODE == kGateUp || MODE == kDown, "grouped modes only");
  constexpr int MS = BM / 32;                        // 32-row MFMA tiles per wavefront
  constexpr int kPD = 4;                             // weight slices in flight
  constexpr int kPA = 2;                             // activation slices in flight
  constexpr int kElem = FP8 ? 1 : 2;
  __shared__ __attribute__((aligned(16))) float upbuf[MODE == kGateUp ? BM * 64 : 1];

  // Workgroup b runs on XCD b % 8. Each XCD takes one contiguous eighth of the live
  // (m-tile, n-tile) pairs, m-tile major: the n-tiles of one row tile run back to back on
  // one XCD, so its activation tile is read from HBM once and then hits that XCD's L2.
  const int total = *p.n_tiles_live * p.n_ntiles;
  const int chunk = (total + 7) / 8;
  const int k8 = blockIdx.x / 8;
  const int id = (blockIdx.x % 8) * chunk + k8;
  if (k8 >= chunk || id >= total) return;
  const int mt = id / p.n_ntiles;
  const int nt = id % p.n_ntiles;
  const int4 t = p.tiles[mt];
  const int expert = t.x, row0 = t.y, row1 = t.z;     // row0 % 32 == 0
  const long RB = long(p.K) * kElem;                  // bytes per operand row
  const int nk = int(RB / kRowBytes);                 // 128-byte K slices
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  // first of the wavefront's 32 weight rows (gate_up: waves 0-1 gate, 2-3 up)
  long wrow;
  int n0;
  if (MODE == kGateUp) {
    n0 = nt * (kBN / 2);
    wrow = long(expert) * 2 * p.N + (wave < 2 ? n0 + 32 * wave : p.N + n0 + 32 * (wave - 2));
  } else {
    n0 = nt * kBN;
    wrow = long(expert) * p.N + n0 + 32 * wave;
  }
  const uint8_t* bsrc = static_cast<const uint8_t*>(p.B) + wrow * RB + lane * 16;
  const uint8_t* asrc[MS];
  const int last_block = (row1 - 1) & ~31;            // 32-row blocks past the tile end
#pragma unroll                                        // re-read its last one
  for (int i = 0; i < MS; ++i)
    asrc[i] = static_cast<const uint8_t*>(p.A) + long(min(row0 + 32 * i, last_block)) * RB + lane * 16;
  auto ld = [](Slice16& f, const uint8_t* src) {
#pragma unroll
    for (int c = 0; c < 4; ++c) f.c[c] = *reinterpret_cast<const int4*>(src + 1024 * c);
  };
  Slice16 wb[kPD];
  Slice16 ab[kPA][MS];
#pragma unroll
  for (int s = 0; s < kPD; ++s) if (s < nk) ld(wb[s], bsrc + long(s) * 4096);
#pragma unroll
  for (int s = 0; s < kPA; ++s) if (s < nk)
#pragma unroll
    for (int i = 0; i < MS; ++i) ld(ab[s][i], asrc[i] + long(s) * 4096);
  floatx16_t acc[MS];
#pragma unroll
  for (int i = 0; i < MS; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;
  auto slice = [&](const Slice16& w, const Slice16 (&a)[MS]) {
    if (!FP8) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(&w.c[s]);
#pragma unroll
        for (int i = 0; i < MS; ++i) acc[i] = mfma(*reinterpret_cast<const bf16x8_t*>(&a[i].c[s]), bv, acc[i]);
      }
    } else {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int4 w0 = w.c[2 * s], w1 = w.c[2 * s + 1];
        const int32x8_t bv = int32x8_t{w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
        for (int i = 0; i < MS; ++i) {
          const int4 lo = a[i].c[2 * s], hi = a[i].c[2 * s + 1];
          acc[i] = mfma(int32x8_t{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w}, bv, acc[i]);
        }
      }
    }
  };
  for (int kb0 = 0; kb0 < nk; kb0 += kPD) {
#pragma unroll
    for (int s = 0; s < kPD; ++s) {
      const int kb = kb0 + s;
      if (kb < nk) {
        slice(wb[s], ab[s % kPA]);
        if (kb + kPD < nk) ld(wb[s], bsrc + long(kb + kPD) * 4096);
        if (kb + kPA < nk)
#pragma unroll
          for (int i = 0; i < MS; ++i) ld(ab[s % kPA][i], asrc[i] + long(kb + kPA) * 4096);
      }
    }
  }
  // accumulator element e of lane (lcol, lgrp) in tile i: row 32 i + 8 (e / 4) + 4 lgrp + e % 4
  const int lcol = lane % 32, lgrp = lane / 32;
  if (MODE == kGateUp) {
    // h = silu(gate) * up, bf16, tiled layout over padded rows; up columns go through LDS
    if (wave >= 2) {
#pragma unroll
      for (int i = 0; i < MS; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
          upbuf[r * 64 + 32 * (wave - 2) + lcol] = acc[i][e];
        }
    }
    __syncthreads();
    if (wave < 2) {
      const int c = 32 * wave + lcol;
      const long hrb = 2L * p.N;
#pragma unroll
      for (int i = 0; i < MS; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
          const int grow = row0 + r;
          if (grow >= row1) continue;
          float g = acc[i][e], u = upbuf[r * 64 + c];
          if (FP8) {
            const float sx = p.a_scale[p.perm[grow] / p.ktop];
            const float* sw = p.b_scale + long(expert) * p.b_scale_ld;
            g = g * sx * sw[n0 + c];
            u = u * sx * sw[p.N + n0 + c];
          }
          *reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(p.C) +
                                       tiled_offset(grow, 2L * (n0 + c), hrb)) = f32_to_bf16(silu(g) * u);
        }
    }
  } else {
    // per-pair expert output, f32, row = pair index (token * K + slot)
    const int c = n0 + 32 * wave + lcol;
#pragma unroll
    for (int i = 0; i < MS; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = 32 * i + 8 * (e / 4) + 4 * lgrp + (e % 4);
        const int grow = row0 + r;
        if (grow >= row1) continue;
        float v = acc[i][e];
        if (FP8) v = v * p.a_scale[grow] * p.b_scale[long(expert) * p.b_scale_ld + c];
        static_cast<float*>(p.C)[long(p.perm[grow]) * p.ldc + c] = v;
      }
  }
}

template <bool FP8, int MODE>
hipError_t run_stream(GemmParams p, int tile_m, hipStream_t s) {
  int grid = p.n_mtiles * p.n_ntiles;
  grid = (grid + 7) / 8 * 8;
  if (tile_m == 32) moe_stream_kernel<32, FP8, MODE><<<grid, kThreads, 0, s>>>(p);
  else if (tile_m == 64) moe_stream_kernel<64, FP8, MODE><<<grid, kThreads, 0, s>>>(p);
  else moe_stream_kernel<128, FP8, MODE><<<grid, kThreads, 0, s>>>(p);
  return hipGetLastError();
}

// ---------------------------------------------------------------- tiled-layout kernels
// pack: row-major [rows, RB bytes] -> tiled; one thread per 16-byte chunk (reads coalesced)
__global__ __launch_bounds__(kThreads) void pack_tiled_kernel(const uint8_t* __restrict__ src,
                                                              uint8_t* __restrict__ dst, long rows,
                                                              long RB) {
  const long q = long(blockIdx.x) * kThreads + threadIdx.x;
  const long per_row = RB / 16;
  if (q >= rows * per_row) return;
  const long r = q / per_row, j = (q % per_row) * 16;
  *reinterpret_cast<int4*>(dst + tiled_offset(r, j, RB)) =
      *reinterpret_cast<const int4*>(src + r * RB + j);
}

// gather: tiled activation rows in padded expert order, row = src[pperm[row] / ktop]
// (zeros for padding rows); one workgroup per 4 KB tile, thread = 16-byte chunk of it
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
  int4 v = make_int4(0, 0, 0, 0);
  if (pair >= 0) v = *reinterpret_cast<const int4*>(src + long(pair / ktop) * RB + j);
  *reinterpret_cast<int4*>(dst + tile * 4096 + threadIdx.x * 16) = v;
}

// ---------------------------------------------------------------- f32 VALU path
// One workgroup per (row tile of 16, column tile of 64); each thread owns 4 outputs.
// Dense: row-major operands. Grouped: weights tiled (f32 element k of row n at byte 4k),
// activations row-major, rows in padded expert order (gate_up reads token rows through
// the padded permutation; down writes pair rows).
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
  const long RB = 4L * K;
  const float* A = static_cast<const float*>(p.A);
  const uint8_t* B = static_cast<const uint8_t*>(p.B);
  auto w = [&](long n, int kk) { return *reinterpret_cast<const float*>(B + tiled_offset(n, 4L * kk, RB)); };
  for (int o = threadIdx.x; o < 16 * 64; o += kThreads) {
    const int r = o / 64, c = o % 64;
    const int grow = row0 + r;
    const int col = nt * 64 + c;
    if (grow >= row1 || col >= p.N) continue;
    if (MODE == kDense) {
      const float* a = A + long(grow) * K;
      const float* b = static_cast<const float*>(p.B) + long(col) * K;
      float s = 0.f;
      for (int kk = 0; kk < K; ++kk) s += a[kk] * b[kk];
      float* dst = static_cast<float*>(p.C) + long(grow) * p.ldc + col;
      if (p.accumulate) s += *dst;
      *dst = s;
    } else if (MODE == kGateUp) {
      const float* a = A + long(p.perm[grow] / p.ktop) * K;
      const long ng = long(expert) * 2 * p.N + col, nu = ng + p.N;
      float g = 0.f, u = 0.f;
      for (int kk = 0; kk < K; ++kk) {
        g += a[kk] * w(ng, kk);
        u += a[kk] * w(nu, kk);
      }
      static_cast<float*>(p.C)[long(grow) * p.ldc + col] = silu(g) * u;
    } else {
      const float* a = A + long(grow) * K;
      const long n = long(expert) * p.N + col;
      float s = 0.f;
      for (int kk = 0; kk < K; ++kk) s += a[kk] * w(n, kk);
      static_cast<float*>(p.C)[long(p.perm[grow]) * p.ldc + col] = s;
    }
  }
}

template <int BM, bool FP8, int MODE>
hipError_t run_mfma(GemmParams p, int grid, hipStream_t s) {
  mfma_gemm_kernel<BM, FP8, MODE><<<grid, kThreads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

// Row-tile height of the grouped expert GEMMs: large enough that an expert of average load
// fits one tile (its weights are then streamed once), as small as that allows.
int moe_tile_m(molt_dtype wdt, int T, int K, int E) {
  if (wdt == MOLT_F32) return 16;
  const long avg = (long(T) * K + E - 1) / E;
  return avg <= 24 ? 32 : avg <= 56 ? 64 : 128;
}

hipError_t launch_gemm(const void* A, const void* Bw, float* C, int M, int N, int K, molt_dtype dt,
                       bool accumulate, hipStream_t s) {
  GemmParams p{};
  p.A = A; p.B = Bw; p.C = C; p.M = M; p.N = N; p.K = K; p.ldc = N;
  p.accumulate = accumulate;
  if (dt == MOLT_F32) {
    p.n_mtiles = (M + 15) / 16;
    p.n_ntiles = (N + 63) / 64;
    f32_gemm_kernel<kDense><<<p.n_mtiles * p.n_ntiles, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  p.n_ntiles = (N + kBN - 1) / kBN;
  p.xcd_remap = 1;
  if (M > 64) {
    p.n_mtiles = (M + 127) / 128;
    return run_mfma<128, false, kDense>(p, p.n_mtiles * p.n_ntiles, s);
  }
  p.n_mtiles = (M + 31) / 32;
  return run_mfma<32, false, kDense>(p, p.n_mtiles * p.n_ntiles, s);
}

hipError_t launch_moe_gate_up(const void* a, const float* a_scale, const int32_t* pperm, int K_top,
                              const void* w_gu, const float* s_gu, int d, int F, molt_dtype wdt,
                              const int32_t* tiles, const int32_t* n_tiles, int max_tiles,
                              int tile_m, void* h, hipStream_t s) {
  GemmParams p{};
  p.n_tiles_live = n_tiles;
  p.A = a; p.B = w_gu; p.C = h; p.N = F; p.K = d; p.ldc = F;
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
  if (wdt == MOLT_FP8_E4M3) return run_stream<true, kGateUp>(p, tile_m, s);
  return run_stream<false, kGateUp>(p, tile_m, s);
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
  if (wdt == MOLT_FP8_E4M3) return run_stream<true, kDown>(p, tile_m, s);
  return run_stream<false, kDown>(p, tile_m, s);
}

hipError_t launch_pack_tiled(const void* src, void* dst, long rows, long row_bytes, hipStream_t s) {
  const long chunks = rows * (row_bytes / 16);
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
