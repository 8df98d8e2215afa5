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
// one expert x 128 output columns; each of the 4 wavefronts owns 32 columns and loads its
// weight fragments straight from global memory into registers, kPD 128-byte K slices
// ahead (a weight element is used by exactly one wavefront: no LDS needed). The
// activation rows (shared by the 4 wavefronts) are prefetched kPD slices ahead into
// registers too and staged through a double-buffered LDS tile, one barrier per slice. A
// lane's MFMA operand chunk for k-step s of a slice is bytes [64 g + 16 s, +16) (bf16,
// g = lane / 32) or [64 g + 32 s, +32) (fp8) of its row, for both operands: each lane
// streams 64 contiguous bytes of its weight row per slice.
constexpr int kPD = 4;   // slices in flight per wavefront

struct Slice16 { int4 c[4]; };   // 64 bytes of one row: 4 x 16 B

template <int BM, bool FP8, int MODE>
__global__ __launch_bounds__(kThreads) void moe_stream_kernel(GemmParams p) {
  constexpr int MS = BM / 32;                        // 32-row MFMA tiles per wavefront
  constexpr int kElem = FP8 ? 1 : 2;
  constexpr int kBK = kRowBytes / kElem;             // K elements per slice
  constexpr int kALoads = BM * 8 / kThreads;         // 16-byte A chunks per thread per slice
  static_assert(kALoads >= 1, "BM too small");
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * BM * kLdsStride];

  int id = blockIdx.x;
  const int G = gridDim.x;
  id = (id % 8) * (G / 8) + id / 8;                   // grid is a multiple of 8: XCD-local order
  if (id >= p.n_mtiles * p.n_ntiles) return;
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
  const long K = p.K;
  const int nk = int(K / kBK);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int lrow = lane % 32, lg = lane / 32;

  // weight row of this lane (column lrow of the wavefront's 32)
  long brow;
  int n0;
  if (MODE == kGateUp) {
    n0 = nt * (kBN / 2);
    brow = long(expert) * 2 * p.N + (wave < 2 ? n0 + 32 * wave + lrow : p.N + n0 + 32 * (wave - 2) + lrow);
  } else {
    n0 = nt * kBN;
    brow = long(expert) * p.N + n0 + 32 * wave + lrow;   // dense: expert 0, N % 128 == 0
  }
  const uint8_t* bsrc = static_cast<const uint8_t*>(p.B) + brow * K * kElem + lg * 64;

  // activation rows staged by all threads: chunk c of row r = tid / 8 + 32 i. Rows past the
  // tile read row row0 (always valid); MFMA rows are independent and those outputs are
  // never stored, so the loads carry no branches and their count stays exact.
  const int chunk = threadIdx.x % 8;
  const uint8_t* a_src[kALoads];
#pragma unroll
  for (int i = 0; i < kALoads; ++i) {
    const int grow = row0 + threadIdx.x / 8 + 32 * i;
    long arow = grow < row1 ? grow : row0;
    if (MODE == kGateUp) arow = p.perm[arow] / p.ktop;
    a_src[i] = static_cast<const uint8_t*>(p.A) + arow * K * kElem + chunk * 16;
  }

  Slice16 wb[kPD];
  auto wload = [&](Slice16& f, int kb) {
    const uint8_t* src = bsrc + long(kb) * kRowBytes;
#pragma unroll
    for (int c = 0; c < 4; ++c) f.c[c] = *reinterpret_cast<const int4*>(src + 16 * c);
  };
  int4 ra[kPD][kALoads];
  auto aload = [&](int4 (&r)[kALoads], int kb) {
#pragma unroll
    for (int i = 0; i < kALoads; ++i)
      r[i] = *reinterpret_cast<const int4*>(a_src[i] + long(kb) * kRowBytes);
  };
  auto astore = [&](const int4 (&r)[kALoads], int buf) {
#pragma unroll
    for (int i = 0; i < kALoads; ++i)
      *reinterpret_cast<int4*>(lds + buf * BM * kLdsStride +
                               (threadIdx.x / 8 + 32 * i) * kLdsStride + chunk * 16) = r[i];
  };

  floatx16_t acc[MS];
#pragma unroll
  for (int i = 0; i < MS; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;

#pragma unroll
  for (int s = 0; s < kPD; ++s)
    if (s < nk) {
      wload(wb[s], s);
      aload(ra[s], s);
    }
  astore(ra[0], 0);
  __syncthreads();

  auto slice = [&](const Slice16& f, int buf) {
    const uint8_t* abase = lds + buf * BM * kLdsStride + lrow * kLdsStride + lg * 64;
    if (!FP8) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(&f.c[s]);
        bf16x8_t av[MS];
#pragma unroll
        for (int i = 0; i < MS; ++i)
          av[i] = *reinterpret_cast<const bf16x8_t*>(abase + i * 32 * kLdsStride + 16 * s);
#pragma unroll
        for (int i = 0; i < MS; ++i) acc[i] = mfma(av[i], bv, acc[i]);
      }
    } else {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int32x8_t bv = int32x8_t{f.c[2 * s].x, f.c[2 * s].y, f.c[2 * s].z, f.c[2 * s].w,
                                       f.c[2 * s + 1].x, f.c[2 * s + 1].y, f.c[2 * s + 1].z,
                                       f.c[2 * s + 1].w};
        int32x8_t av[MS];
#pragma unroll
        for (int i = 0; i < MS; ++i) {
          const uint8_t* q = abase + i * 32 * kLdsStride + 32 * s;
          const int32x4_t lo = *reinterpret_cast<const int32x4_t*>(q);
          const int32x4_t hi = *reinterpret_cast<const int32x4_t*>(q + 16);
          av[i] = int32x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
#pragma unroll
        for (int i = 0; i < MS; ++i) acc[i] = mfma(av[i], bv, acc[i]);
      }
    }
  };

  // slice kb = kb0 + s: stage slice kb+1 (register set (s+1) % kPD) into LDS, compute slice
  // kb from register set s, then refill set s with slice kb + kPD; one barrier per slice
  for (int kb0 = 0; kb0 < nk; kb0 += kPD) {
#pragma unroll
    for (int s = 0; s < kPD; ++s) {
      const int kb = kb0 + s;
      if (kb < nk) {
        if (kb + 1 < nk) astore(ra[(s + 1) % kPD], (kb + 1) & 1);
        slice(wb[s], kb & 1);
        if (kb + kPD < nk) {
          wload(wb[s], kb + kPD);
          aload(ra[s], kb + kPD);
        }
        __syncthreads();
      }
    }
  }

  // ---- epilogue: acc[i][e] is row 32 i + 8 (e/4) + 4 (lane/32) + e%4, column lane%32
  const int lcol = lane % 32, lgrp = lane / 32;
  if (MODE == kGateUp) {
    // the "up" wavefronts (tile columns 64..127) park their values in LDS; the "gate"
    // wavefronts finish h = silu(gate) * up for their columns
    float* upbuf = reinterpret_cast<float*>(lds);   // [BM][64] fits in 2 * BM * 144 bytes
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
          static_cast<uint16_t*>(p.C)[long(grow) * p.ldc + n0 + c] = f32_to_bf16(silu(g) * u);
        }
    }
  } else {
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
        float* dst = static_cast<float*>(p.C) + long(grow) * p.ldc + c;
        if (MODE == kDense && p.accumulate) v += *dst;
        *dst = v;
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

// ---------------------------------------------------------------- f32 VALU path
// One workgroup per (row tile of 16, column tile of 64); each thread owns 4 outputs.
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
    long arow = grow;
    if (MODE == kGateUp) arow = p.perm[grow] / p.ktop;
    const float* a = A + arow * K;
    if (MODE == kGateUp) {
      const float* bg = B + (long(expert) * 2 * p.N + col) * K;
      const float* bu = B + (long(expert) * 2 * p.N + p.N + col) * K;
      float g = 0.f, u = 0.f;
      for (int kk = 0; kk < K; ++kk) {
        g += a[kk] * bg[kk];
        u += a[kk] * bu[kk];
      }
      static_cast<float*>(p.C)[long(grow) * p.ldc + col] = silu(g) * u;
    } else {
      const float* b = B + ((MODE == kDown ? long(expert) * p.N : 0) + col) * K;
      float s = 0.f;
      for (int kk = 0; kk < K; ++kk) s += a[kk] * b[kk];
      float* dst = static_cast<float*>(p.C) + long(grow) * p.ldc + col;
      if (MODE == kDense && p.accumulate) s += *dst;
      *dst = s;
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

hipError_t launch_moe_gate_up(const void* x, const uint8_t* xq, const float* xs, const int32_t* perm,
                              int K_top, const void* w_gu, const float* s_gu, int d, int F,
                              molt_dtype act, molt_dtype wdt, const int32_t* tiles, int max_tiles,
                              int tile_m, void* h, hipStream_t s) {
  GemmParams p{};
  p.A = wdt == MOLT_FP8_E4M3 ? static_cast<const void*>(xq) : x;
  p.B = w_gu; p.C = h; p.N = F; p.K = d; p.ldc = F;
  p.tiles = reinterpret_cast<const int4*>(tiles);
  p.n_mtiles = max_tiles;
  p.perm = perm; p.ktop = K_top;
  p.a_scale = xs; p.b_scale = s_gu; p.b_scale_ld = 2 * F;
  if (wdt == MOLT_F32) {
    p.n_ntiles = (F + 63) / 64;
    f32_gemm_kernel<kGateUp><<<max_tiles * p.n_ntiles, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  p.n_ntiles = F / (kBN / 2);
  if (wdt == MOLT_FP8_E4M3) return run_stream<true, kGateUp>(p, tile_m, s);
  return run_stream<false, kGateUp>(p, tile_m, s);
}

hipError_t launch_moe_down(const void* h, const uint8_t* hq, const float* hs, const void* w_d,
                           const float* s_d, int d, int F, molt_dtype act, molt_dtype wdt,
                           const int32_t* tiles, int max_tiles, int tile_m, float* o,
                           hipStream_t s) {
  GemmParams p{};
  p.A = wdt == MOLT_FP8_E4M3 ? static_cast<const void*>(hq) : h;
  p.B = w_d; p.C = o; p.N = d; p.K = F; p.ldc = d;
  p.tiles = reinterpret_cast<const int4*>(tiles);
  p.n_mtiles = max_tiles;
  p.a_scale = hs; p.b_scale = s_d; p.b_scale_ld = d;
  if (wdt == MOLT_F32) {
    p.n_ntiles = (d + 63) / 64;
    f32_gemm_kernel<kDown><<<max_tiles * p.n_ntiles, kThreads, 0, s>>>(p);
    return hipGetLastError();
  }
  p.n_ntiles = d / kBN;
  if (wdt == MOLT_FP8_E4M3) return run_stream<true, kDown>(p, tile_m, s);
  return run_stream<false, kDown>(p, tile_m, s);
}

}  // namespace molt
