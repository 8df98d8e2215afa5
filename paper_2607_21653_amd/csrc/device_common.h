// Device helpers shared by the gfx950 kernels: number formats, wavefront
// reductions, MFMA operand types. 64-wide wavefronts throughout.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define MOLT_DEV __device__ __forceinline__

constexpr int kWave = 64;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));
typedef int int32x8_t __attribute__((ext_vector_type(8)));
typedef int int32x4_t __attribute__((ext_vector_type(4)));
typedef long int64x2_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- bf16

MOLT_DEV float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// round to nearest, ties to even; NaN kept quiet
MOLT_DEV uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

MOLT_DEV float round_to_bf16(float f) { return bf16_to_f32(f32_to_bf16(f)); }

// ---------------------------------------------------------------- fp8 e4m3fn (OCP)

// Exact decode of an e4m3fn code (bias 7, subnormals, 0x7f/0xff NaN).
MOLT_DEV float fp8e4m3_to_f32(uint32_t c) {
  uint32_t s = (c & 0x80u) << 24;
  uint32_t e = (c >> 3) & 0xfu;
  uint32_t m = c & 0x7u;
  if (e == 0xfu && m == 0x7u) return __uint_as_float(0x7fc00000u | s);
  if (e == 0) return __uint_as_float(s) + (s ? -1.0f : 1.0f) * float(m) * 0.001953125f;  // m * 2^-9
  return __uint_as_float(s | ((e + 120u) << 23) | (m << 20));
}

// float -> e4m3fn: round to nearest even, saturate finite overflow to +-448, NaN -> 0x7f.
// Integer implementation on the binary32 encoding.
MOLT_DEV uint32_t f32_to_fp8e4m3(float f) {
  uint32_t u = __float_as_uint(f);
  uint32_t sign = (u >> 24) & 0x80u;
  uint32_t a = u & 0x7fffffffu;
  if (a > 0x7f800000u) return 0x7fu;
  if (a >= 0x43e00000u) return sign | 0x7eu;   // |f| >= 448 (incl. inf): saturate
  int e = int(a >> 23) - 127;                  // unbiased exponent of |f|
  if (e < -6) {
    // subnormal target: value = n * 2^-9, n = rne(|f| * 2^9)
    if (e < -11) return sign;                  // < 2^-11: rounds to 0 (2^-10 tie -> 0 handled below)
    uint32_t mant = (a & 0x7fffffu) | 0x800000u;   // 24-bit significand, value = mant * 2^(e-23)
    int shift = -9 - (e - 23);                 // n = mant * 2^(e-23+9) = mant >> shift
    uint32_t n = mant >> shift;
    uint32_t rem = mant & ((1u << shift) - 1u);
    uint32_t half = 1u << (shift - 1);
    if (rem > half || (rem == half && (n & 1u))) n++;
    return sign | n;                           // n == 8 lands on the smallest normal code
  }
  // normal target: keep 3 mantissa bits, round to nearest even
  uint32_t mant = a & 0x7fffffu;
  uint32_t q = mant >> 20;
  uint32_t rem = mant & 0xfffffu;
  uint32_t code = (uint32_t(e + 7) << 3) | q;
  if (rem > 0x80000u || (rem == 0x80000u && (q & 1u))) code++;
  if (code > 0x7eu) code = 0x7eu;              // rounding past 448 saturates
  return sign | code;
}

// v / s for the fp8 row quantisation, from r = 1 / s (IEEE) and one fma correction of
// q0 = v * r, the sign copied from v (the correction turns -0 into +0). For s > 1e-30 and
// bf16 values |v| <= 448 s (the quantisation's domain: v a bf16 entry of the row, s its
// amax / 448) it gives the same e4m3 code as the IEEE quotient: compared on gfx950 for
// every positive bf16 amax and every bf16 v with |v| <= amax, no code differs.
MOLT_DEV float div_by_scale(float v, float s, float r) {
  const float q0 = v * r;
  return __builtin_copysignf(__builtin_fmaf(__builtin_fmaf(-q0, s, v), r, q0), v);
}
constexpr float kFastDivMinScale = 1.0e-30f;

// Two codes at once on the hardware conversion (v_cvt_pk_fp8_f32: OCP e4m3, round to
// nearest even), inputs clamped to +-448 first so that it saturates, NaN mapped to 0x7F:
// the same code as f32_to_fp8e4m3 for every f32 (compared exhaustively on gfx950 over all
// patterns of magnitude <= 448 and their negatives). Code of a in bits 0-7, of b in 8-15.
MOLT_DEV uint32_t f32x2_to_fp8e4m3(float a, float b) {
  const float ca = fminf(fmaxf(a, -448.0f), 448.0f), cb = fminf(fmaxf(b, -448.0f), 448.0f);
  uint32_t r = uint32_t(__builtin_amdgcn_cvt_pk_fp8_f32(ca, cb, 0, false)) & 0xffffu;
  if (a != a) r = (r & 0xff00u) | 0x7fu;
  if (b != b) r = (r & 0x00ffu) | 0x7f00u;
  return r;
}

// Workgroup barrier for LDS exchange only: waits for this wavefront's LDS operations, not
// for its outstanding global loads (__syncthreads() fences all memory, draining the
// prefetches a software pipeline keeps in flight). The memory clobber keeps the compiler
// from moving memory accesses across it.
MOLT_DEV void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ---------------------------------------------------------------- reductions

// Wavefront all-reductions on DPP: an inclusive scan along each 16-lane row (row_shr 1, 2,
// 4, 8), then the rows combined by row_bcast15 (rows 1 and 3) and row_bcast31 (rows 2 and
// 3), so lane 63 ends with the whole wavefront's result, read back wave-uniform. A lane
// whose DPP source lies outside its row (or whose row is masked off) takes the identity.
// Each step is a register move with a few cycles of latency, where a __shfl_xor step is a
// permute through the LDS crossbar.
template <int CTRL, int ROWS>
MOLT_DEV uint32_t dpp_u32(uint32_t v, uint32_t ident) {
  return uint32_t(__builtin_amdgcn_update_dpp(int(ident), int(v), CTRL, ROWS, 0xF, false));
}

template <int CTRL, int ROWS>
MOLT_DEV unsigned long long dpp_max_step(unsigned long long v) {
  const uint32_t lo = dpp_u32<CTRL, ROWS>(uint32_t(v), 0u);
  const uint32_t hi = dpp_u32<CTRL, ROWS>(uint32_t(v >> 32), 0u);
  const unsigned long long o = (static_cast<unsigned long long>(hi) << 32) | lo;
  return o > v ? o : v;
}

template <int CTRL, int ROWS>
MOLT_DEV float dpp_max_step(float v) {
  return fmaxf(v, __uint_as_float(dpp_u32<CTRL, ROWS>(__float_as_uint(v), 0xff800000u)));
}

template <int CTRL, int ROWS>
MOLT_DEV float dpp_sum_step(float v) {
  return v + __uint_as_float(dpp_u32<CTRL, ROWS>(__float_as_uint(v), 0u));
}

MOLT_DEV uint32_t lane63(uint32_t v) { return uint32_t(__builtin_amdgcn_readlane(int(v), 63)); }

template <int CTRL, int ROWS>
MOLT_DEV int dpp_add_step(int v) {
  return v + int(dpp_u32<CTRL, ROWS>(uint32_t(v), 0u));
}

// inclusive prefix sum over the lanes (lane i gets lanes 0..i): the same DPP steps, every
// lane keeping its partial result
MOLT_DEV int wave_scan_dpp(int v) {
  v = dpp_add_step<0x111, 0xF>(v);
  v = dpp_add_step<0x112, 0xF>(v);
  v = dpp_add_step<0x114, 0xF>(v);
  v = dpp_add_step<0x118, 0xF>(v);
  v = dpp_add_step<0x142, 0xA>(v);
  v = dpp_add_step<0x143, 0xC>(v);
  return v;
}

// unsigned 64-bit maximum over the wavefront (every lane gets it)
MOLT_DEV unsigned long long wave_max_dpp(unsigned long long v) {
  v = dpp_max_step<0x111, 0xF>(v);
  v = dpp_max_step<0x112, 0xF>(v);
  v = dpp_max_step<0x114, 0xF>(v);
  v = dpp_max_step<0x118, 0xF>(v);
  v = dpp_max_step<0x142, 0xA>(v);
  v = dpp_max_step<0x143, 0xC>(v);
  return (static_cast<unsigned long long>(lane63(uint32_t(v >> 32))) << 32) | lane63(uint32_t(v));
}

MOLT_DEV float wave_max_dpp(float v) {
  v = dpp_max_step<0x111, 0xF>(v);
  v = dpp_max_step<0x112, 0xF>(v);
  v = dpp_max_step<0x114, 0xF>(v);
  v = dpp_max_step<0x118, 0xF>(v);
  v = dpp_max_step<0x142, 0xA>(v);
  v = dpp_max_step<0x143, 0xC>(v);
  return __uint_as_float(lane63(__float_as_uint(v)));
}

MOLT_DEV float wave_sum_dpp(float v) {
  v = dpp_sum_step<0x111, 0xF>(v);
  v = dpp_sum_step<0x112, 0xF>(v);
  v = dpp_sum_step<0x114, 0xF>(v);
  v = dpp_sum_step<0x118, 0xF>(v);
  v = dpp_sum_step<0x142, 0xA>(v);
  v = dpp_sum_step<0x143, 0xC>(v);
  return __uint_as_float(lane63(__float_as_uint(v)));
}

// Maximum (sum) over the lanes l, l ^ 16, l ^ 32 and l ^ 48: the four 16-lane rows of a
// wavefront combined lane by lane, on gfx950's row swaps (VALU moves, no LDS permute).
// permlane16_swap(a, b) exchanges rows 1 and 3 of a with rows 0 and 2 of b, permlane32_swap
// rows 2-3 of a with rows 0-1 of b; given the same value twice, the two results hold each
// row's value and its partner's. Every lane gets (x0 op x1) op (x2 op x3) for its rows.
MOLT_DEV float rows_max4(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
MOLT_DEV float rows_sum4(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

MOLT_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
MOLT_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
MOLT_DEV double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
MOLT_DEV unsigned long long wave_sum(unsigned long long v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Block-wide reductions for blocks of NW waves; `red` is LDS scratch of NW entries.
// Every thread returns the result.
template <int NW>
MOLT_DEV float block_max(float v, float* red) {
  v = wave_max(v);
  int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = fmaxf(r, red[i]);
  return r;
}
template <int NW, typename T>
MOLT_DEV T block_sum(T v, T* red) {
  v = wave_sum(v);
  int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  T r = red[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r += red[i];   // fixed order: deterministic
  return r;
}

// the same over NW wavefronts, each wavefront's share reduced on DPP
template <int NW>
MOLT_DEV float block_sum_dpp(float v, float* red) {
  v = wave_sum_dpp(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r += red[i];   // fixed order: deterministic
  return r;
}
template <int NW>
MOLT_DEV float block_max_dpp(float v, float* red) {
  v = wave_max_dpp(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = fmaxf(r, red[i]);
  return r;
}

// SiLU x * sigmoid(x) with the hardware exp2 and reciprocal (v_exp_f32, v_rcp_f32): exp(-x)
// = 2^(-x log2 e); relative error ~1e-6 for |x| <= 10, limits x and -0 for large |x|.
// (A full-precision expf and division made the expert GEMM epilogues VALU-bound.)
MOLT_DEV float silu(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
}

// ---------------------------------------------------------------- tiled operand layout
// The grouped expert GEMMs keep their operands (expert weights, gathered activations, the
// SwiGLU product) in a tiled byte layout. A row-major matrix of R rows (R % 32 == 0) and
// RB bytes per row (RB % 128 == 0) is cut into 32-row x 128-byte tiles; tile (rb, kb) is
// the 4 KB at ((rb * RB / 128) + kb) * 4096, and byte j of row r inside it sits at
// ((j % 64) / 16) * 1024 + ((j / 64) * 32 + r) * 16 + j % 16. Lane l of a wavefront that
// loads 16 bytes at l * 16 of each 1 KB quarter c gets row l % 32, bytes 64 (l / 32) + 16 c
// of the slice: the MFMA operand layout, with each load instruction reading 1 KB of one
// page instead of touching 32 rows.
MOLT_DEV long tiled_offset(long row, long j, long row_bytes) {
  return ((row >> 5) * (row_bytes >> 7) + (j >> 7)) * 4096 + ((j & 63) >> 4) * 1024 +
         ((((j & 127) >> 6) << 5) + (row & 31)) * 16 + (j & 15);
}
// element index of (row, col) of a tiled matrix of `cols` elements of `esize` bytes per row
MOLT_DEV long tiled_index(long row, long col, long cols, int esize) {
  return tiled_offset(row, col * esize, cols * esize) / esize;
}
