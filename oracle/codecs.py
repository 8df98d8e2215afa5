"""Number formats used by the verify step: bfloat16 and OCP fp8 e4m3fn.

bfloat16: the upper 16 bits of an IEEE binary32; narrowing rounds to nearest,
ties to even. fp8 e4m3fn (OCP 8-bit floating point specification, "E4M3"):
1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 is
subnormal (value m/8 * 2^-6); S.1111.111 is NaN; there is no infinity; the
largest finite magnitude is 1.75 * 2^8 = 448. Narrowing here rounds to nearest,
ties to even, and saturates finite overflow to +-448 (the activation quantiser's
convention; written in the method's fp8 reading).

Pins: tests/test_oracle_codecs.py (brute-force nearest-value search over every
code, torch's own float8_e4m3fn / bfloat16 conversions on in-range values, and
the spec's fixed points such as 448 = 0x7E and 2^-9 = 0x01).
"""
import numpy as np


# ---------------------------------------------------------------- bfloat16

def bf16_bits_to_f32(bits) -> np.ndarray:
    """Widen bf16 bit patterns (uint16/int16) exactly to float32."""
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); NaN stays NaN."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    r = np.where(nan, ((u >> 16) | 0x40) & 0xFFFF, r)
    return r.astype(np.uint16)


def round_bf16(x) -> np.ndarray:
    """Value of x (rounded first to float32) after narrowing to bf16, as float64."""
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(x, dtype=np.float64).astype(np.float32))).astype(np.float64)


# ---------------------------------------------------------------- fp8 e4m3fn

def _e4m3_table() -> np.ndarray:
    vals = np.empty(256, dtype=np.float64)
    for c in range(256):
        s = -1.0 if c & 0x80 else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            vals[c] = np.nan
        elif e == 0:
            vals[c] = s * (m / 8.0) * 2.0 ** -6
        else:
            vals[c] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


E4M3_VALUES = _e4m3_table()
E4M3_MAX = 448.0


def fp8_decode(codes) -> np.ndarray:
    return E4M3_VALUES[np.asarray(codes).astype(np.uint8)]


def fp8_encode(x) -> np.ndarray:
    """float32 -> e4m3fn code: round to nearest, ties to even mantissa, saturate to +-448.

    Works on the binary32 value: |x| is split into an exponent band and scaled so the
    representable neighbours are consecutive integers, then rounded half-to-even."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)  # exact widening
    sign = np.signbit(x)
    a = np.abs(x)
    out = np.zeros(a.shape, dtype=np.int64)
    nan = np.isnan(a)
    a = np.where(nan, 0.0, a)
    # spacing of representable values at |x|: 2^(E-3) for normal band E>=-6, 2^-9 below
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.clip(e, -6, 8)
    # guard log2 rounding at exact band edges
    e = np.where(a >= 2.0 ** (e + 1), e + 1, e)
    e = np.where((a < 2.0 ** e) & (e > -6), e - 1, e)
    step = 2.0 ** (e - 3)
    q = a / step                       # exact (power-of-two scaling)
    n = np.rint(q)                     # numpy rint: round half to even
    val = n * step                     # candidate magnitude
    val = np.minimum(val, E4M3_MAX)    # saturate
    # encode magnitude val (exactly representable now)
    code = np.zeros(a.shape, dtype=np.int64)
    sub = val < 2.0 ** -6
    code = np.where(sub, np.rint(val / 2.0 ** -9), code)
    ee = np.floor(np.log2(np.where(val > 0, val, 1.0)))
    ee = np.where(val >= 2.0 ** (ee + 1), ee + 1, ee)
    ee = np.where(val < 2.0 ** ee, ee - 1, ee)
    mant = np.rint(val / 2.0 ** ee * 8.0) - 8.0
    normal_code = ((ee + 7).astype(np.int64) << 3) | mant.astype(np.int64)
    code = np.where(sub, code, normal_code).astype(np.int64)
    code = np.where(sign, code | 0x80, code)
    code = np.where(nan, 0x7F, code)
    return code.astype(np.uint8)


def fp8_quantize_rows(x_rows) -> tuple:
    """Per-row dynamic quantisation of float32 rows (the method's fp8 reading):
    s = amax(|row|) / 448 in float32, codes = e4m3(row / s) with float32 division.
    A row of zeros gets s = 0 and all-zero codes."""
    xr = np.asarray(x_rows, dtype=np.float32)
    amax = np.abs(xr).max(axis=-1).astype(np.float32)
    s = (amax / np.float32(E4M3_MAX)).astype(np.float32)
    safe = np.where(s > 0, s, np.float32(1.0)).astype(np.float32)
    scaled = (xr / safe[..., None]).astype(np.float32)
    codes = fp8_encode(scaled)
    codes = np.where((s > 0)[..., None], codes, np.uint8(0)).astype(np.uint8)
    return codes, s
