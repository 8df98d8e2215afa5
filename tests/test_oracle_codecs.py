"""Pins of the oracle's number formats: bf16 narrowing against torch's conversion and
a brute-force nearest search; fp8 e4m3fn against the OCP specification's fixed
points, a brute-force nearest-code search over all 254 finite codes (ties to the
even mantissa), torch's float8_e4m3fn conversion for in-range values, and the
per-row quantiser's scale and saturation."""
import numpy as np
import torch

from oracle import codecs


def test_bf16_matches_torch_and_bruteforce():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(size=20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.005859375, 65504.0, 3.4e38]]).astype(np.float32)
    ours = codecs.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert (ours == ref).all()
    # brute force on a slice: nearest of the two bf16 neighbours, ties to even
    for v in x[:300]:
        u = np.float32(v).view(np.uint32)
        lo = (u >> 16) << 16
        hi = lo + (1 << 16)
        a = float(np.uint32(lo).view(np.float32))
        b = float(np.uint32(hi & 0xFFFFFFFF).view(np.float32)) if hi < 2 ** 32 else np.inf
        dv = float(v)
        if abs(dv - a) < abs(b - dv) or (abs(dv - a) == abs(b - dv) and ((lo >> 16) & 1) == 0):
            want = lo >> 16
        else:
            want = hi >> 16
        assert int(codecs.f32_to_bf16_bits(np.float32(v))) == int(want) & 0xFFFF


def test_e4m3_spec_fixed_points():
    v = codecs.E4M3_VALUES
    assert v[0x7E] == 448.0 and v[0xFE] == -448.0          # largest finite
    assert v[0x01] == 2.0 ** -9                            # smallest subnormal
    assert v[0x08] == 2.0 ** -6                            # smallest normal
    assert v[0x38] == 1.0 and v[0x3C] == 1.5
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF])
    assert v[0x00] == 0.0 and v[0x80] == 0.0
    finite = v[~np.isnan(v)]
    assert len(finite) == 254


def _brute_encode(x):
    """Nearest finite code, ties to the code with an even mantissa, saturating."""
    codes = np.array([c for c in range(256) if not np.isnan(codecs.E4M3_VALUES[c])])
    vals = codecs.E4M3_VALUES[codes]
    x = float(x)
    if abs(x) >= 448.0:
        return 0x7E | (0x80 if x < 0 else 0)
    d = np.abs(vals - x)
    best = d.min()
    cand = codes[d == best]
    cand = [c for c in cand if (c & 0x80) == (0x80 if np.signbit(x) else 0)] or list(cand)
    if len(cand) > 1:
        cand = [c for c in cand if (c & 1) == 0]
    return cand[0]


def test_e4m3_encode_bruteforce():
    rng = np.random.default_rng(1)
    vals = codecs.E4M3_VALUES[~np.isnan(codecs.E4M3_VALUES)]
    mids = (np.sort(vals)[1:] + np.sort(vals)[:-1]) / 2      # exact ties
    x = np.concatenate([rng.normal(size=3000) * 2.0 ** rng.integers(-12, 10, 3000),
                        vals, mids, [1000.0, -1000.0, 449.0, 463.99, 464.0, 2.0 ** -10, 2.0 ** -11]])
    x = x.astype(np.float32)
    ours = codecs.fp8_encode(x)
    for xi, c in zip(x, ours):
        want = _brute_encode(np.float64(xi))
        assert codecs.E4M3_VALUES[c] == codecs.E4M3_VALUES[want] or (
            codecs.E4M3_VALUES[c] == 0 and codecs.E4M3_VALUES[want] == 0), (xi, c, want)


def test_e4m3_encode_matches_torch_in_range():
    rng = np.random.default_rng(2)
    x = (rng.normal(size=50000) * 50).astype(np.float32)
    x = x[np.abs(x) < 448]
    ours = codecs.fp8_decode(codecs.fp8_encode(x))
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_row_quantiser():
    rng = np.random.default_rng(3)
    x = (rng.normal(size=(64, 300)) * rng.random((64, 1)) * 10).astype(np.float32)
    x[5] = 0.0
    codes, s = codecs.fp8_quantize_rows(x)
    assert s[5] == 0 and (codes[5] == 0).all()
    rows = np.arange(64) != 5
    # the row maximum maps onto +-448 exactly (up to division rounding) and nothing saturates past it
    dq = codecs.fp8_decode(codes[rows]) * s[rows, None]
    amax = np.abs(x[rows]).max(axis=1)
    np.testing.assert_allclose(np.abs(dq).max(axis=1), amax, rtol=1e-6)
    # relative error of e4m3 rounding is at most 2^-4 for normal values
    big = np.abs(x[rows]) > amax[:, None] * 2.0 ** -6
    rel = np.abs(dq - x[rows]) / np.abs(x[rows])
    assert rel[big].max() <= 2.0 ** -4 + 1e-6
