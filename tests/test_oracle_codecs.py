"""Pins of the oracle's number formats (paper Sec. 3.3) against an independent
integer-arithmetic model, torch's float8_e4m3fn casts and the constants the
paper states."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
import fpmodel as M

FMTS = [("e4m3", O.E4M3), ("e4m11", O.E4M11), ("ue5m3_shift", O.UE5M3_SHIFT),
        ("ue5m11_shift", O.UE5M11_SHIFT), ("ue5m3_exp", O.UE5M3_EXP), ("ue5m11_exp", O.UE5M11_EXP)]


def test_paper_constants():
    # e4m3 overflows beyond 448 (Sec. 3.3): saturate to +-448.
    assert O.round_fmt(O.E4M3, [448.0, 460.0, 464.0, 470.0, 1e6, -1e6]).tolist() == \
        [448.0, 448.0, 448.0, 448.0, 448.0, -448.0]
    assert O.encode_fmt(O.E4M3, [448.0, -448.0]).tolist() == [0x7E, 0xFE]
    # 8-bit exp format: bias chosen so that 11111000 is 1.0, smallest normal
    # 2^-30, smallest subnormal 2^-33 (Sec. 3.3).
    assert O.decode_fmt(O.UE5M3_EXP, [0b11111000, 0b00001000, 0b00000001]).tolist() == \
        [1.0, 2.0 ** -30, 2.0 ** -33]
    # below half the smallest subnormal -> 0; exactly half ties to even -> 0
    assert O.round_fmt(O.UE5M3_EXP, [2.0 ** -34, 1.5 * 2.0 ** -34, 2.0 ** -35]).tolist() == \
        [0.0, 2.0 ** -33, 0.0]
    # shifted logits need the doubled limit 896 (Sec. 3.3): exactly representable
    assert O.round_fmt(O.UE5M3_SHIFT, [896.0]).tolist() == [896.0]
    # e4m11: all codes finite, largest (2 - 2^-11) * 2^8
    assert O.decode_fmt(O.E4M11, [0x7FFF]).tolist() == [511.875]
    assert O.round_fmt(O.E4M11, [600.0, -600.0]).tolist() == [511.875, -511.875]
    # QK-Norm bound: 8*sqrt(2)*maxgain^2 <= 448 gives maxgain <= 6.29 (Sec. 3.3)
    assert abs(np.sqrt(448 / (8 * np.sqrt(2))) - 6.29) < 0.005
    # a few e4m3 roundings (RNE)
    assert O.round_fmt(O.E4M3, [1.0625, 1.1875, 2.0 ** -10, 3 * 2.0 ** -11, -2.0 ** -10]).tolist() == \
        [1.0, 1.25, 0.0, 2.0 ** -9, -0.0]
    assert np.signbit(O.round_fmt(O.E4M3, [-2.0 ** -12]))[0]


def _structured_f32_patterns():
    """Every fp32 exponent x each 4-bit top mantissa x sticky patterns of the
    dropped bits, both signs: covers every (kept bits, round bit, sticky) case
    of rounding to 3 mantissa bits in every binade."""
    exps = np.arange(0, 255, dtype=np.uint32)
    top = np.arange(16, dtype=np.uint32) << 19
    low = np.array([0, 1, 2, 0x3FFFF, 0x40000, 0x40001, 0x7FFFF, 0x12345, 0x7FF, 0x400], dtype=np.uint32)
    b = (exps[:, None, None] << 23) | top[None, :, None] | low[None, None, :]
    b = b.ravel()
    return np.concatenate([b, b | np.uint32(0x80000000)])


def test_e4m3_vs_integer_model_structured_and_random():
    rng = np.random.default_rng(0)
    bits = np.concatenate([_structured_f32_patterns(),
                           rng.integers(0, 2 ** 32, size=2_000_000, dtype=np.uint64).astype(np.uint32)])
    x = bits.view(np.float32).astype(np.float64)
    x = x[~np.isnan(x)]
    got = O.round_fmt(O.E4M3, x)
    ref = M.np_round(x, "e4m3")
    assert np.array_equal(got, ref)
    assert np.array_equal(np.signbit(got), np.signbit(ref))
    assert np.array_equal(O.encode_fmt(O.E4M3, x), M.np_encode(ref, "e4m3").astype(np.uint32))


def test_e4m3_fp32_bit_entry_matches_model():
    """The bulk fp32-pattern entry (used for the GPU's exhaustive check)."""
    for start in (0, 0x3C000000, 0x43E00000, 0xBF800000, 0xFF7FF000):
        cnt = 1 << 16
        got = O.e4m3_of_f32_bits(start, cnt)
        bits = (np.arange(cnt, dtype=np.uint64) + start).astype(np.uint32)
        x = bits.view(np.float32).astype(np.float64)
        ok = ~np.isnan(x)
        ref = M.np_encode(M.np_round(x[ok], "e4m3"), "e4m3")
        assert np.array_equal(got[ok], ref.astype(np.uint8))
        assert np.all(got[~ok] == 0xFF)


def test_e4m3_vs_torch_float8():
    """torch's float8_e4m3fn cast rounds to nearest even; it returns NaN rather
    than saturating above 464, so compare on |x| <= 464."""
    rng = np.random.default_rng(1)
    bits = np.concatenate([_structured_f32_patterns(),
                           rng.integers(0, 2 ** 32, size=1_000_000, dtype=np.uint64).astype(np.uint32)])
    f = bits.view(np.float32)
    f = f[np.isfinite(f) & (np.abs(f) <= 464.0)]
    t = torch.from_numpy(f.copy()).to(torch.float8_e4m3fn)
    ref_codes = t.view(torch.uint8).numpy()
    got = O.encode_fmt(O.E4M3, f.astype(np.float64)).astype(np.uint8)
    assert np.array_equal(got, ref_codes)


def test_e4m3_decode_all_codes_vs_torch():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    ref = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    assert np.array_equal(O.decode_fmt(O.E4M3, codes.astype(np.uint32)), ref)


@pytest.mark.parametrize("name,fid", FMTS)
def test_all_codes_roundtrip(name, fid):
    mbits, emin, maxval, bias, ebits, signed = M.FMT[name]
    ncode = 1 << (ebits + mbits + (1 if signed else 0))
    codes = np.arange(ncode, dtype=np.uint32)
    if name == "e4m3":
        codes = codes[(codes & 0x7F) != 0x7F]          # E4M3FN NaN codes
    vals = O.decode_fmt(fid, codes)
    assert np.all(np.abs(vals) <= maxval)
    assert np.array_equal(O.encode_fmt(fid, vals), codes)
    assert np.array_equal(M.np_encode(vals, name).astype(np.uint32), codes)
    # values are strictly increasing in the (unsigned part of the) code
    pos = codes[(codes >> (ebits + mbits)) == 0] if signed else codes
    assert np.all(np.diff(O.decode_fmt(fid, pos)) > 0)


@pytest.mark.parametrize("name,fid", FMTS)
def test_rounding_vs_integer_model(name, fid):
    mbits, emin, maxval, bias, ebits, signed = M.FMT[name]
    rng = np.random.default_rng(2)
    # grid values, midpoints, neighbours of midpoints, and random magnitudes
    ncode = 1 << (ebits + mbits)
    codes = np.arange(ncode, dtype=np.uint32)
    if name == "e4m3":
        codes = codes[codes != 0x7F]
    g = O.decode_fmt(fid, codes)
    mids = (g[1:] + g[:-1]) / 2
    x = np.concatenate([g, mids, np.nextafter(mids, 0), np.nextafter(mids, np.inf),
                        np.exp(rng.uniform(np.log(2.0 ** (emin - mbits - 3)), np.log(maxval * 1.5), 200_000)),
                        [0.0, maxval, maxval * 1.01, 1e30]])
    if signed:
        x = np.concatenate([x, -x])
    got = O.round_fmt(fid, x)
    ref = M.np_round(x, name)
    assert np.array_equal(got, ref)


def test_fraction_rounding_agrees_with_integer_model():
    """The two independent models agree (cross-check of the test models)."""
    from fractions import Fraction
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(2000) * 40, rng.standard_normal(2000) * 2.0 ** -8])
    for name in ("e4m3", "e4m11"):
        ref = M.np_round(x, name)
        fr = np.array([float(M.frac_fmt(Fraction(float(v)), name)) for v in x])
        assert np.array_equal(np.abs(ref), np.abs(fr))
