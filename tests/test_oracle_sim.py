"""Pins of the oracle's "SIM" precision profile (paper Sec. 4.1: numbers kept
in FP32 with 3- or 11-bit mantissas, recursive FP32 FMA accumulation rounded
after every step, correctly rounded exponentials).

* rounding: against exact Fraction arithmetic, and against the same rounding
  written on the FP32 encoding (round the fraction field at bit 23 - p, ties
  to even, carry into the exponent), over random and tie-making bit patterns,
  FP32 subnormals and the overflow edge;
* shifts: the exact difference rounds correctly even where the fp64
  difference alone would hit a midpoint;
* exponentials: every value on the grid of shifts that can give neither 0 nor
  1 against 160-bit mpmath (tests/fpmodel.py), and the two saturated ends;
* logits: d = 1 is one rounding; small integers give exact sums; Fraction
  brute force of the recursion;
* forward pass: the independent implementation (tests/refimpl.py) in the SIM
  profile at all five thresholds and with both stage variants; +inf on one
  tile is a naive softmax of the SIM logits; threshold 1 never recomputes in
  stage 2; the profile differs from the hardware one where e4m3 saturates.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
import fpmodel as M
import refimpl as R
from paper_2609_39361_amd import workloads as W


def _frac_sim(x, p):
    """Exact reference: RN to p mantissa bits, FP32 exponent range, overflow to inf."""
    r = M.frac_round(Fraction(x), p, -126)
    if abs(r) >= 2 ** 128:
        return math.copysign(math.inf, x)
    return float(r)


def _bits_round(b, p):
    """The rounding on FP32 encodings: RNE of the fraction field at bit 23-p."""
    b = b.astype(np.uint64)
    drop = 23 - p
    lsb = (b >> np.uint64(drop)) & np.uint64(1)
    r = (b + np.uint64((1 << (drop - 1)) - 1) + lsb) & np.uint64(0xFFFFFFFF ^ ((1 << drop) - 1))
    return r.astype(np.uint32)


@pytest.mark.parametrize("p", [3, 11])
def test_round_sim_matches_exact_arithmetic(p):
    rng = np.random.default_rng(40 + p)
    x = rng.standard_normal(3000) * np.exp2(rng.integers(-150, 130, 3000))
    # ties: odd multiples of half the quantum, in normal and subnormal binades
    e = rng.integers(-140, 126, 800)
    k = rng.integers(1 << p, 1 << (p + 1), 800)
    q = np.exp2(np.maximum(e, -126) - p)
    ties = (np.where(e < -126, k % (1 << p), k) + 0.5) * q
    x = np.concatenate([x, ties, -ties, [0.0, -0.0, 2.0 ** 128 * (1 - 2.0 ** -(p + 2)), 3.4e38, 2.0 ** -150]])
    got = O.round_sim(p, x)
    ref = np.array([_frac_sim(v, p) if v != 0 else v for v in x])
    assert np.array_equal(got, ref)
    assert np.array_equal(np.signbit(got[x == 0]), np.signbit(x[x == 0]))


@pytest.mark.parametrize("p", [3, 11])
def test_round_sim_is_the_fp32_encoding_rounding(p):
    rng = np.random.default_rng(50 + p)
    b = rng.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32)
    drop = 23 - p
    tie = (b & np.uint32(0xFFFFFFFF ^ ((1 << drop) - 1))) | np.uint32(1 << (drop - 1))
    sub = rng.integers(0, 1 << 23, 1 << 14, dtype=np.uint64).astype(np.uint32)        # subnormals
    top = np.uint32(0x7F7FFFFF) - rng.integers(0, 1 << 21, 1 << 12, dtype=np.uint64).astype(np.uint32)
    b = np.concatenate([b, tie, sub, sub | np.uint32(1 << 31), top])
    x32 = b.view(np.float32)
    keep = np.isfinite(x32)
    b, x32 = b[keep], x32[keep]
    want = _bits_round(b, p).view(np.float32).astype(np.float64)
    got = O.round_sim(p, x32.astype(np.float64))
    assert np.array_equal(got, want)


def test_shift_sim_rounds_the_exact_difference():
    # mu on a midpoint of the 3-bit grid, y tiny: the fp64 difference is the
    # midpoint itself, the exact one lies on one side
    mu = np.array([1.0625, 1.0625, 1.0625, 1.0625 * 2 ** 60, 1.0625 * 2 ** 60, 5.0])
    y = np.array([2.0 ** -60, -(2.0 ** -60), 0.0, -1.0, 1.0, 5.0 + 2.0 ** -30])
    s = O.shift_sim(3, mu, y)
    assert list(s) == [1.0, 1.125, 1.0, 1.125 * 2 ** 60, 1.0 * 2 ** 60, 0.0]
    assert np.array_equal(R.sim_shift(mu, y, 3), s)
    rng = np.random.default_rng(7)
    for p in (3, 11):
        mu = O.round_sim(11, rng.standard_normal(4000) * np.exp2(rng.integers(-30, 10, 4000)))
        y = O.round_sim(p, rng.standard_normal(4000) * np.exp2(rng.integers(-70, 10, 4000)))
        got = O.shift_sim(p, mu, y)
        # the reference rounds the exact Fraction difference
        ref = [max(float(M.frac_round(Fraction(a) - Fraction(c), p, -126)), 0.0) if a > c else 0.0
               for a, c in zip(mu, y)]
        assert np.array_equal(got, np.array(ref))
        assert np.array_equal(R.sim_shift(mu, y, p), got)


@pytest.mark.parametrize("p", [3, 11])
def test_sim_exp_against_mpmath_on_every_shift(p):
    n = (M.SIM_EMAX - M.SIM_EMIN + 1) << p
    idx = np.arange(n)
    e = M.SIM_EMIN + (idx >> p)
    m = idx & ((1 << p) - 1)
    s = ((1 << p) + m) * np.exp2((e - p).astype(np.float64))
    got = O.sim_exp(p, s)
    assert np.array_equal(got, M.mp_sim_exp(p))
    # the saturated ends: shifts below 2^SIM_EMIN give 1, from 2^(SIM_EMAX+1) on 0
    lo = np.array([0.0, 2.0 ** -149, 2.0 ** (M.SIM_EMIN - 1) * 1.9])
    hi = np.array([2.0 ** (M.SIM_EMAX + 1), 1e4, 3e38])
    assert np.all(O.sim_exp(p, lo) == 1.0) and np.all(O.sim_exp(p, hi) == 0.0)
    assert np.array_equal(got, M.sim_exp_lookup(s, p))
    # values on the grid; the smallest nonzero lies in FP32's subnormal range
    assert np.array_equal(O.round_sim(p, got), got)
    assert got[got > 0].min() < 2.0 ** -126


def _sim_bits(w):
    q, k, v = W.make_inputs(w)
    return O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)


def test_sim_logits_single_channel_and_small_integers():
    rng = np.random.default_rng(3)
    # d = 1: one FP32 product, one rounding (scale 1/sqrt(1) = 1)
    q = (rng.standard_normal((1, 1, 16, 1)) * 8).astype(np.float32)
    k = (rng.standard_normal((1, 1, 16, 1)) * 8).astype(np.float32)
    qb = (q.view(np.uint32) >> 16).astype(np.uint16)
    kb = (k.view(np.uint32) >> 16).astype(np.uint16)
    qf, kf = M.bf16_to_float(qb), M.bf16_to_float(kb)
    for high, p in ((0, 3), (1, 11)):
        y = O.logits_sim(qb, kb, 0, 0, 0, 16, high)[0, 0]
        prod = (qf[0, 0, :, 0][:, None] * kf[0, 0, :, 0][None, :]).astype(np.float32).astype(np.float64)
        assert np.array_equal(y, O.round_sim(p, prod))
    # small integers (d = 16, scale 1/4 exact): every partial sum is on the
    # 3-bit grid when the operands are multiples of 4 of magnitude <= 4
    d = 16
    qi = rng.integers(-1, 2, (1, 1, 8, d)) * 4.0
    ki = rng.integers(-1, 2, (1, 1, 8, d)) * 1.0
    to_b = lambda a: (a.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    y = O.logits_sim(to_b(qi), to_b(ki), 0, 0, 0, 8, 0)[0, 0]
    assert np.array_equal(y, qi[0, 0] @ ki[0, 0].T / 4.0)


@pytest.mark.parametrize("high", [0, 1])
def test_sim_logits_fraction_brute_force(high):
    w = W.small("simlog", N=12, d=24, Hq=1, Hkv=1, bq=12, bk=4, nk=3, causal=0, seed=61, kind="outlier",
                n_outlier=2, outlier_gain=40.0)
    q, k, _ = _sim_bits(w)
    y = O.logits_sim(q, k, 0, 0, 0, w.N, high)[0, 0]
    s = Fraction(float(O.scale(w.d)))
    qt = [[M.rn32(Fraction(float(x)) * s) for x in row] for row in M.bf16_to_float(q[0, 0])]
    kf = [[Fraction(float(x)) for x in row] for row in M.bf16_to_float(k[0, 0])]
    p = 11 if high else 3
    for j in range(w.N):
        for i in range(w.N):
            acc = Fraction(0)
            for c in range(w.d):
                acc = M.rn32(qt[j][c] * kf[i][c] + acc)
                if not high:
                    acc = M.frac_round(acc, 3, -126)
            if high:
                acc = M.frac_round(acc, 11, -126)
            assert y[j, i] == float(acc)
    assert np.abs(y).max() > 448.0      # beyond e4m3's range: the profile does not saturate


SIM_CASES = [
    W.small("s_causal", N=96, d=16, Hq=2, Hkv=1, bq=32, bk=8, nk=4, causal=1, seed=71),
    W.small("s_outlier", N=64, d=32, Hq=1, Hkv=1, bq=32, bk=16, nk=2, causal=0, seed=72, kind="outlier",
            n_outlier=2, outlier_gain=16.0),
    W.small("s_window", N=80, d=8, Hq=1, Hkv=1, bq=16, bk=4, nk=4, causal=1, window=20, seed=73),
]


@pytest.fixture(scope="session")
def mp_tables():
    return M.mp_exp_tables()


@pytest.mark.parametrize("tau", [math.inf, 1.0, 0.5, 2.0 ** -5, 0.0])
@pytest.mark.parametrize("w", SIM_CASES, ids=[w.name for w in SIM_CASES])
def test_sim_fwd_matches_independent_implementation(w, tau, mp_tables):
    q, k, v = _sim_bits(w)
    o, lse, mask = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=O.SIM)
    ro, rlse, rmask = R.ref_fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau,
                                mp_tables, O.scale(w.d), flags=O.SIM)
    assert np.array_equal(mask, rmask)
    np.testing.assert_allclose(o, ro, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)
    if tau == 1.0:
        assert not np.any(mask == 2)


@pytest.mark.parametrize("flags", [O.STAGE1_OFF, O.MU_TRUNC])
def test_sim_with_stage_variants(flags, mp_tables):
    w = SIM_CASES[0]
    q, k, v = _sim_bits(w)
    f = flags | O.SIM
    o, lse, mask = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 2.0 ** -5, flags=f)
    ro, rlse, rmask = R.ref_fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 2.0 ** -5,
                                mp_tables, O.scale(w.d), flags=f)
    assert np.array_equal(mask, rmask)
    np.testing.assert_allclose(o, ro, rtol=1e-9, atol=1e-12)


def test_trunc_sim3():
    x = np.array([1.0625, -1.99, 1000.0, 2.0 ** -127 * 1.7, math.inf, -math.inf, 0.0])
    got = np.array([O.trunc_sim3(v) for v in x])
    assert np.array_equal(got, np.array([1.0, -1.875, 960.0, 2.0 ** -127 * 1.5, math.inf, -math.inf, 0.0]))
    assert np.array_equal(R._trunc_sim3(x), got)


def test_sim_pure8_single_tile_is_naive_softmax():
    w = W.CONFIGS[1]
    q, k, v = _sim_bits(w)
    o, lse, mask = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, math.inf, flags=O.SIM)
    assert np.all(mask == 0)
    y8 = O.logits_sim(q, k, 0, 0, 0, w.N, 0)[0, 0]            # [j, i]
    mx = y8.max(axis=1, keepdims=True)
    E = M.sim_exp_lookup(R.sim_shift(mx, y8, 3), 3)
    vf = M.bf16_to_float(v[0, 0])
    S = np.zeros(w.N)
    for i in range(w.N):
        S = S + E[:, i]
    np.testing.assert_allclose(o[0, 0], (E @ vf) / S[:, None], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse[0, 0], mx[:, 0] + np.log(S), rtol=0, atol=1e-12)


def test_sim_differs_from_hardware_profile_where_e4m3_saturates():
    w = W.small("s_sat", N=64, d=32, Hq=1, Hkv=1, bq=32, bk=16, nk=2, causal=0, seed=74, kind="outlier",
                n_outlier=2, outlier_gain=40.0)   # outlier channels: logits beyond 448
    q, k, v = _sim_bits(w)
    y_hw = M.np_decode(O.logits8(q, k, 0, 0, 0, w.N)[0, 0].astype(np.int64), "e4m3")
    y_sim = O.logits_sim(q, k, 0, 0, 0, w.N, 0)[0, 0]
    assert np.abs(y_hw).max() == 448.0 and np.abs(y_sim).max() > 448.0
    o1 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.5)[0]
    o2 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.5, flags=O.SIM)[0]
    assert not np.array_equal(o1, o2)
