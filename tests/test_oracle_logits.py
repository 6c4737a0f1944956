"""Pins of the oracle's logits.

Y8 (paper Sec. 4.1, Alg. 1): recursive summation with one FP32 FMA per step,
the running sum rounded to e4m3 after every step, channels ascending.
Y16: FP32 FMA chain rounded once to e4m11; and the alternative reading with
e4m11 as the accumulator (rounded after every FMA).  All are re-derived here with
exact rational arithmetic (Python Fractions), a different method from the
oracle's float code."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
import fpmodel as M
from paper_2609_39361_amd import workloads as W


def _frac_y8(qrow_bits, krow_bits, s):
    acc = Fraction(0)
    for qb, kb in zip(qrow_bits, krow_bits):
        qt = M.rn32(Fraction(float(M.bf16_to_float(qb))) * Fraction(float(s)))
        acc = M.frac_fmt(M.rn32(qt * Fraction(float(M.bf16_to_float(kb))) + acc), "e4m3")
    return acc


def _frac_y16(qrow_bits, krow_bits, s):
    acc = Fraction(0)
    for qb, kb in zip(qrow_bits, krow_bits):
        qt = M.rn32(Fraction(float(M.bf16_to_float(qb))) * Fraction(float(s)))
        acc = M.rn32(qt * Fraction(float(M.bf16_to_float(kb))) + acc)
    return M.frac_fmt(acc, "e4m11")


def _frac_y16_step(qrow_bits, krow_bits, s):
    """The literal Sec. 3.3 reading: e4m11 as the accumulator, every FP32 FMA
    result rounded to e4m11 (saturating) before the next step."""
    acc = Fraction(0)
    for qb, kb in zip(qrow_bits, krow_bits):
        qt = M.rn32(Fraction(float(M.bf16_to_float(qb))) * Fraction(float(s)))
        acc = M.frac_fmt(M.rn32(qt * Fraction(float(M.bf16_to_float(kb))) + acc), "e4m11")
    return acc


def _inputs(d, N, seed, gain=1.0, kind="gauss"):
    w = W.small(N=N, d=d, Hq=1, Hkv=1, bq=N, bk=N, nk=1, seed=seed, kind=kind, causal=0,
                extra={"gain": gain})
    q, k, v = W.make_inputs(w)
    return O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)


def test_y8_d1_is_single_rounding():
    """d = 1: Y8 = RN_e4m3(RN32(q_tilde * k))."""
    q, k, _ = _inputs(1, 64, 0, gain=30.0)
    s = O.scale(1)
    y = O.logits8(q, k, 0, 0, 0, 64)
    qf = M.bf16_to_float(q[0, 0, :, 0])
    kf = M.bf16_to_float(k[0, 0, :, 0])
    qt = (qf * s).astype(np.float32).astype(np.float64)
    prod = (qt[:, None] * kf[None, :]).astype(np.float32).astype(np.float64)   # exact product, RN32
    ref = M.np_encode(M.np_round(prod, "e4m3"), "e4m3")
    assert np.array_equal(y[0, 0].astype(np.int64), ref)


def test_y8_small_integers_exact():
    """Small-integer inputs with d = 64 (scale 1/8 exact): every partial sum
    is a multiple of 1/8 bounded by 16 and so exactly representable in e4m3
    below 16 only if it has <= 4 significant bits; restrict to d = 4, values
    in {-1, 0, 1} where all partial sums are in {-4/8..4/8} (exact)."""
    w = W.small(N=64, d=4, Hq=1, Hkv=1, bq=64, bk=64, nk=1, kind="small_int", causal=0,
                extra={"lim": 1})
    q, k, v = W.make_inputs(w)
    qb, kb = O.bf16_bits(q), O.bf16_bits(k)
    y = O.logits8(qb, kb, 0, 0, 0, 64)
    val = O.decode_fmt(O.E4M3, y.astype(np.uint32))[0, 0]
    exact = (q[0, 0].double() * 0.5) @ k[0, 0].double().T          # s = RN32(1/2) = 0.5
    assert np.array_equal(val, exact.numpy())


@pytest.mark.parametrize("d,seed,gain", [(8, 1, 1.0), (16, 2, 3.0), (64, 3, 1.0), (64, 4, 6.0), (128, 5, 2.0)])
def test_y8_vs_fraction_bruteforce(d, seed, gain):
    N = 16
    q, k, _ = _inputs(d, N, seed, gain)
    s = O.scale(d)
    y = O.logits8(q, k, 0, 0, 0, N)
    val = O.decode_fmt(O.E4M3, y.astype(np.uint32))[0, 0]
    for j in range(0, N, 3):
        for i in range(N):
            ref = _frac_y8(q[0, 0, j], k[0, 0, i], s)
            assert val[j, i] == float(ref), (j, i, val[j, i], float(ref))


@pytest.mark.parametrize("d,seed,gain", [(8, 6, 1.0), (64, 7, 1.0), (128, 8, 4.0)])
def test_y16_vs_fraction_bruteforce(d, seed, gain):
    N = 12
    q, k, _ = _inputs(d, N, seed, gain)
    s = O.scale(d)
    y = O.logits16(q, k, 0, 0, 0, N)
    val = O.decode_fmt(O.E4M11, y.astype(np.uint32))[0, 0]
    for j in range(N):
        for i in range(0, N, 2):
            ref = _frac_y16(q[0, 0, j], k[0, 0, i], s)
            assert val[j, i] == float(ref)
            # and close to the correctly rounded exact dot product: the FP32
            # chain is off by at most d * 2^-24 * sum|products|
            qt = [M.rn32(Fraction(float(M.bf16_to_float(a))) * Fraction(float(s))) for a in q[0, 0, j]]
            prods = [a * Fraction(float(M.bf16_to_float(b))) for a, b in zip(qt, k[0, 0, i])]
            ex = sum(prods)
            bound = d * 2.0 ** -24 * float(sum(abs(p) for p in prods))
            assert abs(val[j, i] - float(ex)) <= bound + 2.0 ** -12 * abs(float(ex)) + 2.0 ** -18


def test_y8_saturation_and_sign_of_zero():
    """Outlier-scaled inputs saturate at +-448; an all-zero key gives +0."""
    q, k, _ = _inputs(64, 16, 9, gain=40.0)
    k[0, 0, 3, :] = 0
    y = O.logits8(q, k, 0, 0, 0, 16)
    val = O.decode_fmt(O.E4M3, y.astype(np.uint32))[0, 0]
    assert np.all(np.abs(val) <= 448.0)
    assert np.any(np.abs(val) == 448.0)
    assert np.all(y[0, 0, :, 3] == 0x00)
    for j in range(0, 16, 5):
        for i in (0, 5, 11):
            assert val[j, i] == float(_frac_y8(q[0, 0, j], k[0, 0, i], O.scale(64)))


def test_visibility_conventions():
    """Causal: key i visible to query j iff i <= j; window W: also i > j - W."""
    w = W.small(N=32, d=8, Hq=2, Hkv=1, bq=32, bk=8, nk=4, causal=1)
    q, k, _ = W.make_inputs(w)
    qb, kb = O.bf16_bits(q), O.bf16_bits(k)
    yc = O.logits8(qb, kb, 1, 0, 0, 32)
    yw = O.logits8(qb, kb, 1, 5, 0, 32)
    j = np.arange(32)[:, None]
    i = np.arange(32)[None, :]
    assert np.array_equal(yc[0, 0] == 0xFF, i > j)
    assert np.array_equal(yw[0, 0] == 0xFF, (i > j) | (i <= j - 5))
    # GQA: both query heads read kv head 0
    y1 = O.logits8(qb[:, 1:2].copy(), kb, 1, 0, 0, 32)
    assert np.array_equal(y1[0, 0], yc[0, 1])


@pytest.mark.parametrize("d,seed,gain", [(8, 21, 1.0), (64, 22, 1.0), (128, 23, 4.0), (128, 24, 30.0)])
def test_y16_step_vs_fraction_bruteforce(d, seed, gain):
    """The per-FMA e4m11 reading (ORACLE_Y16_STEP) against exact rational
    arithmetic, including inputs large enough to saturate at 511.875; and it
    differs from the FP32-chain reading somewhere (the readings are distinct)."""
    N = 12
    q, k, _ = _inputs(d, N, seed, gain)
    s = O.scale(d)
    y = O.logits16_step(q, k, 0, 0, 0, N)
    val = O.decode_fmt(O.E4M11, y.astype(np.uint32))[0, 0]
    for j in range(0, N, 2):
        for i in range(N):
            ref = _frac_y16_step(q[0, 0, j], k[0, 0, i], s)
            assert val[j, i] == float(ref), (j, i, val[j, i], float(ref))
    if d >= 64:
        chain = O.decode_fmt(O.E4M11, O.logits16(q, k, 0, 0, 0, N).astype(np.uint32))[0, 0]
        assert np.any(chain != val)
    if gain >= 30.0:
        assert np.any(np.abs(val) == 511.875)
