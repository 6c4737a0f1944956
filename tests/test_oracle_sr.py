"""Pins of the oracle's stochastic rounding of the 8-bit accumulation (the
alternative to round-to-nearest that Sec. 3.3 names against swamping).

Readings (the paper fixes neither generator nor bit count): each FP32 FMA
result is rounded to one of its two e4m3 neighbours, away from zero when
floor(2^16 * distance to the lower one / spacing) + r >= 2^16 for a 16-bit
uniform r, saturating at 448; r comes from Philox4x32-10 keyed by (seed mod
2^32, seed / 2^32) at counter (query row, key, b*Hq + h, channel / 8): the
low (even channel) or high (odd channel) half of word (channel mod 8) / 2.

Pinned by: the library routine rocRAND's Philox4x32-10 stream on the GPU machine
(tests/test_gpu_rocrand.py: counter (n, 0, 0, 0), key = the seed's halves),
and here by what any correct Philox4x32-10 has (every output bit balanced,
the 16-bit fields uniform, one flipped counter or key bit flipping half the
output bits) and a second implementation written apart (tests/refimpl.py);
the rounding against the enumerated e4m3 grid and a second rounding written
with a grid search; exact unbiasedness over all 2^16 random integers; the
8-bit logits and the whole forward pass against the independent
implementation; a swamping example in which round-to-nearest loses every
small term while the stochastic mean keeps the exact sum.
"""
import math

import numpy as np
import pytest

from oracle import oracle as O
import fpmodel as M
import refimpl as R
from paper_2609_39361_amd import workloads as W


@pytest.fixture(scope="session")
def mp_tables():
    return M.mp_exp_tables()


PHILOX_CASES = [
    ([0, 0, 0, 0], [0, 0]),
    ([1, 0, 0, 0], [0, 0]),
    ([5, 7, 9, 11], [0x1234, 0x5678]),
    ([2 ** 32 - 1, 2 ** 32 - 1, 3, 0], [2 ** 32 - 1, 2 ** 32 - 1]),
    ([123456789, 42, 31, 15], [0xCAFEF00D, 0xDEADBEEF]),
]


@pytest.mark.parametrize("ctr,key", PHILOX_CASES)
def test_philox_matches_the_second_implementation(ctr, key):
    got = O.philox4x32_10(ctr, key)
    want = R.philox4x32(np.array(ctr, dtype=np.uint64), (key[0], key[1]))
    assert np.array_equal(got.astype(np.uint64), want)


def test_philox_output_statistics():
    """Over 2^13 consecutive counters: each of the 128 output bits is set in
    half the calls (within 5 standard deviations), the 16-bit fields are
    uniform (chi-square over 16 bins of their top nibble), and flipping any
    one of the 192 counter and key bits flips 64 of the 128 output bits on
    average (within 4 of 64 over 64 random inputs per bit)."""
    n = 1 << 13
    ctr = np.zeros((n, 4), dtype=np.uint64)
    ctr[:, 0] = np.arange(n)
    ctr[:, 2] = 7
    key = (0x9E3779B9, 0x243F6A88)
    out = R.philox4x32(ctr, key)
    for t in range(4):
        c = np.array([O.philox4x32_10(ctr[t * 997], key)], dtype=np.uint64)
        assert np.array_equal(c[0], out[t * 997])
    bits = ((out[:, :, None] >> np.arange(32, dtype=np.uint64)) & np.uint64(1)).reshape(n, 128)
    frac = bits.mean(axis=0)
    assert np.all(np.abs(frac - 0.5) < 5 * 0.5 / np.sqrt(n))
    fields = np.concatenate([out & np.uint64(0xFFFF), out >> np.uint64(16)]).ravel()
    hist = np.bincount((fields >> np.uint64(12)).astype(np.int64), minlength=16)
    expect = fields.size / 16
    chi2 = ((hist - expect) ** 2 / expect).sum()
    assert chi2 < 50.0                                  # 15 degrees of freedom: p ~ 1e-5
    rng = np.random.default_rng(3)
    base = rng.integers(0, 2 ** 32, (64, 4), dtype=np.uint64)
    keys = rng.integers(0, 2 ** 32, (64, 2), dtype=np.uint64)
    ref = np.stack([O.philox4x32_10(base[m], keys[m]) for m in range(64)]).astype(np.uint64)
    def popcount(x):
        return sum(((x >> np.uint64(b)) & np.uint64(1)) for b in range(32)).sum(axis=-1)
    for bit in range(192):
        flipped = []
        for m in range(64):
            c, k = base[m].copy(), keys[m].copy()
            if bit < 128:
                c[bit // 32] ^= np.uint64(1 << (bit % 32))
            else:
                k[(bit - 128) // 32] ^= np.uint64(1 << (bit % 32))
            flipped.append(O.philox4x32_10(c, k).astype(np.uint64))
        d = popcount(np.stack(flipped) ^ ref)
        assert abs(d.mean() - 64.0) < 4.0, bit


def _f32_values(rng, n):
    # FP32 numbers over the e4m3 range and beyond: normal, subnormal-range, saturating, zero
    mag = np.concatenate([2.0 ** rng.uniform(-6, 8.8, n), 2.0 ** rng.uniform(-14, -6, n // 4),
                          rng.uniform(448, 600, n // 8), [0.0, 448.0, 2.0 ** -9, 2.0 ** -6, 1.0]])
    t = (mag * rng.choice([-1.0, 1.0], mag.size)).astype(np.float32).astype(np.float64)
    return t


def test_sr_picks_a_neighbour_on_the_grid():
    rng = np.random.default_rng(7)
    t = _f32_values(rng, 4000)
    r = rng.integers(0, 1 << 16, t.size).astype(np.uint32)
    y = O.sr_e4m3(t, r)
    mags = R.e4m3_mags()
    a = np.minimum(np.abs(t), 448.0)
    idx = np.searchsorted(mags, a, side="right") - 1
    lo, hi = mags[idx], mags[np.minimum(idx + 1, mags.size - 1)]
    assert np.all((np.abs(y) == lo) | (np.abs(y) == hi))
    assert np.all(np.signbit(y) == np.signbit(t))
    # every result is an e4m3 value (round-to-nearest leaves it unchanged)
    assert np.array_equal(O.round_fmt(O.E4M3, y), y)
    # r = 0 truncates toward zero; grid values and saturation are fixed points
    assert np.array_equal(np.abs(O.sr_e4m3(t, 0)), lo)
    on_grid = a == lo
    for rr in (0, 1, 1 << 15, (1 << 16) - 1):
        assert np.array_equal(np.abs(O.sr_e4m3(t, rr))[on_grid], lo[on_grid])
    assert np.all(np.abs(O.sr_e4m3(t[np.abs(t) >= 448], (1 << 16) - 1)) == 448.0)
    # the independent rounding agrees everywhere
    assert np.array_equal(y, R.sr_round(t, r))


def test_sr_is_unbiased_over_all_random_integers():
    """Mean over r in [0, 2^16) equals t exactly where t is a multiple of
    2^-16 of the e4m3 spacing (FP32 values whose 4 lowest of the 20 bits below
    e4m3's last bit are zero), and the value with the distance cut to 16 bits
    where it is not."""
    r = np.arange(1 << 16, dtype=np.uint32)

    def cut4(x):
        b = np.float32(x).view(np.uint32) & np.uint32(0xFFFFFFF0)
        return float(b.view(np.float32))
    for t in (1.0 + 2 ** -19, cut4(3.14159274101257324), cut4(17.3), -cut4(200.123), cut4(447.9), cut4(0.0157),
              2.0 ** -6 + 2 ** -25, -(2.0 ** -7 + 2.0 ** -25)):
        y = O.sr_e4m3(np.full(r.size, t), r)
        assert math.fsum(y) / r.size == t, t
    for t, cut in ((1.0 + 2 ** -23, 1.0), (float(np.float32(2.0 ** -7 + 2.0 ** -30)), 2.0 ** -7)):
        y = O.sr_e4m3(np.full(r.size, t), r)
        assert math.fsum(y) / r.size == cut


def _bits(w):
    q, k, v = W.make_inputs(w)
    return O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)


def _codes_of(vals):
    mags = R.e4m3_mags()
    idx = np.searchsorted(mags, np.abs(vals))
    assert np.array_equal(mags[idx], np.abs(vals))
    return (idx | np.where(np.signbit(vals), 0x80, 0)).astype(np.uint8)


@pytest.mark.parametrize("d,causal,window,seed", [(32, 1, 0, 11), (16, 1, 9, 2 ** 63 + 3), (24, 0, 0, 0)])
def test_logits8_sr_match_independent_implementation(d, causal, window, seed):
    w = W.small("sr", N=40, d=d, Hq=2, Hkv=1, causal=causal, window=window, seed=5, kind="outlier",
                n_outlier=2, outlier_gain=8.0)
    q, k, _ = _bits(w)
    got = O.logits8_sr(q, k, causal, window, 0, w.N, seed)
    s = O.scale(d)
    for h in range(2):
        qt = (M.bf16_to_float(q[0, h]) * np.float64(s)).astype(np.float32).astype(np.float64)
        kf = M.bf16_to_float(k[0, 0])
        keys = np.arange(w.N)
        Y = R.y8_tile_sr(qt, kf, seed, h, keys, keys)          # [key, row]
        want = _codes_of(Y.T)
        jj, ii = np.meshgrid(keys, keys, indexing="ij")
        vis = np.ones_like(jj, dtype=bool)
        if causal:
            vis &= ii <= jj
        if window:
            vis &= ii > jj - window
        assert np.array_equal(got[0, h][vis], want[vis])
        assert np.all(got[0, h][~vis] == 0xFF)
    # a different seed changes some logits, the same seed none; round-to-nearest differs too
    assert np.array_equal(O.logits8_sr(q, k, causal, window, 0, w.N, seed), got)
    assert not np.array_equal(O.logits8_sr(q, k, causal, window, 0, w.N, seed + 1), got)
    assert not np.array_equal(O.logits8(q, k, causal, window, 0, w.N), got)


def test_sr_keeps_the_small_terms_that_rounding_to_nearest_swamps():
    """One product of 16 followed by 255 products of 2^-5: round-to-nearest
    stays at 16 (each term is below half the spacing 2 of e4m3 at 16), while
    the mean of the stochastic logits over 4096 independent pairs is the exact
    sum 16 + 255/32 within 3 standard errors."""
    d, N = 256, 64
    def bf(x):
        return (np.array(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)
    qrow = np.full(d, 2.0)
    qrow[0] = 64.0                                   # x 1/16 (exact for d = 256): 4, then 1/8
    krow = np.full(d, 0.25)
    krow[0] = 4.0
    q = np.broadcast_to(bf(qrow), (1, 1, N, d)).copy()
    k = np.broadcast_to(bf(krow), (1, 1, N, d)).copy()
    exact = 16.0 + 255 / 32.0
    rn = O.decode_fmt(O.E4M3, O.logits8(q, k, 0, 0, 0, N).astype(np.uint32))
    assert np.all(rn == 16.0)
    y = O.decode_fmt(O.E4M3, O.logits8_sr(q, k, 0, 0, 0, N, 2024).astype(np.uint32)).ravel()
    assert abs(y.mean() - exact) < 3 * y.std() / math.sqrt(y.size)
    assert y.min() >= 16.0                            # the terms are positive: never below the first


SR_CASES = [
    W.small("sr_causal", N=64, d=16, Hq=2, Hkv=1, bq=32, bk=8, nk=4, causal=1, seed=41),
    W.small("sr_ragged_outlier", N=50, d=24, Hq=1, Hkv=1, bq=16, bk=8, nk=2, causal=0, seed=42, kind="outlier",
            n_outlier=2, outlier_gain=16.0),
]


@pytest.mark.parametrize("flags", [O.SR8, O.SR8 | O.STAGE1_OFF, O.SR8 | O.MU_TRUNC])
@pytest.mark.parametrize("tau", [math.inf, 0.5, 2.0 ** -5])
@pytest.mark.parametrize("w", SR_CASES, ids=[w.name for w in SR_CASES])
def test_fwd_sr_matches_independent_implementation(w, tau, flags, mp_tables):
    q, k, v = _bits(w)
    seed = 99
    o, lse, mask = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=flags, seed=seed)
    ro, rlse, rmask = R.ref_fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau,
                                mp_tables, O.scale(w.d), flags=flags, seed=seed)
    assert np.array_equal(mask, rmask)
    np.testing.assert_allclose(o, ro, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)


def test_fwd_sr_leaves_the_all_16bit_mode_alone_and_refuses_the_sim_profile():
    w = SR_CASES[0]
    q, k, v = _bits(w)
    a = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.0, flags=O.SR8, seed=5)
    b = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.0)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    with pytest.raises(ValueError):
        O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.5, flags=O.SR8 | O.SIM, seed=5)
