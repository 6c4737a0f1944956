"""Pins of the oracle's variants of Algorithm 1.

* first stage disabled (the paper's appendix on first-stage recomputation):
  mu_hat from the 8-bit maxima, stage 2 alone recomputes;
* 8-bit shifts against mu_hat truncated to e4m3 (Sec. 3.3, hardware
  co-design: the running maxima may be rounded to e4m3 for the low-precision
  shifts by dropping the low mantissa bits).

Pinned by: the truncation against its definition on every e4m11 value; the
independent implementation (tests/refimpl.py) on small problems; with the
first stage off and threshold 1 the second stage never recomputes (xi <=
omega_hat^2 always), so the pass is the pure 8-bit path exactly; neither
flag changes the two end modes.
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


def _bits(w):
    q, k, v = W.make_inputs(w)
    return O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)


def test_trunc_e4m3_every_e4m11_value():
    codes = np.arange(1 << 16, dtype=np.uint32)
    x = O.decode_fmt(O.E4M11, codes)
    t = np.array([O.trunc_e4m3(v) for v in x])
    # on the e4m3 grid, same sign, not larger in magnitude
    assert np.array_equal(O.round_fmt(O.E4M3, t), t)
    assert np.all((np.sign(t) == np.sign(x)) | (t == 0))
    assert np.all(np.abs(t) <= np.minimum(np.abs(x), 448.0))
    # the next e4m3 magnitude above |t| exceeds |x| (toward zero), unless saturated
    mags = np.unique(np.abs(O.decode_fmt(O.E4M3, np.arange(0, 0x7F, dtype=np.uint32))))
    nxt = mags[np.minimum(np.searchsorted(mags, np.abs(t), side="right"), mags.size - 1)]
    sat = np.abs(x) >= 448.0
    assert np.all(sat | (nxt > np.abs(x)))
    assert np.all(np.abs(t[sat]) == 448.0)
    # e4m3 values are fixed points; an independent integer-grid rendering agrees
    e3 = O.decode_fmt(O.E4M3, np.arange(0, 0x7F, dtype=np.uint32))
    assert np.array_equal(np.array([O.trunc_e4m3(v) for v in e3]), e3)
    assert np.array_equal(R._trunc_e4m3(x), t)
    assert O.trunc_e4m3(-math.inf) == -math.inf


VCASES = [
    W.small("v_causal", N=96, d=16, Hq=2, Hkv=1, bq=32, bk=8, nk=4, causal=1, seed=31),
    W.small("v_nc_outlier", N=64, d=32, Hq=1, Hkv=1, bq=32, bk=16, nk=2, causal=0, seed=32, kind="outlier",
            n_outlier=2, outlier_gain=16.0),
    W.small("v_window", N=96, d=8, Hq=1, Hkv=1, bq=16, bk=4, nk=4, causal=1, window=20, seed=33),
]


@pytest.mark.parametrize("flags", [O.STAGE1_OFF, O.MU_TRUNC, O.STAGE1_OFF | O.MU_TRUNC])
@pytest.mark.parametrize("tau", [1.0, 0.5, 2.0 ** -5])
@pytest.mark.parametrize("w", VCASES, ids=[w.name for w in VCASES])
def test_variants_match_independent_implementation(w, tau, flags, mp_tables):
    q, k, v = _bits(w)
    o, lse, mask = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=flags)
    ro, rlse, rmask = R.ref_fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau,
                                mp_tables, O.scale(w.d), flags=flags)
    assert np.array_equal(mask, rmask)
    np.testing.assert_allclose(o, ro, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)
    if flags & O.STAGE1_OFF:
        assert not np.any(mask == 1)


def test_stage1_off_at_threshold_one_is_the_pure_8bit_path():
    w = W.small("v_t1", N=128, d=32, Hq=2, Hkv=1, bq=32, bk=8, nk=4, causal=1, seed=34)
    q, k, v = _bits(w)
    o1, l1, m1 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 1.0, flags=O.STAGE1_OFF)
    o8, l8, m8 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, math.inf)
    assert np.array_equal(m1, m8)
    assert np.array_equal(o1, o8) and np.array_equal(l1, l8)


def test_stage1_off_recomputes_only_in_stage2_and_trunc_changes_exponentials():
    w = W.small("v_mix", N=128, d=32, Hq=2, Hkv=1, bq=32, bk=8, nk=4, causal=1, seed=36)
    q, k, v = _bits(w)
    o0, _, m0 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 2.0 ** -5)
    o1, _, m1 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 2.0 ** -5, flags=O.STAGE1_OFF)
    o2, _, m2 = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 2.0 ** -5, flags=O.MU_TRUNC)
    assert np.any(m0 == 1) and not np.any(m1 == 1) and np.any(m1 == 2)
    assert not np.array_equal(o0, o2)          # truncation moves some 8-bit exponentials


@pytest.mark.parametrize("tau", [math.inf, 0.0])
def test_flags_do_not_change_the_end_modes(tau):
    w = W.small("v_end", N=64, d=16, Hq=1, Hkv=1, bq=32, bk=8, nk=4, causal=1, seed=36)
    q, k, v = _bits(w)
    ref = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau)
    got = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=O.STAGE1_OFF | O.MU_TRUNC)
    for a, b in zip(ref, got):
        assert np.array_equal(a, b)
