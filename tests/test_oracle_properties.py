"""Property tests of the oracle: the C oracle against the independent Python
implementation (tests/refimpl.py) on shapes, thresholds, margins, flags and
input scales drawn by hypothesis, and invariants that hold for any input.

Drawn: B, Hkv, the GQA group, N (ragged against every block size), d, bq, bk,
nk, causal/window, tau (0, inf, 1, powers of two and arbitrary values in
(0, 1)), delta, the flags (first stage off, mu_hat truncated, the SIM
profile, the per-FMA e4m11 reading, stochastic rounding with a drawn seed)
and an input gain that reaches the saturating range of e4m3 and e4m11.
Compared: the mask byte for byte, the statistics words exactly, O and the
log-sum-exp to fp64 rounding.  The draws are derandomized, so a failure
reproduces on every run."""
import math

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import oracle as O
import fpmodel as M
import refimpl as R
from paper_2609_39361_amd import workloads as W

_TABLES = None


def _tables():
    global _TABLES
    if _TABLES is None:
        _TABLES = M.mp_exp_tables()
    return _TABLES


@st.composite
def problems(draw):
    B = draw(st.integers(1, 2))
    Hkv = draw(st.integers(1, 2))
    G = draw(st.integers(1, 2))
    d = draw(st.sampled_from([4, 8, 16]))
    bq = draw(st.sampled_from([8, 16, 32]))
    bk = draw(st.sampled_from([4, 8]))
    nk = draw(st.integers(1, 4))
    N = draw(st.integers(1, 72))
    causal = draw(st.integers(0, 1))
    window = draw(st.integers(0, N + 2)) if causal and draw(st.booleans()) else 0
    tau = draw(st.one_of(st.sampled_from([0.0, math.inf, 1.0, 0.5, 2.0 ** -5]),
                         st.floats(0.0, 1.0, allow_nan=False, exclude_min=True)))
    delta = draw(st.sampled_from([0.0, 2.0 ** -8, 2.0 ** -4]))
    flags = 0
    for bit in (1, 2, 4, 16):
        if draw(st.booleans()):
            flags |= bit
    seed = 0
    if not flags & 4 and draw(st.integers(0, 3)) == 0:
        flags |= 8
        seed = draw(st.integers(0, 2 ** 64 - 1))
    gain = draw(st.sampled_from([1.0, 1.0, 4.0, 24.0]))
    wseed = draw(st.integers(0, 2 ** 31 - 1))
    kind = draw(st.sampled_from(["gauss", "rope_lognormal"]))
    w = W.small("drawn", B=B, Hq=Hkv * G, Hkv=Hkv, N=N, d=d, causal=causal, window=window, bq=bq, bk=bk, nk=nk,
                seed=wseed, kind=kind, extra={"gain": gain})
    return w, tau, delta, flags, seed


def _stat_vector(s, nk):
    return [s["tiles"], s["stage1"], s["stage2"], s["inactive"], s["sat8"], s["sat16"], 0, 0] + s["hist"]


@settings(max_examples=40, deadline=None, derandomize=True, database=None,
          suppress_health_check=[HealthCheck.too_slow])
@given(problems())
def test_oracle_matches_independent_implementation_on_drawn_problems(prob):
    w, tau, delta, flags, seed = prob
    q, k, v = (O.bf16_bits(t) for t in W.make_inputs(w))
    o, lse, mask, s = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, delta, tau, flags=flags, seed=seed,
                            stats=True)
    ro, rlse, rmask, rs = R.ref_fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, delta, tau, _tables(),
                                    O.scale(w.d), flags=flags, seed=seed, stats=True)
    assert np.array_equal(mask, rmask)
    assert s.tolist() == _stat_vector(rs, w.nk)
    np.testing.assert_allclose(o, ro, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)


@settings(max_examples=40, deadline=None, derandomize=True, database=None,
          suppress_health_check=[HealthCheck.too_slow])
@given(problems())
def test_invariants_on_drawn_problems(prob):
    """For any input: O and the log-sum-exp are finite; every row of O lies in
    the box spanned by the value rows it can see (a convex combination); the
    mask marks exactly the sub-blocks holding no visible key inactive; the
    statistics words count the mask; tau = inf recomputes nothing and tau = 0
    everything visible."""
    w, tau, delta, flags, seed = prob
    q, k, v = (O.bf16_bits(t) for t in W.make_inputs(w))
    o, lse, mask, s = O.fwd(q, k, v, w.causal, w.window, w.bq, w.bk, w.nk, delta, tau, flags=flags, seed=seed,
                            stats=True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    vf = M.bf16_to_float(v)
    G = w.Hq // w.Hkv
    j = np.arange(w.N)[:, None]
    i = np.arange(w.N)[None, :]
    vis = np.ones((w.N, w.N), dtype=bool)
    if w.causal:
        vis &= i <= j
        if w.window:
            vis &= i > j - w.window
    for b in range(w.B):
        for h in range(w.Hq):
            vv = vf[b, h // G]
            for r in range(w.N):
                rows = vv[vis[r]]
                lo, hi = rows.min(axis=0), rows.max(axis=0)
                slack = 1e-12 * np.maximum(1.0, np.abs(rows).max(axis=0))
                assert np.all(o[b, h, r] >= lo - slack) and np.all(o[b, h, r] <= hi + slack)
    # a sub-block is active iff some row of its query block sees one of its keys
    T = w.bk * w.nk
    nqb, ntiles = -(-w.N // w.bq), -(-w.N // T)
    for qb in range(nqb):
        rr = vis[qb * w.bq: min(w.N, (qb + 1) * w.bq)]
        for sb in range(ntiles * w.nk):
            seen = rr[:, sb * w.bk: min(w.N, (sb + 1) * w.bk)].any() if sb * w.bk < w.N else False
            assert np.all((mask[:, :, qb, sb] != 3) == seen)
    m = mask.reshape(-1, w.nk)
    assert s[0] == (m != 3).any(axis=1).sum()
    assert s[1] == (mask == 1).sum() and s[2] == (mask == 2).sum() and s[3] == (mask == 3).sum()
    if math.isinf(tau):
        assert not np.any((mask == 1) | (mask == 2))
    if tau == 0.0:
        assert not np.any(mask == 0)
