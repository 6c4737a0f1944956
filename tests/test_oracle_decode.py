"""Pins of the oracle's vector-LAMP decode pass (paper Sec. 2, the two-step
look-ahead and the greedy knapsack of Eq. (6)), for query rows against a
key/value cache.

* an independent implementation (tests/refimpl.py) reproduces the masks and
  O / lse, and on every tile checks the greedy against the exact optimum of
  the uniform-value knapsack;
* threshold +inf and 0 equal the last rows of the block pass (Algorithm 1)
  run as a prefill with the same key tiles (both are then plain 8-bit /
  16-bit online softmax);
* threshold +inf on a single tile is a naive softmax of the rounded logits;
* threshold 1 never recomputes by the knapsack (sum p (1 - p) <= sum p <= 1);
* fewer knapsack recomputes as the threshold grows; a row subset equals the
  same rows of the full run; rows of P sum to one.
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


def _dec(w):
    q, k, v = W.make_inputs(w)
    return O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)


DCASES = [
    W.small("d_causal", B=1, Hq=4, Hkv=2, N=100, d=16, causal=1, seed=81, M=3, bk=8),
    W.small("d_window", B=1, Hq=2, Hkv=1, N=90, d=16, causal=1, window=30, seed=82, M=2, bk=8),
    W.small("d_noncausal", B=2, Hq=2, Hkv=2, N=64, d=8, causal=0, seed=83, M=2, bk=16, scale_sigma=1.5),
]


@pytest.mark.parametrize("tau", [math.inf, 1.0, 0.5, 2.0 ** -5, 0.0])
@pytest.mark.parametrize("w", DCASES, ids=[w.name for w in DCASES])
def test_decode_matches_independent_implementation(w, tau, mp_tables):
    q, k, v = _dec(w)
    o, lse, mask = O.decode(q, k, v, w.causal, w.window, w.bk, w.delta, tau)
    ro, rlse, rmask = R.ref_decode(q, k, v, w.causal, w.window, w.bk, w.delta, tau, mp_tables, O.scale(w.d))
    assert np.array_equal(mask, rmask)
    np.testing.assert_allclose(o, ro, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)
    if tau == 1.0 or math.isinf(tau):
        assert not np.any(mask == 2)
    if 0 < tau < math.inf:
        # the first tile of every row starts from mu = -inf: its maximizer
        # fails the look-ahead test and is recomputed
        tiles = mask.reshape(mask.shape[:3] + (-1, w.bk))
        first = np.argmax((tiles != 3).any(axis=-1), axis=-1)          # first tile with a visible key
        ft = np.take_along_axis(tiles, first[..., None, None], axis=3)[..., 0, :]
        assert np.all((ft == 1).sum(axis=-1) == 1)


@pytest.mark.parametrize("tau", [math.inf, 0.0])
def test_decode_end_modes_equal_the_block_pass(tau):
    """The decode rows against the prefill's last rows with one-key
    sub-blocks in tiles of the same length: with no look-ahead decisions both
    are plain online softmax, so every value agrees bit for bit."""
    N, M, tk = 96, 4, 16
    wp = W.small("dp", B=1, Hq=2, Hkv=1, N=N, d=16, causal=1, seed=84)
    q, k, v = (O.bf16_bits(t) for t in W.make_inputs(wp))
    o_p, lse_p, _ = O.fwd(q, k, v, 1, 0, 16, 1, tk, wp.delta, tau)
    o_d, lse_d, mask_d = O.decode(q[:, :, N - M:], k, v, 1, 0, tk, wp.delta, tau)
    assert np.array_equal(o_d, o_p[:, :, N - M:])
    assert np.array_equal(lse_d, lse_p[:, :, N - M:])


def test_decode_pure8_single_tile_is_naive_softmax(mp_tables):
    w = W.small("d1", B=1, Hq=1, Hkv=1, N=48, d=16, causal=0, seed=86, M=4, bk=64)
    q, k, v = _dec(w)
    o, lse, mask = O.decode(q, k, v, 0, 0, 64, w.delta, math.inf)
    qt = (M.bf16_to_float(q[0, 0]) * np.float64(O.scale(w.d))).astype(np.float32).astype(np.float64)
    y8 = R.y8_tile(qt, M.bf16_to_float(k[0, 0])).T                 # [row, key]
    mx = y8.max(axis=1, keepdims=True)
    sc = M.np_encode(M.np_round(mx - y8, "ue5m3_shift"), "ue5m3_shift")
    E = M.np_decode(mp_tables[0][sc], "ue5m3_exp")
    ref = (E @ M.bf16_to_float(v[0, 0])) / E.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(o[0, 0], ref, rtol=1e-12, atol=1e-13)
    assert np.all(mask[0, 0, :, :48] == 0) and np.all(mask[0, 0, :, 48:] == 3)


def test_decode_threshold_monotone_and_rows_subset():
    w = W.small("dm", B=2, Hq=4, Hkv=2, N=256, d=32, causal=1, seed=87, M=4, bk=32, scale_sigma=1.2)
    q, k, v = _dec(w)
    counts = []
    for tau in (2.0 ** -8, 2.0 ** -5, 2.0 ** -3, 0.5):
        _, _, mask = O.decode(q, k, v, 1, 0, 32, w.delta, tau)
        counts.append(int((mask == 2).sum()))
    assert counts == sorted(counts, reverse=True) and counts[0] > counts[-1]
    o, lse, mask = O.decode(q, k, v, 1, 0, 32, w.delta, 2.0 ** -5)
    rows = [0, 5, 13, 31]
    os_, ls_, ms_ = O.decode(q, k, v, 1, 0, 32, w.delta, 2.0 ** -5, rows=rows)
    flat = o.reshape(-1, w.d)
    assert np.array_equal(os_.reshape(-1, w.d)[rows], flat[rows])
    assert np.array_equal(ms_.reshape(len(flat), -1)[rows], mask.reshape(len(flat), -1)[rows])
    # O is a convex combination of the V rows of its key/value head
    vf = np.repeat(M.bf16_to_float(v), w.Hq // w.Hkv, axis=1)          # [B, Hq, N, d]
    assert np.all(o <= vf.max(axis=2, keepdims=True) + 1e-12)
    assert np.all(o >= vf.min(axis=2, keepdims=True) - 1e-12)
