"""GPU parity of the stochastically rounded 8-bit accumulation (Sec. 3.3's
alternative to round-to-nearest) through the C ABI against the CPU oracle.

Bar as for the round-to-nearest path: 8-bit logit codes and recompute masks
bit-exact (the random numbers come from the same counter-based generator on
both sides, written separately); O within 2e-3 of max|O|; lse within 1e-4.
"""
import math
import sys
import time

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_39361_amd import workloads as W

pytestmark = pytest.mark.gpu

O_TOL = 2e-3
LSE_TOL = 1e-4
SEEDS = (7, 2 ** 63 + 12345)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_39361_amd import lamp
    lamp.init(0)
    return lamp


def _inputs(w):
    q, k, v = W.make_inputs(w)
    return q.cuda(), k.cuda(), v.cuda(), O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)


LOGIT_CASES = [
    W.small("sr_l_nc_d64", N=128, d=64, Hq=2, Hkv=1, causal=0, seed=401),
    W.small("sr_l_causal_d128_n80", N=80, d=128, Hq=2, Hkv=1, causal=1, seed=402),      # N % 64 != 0
    W.small("sr_l_window_d128", N=192, d=128, Hq=1, Hkv=1, causal=1, window=50, seed=403),
    W.small("sr_l_saturate_d128", N=64, d=128, Hq=1, Hkv=1, causal=0, seed=404, extra={"gain": 12.0}),
    W.small("sr_l_d256", N=64, d=256, Hq=2, Hkv=2, causal=1, seed=405, kind="outlier", n_outlier=2,
            outlier_gain=16.0),
]


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("w", LOGIT_CASES, ids=[w.name for w in LOGIT_CASES])
def test_logits8_sr_bitexact(L, w, seed):
    qd, kd, _, qb, kb, _ = _inputs(w)
    got = L.logits8(qd, kd, w.causal, w.window, sr_seed=seed).cpu().numpy()
    ref = O.logits8_sr(qb, kb, w.causal, w.window, 0, w.N, seed)
    assert np.array_equal(got, ref), "%d codes differ" % (got != ref).sum()
    # a row range reads the same numbers (they depend on the logit alone)
    part = L.logits8(qd, kd, w.causal, w.window, row0=w.N // 2, nrows=w.N // 4, sr_seed=seed).cpu().numpy()
    assert np.array_equal(part, ref[:, :, w.N // 2: w.N // 2 + w.N // 4])


def _compare(L, w, tau, flags=0, seed=SEEDS[0], qblocks=None):
    qd, kd, vd, qb, kb, vb = _inputs(w)
    o, lse, mask = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=flags,
                              sr_seed=seed)
    torch.cuda.synchronize()
    ro, rlse, rmask = O.fwd(qb, kb, vb, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, qblocks=qblocks,
                            flags=flags | O.SR8, seed=seed)
    o, lse, mask = o.cpu().numpy(), lse.cpu().numpy(), mask.cpu().numpy()
    if qblocks is not None:
        nqb = -(-w.N // w.bq)
        sel = np.zeros((w.B, w.Hq, nqb), dtype=bool)
        for f in qblocks:
            sel.reshape(-1)[f] = True
        rows = np.repeat(sel, w.bq, axis=2)[:, :, :w.N]
        o, ro, lse, rlse = o[rows], ro[rows], lse[rows], rlse[rows]
        mask, rmask = mask[sel], rmask[sel]
    assert np.array_equal(mask, rmask), "%d mask bytes differ" % (mask != rmask).sum()
    # a row whose every exponential underflows (omega = 0: see
    # test_fwd_sr_row_with_every_exponential_underflowing) is 0/0 on both sides
    nan = np.isnan(ro)
    assert np.array_equal(np.isnan(o), nan)
    assert np.array_equal(lse[np.isinf(rlse)], rlse[np.isinf(rlse)])
    fin = ~np.isinf(rlse)
    scale = np.abs(ro[~nan]).max()
    err = np.abs(o[~nan] - ro[~nan]).max() / scale
    assert err <= O_TOL, "O max-abs error %.3g of max|O| %.3g" % (err, scale)
    assert np.abs(lse[fin] - rlse[fin]).max() <= LSE_TOL
    return err, mask


FWD_CASES = [
    W.small("sr_f_causal_d128_bq128", N=256, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=411),
    W.small("sr_f_causal_d64_bq64", N=256, d=64, Hq=2, Hkv=2, bq=64, bk=16, nk=4, causal=1, seed=412),
    W.small("sr_f_nc_d64_bk64", N=256, d=64, Hq=1, Hkv=1, bq=64, bk=64, nk=4, causal=0, seed=413,
            kind="outlier", n_outlier=2, outlier_gain=16.0),
    W.small("sr_f_window_d128_bq64", N=384, d=128, Hq=1, Hkv=1, bq=64, bk=16, nk=4, causal=1, window=100, seed=414),
    W.small("sr_f_gqa_d128_bk64", N=256, d=128, Hq=4, Hkv=2, bq=128, bk=64, nk=4, causal=1, seed=415),
    W.small("sr_f_d256", N=256, d=256, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=416),
    W.small("sr_f_ragged_d128_n300", N=300, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=417),
    W.small("sr_f_ragged_d256_bk64_n150", N=150, d=256, Hq=1, Hkv=1, bq=64, bk=64, nk=4, causal=0, seed=418),
]


@pytest.mark.parametrize("tau", [math.inf, 0.5, 2.0 ** -5])
@pytest.mark.parametrize("w", FWD_CASES, ids=[w.name for w in FWD_CASES])
def test_fwd_sr_parity(L, w, tau):
    _compare(L, w, tau)


@pytest.mark.parametrize("flags", [1, 2, 3])
@pytest.mark.parametrize("w", [FWD_CASES[0], FWD_CASES[2], FWD_CASES[5]], ids=lambda w: w.name)
def test_fwd_sr_variants(L, w, flags):
    _compare(L, w, 0.5, flags=flags, seed=SEEDS[1])


def test_fwd_sr_row_with_every_exponential_underflowing(L):
    """With the first stage off, mu_hat is the largest 8-bit logit; here
    (seed 3, query row 123) a stochastically rounded 8-bit logit overshoots its
    16-bit value by 31.9 (352 vs 320.125), the knapsack recomputes that
    sub-block and one other, and every 16-bit and remaining 8-bit exponential
    of the row underflows against mu_hat: omega = 0, so O is 0/0 (NaN) and
    lse is -inf, on both sides."""
    w = FWD_CASES[2]
    qd, kd, vd, *_ = _inputs(w)
    err, mask = _compare(L, w, 0.5, flags=1, seed=3)
    assert list(mask[0, 0, 1]) == [0, 2, 2, 0]
    o, lse, _ = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.5, flags=1, sr_seed=3)
    assert lse[0, 0, 123].item() == -math.inf and torch.isnan(o[0, 0, 123]).all()


def test_fwd_sr_seed_changes_the_logits_not_the_all16_mode(L):
    w = FWD_CASES[0]
    qd, kd, vd, *_ = _inputs(w)
    args = (qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta)
    a = [t.cpu() for t in L.attn_fwd(*args, math.inf, sr_seed=1)]
    b = [t.cpu() for t in L.attn_fwd(*args, math.inf, sr_seed=2)]
    assert not torch.equal(a[0], b[0])
    c = [t.cpu() for t in L.attn_fwd(*args, 0.0, sr_seed=1)]
    d = [t.cpu() for t in L.attn_fwd(*args, 0.0)]
    for x, y in zip(c, d):
        assert torch.equal(x, y)


def test_fwd_sr_refuses_the_sim_profile(L):
    w = FWD_CASES[0]
    qd, kd, vd, *_ = _inputs(w)
    with pytest.raises(Exception, match="SIM"):
        L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, 0.5, flags=4, sr_seed=1)


def test_fwd_sr_config3_sampled(L):
    """The Qwen3-8B-shaped prefill (32/8 heads, d=128, N=8192, causal) at full
    size with stochastic rounding; the oracle computes the last query block of
    head 0 and an early one of head 31."""
    w = W.CONFIGS[3]
    nqb = w.N // w.bq
    qbl = [nqb - 1, 31 * nqb + 9]
    t0 = time.time()
    err, mask = _compare(L, w, w.tau, qblocks=qbl)
    _say("config 3 sampled with stochastic rounding: O err %.2e, mask %s (%.1f s)"
         % (err, np.bincount(mask.ravel(), minlength=4), time.time() - t0))
