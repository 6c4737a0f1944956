"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar: e4m3 / e4m11 logit codes, exponential tables, the fp64 rescale
exponential and the recompute masks bit-exact; O within 2e-3 * max|O|
(fp32 matrix-core accumulation vs the oracle's fp64); lse within 1e-4.
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


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def L():
    _need_gpu()
    from paper_2609_39361_amd import lamp
    lamp.init(0)
    return lamp


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


# ------------------------------------------------------------------ codecs
def test_e4m3_exhaustive_vs_oracle(L):
    """Every fp32 bit pattern: the device rounding sequence equals the oracle.
    The emulator relies on two facts about the non-saturating hardware
    conversion, checked here as well: it returns either the correct code or a
    NaN code (never a wrong finite code), and a NaN input gives a NaN code."""
    chunk = 1 << 28
    dev = torch.device("cuda:0")
    t0 = time.time()
    nan_lo = np.inf
    for c in range(16):
        start = c * chunk
        bits = (torch.arange(chunk, dtype=torch.int64, device=dev) + start).to(torch.int32)
        x = bits.view(torch.float32)
        out, raw = L.selftest_e4m3(x)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        rawh = raw.cpu().numpy()
        ref = O.e4m3_of_f32_bits(start, chunk)
        xf = x.cpu().numpy()
        isnan = np.isnan(xf)
        mism = (got != ref) & ~isnan
        assert not mism.any(), "chunk %d: %d mismatches, first at bits 0x%08x" % (
            c, mism.sum(), start + int(np.argmax(mism)))
        rawnan = (rawh & 0x7F) == 0x7F
        assert np.all(rawnan[isnan]), "chunk %d: a NaN input gave a finite code" % c
        bad = ~rawnan & ~isnan & (rawh != ref)
        assert not bad.any(), "chunk %d: raw conversion gave a wrong finite code at 0x%08x" % (
            c, start + int(np.argmax(bad)))
        fin = rawnan & ~isnan
        if fin.any():
            nan_lo = min(nan_lo, float(np.abs(xf[fin]).min()))
        _say("e4m3 chunk %d/16 ok (%.1fs)" % (c + 1, time.time() - t0))
        del bits, x, out, raw
    _say("smallest |x| whose raw conversion is NaN: %r" % nan_lo)
    assert nan_lo > 448.0

def test_tables_match_oracle(L):
    lut8, exp16 = L.get_tables(0)
    olut8, oexp16 = O.tables()
    assert np.array_equal(lut8, olut8)
    assert np.array_equal(exp16, oexp16)


def test_exp16_parts_sum_to_table(L):
    """The bf16 high/low pairs the forward pass reads sum exactly to the
    oracle's 16-bit exponentials; the high part is the truncated value."""
    _, oexp16 = O.tables()
    parts = L.get_exp16_parts(0)
    hi = ((parts & 0xFFFF) << 16).view(np.float32).astype(np.float64)
    lo = ((parts >> 16) << 16).view(np.float32).astype(np.float64)
    ref = O.decode_fmt(O.UE5M11_EXP, oexp16.astype(np.uint32))
    assert np.array_equal(hi + lo, ref)
    ref32 = ref.astype(np.float32).view(np.uint32)
    assert np.array_equal((parts & 0xFFFF), ref32 >> 16)


def test_exp_doc_bitexact(L):
    rng = np.random.default_rng(5)
    x = np.concatenate([-rng.uniform(0, 720, 500_000), -rng.uniform(0, 2, 200_000),
                        -np.ldexp(1.0, -rng.integers(1, 60, 10_000)), [0.0, -700.0, -700.0000001, -1e-300]])
    y = L.selftest_exp_doc(torch.from_numpy(x).cuda()).cpu().numpy()
    ref = O.exp_doc(x)
    assert np.array_equal(y.view(np.uint64), ref.view(np.uint64))


# ------------------------------------------------------------------ logits
LOGIT_CASES = [
    W.small("l_nc_d64", N=128, d=64, Hq=2, Hkv=1, causal=0, seed=101),
    W.small("l_causal_d128", N=192, d=128, Hq=4, Hkv=2, causal=1, seed=102),
    W.small("l_window_d128", N=256, d=128, Hq=1, Hkv=1, causal=1, window=40, seed=103),
    W.small("l_outlier_d64", N=128, d=64, Hq=1, Hkv=1, causal=0, seed=104, kind="outlier",
            n_outlier=2, outlier_gain=16.0),
    W.small("l_saturate_d128", N=64, d=128, Hq=1, Hkv=1, causal=0, seed=105, extra={"gain": 12.0}),
    W.small("l_d256", N=64, d=256, Hq=2, Hkv=2, causal=1, seed=106),
]


@pytest.mark.parametrize("w", LOGIT_CASES, ids=[w.name for w in LOGIT_CASES])
def test_logits8_bitexact(L, w):
    q, k, v = W.make_inputs(w)
    ref = O.logits8(O.bf16_bits(q), O.bf16_bits(k), w.causal, w.window, 0, w.N)
    got = L.logits8(q.cuda(), k.cuda(), w.causal, w.window, 0, w.N).cpu().numpy()
    assert np.array_equal(got, ref), "%d mismatching codes" % (got != ref).sum()


@pytest.mark.parametrize("w", LOGIT_CASES[:4] + LOGIT_CASES[5:], ids=[w.name for w in LOGIT_CASES[:4] + LOGIT_CASES[5:]])
def test_logits16_bitexact(L, w):
    q, k, v = W.make_inputs(w)
    ref = O.logits16(O.bf16_bits(q), O.bf16_bits(k), w.causal, w.window, 0, w.N)
    got = L.logits16(q.cuda(), k.cuda(), w.causal, w.window, 0, w.N).cpu().numpy().view(np.uint16)
    vis = ref != 0xFFFF
    assert np.array_equal(got[vis], ref[vis])


def test_logits8_row_range_and_ragged_rows(L):
    w = W.small("rows", N=256, d=128, Hq=2, Hkv=1, causal=1, seed=107)
    q, k, v = W.make_inputs(w)
    ref = O.logits8(O.bf16_bits(q), O.bf16_bits(k), 1, 0, 37, 91)
    got = L.logits8(q.cuda(), k.cuda(), 1, 0, 37, 91).cpu().numpy()
    assert np.array_equal(got, ref)


# ------------------------------------------------------------------ forward
_INPUTS = {}


def _inputs(w, keep=False):
    """(q, k, v) on the GPU and their bf16 bit patterns on the host; kept for
    reuse across thresholds when `keep`."""
    if w.name in _INPUTS:
        return _INPUTS[w.name]
    q, k, v = W.make_inputs(w)
    r = (q.cuda(), k.cuda(), v.cuda(), O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v))
    if keep:
        _INPUTS.clear()
        _INPUTS[w.name] = r
    return r


def _compare_fwd(L, w, tau, delta=None, qblocks=None, keep=False, flags=0):
    delta = w.delta if delta is None else delta
    qd, kd, vd, qb, kb, vb = _inputs(w, keep)
    o, lse, mask = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, delta, tau, flags=flags)
    torch.cuda.synchronize()
    ro, rlse, rmask = O.fwd(qb, kb, vb, w.causal, w.window, w.bq, w.bk, w.nk, delta, tau, qblocks=qblocks,
                            flags=flags)
    o, lse, mask = o.cpu().numpy(), lse.cpu().numpy(), mask.cpu().numpy()
    if qblocks is not None:
        nqb = w.N // w.bq
        sel = np.zeros((w.B, w.Hq, nqb), dtype=bool)
        for f in qblocks:
            sel.reshape(-1)[f] = True
        rows = np.repeat(sel, w.bq, axis=2)
        o, ro = o[rows], ro[rows]
        lse, rlse = lse[rows], rlse[rows]
        mask, rmask = mask[sel], rmask[sel]
    assert np.array_equal(mask, rmask), "%d mask bytes differ" % (mask != rmask).sum()
    scale = np.abs(ro).max()
    err = np.abs(o - ro).max() / scale
    assert err <= O_TOL, "O max-abs error %.3g of max|O| %.3g" % (err, scale)
    assert np.abs(lse - rlse).max() <= LSE_TOL
    return err, mask


FWD_CASES = [
    W.small("f_causal_d128_bq128", N=256, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=201),
    W.small("f_causal_d64_bq64", N=256, d=64, Hq=2, Hkv=2, bq=64, bk=16, nk=4, causal=1, seed=202),
    W.small("f_noncausal_d64_bk64", N=256, d=64, Hq=1, Hkv=1, bq=64, bk=64, nk=4, causal=0, seed=203,
            kind="outlier", n_outlier=2, outlier_gain=16.0),
    W.small("f_window_d128", N=512, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, window=100, seed=204),
    W.small("f_gqa_d128_bk64", N=512, d=128, Hq=4, Hkv=2, bq=128, bk=64, nk=4, causal=1, seed=205),
    W.small("f_d256", N=256, d=256, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=206),
]


@pytest.mark.parametrize("tau", [math.inf, 1.0, 0.5, 2.0 ** -5, 0.0])
@pytest.mark.parametrize("w", FWD_CASES, ids=[w.name for w in FWD_CASES])
def test_fwd_parity_small(L, w, tau):
    _compare_fwd(L, w, tau)


VARIANT_CASES = [FWD_CASES[0], FWD_CASES[1], FWD_CASES[2], FWD_CASES[3], FWD_CASES[5]]


@pytest.mark.parametrize("flags", [1, 2, 3])
@pytest.mark.parametrize("tau", [1.0, 0.5, 2.0 ** -5])
@pytest.mark.parametrize("w", VARIANT_CASES, ids=[w.name for w in VARIANT_CASES])
def test_fwd_variants_small(L, w, tau, flags):
    """First stage off (1), mu_hat truncated for the 8-bit shifts (2), both."""
    _compare_fwd(L, w, tau, flags=flags)


@pytest.mark.parametrize("flags", [1, 2])
def test_fwd_variants_config3_sampled(L, flags):
    w = W.CONFIGS[3]
    nqb = w.N // w.bq
    qbl = [nqb - 1, 17, 31 * nqb + 40]
    err, mask = _compare_fwd(L, w, 2.0 ** -5, qblocks=qbl, flags=flags)
    _say("config 3 flags %d tau 2^-5 sampled: O err %.2e, mask %s" % (flags, err, np.bincount(mask.ravel(), minlength=4)))


@pytest.mark.parametrize("delta", [2.0 ** -4, 0.003, 0.0])
@pytest.mark.parametrize("w", [FWD_CASES[0], FWD_CASES[1]], ids=[FWD_CASES[0].name, FWD_CASES[1].name])
def test_fwd_delta_variant(L, w, delta):
    """Safety margins that are powers of two or zero (the kernels test them
    in fixed point) and one that is not (fp64 test)."""
    _compare_fwd(L, w, 0.5, delta=delta)


def test_fwd_config1_full(L):
    w = W.CONFIGS[1]
    err, mask = _compare_fwd(L, w, w.tau)
    _say("config 1: O err %.2e, mask %s" % (err, np.bincount(mask.ravel(), minlength=4)))


def test_fwd_config2_full(L):
    w = W.CONFIGS[2]
    err, mask = _compare_fwd(L, w, w.tau)
    _say("config 2: O err %.2e, mask %s" % (err, np.bincount(mask.ravel(), minlength=4)))


def _sample_blocks(w, n_per_head=2, heads=(0,)):
    nqb = w.N // w.bq
    out = []
    for b in range(w.B):
        for h in heads:
            for qb in (nqb - 1, nqb // 3)[:n_per_head]:
                out.append((b * w.Hq + h) * nqb + qb)
    return out


def test_fwd_config3_sampled(L):
    """Qwen3-8B-shaped prefill at full size; the oracle computes sampled query
    blocks (the last block of heads 0 and 31, and a middle one of head 0)."""
    w = W.CONFIGS[3]
    nqb = w.N // w.bq
    qbl = [0 * nqb + nqb - 1, 0 * nqb + 21, 31 * nqb + nqb - 1]
    err, mask = _compare_fwd(L, w, w.tau, qblocks=qbl)
    _say("config 3 sampled: O err %.2e, mask %s" % (err, np.bincount(mask.ravel(), minlength=4)))


@pytest.mark.parametrize("cfg", [4, 40])
def test_fwd_config4_sampled(L, cfg):
    """Gemma-3-shaped d=256 layers at full size (N=16384): the sliding-window
    (1024) local layer and the global causal layer; the oracle computes the
    last query block and an early one of the first and last query head."""
    w = W.CONFIGS[cfg]
    nqb = w.N // w.bq
    qbl = [nqb - 1, 9, (w.Hq - 1) * nqb + nqb - 1, (w.Hq - 1) * nqb + nqb // 2]
    t0 = time.time()
    err, mask = _compare_fwd(L, w, w.tau, qblocks=qbl)
    _say("config %d sampled: O err %.2e, mask %s (%.1f s)" % (cfg, err, np.bincount(mask.ravel(), minlength=4),
                                                              time.time() - t0))


@pytest.mark.parametrize("tau", W.TAU_SWEEP)
def test_fwd_config5_sampled(L, tau):
    """Long-context batch (B=4, 32/8 heads, N=32768, Student-t channel scales)
    at full size for every threshold of the sweep; the oracle computes the
    last query block of batch 0 head 0 and of batch 3 head 31, and an early
    block of batch 1 head 7 and batch 2 head 20."""
    w = W.CONFIGS[5]
    nqb = w.N // w.bq
    qbl = [nqb - 1, (3 * w.Hq + 31) * nqb + nqb - 1, (1 * w.Hq + 7) * nqb + 5, (2 * w.Hq + 20) * nqb + nqb // 4]
    t0 = time.time()
    err, mask = _compare_fwd(L, w, tau, qblocks=qbl, keep=True)
    _say("config 5 tau %s sampled: O err %.2e, mask %s (%.1f s)" % (tau, err, np.bincount(mask.ravel(), minlength=4),
                                                                   time.time() - t0))


# ------------------------------------------------------------------ edge cases
RAGGED_CASES = [
    W.small("r_d128_n300", N=300, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=301),
    W.small("r_d128_n77", N=77, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=302),
    W.small("r_d128_nc_n200", N=200, d=128, Hq=1, Hkv=1, bq=64, bk=16, nk=4, causal=0, seed=303),
    W.small("r_d128_win_n333", N=333, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, window=70, seed=304),
    W.small("r_d64_n200", N=200, d=64, Hq=2, Hkv=2, bq=64, bk=16, nk=4, causal=1, seed=305),
    W.small("r_d128_bk64_n300", N=300, d=128, Hq=2, Hkv=1, bq=128, bk=64, nk=4, causal=1, seed=306),
    W.small("r_d256_n150", N=150, d=256, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=307),
]


@pytest.mark.parametrize("tau", [math.inf, 0.5, 2.0 ** -5, 0.0])
@pytest.mark.parametrize("w", RAGGED_CASES, ids=[w.name for w in RAGGED_CASES])
def test_fwd_ragged_lengths(L, w, tau):
    """N not a multiple of b_q or of the key tile: partial last query block
    and key tile, through both kernels."""
    _compare_fwd(L, w, tau)


def test_fwd_maximum_length(L):
    """N = 2^20, the longest sequence the library accepts, through the
    pipelined kernel (d=128, 16-key sub-blocks) with a 256-key sliding window
    (so the pass stays short): the oracle computes the first, a middle and the
    last query block; their rows of O, lse and their mask bytes (65536
    sub-blocks each) must match."""
    w = W.small("max_n_window", N=1 << 20, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, window=256,
                seed=321, kind="gauss")
    nqb = w.N // w.bq
    t0 = time.time()
    err, mask = _compare_fwd(L, w, 0.5, qblocks=[0, nqb // 2, nqb - 1])
    _say("N = 2^20 sampled: O err %.2e, mask %s (%.1f s)" % (err, np.bincount(mask.ravel(), minlength=4),
                                                             time.time() - t0))


def test_fwd_empty_inputs(L):
    for shape_q, shape_k in (((1, 2, 0, 128), (1, 1, 0, 128)), ((0, 2, 256, 128), (0, 1, 256, 128))):
        q = torch.zeros(shape_q, dtype=torch.bfloat16, device="cuda")
        k = torch.zeros(shape_k, dtype=torch.bfloat16, device="cuda")
        o, lse, mask = L.attn_fwd(q, k, k, True, 0, 128, 16, 4, 2.0 ** -8, 0.5)
        torch.cuda.synchronize()
        assert o.numel() == 0 and lse.numel() == 0 and mask.numel() == 0


DEGENERATE = [
    # all queries zero: every logit is 0, |mu_hat| delta = 0, so the margin
    # test fails on every tile and everything is recomputed in stage 1
    W.small("g_zero_q", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=311, extra={"zero_q": 1}),
    # constant rows: all logits of a row equal, every threat ties
    W.small("g_const", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=312, extra={"const": 1}),
    # large magnitudes: e4m3 and e4m11 saturate on most logits
    W.small("g_saturate", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=313, extra={"gain": 8.0}),
    W.small("g_saturate_d64_bk64", N=256, d=64, Hq=1, Hkv=1, bq=64, bk=64, nk=4, causal=0, seed=314,
            extra={"gain": 8.0}),
]


@pytest.mark.parametrize("tau", [math.inf, 0.5, 0.0])
@pytest.mark.parametrize("w", DEGENERATE, ids=[w.name for w in DEGENERATE])
def test_fwd_degenerate_inputs(L, w, tau):
    err, mask = _compare_fwd(L, w, tau)
    if "zero_q" in w.extra and tau == 0.5:
        assert np.all((mask == 1) | (mask == 3))


# ------------------------------------------------------------------ SIM profile
def _sim_grid(p, emin, emax):
    idx = np.arange((emax - emin + 1) << p)
    e = emin + (idx >> p)
    m = idx & ((1 << p) - 1)
    return ((1 << p) + m) * np.exp2((e - p).astype(np.float64))


def test_sim_tables_match_oracle(L):
    """The SIM profile's exponential tables, entry by entry, against the
    oracle's correctly rounded exponentials; shifts below the first row give
    1 and beyond the last 0 in the oracle, as the kernel's clamping assumes."""
    sim8, sim16 = L.get_sim_tables(0)
    for p, emin, emax, got in ((3, -6, 7, (sim8.astype(np.uint32) << 16).view(np.float32)),
                               (11, -14, 7, sim16.view(np.float32))):
        s = _sim_grid(p, emin, emax)
        ref = O.sim_exp(p, s)
        assert np.array_equal(got.astype(np.float64), ref)
        assert np.all(ref[: 1 << p] == 1.0) and np.all(ref[-(1 << p):] == 0.0)
        below = _sim_grid(p, -40, emin - 1)
        above = _sim_grid(p, emax + 1, emax + 3)
        assert np.all(O.sim_exp(p, below) == 1.0) and np.all(O.sim_exp(p, above) == 0.0)


SIM_LOGIT_CASES = [LOGIT_CASES[0], LOGIT_CASES[1], LOGIT_CASES[2], LOGIT_CASES[3], LOGIT_CASES[4], LOGIT_CASES[5]]


@pytest.mark.parametrize("high", [0, 1])
@pytest.mark.parametrize("w", SIM_LOGIT_CASES, ids=[w.name for w in SIM_LOGIT_CASES])
def test_logits_sim_bitexact(L, w, high):
    q, k, v = W.make_inputs(w)
    ref = O.logits_sim(O.bf16_bits(q), O.bf16_bits(k), w.causal, w.window, 0, w.N, high)
    got = L.logits_sim(q.cuda(), k.cuda(), high, w.causal, w.window, 0, w.N).cpu().numpy().astype(np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    vis = ~np.isnan(ref)
    assert np.array_equal(got[vis], ref[vis]), "%d values differ" % (got[vis] != ref[vis]).sum()


SIM_FWD_CASES = [FWD_CASES[0], FWD_CASES[3], FWD_CASES[5],
                 W.small("s_gqa_d128_bq64", N=384, d=128, Hq=4, Hkv=2, bq=64, bk=16, nk=4, causal=1, seed=211),
                 W.small("s_outlier_d128", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=0, seed=212,
                         kind="outlier", n_outlier=2, outlier_gain=40.0)]


@pytest.mark.parametrize("tau", [math.inf, 1.0, 0.5, 2.0 ** -5, 0.0])
@pytest.mark.parametrize("w", SIM_FWD_CASES, ids=[w.name for w in SIM_FWD_CASES])
def test_fwd_sim_small(L, w, tau):
    _compare_fwd(L, w, tau, flags=O.SIM)


@pytest.mark.parametrize("flags", [O.SIM | O.STAGE1_OFF, O.SIM | O.MU_TRUNC])
@pytest.mark.parametrize("w", [FWD_CASES[0], FWD_CASES[5]], ids=[FWD_CASES[0].name, FWD_CASES[5].name])
def test_fwd_sim_variants(L, w, flags):
    _compare_fwd(L, w, 2.0 ** -5, flags=flags)


@pytest.mark.parametrize("tau", [math.inf, 0.5, 0.0])
@pytest.mark.parametrize("w", [RAGGED_CASES[0], RAGGED_CASES[2], RAGGED_CASES[3], RAGGED_CASES[6]] + DEGENERATE[:3],
                         ids=[w.name for w in [RAGGED_CASES[0], RAGGED_CASES[2], RAGGED_CASES[3], RAGGED_CASES[6]]
                              + DEGENERATE[:3]])
def test_fwd_sim_ragged_and_degenerate(L, w, tau):
    _compare_fwd(L, w, tau, flags=O.SIM)


@pytest.mark.parametrize("tau", [0.5, 2.0 ** -5])
def test_fwd_sim_config3_sampled(L, tau):
    w = W.CONFIGS[3]
    nqb = w.N // w.bq
    qbl = [nqb - 1, 21, 31 * nqb + nqb - 1]
    err, mask = _compare_fwd(L, w, tau, qblocks=qbl, flags=O.SIM)
    _say("config 3 SIM tau %s sampled: O err %.2e, mask %s" % (tau, err, np.bincount(mask.ravel(), minlength=4)))


def test_fwd_sim_config4_global_sampled(L):
    w = W.CONFIGS[40]
    nqb = w.N // w.bq
    qbl = [nqb - 1, (w.Hq - 1) * nqb + nqb // 2]
    err, mask = _compare_fwd(L, w, w.tau, qblocks=qbl, flags=O.SIM)
    _say("config 40 SIM sampled: O err %.2e, mask %s" % (err, np.bincount(mask.ravel(), minlength=4)))


@pytest.mark.parametrize("tau", W.TAU_SWEEP)
def test_fwd_sim_config5_sampled(L, tau):
    w = W.CONFIGS[5]
    nqb = w.N // w.bq
    qbl = [nqb - 1, (3 * w.Hq + 31) * nqb + nqb - 1, (2 * w.Hq + 20) * nqb + nqb // 4]
    t0 = time.time()
    err, mask = _compare_fwd(L, w, tau, qblocks=qbl, keep=True, flags=O.SIM)
    _say("config 5 SIM tau %s sampled: O err %.2e, mask %s (%.1f s)" % (
        tau, err, np.bincount(mask.ravel(), minlength=4), time.time() - t0))


NO_MASS = [
    W.small("nm_pipelined", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=313, extra={"gain": 8.0}),
    W.small("nm_general", N=256, d=64, Hq=1, Hkv=1, bq=64, bk=64, nk=4, causal=0, seed=314, extra={"gain": 8.0}),
    W.small("nm_general_d64_bk16", N=256, d=64, Hq=2, Hkv=1, bq=64, bk=16, nk=4, causal=1, seed=315,
            extra={"gain": 8.0}),
]


@pytest.mark.parametrize("tau", [0.5, 2.0 ** -5])
@pytest.mark.parametrize("w", NO_MASS, ids=[w.name for w in NO_MASS])
def test_fwd_tiles_adding_no_mass(L, w, tau):
    """First stage off on saturating inputs: the 8-bit maximum can overshoot a
    row's 16-bit logits so far that a tile adds no mass (every exponential
    underflows) while the rescale factor is below fp32's range.  O keeps its
    ratio to omega (O finite wherever the oracle's is; NaN with lse = -inf
    only for rows that never receive mass)."""
    qd, kd, vd, qb, kb, vb = _inputs(w)
    o, lse, mask = [t.cpu().numpy() for t in
                    L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=1)]
    ro, rlse, rmask = O.fwd(qb, kb, vb, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=1)
    assert np.array_equal(mask, rmask)
    assert np.array_equal(np.isnan(o), np.isnan(ro)), "NaN rows differ"
    assert np.array_equal(np.isneginf(lse), np.isneginf(rlse))
    fin = ~np.isnan(ro)
    assert np.abs(o[fin] - ro[fin]).max() <= O_TOL * np.abs(ro[fin]).max()
    fl = np.isfinite(rlse)
    assert np.abs(lse[fl] - rlse[fl]).max() <= LSE_TOL
