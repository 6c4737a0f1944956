"""The compact register layout (Sec. 3.3, "Register layout"; flag
LAMP_COMPACT): 8-bit accumulators four per register, one 16-bit sub-block in
the fused pass, a sequential 16-bit pass for disruptive tiles.  A schedule of
the pipelined kernel only: its outputs must equal the oracle's to the usual
bar, be bit-identical to the default layout's, and its own 8-bit and 16-bit
codes must equal the oracle's."""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_39361_amd import workloads as W
import test_gpu_observe as OBS

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_39361_amd import lamp
    lamp.init(0)
    return lamp


def _bits_equal(a, b):
    return torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                       b.view(torch.int32) if b.dtype == torch.float32 else b)


CASES = [
    W.small("c_d128", N=384, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=701),
    W.small("c_d256", N=384, d=256, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=702),
    W.small("c_d256_window_ragged", N=333, d=256, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, window=70, seed=703),
    W.small("c_d128_noncausal_outlier", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=0, seed=704,
            kind="outlier", n_outlier=2, outlier_gain=16.0),
    W.small("c_saturate", N=256, d=128, Hq=1, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=313, extra={"gain": 8.0}),
]


@pytest.mark.parametrize("flags", [0, 1, 2])
@pytest.mark.parametrize("tau", [1.0, 0.5, 2.0 ** -5])
@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_compact_matches_oracle_and_safe_layout(L, w, tau, flags):
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    s0 = torch.zeros(L.stats_words(w.nk), dtype=torch.int64, device="cuda")
    s1 = torch.zeros_like(s0)
    safe = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=flags, stats=s0)
    comp = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, flags=flags | L.COMPACT,
                      stats=s1)
    torch.cuda.synchronize()
    for a, b in zip(safe, comp):
        assert _bits_equal(a, b)
    # statistics equal except the schedule words (6, 7)
    sel = [0, 1, 2, 3, 4, 5] + list(range(8, 8 + w.nk + 1))
    assert s0[sel].tolist() == s1[sel].tolist()
    ro, rlse, rmask = O.fwd(O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v), w.causal, w.window, w.bq, w.bk, w.nk,
                            w.delta, tau, flags=flags)
    o, lse, mask = [t.cpu().numpy() for t in comp]
    assert np.array_equal(mask, rmask)
    # a row whose exponentials all underflow (possible with the first stage
    # off) is O = NaN, lse = -inf on both sides
    assert np.array_equal(np.isnan(o), np.isnan(ro)) and np.array_equal(np.isinf(lse), np.isinf(rlse))
    fin = ~np.isnan(ro)
    assert np.abs(o[fin] - ro[fin]).max() <= 2e-3 * np.abs(ro[fin]).max()
    fl = np.isfinite(rlse)
    assert np.abs(lse[fl] - rlse[fl]).max() <= 1e-4


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_compact_observables(L, w):
    """The compact instantiation's own 8-bit codes and used 16-bit codes."""
    OBS._check_observables(L, w, 0.5, 0, -(-w.N // w.bq), flags=L.COMPACT)


@pytest.mark.parametrize("cfg", [3, 4, 40])
def test_compact_full_size_sampled(L, cfg):
    """Configs 3 and 4 (local, global) at full size with the compact layout:
    bit-identical to the default layout on every output, and the oracle on
    sampled query blocks."""
    w = W.CONFIGS[cfg]
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    safe = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, w.tau)
    comp = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, w.tau, flags=L.COMPACT)
    torch.cuda.synchronize()
    for a, b in zip(safe, comp):
        assert _bits_equal(a, b)
    nqb = w.N // w.bq
    qbl = [nqb - 1, 9, (w.Hq - 1) * nqb + nqb // 2]
    ro, rlse, rmask = O.fwd(O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v), w.causal, w.window, w.bq, w.bk, w.nk,
                            w.delta, w.tau, qblocks=qbl)
    o, lse, mask = [t.cpu().numpy() for t in comp]
    sel = np.zeros((w.B, w.Hq, nqb), dtype=bool)
    sel.reshape(-1)[qbl] = True
    rows = np.repeat(sel, w.bq, axis=2)
    assert np.array_equal(mask[sel], rmask[sel])
    assert np.abs(o[rows] - ro[rows]).max() <= 2e-3 * np.abs(ro[rows]).max()
    print("config %d compact: bit-identical to the default layout; sampled blocks match the oracle" % cfg,
          flush=True)
