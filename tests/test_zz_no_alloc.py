"""The allocation-free entry point lamp_attn_fwd_noalloc, through the C ABI:
two calls in a row (the second on a smaller input) against lamp_attn_fwd on
the same inputs -- bit-identical O, lse and mask (same kernels, so the
oracle's bar holds a fortiori) -- and the oracle itself on the small call;
no device memory is taken during the calls; sizes beyond the fixed scratch
are refused."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_39361_amd import workloads as W

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


def _outs(w):
    dev = torch.device("cuda:0")
    return (torch.empty((w.B, w.Hq, w.N, w.d), dtype=torch.float32, device=dev),
            torch.empty((w.B, w.Hq, w.N), dtype=torch.float32, device=dev),
            torch.empty((w.B, w.Hq, -(-w.N // w.bq), -(-w.N // (w.bk * w.nk)) * w.nk), dtype=torch.uint8,
                        device=dev))


def test_noalloc_two_calls_match_lamp_attn_fwd(L):
    big = W.small("na_big", N=4096, d=128, Hq=8, Hkv=2, bq=128, bk=16, nk=4, causal=1, seed=601)
    small = W.small("na_small", N=300, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=602)
    # a first call loads the kernels' code (the runtime may take memory for
    # that); the two checked calls follow
    tiny = W.small("na_tiny", N=64, d=128, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=600)
    q, k, v = W.make_inputs(tiny)
    L.attn_fwd_noalloc(q.cuda(), k.cuda(), v.cuda(), _outs(tiny), True, 0, 128, 16, 4, 2.0 ** -8, 0.5)
    torch.cuda.synchronize()
    runs = []
    for w in (big, small):
        q, k, v = W.make_inputs(w)
        qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
        out = _outs(w)
        st = torch.zeros(L.stats_words(w.nk), dtype=torch.int64, device="cuda")
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info(0)[0]
        L.attn_fwd_noalloc(qd, kd, vd, out, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, w.tau, stats=st)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info(0)[0]
        # the workspace of the big call is about 40 MiB: none of it may come from new device memory
        assert free0 - free1 < (8 << 20), (free0, free1)
        runs.append((w, q, k, v, qd, kd, vd, [t.clone() for t in out], st.clone()))
    for w, q, k, v, qd, kd, vd, got, st in runs:
        st2 = torch.zeros_like(st)
        ref = L.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, w.tau, stats=st2)
        torch.cuda.synchronize()
        for a, b in zip(got, ref):
            assert _bits_equal(a, b)
        assert torch.equal(st, st2)
    w, q, k, v, qd, kd, vd, got, st = runs[1]
    ro, rlse, rmask = O.fwd(O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v), w.causal, w.window, w.bq, w.bk, w.nk,
                            w.delta, w.tau)
    assert np.array_equal(got[2].cpu().numpy(), rmask)
    ro_ = got[0].cpu().numpy()
    assert np.abs(ro_ - ro).max() <= 2e-3 * np.abs(ro).max()
    assert np.abs(got[1].cpu().numpy() - rlse).max() <= 1e-4


def test_noalloc_refuses_sizes_beyond_the_scratch(L):
    """Four Qwen3-8B-shaped 8K sequences need 704 MiB of workspace: refused
    before any device work, with the fixed size in the message."""
    B, Hq, Hkv, N, d = 4, 32, 8, 8192, 128
    assert L.fwd_workspace_size(B, Hq, Hkv, N, d) > L.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((B, Hq, N, d), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((B, Hkv, N, d), dtype=torch.bfloat16, device="cuda")
    w = W.small("na_huge", B=B, N=N, d=d, Hq=Hq, Hkv=Hkv, bq=128, bk=16, nk=4, causal=1, seed=0)
    out = _outs(w)
    with pytest.raises(L.LampError) as ei:
        L.attn_fwd_noalloc(q, k, k, out, True, 0, 128, 16, 4, 2.0 ** -8, 0.5)
    assert ei.value.status == L.LAMP_ERR_WORKSPACE
    with pytest.raises(L.LampError) as ei:
        ks = k[:1, :1, :256].contiguous()
        L.attn_fwd_noalloc(q[:1, :2, :256].contiguous(), ks, ks, _outs(
            W.small("na_s", N=256, d=d, Hq=2, Hkv=1, bq=128, bk=16, nk=4, causal=1, seed=0)),
            True, 0, 128, 16, 4, 2.0 ** -8, 0.5, flags=L.CHECK_FINITE)
    assert ei.value.status == 2
