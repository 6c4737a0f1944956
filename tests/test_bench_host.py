"""Host-side logic of bench.py (no GPU): the count of visible pairs inside the
recomputed sub-blocks (the 16-bit multiply-adds of the roofline figures)
against brute force, the workloads' visible-pair and effective-FLOP counts
against brute force, and the refusal of a multi-GPU run."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_39361_amd import workloads as W  # noqa: E402


def _visible(w, j, i):
    if i >= w.N or j >= w.N:
        return False
    if w.causal and i > j:
        return False
    if w.window > 0 and i <= j - w.window:
        return False
    return True


@pytest.mark.parametrize("causal,window,N,bq,bk", [(1, 0, 256, 64, 16), (0, 0, 192, 64, 16), (1, 40, 256, 64, 16),
                                                   (1, 0, 256, 128, 64)])
def test_visible_in_mask_matches_brute_force(causal, window, N, bq, bk):
    w = W.small("t", B=1, Hq=2, Hkv=1, N=N, d=64, causal=causal, window=window, bq=bq, bk=bk, nk=4)
    rng = np.random.default_rng(3)
    nqb, nkb = N // bq, N // bk
    mask = rng.integers(0, 4, size=(w.B, w.Hq, nqb, nkb)).astype(np.uint8)
    want = 0
    for b in range(w.B):
        for h in range(w.Hq):
            for qb in range(nqb):
                for kb in range(nkb):
                    if mask[b, h, qb, kb] in (1, 2):
                        want += sum(_visible(w, qb * bq + dj, kb * bk + di) for dj in range(bq) for di in range(bk))
    assert bench.visible_in_mask(w, mask) == want


@pytest.mark.parametrize("causal,window", [(1, 0), (0, 0), (1, 100), (1, 1000)])
def test_visible_logits_and_flops(causal, window):
    w = W.small("t", B=2, Hq=3, Hkv=1, N=300, d=64, causal=causal, window=window)
    brute = sum(_visible(w, j, i) for j in range(w.N) for i in range(w.N))
    assert w.visible_logits == w.B * w.Hq * brute
    assert w.macs == w.visible_logits * w.d
    full = 4.0 * w.B * w.Hq * w.N * w.N * w.d
    assert w.eff_flops == (full / 2 if causal else full)


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_profile_records_need_the_current_sources():
    """Counter figures are reported only while the kernel sources hash to the
    value recorded beside them."""
    h = bench.kernel_source_hash()
    assert len(h) == 64
    assert bench._profile_record(bench.TRAFFIC_FILE, "traffic-json", "no_such_workload", 0.5) is None
