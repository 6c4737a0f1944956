"""How much the reading of the 16-bit accumulation changes the decisions.

TEST INFRASTRUCTURE ONLY (runs the oracle alone, on the CPU).  The library
takes the 16-bit logit as the FP32 FMA chain rounded once to e4m11 (FP32
accumulation); the literal reading of Sec. 3.3 makes e4m11 itself the
accumulator, every FMA result rounded to e4m11 (oracle flag Y16_STEP).  This
script runs the oracle both ways on seeded query blocks of a workload and
prints how many mask bytes, and which recompute counts, differ.

    python oracle/reading_y16_step.py [--config 3] [--blocks 48] [--tau 0.5]
"""
import argparse
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2609_39361_amd import workloads as W  # noqa: E402


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--blocks", type=int, default=48)
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--seed", type=int, default=0)
    a = ap.parse_args()
    w = W.CONFIGS[a.config]
    tau = w.tau if a.tau is None else a.tau
    q, k, v = W.make_inputs(w)
    qb, kb, vb = O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)
    nqb = -(-w.N // w.bq)
    blocks = sorted(int(x) for x in np.random.default_rng(a.seed).permutation(w.B * w.Hq * nqb)[:a.blocks])
    res = {}
    for name, flags in (("fp32 chain, one rounding", 0), ("e4m11 accumulator", O.Y16_STEP)):
        t0 = time.perf_counter()
        o, lse, mask, st = O.fwd(qb, kb, vb, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, qblocks=blocks,
                                 flags=flags, stats=True)
        res[name] = (o, lse, mask, st)
        print("%-26s %.1f s  stats %s" % (name, time.perf_counter() - t0, st.tolist()))
    (o0, l0, m0, s0), (o1, l1, m1, s1) = res.values()
    sel = np.zeros((w.B, w.Hq, nqb), dtype=bool)
    sel.reshape(-1)[blocks] = True
    m0, m1 = m0[sel], m1[sel]
    active = m0 != 3
    diff = m0 != m1
    rows = np.repeat(sel, w.bq, axis=2)[:, :, :w.N]
    do = np.abs(o0[rows] - o1[rows]).max() / np.abs(o0[rows]).max()
    print("workload %s, tau %g, %d query blocks: %d of %d active mask bytes differ (%.3f%%); "
          "recomputed sub-blocks %d vs %d; max |dO| / max|O| = %.3g; max |d lse| = %.3g" % (
              w.name, tau, len(blocks), diff.sum(), active.sum(), 100.0 * diff.sum() / active.sum(),
              int(s0[1] + s0[2]), int(s1[1] + s1[2]), do, np.abs(l0[rows] - l1[rows]).max()))


if __name__ == "__main__":
    main()
