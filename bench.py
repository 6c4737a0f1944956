#!/usr/bin/env python3
"""Benchmark of the LampAttention forward pass on one MI355X.

One step is one full forward pass (lamp_attn_fwd: prepass + the forward
kernel) over the Qwen3-8B-shaped causal prefill (B=1, 32 query heads / 8 KV
heads, d=128, N=8192, b_q=128, b_k=16, N_k=4, delta=2^-8, tau=2^-1) with
synthetic inputs resident in HBM.  Prints one JSON line with the effective
attention TFLOP/s (4*B*H*N^2*d, halved for causal), the recomputed-sub-block
fraction, the VALU roofline of the forward kernel and the CPU oracle timed on
a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X peaks (public figures): 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz of
# VALU issue (one fp32 FMA or conversion per lane per cycle), the unit-count
# model of one operation per multiply-add; and the published fp32 vector
# peak, 157.3 TFLOP/s (packed FMAs: 2 flops on 2 values per lane and cycle).
VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9          # 39.3e12 lane-instructions / s
FP32_PEAK_FLOPS = 157.3e12
# Fewest VALU lane-instructions per emulated 8-bit multiply-add on gfx950: one
# fp32 FMA, half a packed round-to-e4m3 and half a packed decode.
OPS_PER_MAC8 = 2.0
# 16-bit recompute: one fp32 FMA per multiply-add.
OPS_PER_MAC16 = 1.0
# SIM precision profile (flag 4): the 8-bit step is one fp32 FMA and a
# round-to-nearest-even of the FP32 encoding to 3 mantissa bits (bit-field
# extract of the last kept bit, one 3-input add, one mask): 4 per MAC.
OPS_PER_MAC8_SIM = 4.0
SIM_FLAG = 4


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "lamp_fwd16_kernel.qwen3-8b-prefill-8k.hbm_traffic.md")
VALU_FILE = os.path.join(ROOT, "profiles", "lamp_fwd16_kernel.qwen3-8b-prefill-8k.valu_issue.md")
DEC_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "lamp_decode.qwen3-8b-decode-b32-kv8k.hbm_traffic.md")
KERNEL_SOURCES = ["lamp_fwd.hip", "lamp_fwd16.hip", "lamp_loops.h", "lamp_sr.h", "lamp_device.h", "lamp_kernels.h", "lamp_stats.h"]
DEC_SOURCES = ["lamp_decode.hip", "lamp_decode.h", "lamp_device.h", "lamp_loops.h", "lamp_host.cpp"]


def kernel_source_hash(sources=None):
    """sha256 over the forward kernel's sources (or the given ones), to tie
    counter readings to them."""
    h = hashlib.sha256()
    for name in sources or KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_39361_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _mode_of(tau):
    """Template mode of the pipelined kernel: 0 threshold, 1 pure 8-bit, 2 all 16-bit."""
    return 1 if math.isinf(tau) else (2 if tau == 0 else 0)


def _profile_record(path, tag, workload, tau, flags=0, sources=None):
    """The `tag: {json}` line of a committed profile summary, when it was taken
    on the current kernel sources and on this workload; else None."""
    try:
        with open(path) as f:
            text = f.read()
    except OSError:
        return None
    for line in text.splitlines():
        if line.startswith(tag + ": "):
            rec = json.loads(line[len(tag) + 2:])
            if rec.get("source_sha256") == kernel_source_hash(sources) and rec.get("workload") == workload \
                    and rec.get("tau") == tau and rec.get("flags", 0) == flags:
                return rec
    return None


def measured_traffic(workload, tau, flags=0):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE runs."""
    rec = _profile_record(TRAFFIC_FILE, "traffic-json", workload, tau, flags)
    return None if rec is None else rec["bytes_per_launch"]


def measured_decode_traffic(workload, tau, flags=0):
    """HBM bytes per decode step (all its kernels) from the committed
    FETCH_SIZE / WRITE_SIZE runs."""
    rec = _profile_record(DEC_TRAFFIC_FILE, "traffic-json", workload, tau, flags, DEC_SOURCES)
    return None if rec is None else rec["bytes_per_step"]


def copy_calibration(mib, dev):
    """One plain negating copy of `mib` MiB of fp32 (reads and writes that many
    bytes), whose counter readings calibrate the HBM byte counters."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


def measured_valu_issue(workload, tau, flags=0):
    """SQ_INSTS_VALU over the launch's VALU issue capacity, from the committed
    counter run."""
    rec = _profile_record(VALU_FILE, "valu-json", workload, tau, flags)
    return None if rec is None else rec["valu_issue_fraction"]


def visible_in_mask(w, mask):
    """Visible (query, key) pairs inside the recomputed sub-blocks."""
    m = mask.reshape(w.B * w.Hq, w.N // w.bq, w.N // w.bk)
    rec = (m == 1) | (m == 2)
    qb = np.arange(w.N // w.bq)[:, None]
    kb = np.arange(w.N // w.bk)[None, :]
    # count visible pairs of each (query block, key sub-block) in closed form
    j0 = qb * w.bq
    i0 = kb * w.bk
    cnt = np.zeros((w.N // w.bq, w.N // w.bk), dtype=np.int64)
    for dj in range(w.bq):
        j = j0 + dj
        lo = np.maximum(i0, (j - w.window + 1) if w.window > 0 else i0)
        hi = np.minimum(i0 + w.bk - 1, j if w.causal else i0 + w.bk - 1)
        cnt += np.maximum(hi - lo + 1, 0)
    return int((rec * cnt[None]).sum())


def cpu_baseline(w, tau, q, k, v, budget_s=15.0, seed=0, flags=0, sr_seed=None, gpu=None):
    """The CPU oracle on a bounded, stated sample of query blocks (with
    sr_seed: the stochastically rounded 8-bit accumulation).  With gpu =
    (o, lse, mask) numpy arrays of the same run, the sampled blocks are also
    compared with them: returns (baseline, parity)."""
    from oracle import oracle as O
    rng = np.random.default_rng(seed)
    nqb = w.N // w.bq
    qbits, kbits, vbits = O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)
    threads = O.max_threads()
    # calibrate: one block of the median position, then as many as fit the budget
    order = rng.permutation(w.B * w.Hq * nqb)
    picked, spent, flops = [], 0.0, 0.0
    first = True
    par = {"blocks": 0, "mask_mismatch": 0, "o_err": 0.0, "lse_err": 0.0}
    while spent < budget_s and len(picked) < len(order):
        n = 1 if first else max(1, min(threads, int((budget_s - spent) / max(spent / len(picked), 1e-3))))
        batch = [int(x) for x in order[len(picked):len(picked) + n]]
        t0 = time.perf_counter()
        ro, rlse, rmask = O.fwd(qbits, kbits, vbits, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau,
                                qblocks=batch, nthreads=threads, flags=flags | (O.SR8 if sr_seed is not None else 0),
                                seed=sr_seed if sr_seed is not None else 0)
        spent += time.perf_counter() - t0
        if gpu is not None:   # the sampled blocks of the GPU outputs of this run, outside the timing
            go, glse, gmask = gpu
            for f in batch:
                bh, qb = divmod(f, nqb)
                b, h = divmod(bh, w.Hq)
                rows = slice(qb * w.bq, min((qb + 1) * w.bq, w.N))
                ref_o = ro[b, h, rows]
                par["blocks"] += 1
                par["mask_mismatch"] += int((gmask[b, h, qb] != rmask[b, h, qb]).sum())
                par["o_err"] = max(par["o_err"], float(np.abs(go[b, h, rows] - ref_o).max() / np.abs(ref_o).max()))
                par["lse_err"] = max(par["lse_err"], float(np.abs(glse[b, h, rows] - rlse[b, h, rows]).max()))
        for f in batch:
            qb = f % nqb
            vis = 0
            for dj in range(w.bq):
                j = qb * w.bq + dj
                lo = max(0, j - w.window + 1) if w.window > 0 else 0
                hi = j if w.causal else w.N - 1
                vis += hi - lo + 1
            flops += 4.0 * vis * w.d
        picked += batch
        first = False
    base = {
        "value": flops / spent / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "%d of %d query blocks (seeded random over heads and positions), %.1f s, "
                  "effective FLOP counted over the sampled blocks' visible pairs" % (
                      len(picked), w.B * w.Hq * nqb, spent),
    }
    if gpu is None:
        return base
    par["ok"] = par["mask_mismatch"] == 0 and par["o_err"] <= 2e-3 and par["lse_err"] <= 1e-4
    par["bar"] = "masks bit-exact, O within 2e-3 of max|O| per block, lse within 1e-4"
    return base, par


HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, public figure


def cpu_baseline_decode(w, tau, q, k, v, budget_s=15.0, seed=0):
    """The CPU oracle of the decode form on a bounded, stated sample of query rows."""
    from oracle import oracle as O
    rng = np.random.default_rng(seed)
    nrows = w.B * w.Hq * w.M
    qbits, kbits, vbits = O.bf16_bits(q), O.bf16_bits(k), O.bf16_bits(v)
    threads = O.max_threads()
    order = rng.permutation(nrows)
    picked, spent = [], 0.0
    first = True
    while spent < budget_s and len(picked) < nrows:
        n = 1 if first else max(1, min(4 * threads, int((budget_s - spent) / max(spent / len(picked), 1e-3))))
        batch = [int(x) for x in order[len(picked):len(picked) + n]]
        t0 = time.perf_counter()
        O.decode(qbits, kbits, vbits, w.causal, w.window, w.bk, w.delta, tau, rows=batch, nthreads=threads)
        spent += time.perf_counter() - t0
        picked += batch
        first = False
    flops = w.eff_flops * len(picked) / nrows
    return {"value": flops / spent / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": "%d of %d query rows (seeded random), %.1f s, effective FLOP of the sampled rows" % (
                len(picked), nrows, spent)}


def main_decode(args, w, tau, flags=0):
    """Bench line of the decode form (vector LAMP, Sec. 2, Eq. (6)); flags: 0 (the key-chunk
    pipeline) or lamp.DECODE_SERIAL."""
    import torch
    from paper_2609_39361_amd import lamp, workloads as W
    dev = torch.device("cuda:0")
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    tk = w.bk
    o = torch.empty((w.B, w.Hq, w.M, w.d), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.Hq, w.M), dtype=torch.float32, device=dev)
    mask = torch.empty((w.B, w.Hq, w.M, -(-w.N // tk) * tk), dtype=torch.uint8, device=dev)

    def step():
        lamp.attn_decode(qd, kd, vd, w.causal, w.window, tk, w.delta, tau, out=(o, lse, mask), flags=flags)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    lamp.timing_read()
    lamp.timing_enable(True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record()
        step()
        ends[i].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    lamp.timing_enable(False)
    launches, kern_ms_sum, pre_ms_sum = lamp.timing_read()
    kernel_ms = kern_ms_sum / launches
    ms = float(np.mean([s_.elapsed_time(e_) for s_, e_ in zip(starts, ends)]))
    m = mask.cpu().numpy()
    vis = int((m != 3).sum())
    s1, s2 = int((m == 1).sum()), int((m == 2).sum())
    # algorithmic HBM bytes: the cache (K and V of every key/value head), the
    # queries, and the outputs (O, lse, one mask byte per key and row)
    nbytes = (2 * w.B * w.Hkv * w.N * w.d * 2 + w.B * w.Hq * w.M * w.d * 2
              + w.B * w.Hq * w.M * (w.d * 4 + 4) + m.size)
    achieved = nbytes / (kernel_ms * 1e-3) / 1e9
    mac8 = 0 if tau == 0 else w.macs
    mac16 = (s1 + s2) * w.d
    serial = flags == lamp.DECODE_SERIAL
    md = _mode_of(tau)
    rows = w.Hq // w.Hkv * w.M
    if serial or rows > 8:
        kernels = ["dec_logits_kernel<%d,%d>" % (w.d, md), "dec_lamp_kernel<%d,%d>" % (w.d, md),
                   "dec_pv_kernel<%d,%d>" % (w.d, 4 if rows <= 4 else 8 if rows <= 8 else 16)]
    else:
        kernels = ["dec_stage_kernel<%d,%d,%d>" % (w.d, md, 4 if rows <= 4 else 8)]
    kernels += ["dec_reduce_kernel<%d>" % w.d]
    result = {
        "metric": "effective attention TFLOP/s (4*d per visible (query, key) pair), decode form, 1 GPU",
        "value": w.eff_flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "e4m3/e4m11 emulated (fp32 FMA + fp8 conversions), bf16 cache, fp32 output",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "M": w.M, "N": w.N, "d": w.d,
                   "causal": w.causal, "window": w.window, "tk": tk, "delta": w.delta, "tau": tau,
                   "form": "serial" if serial else "pipelined"},
        "tokens_per_s": w.B * w.M / (ms * 1e-3),
        "recompute_fraction": (s1 + s2) / vis,
        "lookahead_recomputes": s1, "knapsack_recomputes": s2,
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": measured_decode_traffic(w.name, tau, flags),
            "kernel": " + ".join(kernels),
            "kernel_ms": kernel_ms, "prepass_ms": pre_ms_sum / launches,
            "bytes_per_launch": nbytes,
            "valu_frac_algorithmic": (OPS_PER_MAC8 * mac8 + OPS_PER_MAC16 * mac16) / (kernel_ms * 1e-3) / VALU_LANE_OPS,
        },
        "wall_s_timed_region": wall,
    }
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline_decode(w, tau, q, k, v, budget_s=args.cpu_budget)
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=3, help="config id (1, 2, 3, 4, 40, 5; 6 decode form)")
    ap.add_argument("--tau", type=str, default=None,
                    help="threshold, or a comma-separated sweep (one JSON line each, inputs drawn once)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--flags", type=str, default="0",
                    help="variants: 1 first stage off, 2 mu_hat truncation, 4 SIM precision profile; "
                         "a comma-separated list sweeps them (outer loop)")
    ap.add_argument("--sr-seed", type=int, default=None,
                    help="round the 8-bit accumulation stochastically with this seed (lamp_attn_fwd_sr)")
    ap.add_argument("--phase-timer", action="store_true",
                    help="load liblamp_phase.so (built by `python -m paper_2609_39361_amd.build --phase-timer`) and "
                         "report the pipelined kernel's share of wave time per phase (instrumented: not a timing)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="before the timed steps, run one plain negating copy of this many MiB "
                         "(fp32 in, fp32 out) to calibrate the HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the forward pass is not sharded across GPUs "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.phase_timer:
        os.environ["LAMP_LIBRARY"] = os.path.join(ROOT, "paper_2609_39361_amd", "liblamp_phase.so")
    import torch
    from paper_2609_39361_amd import lamp, workloads as W

    w = W.CONFIGS[args.workload]
    taus = [w.tau] if args.tau is None else [float(x) for x in args.tau.split(",")]
    flags_list = [int(x) for x in args.flags.split(",")]
    if w.M > 0:
        if any(f not in (0, lamp.DECODE_SERIAL) for f in flags_list) or args.sr_seed is not None:
            raise SystemExit("the decode form takes flags 0 or %d (serial) and no stochastic rounding"
                             % lamp.DECODE_SERIAL)
        if args.copy_calib_mib > 0:
            copy_calibration(args.copy_calib_mib, torch.device("cuda:0"))
        for flags in flags_list:
            for tau in taus:
                main_decode(args, w, tau, flags)
        return
    dev = torch.device("cuda:0")
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    o = torch.empty((w.B, w.Hq, w.N, w.d), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.Hq, w.N), dtype=torch.float32, device=dev)
    mask = torch.empty((w.B, w.Hq, -(-w.N // w.bq), -(-w.N // (w.bk * w.nk)) * w.nk), dtype=torch.uint8, device=dev)
    out = (o, lse, mask)
    if args.copy_calib_mib > 0:
        copy_calibration(args.copy_calib_mib, dev)
    for flags in flags_list:
        for tau in taus:
            run_fwd(args, w, tau, flags, (q, k, v), (qd, kd, vd), out, dev)


def run_fwd(args, w, tau, flags, host_inputs, dev_inputs, out, dev):
    """One bench line of the forward pass at threshold tau and variant flags."""
    import torch
    from paper_2609_39361_amd import lamp
    q, k, v = host_inputs
    qd, kd, vd = dev_inputs
    o, lse, mask = out

    sr = args.sr_seed is not None and tau != 0.0   # threshold 0 computes no 8-bit logit

    def step():
        lamp.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, out=out, flags=flags,
                      sr_seed=args.sr_seed)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    lamp.timing_read()
    if args.phase_timer:
        lamp.phase_read(reset=True)
    lamp.timing_enable(True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        step()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    phases = None
    if args.phase_timer:
        cyc, waves = lamp.phase_read(reset=True)
        tot = float(sum(cyc.values()))
        phases = {"share_of_wave_time": {k: v / tot for k, v in cyc.items()}, "waves": waves,
                  "note": "instrumented build (liblamp_phase.so): shares of the cycles each wave spends per phase; "
                          "the kernel time of this run is not the benchmark's"}
    lamp.timing_enable(False)
    launches, fwd_ms_sum, pre_ms_sum = lamp.timing_read()
    if launches != args.steps:
        raise RuntimeError("kernel timing recorded %d launches for %d steps" % (launches, args.steps))
    kernel_ms = fwd_ms_sum / launches
    ev_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    ms = float(np.mean(ev_ms))

    st = lamp.mask_stats(mask, w.nk)
    mask_np = mask.cpu().numpy()
    # the statistics words of one more call, outside the timed region
    # (saturations: how often the accumulations leave the formats' range,
    # which Sec. 3.3 assumes QK-Norm prevents)
    stw = torch.zeros(lamp.stats_words(w.nk), dtype=torch.int64, device=dev)
    lamp.attn_fwd(qd, kd, vd, w.causal, w.window, w.bq, w.bk, w.nk, w.delta, tau, out=out, flags=flags,
                  sr_seed=args.sr_seed, stats=stw)
    stats = lamp.stats_dict(stw, w.nk)
    mac8 = 0 if tau == 0 else w.macs
    mac16 = visible_in_mask(w, mask_np) * w.d
    sim = bool(flags & SIM_FLAG)
    # the multiply-adds alone at the issue rates measured on this device: one
    # emulated 8-bit step is two multiply-adds per lane (128 per wave), one
    # SIM step one (64 per wave), one 16-bit FMA with its broadcast key one
    rates = lamp.issue_rates()
    simds = 4 * torch.cuda.get_device_properties(dev).multi_processor_count
    step8 = rates["emulated_step_sim"] / 64.0 if sim else rates["emulated_step"] / 128.0
    floor_ms = (mac8 * step8 + mac16 / 64.0 * rates["fmac_f32_dpp"]) / simds * 1e-6
    issue_floor = None if sr else {
        "ms": floor_ms, "frac": floor_ms / kernel_ms,
        "ns_per_wave_instruction_per_simd": rates,
        "counts": "emulated 8-bit steps (%s) of every visible logit and 16-bit FMAs of the recomputed sub-blocks "
                  "(not the speculative ones); exponentials, stage logic and P.V not included"
                  % ("SIM profile" if sim else "hardware formats"),
    }
    alg_ops = (OPS_PER_MAC8_SIM if sim else OPS_PER_MAC8) * mac8 + OPS_PER_MAC16 * mac16
    macs_per_s = (mac8 + mac16) / (kernel_ms * 1e-3)
    achieved = macs_per_s / 1e12
    peak = VALU_LANE_OPS / 1e12
    fmac_rate = 64.0 / (rates["fmac_f32"] * 1e-9) * simds   # measured lane-FMAs per second
    result = {
        "metric": "effective attention TFLOP/s (4*B*H*N^2*d, halved for causal), 1 GPU",
        "value": w.eff_flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("SIM profile: fp32 with 3/11-bit mantissas (fp32 FMA + integer rounding), bf16 inputs, fp32 output"
                  if sim else
                  "e4m3 stochastically rounded (fp32 FMA + Philox4x32-10 bits), e4m11, bf16 inputs, fp32 output"
                  if sr else "e4m3/e4m11 emulated (fp32 FMA + fp8 conversions), bf16 inputs, fp32 output"),
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "N": w.N, "d": w.d,
                   "causal": w.causal, "window": w.window, "bq": w.bq, "bk": w.bk, "nk": w.nk,
                   "delta": w.delta, "tau": tau, "flags": flags,
                   "rounding_8bit": ("stochastic, seed %d" % args.sr_seed) if sr else "nearest-even"},
        "visible_pair_tflops": 4.0 * w.macs / (ms * 1e-3) / 1e12,   # 4*d per visible (query, key) pair
        "recompute_fraction": st["recompute_fraction"],
        "tile_hist": st["tile_hist"],
        "stats": stats,
        "roofline": {
            "bound": "alu",
            "achieved": achieved,
            "peak": peak,
            "unit": "T multiply-adds/s (one VALU lane-op per 8-bit or 16-bit MAC)",
            "frac": achieved / peak,
            "frac_2op_per_mac8": alg_ops / (kernel_ms * 1e-3) / VALU_LANE_OPS,
            "frac_vs_fp32_published": 2.0 * macs_per_s / FP32_PEAK_FLOPS,
            "frac_vs_measured_fmac_rate": macs_per_s / fmac_rate,
            "measured_fmac_lane_ops_per_s": fmac_rate,
            "traffic": None if sr else measured_traffic(w.name, tau, flags),
            "kernel": ("lamp_fwd16_kernel<%d,%d,%d,%s%s>" % (w.d, w.bq, _mode_of(tau), "true" if sim else "false",
                                                             ",SR" if sr and _mode_of(tau) != 2 else ""))
                      if (w.bk == 16 and w.d >= 128)
                      else ("lamp_fwd_kernel<%d,%d,%d,%d%s>" % (w.d, w.bq, w.bk, w.nk, ",SR" if sr else "")),
            "kernel_ms": kernel_ms,
            "prepass_ms": pre_ms_sum / launches,
            "macs_per_launch": {"mac8": mac8, "mac16": mac16},
            "ops_per_unit": ("1 per MAC for frac; frac_2op_per_mac8 charges %d per emulated 8-bit MAC "
                             "(this emulation's cost) and 1 per 16-bit MAC" % (OPS_PER_MAC8_SIM if sim else OPS_PER_MAC8)),
            "valu_issue_frac_counters": None if sr else measured_valu_issue(w.name, tau, flags),
            "issue_floor": issue_floor,
        },
        "wall_s_timed_region": wall,
    }
    if phases is not None:
        result["phases"] = phases
    if not args.no_cpu:
        gpu = (o.cpu().numpy(), lse.cpu().numpy(), mask_np)
        result["cpu_baseline"], result["parity"] = cpu_baseline(w, tau, q, k, v, budget_s=args.cpu_budget,
                                                                flags=flags, sr_seed=args.sr_seed if sr else None,
                                                                gpu=gpu)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
