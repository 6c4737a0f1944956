"""A second, independent implementation of LampAttention (paper Sec. 3.1-3.2,
Algorithm 1) for tiny inputs, used to pin the C oracle.

Written separately from the oracle with different methods:
  * numpy vectorised over a whole tile instead of scalar loops;
  * the FP32 FMAs of the 8- and 16-bit accumulations are emulated exactly
    from fp64 products and a TwoSum correction instead of calling fmaf;
  * rounding to the formats with the integer model of fpmodel.py;
  * exponential tables from mpmath, lambda_hat from math.exp;
  * the SIM profile's exact shift rounding from a TwoSum and a midpoint test;
  * the stage-2 knapsack by brute force over every g in {0,1}^N_k.
It asserts the stage-1 invariant (every 8-bit sub-block passes the margin test
against the final running maximum) on every tile.
"""
import math

import numpy as np

import fpmodel as M


def _two_sum(a, b):
    s = a + b
    bb = s - a
    e = (a - (s - bb)) + (b - bb)
    return s, e


def rn32_sum(p, c):
    """RN32(p + c) for fp64 arrays p (exact products) and c (fp32 values)."""
    s, e = _two_sum(p, c)
    r = s.astype(np.float32).astype(np.float64)
    inexact = r != s
    # neighbour on the other side of s
    toward = np.where(s > r, np.inf, -np.inf).astype(np.float32)
    r2 = np.nextafter(r.astype(np.float32), toward).astype(np.float64)
    mid = (r + r2) / 2
    # Only when s is exactly an fp32 midpoint can the exact sum s + e round
    # differently from s (any other midpoint is an fp64 number strictly closer
    # to s + e than s, impossible).  Then the sign of e decides.
    tie = inexact & (s == mid) & (e != 0)
    go_r2 = tie & (np.sign(e) == np.sign(r2 - r))
    return np.where(go_r2, r2, r)


def _clamped(t, fmt):
    """Where rounding t to fmt (e4m3 or e4m11) exceeds the largest value, so
    that the saturating rounding clamps it: the rounding is repeated on a grid
    without a largest value (same mantissa bits and smallest normal)."""
    mbits, emin, maxval = M.FMT[fmt][:3]
    q = M.np_quantum(np.where(t != 0, t, 1.0), fmt)
    r = np.round(np.abs(t) / q) * q                     # numpy rounds halves to even
    return (r > maxval) & (t != 0)


def y8_tile(qt, kf, fmt="e4m3", sat=None):
    """qt [bq, d] fp32 values (as fp64), kf [T, d] -> Y8 values [T, bq]
    (fmt "sim3" for the SIM profile).  sat: an optional bool array [T, bq]
    or-ed with the chains clamped in some step."""
    acc = np.zeros((kf.shape[0], qt.shape[0]))
    for c in range(qt.shape[1]):
        p = kf[:, c][:, None] * qt[:, c][None, :]          # exact in fp64
        t = rn32_sum(p, acc)
        if sat is not None and fmt == "e4m3":
            sat |= _clamped(t, fmt)
        acc = M.np_round(t, fmt)
    return acc


# ---- stochastic rounding of the 8-bit accumulation (Sec. 3.3's alternative
# to round-to-nearest).  Written apart from the oracle: Philox4x32-10 on numpy
# arrays of 64-bit integers (all counters of a tile at once), the e4m3
# neighbours from a search of the enumerated e4m3 magnitudes.
_E4M3_MAGS = None


def e4m3_mags():
    global _E4M3_MAGS
    if _E4M3_MAGS is None:
        # e4m3: bias 7, 3 stored bits, subnormals below 2^-6, 0x7F the NaN
        vals = []
        for code in range(0x7F):
            e, m = code >> 3, code & 7
            vals.append(m * 2.0 ** -9 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7))
        _E4M3_MAGS = np.array(vals)
    return _E4M3_MAGS


def philox4x32(ctr, key, rounds=10):
    """Philox4x32 (Salmon et al., SC 2011) of counters ctr [..., 4] under key
    (k0, k1); numpy uint64 arithmetic, every word kept below 2^32."""
    mask = np.uint64(0xFFFFFFFF)
    x = [np.asarray(ctr[..., t], dtype=np.uint64) & mask for t in range(4)]
    k0, k1 = np.uint64(key[0] & 0xFFFFFFFF), np.uint64(key[1] & 0xFFFFFFFF)
    mul = (np.uint64(0xD2511F53), np.uint64(0xCD9E8D57))
    weyl = (np.uint64(0x9E3779B9), np.uint64(0xBB67AE85))
    for rnd in range(rounds):
        if rnd:
            k0, k1 = (k0 + weyl[0]) & mask, (k1 + weyl[1]) & mask
        p0 = mul[0] * x[0]                      # < 2^64: exact in uint64
        p1 = mul[1] * x[2]
        x = [(p1 >> np.uint64(32)) ^ x[1] ^ k0, p1 & mask, (p0 >> np.uint64(32)) ^ x[3] ^ k1, p0 & mask]
    return np.stack(x, axis=-1)


def sr_r16(seed, j, i, bh, c):
    """16-bit random integers of channel c for arrays of query rows j and keys
    i: Philox4x32-10 at counter (j, i, bh, c // 8), key (seed mod 2^32,
    seed // 2^32); the low (c even) or high (c odd) half of word (c mod 8) // 2."""
    j, i = np.broadcast_arrays(np.asarray(j, dtype=np.uint64), np.asarray(i, dtype=np.uint64))
    ctr = np.stack([j, i, np.full(j.shape, bh, dtype=np.uint64), np.full(j.shape, c // 8, dtype=np.uint64)], -1)
    w = philox4x32(ctr, (seed & 0xFFFFFFFF, seed >> 32))[..., (c % 8) // 2]
    return ((w >> np.uint64(16 * (c & 1))) & np.uint64(0xFFFF)).astype(np.float64)


def sr_round(t, r):
    """Stochastic rounding of fp64 values t (fp32 numbers) to e4m3, random integers r < 2^16."""
    mags = e4m3_mags()
    a = np.minimum(np.abs(t), 448.0)
    idx = np.searchsorted(mags, a, side="right") - 1
    lo = mags[idx]
    hi = mags[np.minimum(idx + 1, mags.size - 1)]
    u = np.where(hi > lo, hi - lo, 1.0)
    frac16 = np.floor((a - lo) / u * 2.0 ** 16)
    res = np.where(frac16 + r >= 2.0 ** 16, hi, lo)
    return np.copysign(res, t)


def y8_tile_sr(qt, kf, seed, bh, rows, keys, sat=None):
    """Y8 values [T, bq] with stochastic rounding; rows / keys: the query and
    key indices of qt's rows and kf's rows.  sat: as in y8_tile (a step with
    |t| > 448)."""
    d = qt.shape[1]
    ii, jj = np.meshgrid(np.asarray(keys), np.asarray(rows), indexing="ij")   # [T, bq]
    acc = np.zeros((kf.shape[0], qt.shape[0]))
    for c in range(d):
        p = kf[:, c][:, None] * qt[:, c][None, :]          # exact in fp64
        t = rn32_sum(p, acc)
        if sat is not None:
            sat |= np.abs(t) > 448.0
        acc = sr_round(t, sr_r16(seed, jj, ii, bh, c))
    return acc


def y16_tile(qt, kf, fmt="e4m11", sat=None, step=False):
    """Y16 values [T, bq]: the FP32 FMA chain rounded once to fmt, or, with
    `step`, rounded to fmt after every FMA (e4m11 as the accumulator).  sat:
    as in y8_tile."""
    acc = np.zeros((kf.shape[0], qt.shape[0]))
    for c in range(qt.shape[1]):
        p = kf[:, c][:, None] * qt[:, c][None, :]           # exact in fp64
        acc = rn32_sum(p, acc)                               # FP32 FMA step
        if step:
            if sat is not None and fmt == "e4m11":
                sat |= _clamped(acc, fmt)
            acc = M.np_round(acc, fmt)
    if step:
        return acc
    if sat is not None and fmt == "e4m11":
        sat |= _clamped(acc, fmt)
    return M.np_round(acc, fmt)


def sim_shift(muh, y, p):
    """RN_p(max(0, muh - y)) of the exact difference in the SIM profile: the
    fp64 difference and its TwoSum error; only an fp64 result exactly halfway
    between two grid values can round differently, then the error's sign
    decides."""
    fmt = "sim3" if p == 3 else "sim11"
    hi, lo = _two_sum(np.asarray(muh, dtype=np.float64), -np.asarray(y, dtype=np.float64))
    r = M.np_round(hi, fmt)
    with np.errstate(invalid="ignore"):
        q = M.np_quantum(np.where(hi != 0, hi, 1.0), fmt)
        t = np.abs(hi) / q
        mid = (t - np.floor(t) == 0.5) & (lo != 0) & (hi != 0)
        away = (lo > 0) == (hi > 0)
        adj = np.copysign(np.where(away, np.floor(t) + 1, np.floor(t)) * q, hi)
    r = np.where(mid, adj, r)
    return np.where(hi > 0, r, 0.0)


def _shift_exp(muh, y, high, tabs, sim=False):
    if sim:
        p = 11 if high else 3
        return M.sim_exp_lookup(sim_shift(muh[None, :], y, p), p)
    x = np.maximum(muh[None, :] - y, 0.0)
    if high:
        code = M.np_encode(M.np_round(x, "ue5m11_shift"), "ue5m11_shift")
        e = tabs[1][code]
        return M.np_decode(e, "ue5m11_exp")
    code = M.np_encode(M.np_round(x, "ue5m3_shift"), "ue5m3_shift")
    return M.np_decode(tabs[0][code], "ue5m3_exp")


def _trunc_e4m3(x):
    """Round toward zero onto the e4m3 grid (3 stored mantissa bits, smallest
    normal 2^-6), saturating at 448; infinities kept."""
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    fin = np.isfinite(ax) & (ax > 0)
    _, ex = np.frexp(np.where(fin, ax, 1.0))
    e = np.maximum(ex - 1, -6)
    quantum = np.ldexp(1.0, e - 3)
    t = np.floor(ax / quantum) * quantum
    t = np.where(ax >= 448.0, 448.0, t)
    return np.where(fin, np.copysign(t, x), x)


def _trunc_sim3(x):
    """Round toward zero to 3 mantissa bits in FP32's exponent range."""
    x = np.asarray(x, dtype=np.float64)
    fin = np.isfinite(x) & (x != 0)
    q = M.np_quantum(np.where(fin, x, 1.0), "sim3")
    return np.where(fin, np.copysign(np.floor(np.abs(x) / q) * q, x), x)


def _colsum(E):
    """Sum over keys in ascending order, one fp64 addition at a time."""
    S = np.zeros(E.shape[1])
    for r in range(E.shape[0]):
        S = S + E[r]
    return S


def ref_fwd(q, k, v, causal, window, bq, bk, nk, delta, tau, tabs, scale, flags=0, seed=0, stats=False):
    """q [B,Hq,N,d], k/v [B,Hkv,N,d] bf16 bit patterns.  Returns o, lse, mask
    (and, with `stats`, a dict of the statistics: tiles, stage1, stage2,
    inactive, sat8, sat16, hist).  flags: 1 = first stage disabled, 2 = 8-bit
    shifts against mu_hat truncated to e4m3 (both only for 0 < tau < inf),
    4 = the SIM precision profile (Sec. 4.1) in every mode, 8 = the 8-bit
    accumulation rounded stochastically with random words keyed by `seed`,
    16 = the 16-bit logits with e4m11 (SIM: 11 bits) as the accumulator."""
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    T = bk * nk
    o = np.zeros((B, Hq, N, d))
    lse = np.zeros((B, Hq, N))
    nqb, ntiles = -(-N // bq), -(-N // T)          # ragged lengths: keys and rows beyond N do not exist
    mask = np.full((B, Hq, nqb, ntiles * nk), 3, dtype=np.uint8)
    pure8 = math.isinf(tau)
    all16 = tau == 0.0
    stage1_off = (not pure8) and (not all16) and bool(flags & 1)
    mu_trunc = (not pure8) and (not all16) and bool(flags & 2)
    sim = bool(flags & 4)
    step16 = bool(flags & 16)
    f8, f16 = ("sim3", "sim11") if sim else ("e4m3", "e4m11")
    st = {"tiles": 0, "stage1": 0, "stage2": 0, "inactive": 0, "sat8": 0, "sat16": 0, "hist": [0] * (nk + 1)}
    trunc8 = _trunc_sim3 if sim else _trunc_e4m3
    for b in range(B):
        for h in range(Hq):
            kf_all = M.bf16_to_float(k[b, h // G])
            vf_all = M.bf16_to_float(v[b, h // G])
            for qb in range(nqb):
                q0 = qb * bq
                nr = min(bq, N - q0)
                qf = np.zeros((bq, d))
                qf[:nr] = M.bf16_to_float(q[b, h, q0:q0 + nr])
                qt = (qf * np.float64(scale)).astype(np.float32).astype(np.float64)
                mu = np.full(bq, -np.inf)
                om = np.zeros(bq)
                O = np.zeros((bq, d))
                jj = q0 + np.arange(bq)
                for t in range(ntiles):
                    ii = t * T + np.arange(T)
                    vis = (ii[:, None] < N) & (jj[None, :] < N)
                    if causal:
                        vis &= ii[:, None] <= jj[None, :]
                    if window > 0:
                        vis &= ii[:, None] > jj[None, :] - window
                    act = np.array([vis[th * bk:(th + 1) * bk].any() for th in range(nk)])
                    if not act.any():
                        continue
                    kf = kf_all[np.minimum(ii, N - 1)]
                    prec = np.where(act, 0, 3)
                    Y = np.full((T, bq), np.nan)
                    sat8 = np.zeros((T, bq), dtype=bool)
                    if not all16 and flags & 8:
                        Y = y8_tile_sr(qt, kf, seed, b * Hq + h, jj, ii, sat=sat8)
                    elif not all16:
                        Y = y8_tile(qt, kf, f8, sat=sat8)
                    st["sat8"] += int((sat8 & vis).sum())
                    Yv = np.where(vis, Y, -np.inf)
                    m8 = np.array([Yv[th * bk:(th + 1) * bk].max(axis=0) for th in range(nk)])
                    muh = mu.copy()
                    Y16 = None
                    sat16 = np.zeros((T, bq), dtype=bool)

                    def y16():
                        nonlocal Y16
                        if Y16 is None:
                            Y16 = y16_tile(qt, kf, f16, sat=sat16, step=step16)
                        return Y16

                    if pure8 or stage1_off:
                        for th in range(nk):
                            if act[th]:
                                muh = np.maximum(muh, m8[th])
                    elif all16:
                        for th in range(nk):
                            if act[th]:
                                prec[th] = 1
                                sl = slice(th * bk, (th + 1) * bk)
                                Y[sl] = y16()[sl]
                                muh = np.maximum(muh, np.where(vis[sl], Y[sl], -np.inf).max(axis=0))
                    else:
                        thr = {}
                        for th in range(nk):
                            if act[th]:
                                m = m8[th]
                                ok = m > -np.inf
                                thr[th] = (m[ok] - mu[ok]).max()
                        order = sorted(thr, key=lambda th: (-thr[th], th))
                        for th in order:
                            m = m8[th]
                            ok = m > -np.inf
                            margin = muh[ok] > m[ok] + np.abs(muh[ok]) * delta
                            if margin.all():
                                continue
                            prec[th] = 1
                            sl = slice(th * bk, (th + 1) * bk)
                            Y[sl] = y16()[sl]
                            muh = np.maximum(muh, np.where(vis[sl], Y[sl], -np.inf).max(axis=0))
                        # stage-1 invariant against the final mu_hat
                        for th in range(nk):
                            if act[th] and prec[th] == 0:
                                m = m8[th]
                                ok = m > -np.inf
                                assert np.all(muh[ok] > m[ok] + np.abs(muh[ok]) * delta)
                    E = np.zeros((T, bq))
                    for th in range(nk):
                        if prec[th] == 3:
                            continue
                        sl = slice(th * bk, (th + 1) * bk)
                        high = prec[th] == 1
                        ref = trunc8(muh) if (mu_trunc and not high) else muh
                        e = _shift_exp(ref, np.where(vis[sl], Y[sl], 0.0), high, tabs, sim)
                        E[sl] = np.where(vis[sl], e, 0.0)
                    lam = np.where(muh == -np.inf, 1.0,
                                   np.where(mu == -np.inf, 0.0,
                                            np.exp(np.where(np.isfinite(mu) & np.isfinite(muh), mu - muh, 0.0))))
                    omh = lam * om + _colsum(E)
                    if not pure8 and not all16:
                        F = [th for th in range(nk) if prec[th] == 0]
                        cost = {}
                        for th in F:
                            c = np.zeros(bq)
                            for r in range(th * bk, (th + 1) * bk):
                                c = c + np.where(vis[r], E[r] * (omh - E[r]), 0.0)
                            cost[th] = c
                        lim = (tau * omh) * omh
                        best = None
                        for g in range(1 << len(F)):           # g: kept (8-bit) subset of F
                            keep = [F[a] for a in range(len(F)) if g >> a & 1]
                            xi = np.zeros(bq)
                            for th in sorted(keep):
                                xi = xi + cost[th]
                            if not np.all(xi <= lim):
                                continue
                            rmask = sum(1 << th for th in F if th not in keep)
                            key = (len(keep), -rmask)
                            if best is None or key > best[0]:
                                best = (key, rmask)
                        rmask = best[1]
                        for th in range(nk):
                            if rmask >> th & 1:
                                prec[th] = 2
                                sl = slice(th * bk, (th + 1) * bk)
                                Y[sl] = y16()[sl]
                                e = _shift_exp(muh, np.where(vis[sl], Y[sl], 0.0), True, tabs, sim)
                                E[sl] = np.where(vis[sl], e, 0.0)
                    om = lam * om + _colsum(E)
                    O = O * lam[:, None] + E.T @ vf_all[np.minimum(ii, N - 1)]
                    mu = muh
                    mask[b, h, qb, t * nk:(t + 1) * nk] = prec
                    rec = [th for th in range(nk) if prec[th] in (1, 2)]
                    st["tiles"] += 1
                    st["stage1"] += int((prec == 1).sum())
                    st["stage2"] += int((prec == 2).sum())
                    st["hist"][len(rec)] += 1
                    for th in rec:
                        sl = slice(th * bk, (th + 1) * bk)
                        st["sat16"] += int((sat16[sl] & vis[sl]).sum())
                with np.errstate(invalid="ignore", divide="ignore"):
                    o[b, h, q0:q0 + nr] = (O / om[:, None])[:nr]
                    lse[b, h, q0:q0 + nr] = (mu + np.log(om))[:nr]
    st["inactive"] = int((mask == 3).sum())
    if stats:
        return o, lse, mask, st
    return o, lse, mask


def ref_decode(q, k, v, causal, window, tk, delta, tau, tabs, scale):
    """The vector-LAMP decode pass (Sec. 2, Eq. (6)), independently: q
    [B,Hq,M,d] rows at positions N-M .. N-1, k/v [B,Hkv,N,d] bf16 patterns.
    The greedy knapsack is checked on every tile against the exact optimum
    (largest number of 8-bit logits whose exact cost sum fits the limit)."""
    from fractions import Fraction
    B, Hq, Mr, d = q.shape
    Hkv, N = k.shape[1], k.shape[2]
    G = Hq // Hkv
    ntiles = -(-N // tk)
    o = np.zeros((B, Hq, Mr, d))
    lse = np.zeros((B, Hq, Mr))
    mask = np.full((B, Hq, Mr, ntiles * tk), 3, dtype=np.uint8)
    pure8, all16 = math.isinf(tau), tau == 0.0
    for b in range(B):
        for h in range(Hq):
            kf_all = M.bf16_to_float(k[b, h // G])
            vf_all = M.bf16_to_float(v[b, h // G])
            for r in range(Mr):
                P = N - Mr + r
                qt = (M.bf16_to_float(q[b, h, r]) * np.float64(scale)).astype(np.float32).astype(np.float64)
                mu, om = -np.inf, 0.0
                O = np.zeros(d)
                for t in range(ntiles):
                    ii = t * tk + np.arange(tk)
                    vis = ii < N
                    if causal:
                        vis &= ii <= P
                    if window > 0:
                        vis &= ii > P - window
                    if not vis.any():
                        continue
                    kf = kf_all[np.minimum(ii, N - 1)]
                    prec = np.where(vis, 0, 3)
                    Y16 = y16_tile(qt[None, :], kf)[:, 0]
                    if all16:
                        Y = Y16.copy()
                        prec[vis] = 1
                        muh = max(mu, Y[vis].max())
                    else:
                        Y = y8_tile(qt[None, :], kf)[:, 0]
                        yv = np.where(vis, Y, -np.inf)
                        c = int(np.argmax(yv))            # first index of the maximum
                        if pure8:
                            muh = max(mu, Y[c])
                        elif mu > Y[c] + abs(mu) * delta:
                            muh = mu
                        else:
                            Y[c] = Y16[c]
                            prec[c] = 1
                            muh = max(mu, Y[c])
                    E = np.zeros(tk)
                    for i in np.nonzero(vis)[0]:
                        E[i] = _shift_exp(np.array([muh]), np.array([[Y[i]]]), prec[i] == 1, tabs)[0, 0]
                    lam = 0.0 if mu == -np.inf else math.exp(mu - muh)
                    omh = lam * om + _colsum(E[:, None])[0]
                    if not pure8 and not all16:
                        F = [i for i in range(tk) if prec[i] == 0]
                        kap = {i: E[i] * (omh - E[i]) for i in F}
                        order = sorted(F, key=lambda i: (kap[i], i))
                        lim = (tau * omh) * omh
                        xi, nkeep = 0.0, 0
                        for i in order:
                            if not (xi + kap[i] <= lim):
                                break
                            xi += kap[i]
                            nkeep += 1
                        # exact optimum of the uniform-value knapsack
                        exact = sorted(Fraction(kap[i]) for i in F)
                        acc, best = Fraction(0), 0
                        for x in exact:
                            if acc + x > Fraction(lim):
                                break
                            acc += x
                            best += 1
                        assert nkeep == best, (b, h, r, t, nkeep, best)
                        for i in order[nkeep:]:
                            prec[i] = 2
                            Y[i] = Y16[i]
                            E[i] = _shift_exp(np.array([muh]), np.array([[Y[i]]]), True, tabs)[0, 0]
                    om = lam * om + _colsum(E[:, None])[0]
                    O = O * lam + E @ vf_all[np.minimum(ii, N - 1)]
                    mu = muh
                    mask[b, h, r, t * tk:(t + 1) * tk] = prec
                o[b, h, r] = O / om
                lse[b, h, r] = mu + math.log(om)
    return o, lse, mask
