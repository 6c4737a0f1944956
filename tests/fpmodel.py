"""Independent reference models used to pin the oracle.

Nothing here calls the oracle.  The rounding models use integer arithmetic
(numpy int64 on decomposed significands, or Python Fractions), a different
method from the oracle's frexp/nearbyint rounding, and the exponential tables
are derived from mpmath at 60 significant digits.
"""
from fractions import Fraction
import functools

import numpy as np

# (mbits, emin, maxval, bias, ebits, signed) of the method's formats
# (paper Sec. 3.3); emin is the smallest normal exponent.
FMT = {
    "e4m3": (3, -6, 448.0, 7, 4, True),
    "e4m11": (11, -6, 511.875, 7, 4, True),
    "ue5m3_shift": (3, -14, 122880.0, 15, 5, False),
    "ue5m11_shift": (11, -14, 131040.0, 15, 5, False),
    "ue5m3_exp": (3, -30, 1.875, 31, 5, False),
    "ue5m11_exp": (11, -30, 2.0 - 2.0 ** -11, 31, 5, False),
    # the "SIM" profile (Sec. 4.1): FP32's exponent range and gradual
    # underflow, 3 or 11 mantissa bits, no saturation (overflow gives inf)
    "sim3": (3, -126, np.inf, 127, 8, True),
    "sim11": (11, -126, np.inf, 127, 8, True),
}


def np_round(x, fmt):
    """Round doubles to a format with integer arithmetic (RNE, subnormals, saturation)."""
    mbits, emin, maxval = FMT[fmt][:3]
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    m, e = np.frexp(ax)                                 # ax = m * 2^e, m in [0.5, 1)
    S = np.round(m * 2.0 ** 53).astype(np.int64)         # exact 53-bit significand
    E = e.astype(np.int64) - 53                          # ax = S * 2^E
    te = np.maximum(e.astype(np.int64) - 1, emin) - mbits  # exponent of the quantum
    shift = te - E                                       # >= 1 for these formats
    big = shift >= 60
    sh = np.where(big, 1, shift)
    n = S >> sh
    rem = S & ((np.int64(1) << sh) - 1)
    half = np.int64(1) << (sh - 1)
    up = (rem > half) | ((rem == half) & ((n & 1) == 1))
    n = n + up.astype(np.int64)
    n = np.where(big, 0, n)
    r = n.astype(np.float64) * np.exp2(te.astype(np.float64))
    r = np.where(ax == 0, 0.0, r)
    r = np.minimum(r, maxval)
    if np.isinf(maxval):
        r = np.where(r >= 2.0 ** 128, np.inf, r)         # FP32 overflow
    r = np.where(np.isinf(ax), maxval, r)
    return np.copysign(r, x)


def np_quantum(x, fmt):
    """Grid spacing of a format in the binade of each |x| (x != 0)."""
    mbits, emin = FMT[fmt][:2]
    _, e = np.frexp(np.abs(np.asarray(x, dtype=np.float64)))
    return np.exp2((np.maximum(e.astype(np.int64) - 1, emin) - mbits).astype(np.float64))


def np_encode(v, fmt):
    """Codes of values that lie on the grid (integer construction)."""
    mbits, emin, maxval, bias, ebits, signed = FMT[fmt]
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    sign = (np.signbit(v) & signed).astype(np.int64)
    m, e = np.frexp(a)
    eu = e.astype(np.int64) - 1
    normal = a >= 2.0 ** emin
    man_n = np.round(a / np.exp2((eu - mbits).astype(np.float64))).astype(np.int64) - (1 << mbits)
    man_s = np.round(a / 2.0 ** (emin - mbits)).astype(np.int64)
    code = np.where(normal, ((eu + bias) << mbits) | man_n, man_s)
    return (sign << (ebits + mbits)) | code


def np_decode(code, fmt):
    """Values of codes (integer construction)."""
    mbits, emin, maxval, bias, ebits, signed = FMT[fmt]
    c = np.asarray(code, dtype=np.int64)
    m = c & ((1 << mbits) - 1)
    e = (c >> mbits) & ((1 << ebits) - 1)
    sign = ((c >> (ebits + mbits)) & 1) if signed else np.zeros_like(c)
    v = np.where(e == 0, m * 2.0 ** (emin - mbits),
                 ((1 << mbits) | m) * np.exp2((e - bias - mbits).astype(np.float64)))
    return np.where(sign == 1, -v, v)


def frac_round(x: Fraction, mbits, emin, maxval=None):
    """Round a Fraction to a binary grid with `mbits` mantissa bits and smallest
    normal exponent `emin` (RNE; saturating at maxval when given)."""
    if x == 0:
        return Fraction(0)
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    e = max(e, emin)
    q = Fraction(2) ** (e - mbits)
    r = round(a / q) * q                    # round() on a Fraction is half-to-even
    if maxval is not None and r > maxval:
        r = Fraction(maxval)
    return r if x > 0 else -r


def frac_fmt(x, fmt):
    mbits, emin, maxval = FMT[fmt][:3]
    return frac_round(Fraction(x), mbits, emin, Fraction(maxval))


def rn32(x: Fraction):
    return frac_round(x, 23, -126)


def rn64(x: Fraction):
    return frac_round(x, 52, -1022)


def bf16_to_float(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


SIM_EMIN, SIM_EMAX = -20, 8   # shifts below 2^-20 give 1, from 2^9 on 0, in both SIM widths


@functools.lru_cache(maxsize=None)
def mp_sim_exp(p):
    """RN_p(exp(-s)) in the SIM profile for every shift s = (2^p + m) 2^(e-p),
    e in [SIM_EMIN, SIM_EMAX], m in [0, 2^p), from mpmath; flat index
    (e - SIM_EMIN) 2^p + m.  Every value is certified far from a midpoint."""
    import mpmath as mp
    mp.mp.prec = 160
    n = (SIM_EMAX - SIM_EMIN + 1) << p
    tab = np.empty(n)
    for idx in range(n):
        e, m = SIM_EMIN + (idx >> p), idx & ((1 << p) - 1)
        s = Fraction((1 << p) | m) * Fraction(2) ** (e - p)
        y = mp.exp(-mp.mpf(s.numerator) / s.denominator)
        man, ex = mp.mpf(y).man_exp
        yf = Fraction(int(man)) * Fraction(2) ** int(ex)
        r = frac_round(yf, p, -126)
        ey = yf.numerator.bit_length() - yf.denominator.bit_length()
        if Fraction(2) ** ey > yf:
            ey -= 1
        qy = Fraction(2) ** (max(ey, -126) - p)
        t = yf / qy - (yf // qy)
        assert abs(t - Fraction(1, 2)) * qy > yf * Fraction(1, 2 ** 120)
        tab[idx] = float(r)
    return tab


def sim_exp_lookup(s, p):
    """RN_p(exp(-s)) for shifts s >= 0 on the SIM p-bit grid, from mp_sim_exp."""
    tab = mp_sim_exp(p)
    s = np.asarray(s, dtype=np.float64)
    fr, e = np.frexp(np.where(s > 0, s, 1.0))
    e = e.astype(np.int64) - 1
    m = np.round((fr * 2.0) * (1 << p)).astype(np.int64) - (1 << p)
    idx = (np.clip(e, SIM_EMIN, SIM_EMAX) - SIM_EMIN) * (1 << p) + m
    v = tab[np.clip(idx, 0, tab.size - 1)]
    v = np.where(e < SIM_EMIN, 1.0, np.where(e > SIM_EMAX, 0.0, v))
    return np.where(s > 0, v, 1.0)


@functools.lru_cache(maxsize=None)
def mp_exp_tables():
    """(LUT8, EXP16) from mpmath: E = RN_exp(exp(-s)) for every shift code."""
    import mpmath as mp
    mp.mp.prec = 160
    out = {}
    for name, shift_fmt, exp_fmt, n in (("lut8", "ue5m3_shift", "ue5m3_exp", 256),
                                        ("exp16", "ue5m11_shift", "ue5m11_exp", 65536)):
        smb, semin = FMT[shift_fmt][:2]
        emb, eemin = FMT[exp_fmt][:2]
        tab = np.empty(n, dtype=np.uint32)
        for c in range(n):
            e_field, m_field = c >> smb, c & ((1 << smb) - 1)
            if e_field == 0:
                s = Fraction(m_field) * Fraction(2) ** (semin - smb)
            else:
                s = Fraction((1 << smb) | m_field) * Fraction(2) ** (e_field - FMT[shift_fmt][3] - smb)
            if s > 40:          # exp(-40) < 2^-57: rounds to 0 in both formats
                tab[c] = 0
                continue
            y = mp.exp(-mp.mpf(s.numerator) / s.denominator)
            man, ex = mp.mpf(y).man_exp if y != 0 else (0, 0)
            yf = Fraction(int(man)) * Fraction(2) ** int(ex) if y != 0 else Fraction(0)
            r = frac_round(yf, emb, eemin)
            # the 200-bit value must be far from a rounding midpoint (odd
            # multiples of half the quantum of its binade)
            if yf != 0:
                ey = yf.numerator.bit_length() - yf.denominator.bit_length()
                if Fraction(2) ** ey > yf:
                    ey -= 1
                qy = Fraction(2) ** (max(ey, eemin) - emb)
                t = yf / qy - (yf // qy)
                assert abs(t - Fraction(1, 2)) * qy > yf * Fraction(1, 2 ** 120)
            tab[c] = int(np_encode(float(r), exp_fmt))
        out[name] = tab
    return out["lut8"].astype(np.uint8), out["exp16"].astype(np.uint16)
