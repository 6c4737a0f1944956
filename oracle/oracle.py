"""ctypes wrapper around the CPU oracle (oracle/lamp_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's cpu_baseline leg, never by the product path.  It shares no code
with the GPU library.

All functions take numpy arrays on the host.  Q, K and V are passed as bf16 bit
patterns (uint16); see `bf16_bits` for the conversion from a torch tensor.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblamp_oracle.so")

# Format ids understood by the oracle's codec entry points.
E4M3, E4M11, UE5M3_SHIFT, UE5M11_SHIFT, UE5M3_EXP, UE5M11_EXP = range(6)

MASK_LOW, MASK_STAGE1, MASK_STAGE2, MASK_INACTIVE = 0, 1, 2, 3

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            import importlib.util
            spec = importlib.util.spec_from_file_location("_oracle_build", os.path.join(HERE, "build.py"))
            mod = importlib.util.module_from_spec(spec)
            spec.loader.exec_module(mod)
            mod.build()
        _lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        _lib.lamp_oracle_fwd.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32,
                                         f64, f64, ctypes.c_uint, P, P, P, P, i64, i32]
        _lib.oracle_trunc_e4m3.argtypes = [f64]
        _lib.oracle_trunc_e4m3.restype = f64
        _lib.lamp_oracle_fwd.restype = i32
        _lib.lamp_oracle_fwd_seeded.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32,
                                                f64, f64, ctypes.c_uint, ctypes.c_uint64, P, P, P, P, i64, i32]
        _lib.lamp_oracle_fwd_seeded.restype = i32
        _lib.lamp_oracle_fwd_ex.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32,
                                            f64, f64, ctypes.c_uint, ctypes.c_uint64, P, P, P, P, i64, i32, P]
        _lib.lamp_oracle_fwd_ex.restype = i32
        _lib.oracle_philox4x32_10.argtypes = [P, P, P]
        _lib.oracle_philox4x32_10.restype = None
        _lib.oracle_sr_e4m3.argtypes = [P, P, P, i64]
        _lib.oracle_sr_e4m3.restype = i32
        _lib.oracle_logits8_sr.argtypes = [P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, ctypes.c_uint64, P, i32]
        _lib.oracle_logits8_sr.restype = i32
        for name in ("oracle_logits8", "oracle_logits16", "oracle_logits16_step"):
            fn = getattr(_lib, name)
            fn.argtypes = [P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, P, i32]
            fn.restype = i32
        for name in ("oracle_round_fmt", "oracle_encode_fmt", "oracle_decode_fmt"):
            fn = getattr(_lib, name)
            fn.argtypes = [i32, P, P, i64]
            fn.restype = i32
        _lib.oracle_e4m3_of_f32_bits.argtypes = [ctypes.c_uint64, i64, P, i32]
        _lib.oracle_e4m3_of_f32_bits.restype = i32
        _lib.oracle_exp_doc.argtypes = [P, P, i64]
        _lib.oracle_exp_doc.restype = i32
        _lib.oracle_exp_doc_constants.argtypes = [P]
        _lib.oracle_exp_doc_constants.restype = i32
        _lib.oracle_tables.argtypes = [P, P]
        _lib.oracle_tables.restype = i32
        _lib.oracle_scale.argtypes = [i32]
        _lib.oracle_scale.restype = ctypes.c_float
        for name in ("oracle_round_sim", "oracle_sim_exp"):
            fn = getattr(_lib, name)
            fn.argtypes = [i32, P, P, i64]
            fn.restype = i32
        _lib.oracle_shift_sim.argtypes = [i32, P, P, P, i64]
        _lib.oracle_shift_sim.restype = i32
        _lib.oracle_trunc_sim3.argtypes = [f64]
        _lib.oracle_trunc_sim3.restype = f64
        _lib.oracle_logits_sim.argtypes = [P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, P, i32]
        _lib.oracle_logits_sim.restype = i32
        _lib.lamp_oracle_decode.argtypes = [P, P, P] + [i32] * 9 + [f64, f64, ctypes.c_uint, P, P, P, P, i64, i32]
        _lib.lamp_oracle_decode.restype = i32
        _lib.oracle_max_threads.argtypes = []
        _lib.oracle_max_threads.restype = i32
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def bf16_bits(t):
    """uint16 numpy array of the bf16 bit patterns of a torch bf16 tensor."""
    import torch
    assert t.dtype == torch.bfloat16
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


# ---------------------------------------------------------------- codecs
def round_fmt(fmt, x):
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    assert lib().oracle_round_fmt(fmt, _ptr(x), _ptr(y), x.size) == 0
    return y


def encode_fmt(fmt, x):
    x = np.ascontiguousarray(x, dtype=np.float64)
    c = np.empty(x.shape, dtype=np.uint32)
    assert lib().oracle_encode_fmt(fmt, _ptr(x), _ptr(c), x.size) == 0
    return c


def decode_fmt(fmt, c):
    c = np.ascontiguousarray(c, dtype=np.uint32)
    y = np.empty(c.shape, dtype=np.float64)
    assert lib().oracle_decode_fmt(fmt, _ptr(c), _ptr(y), c.size) == 0
    return y


def e4m3_of_f32_bits(start, count, nthreads=0):
    out = np.empty(count, dtype=np.uint8)
    assert lib().oracle_e4m3_of_f32_bits(start, count, _ptr(out), nthreads) == 0
    return out


def exp_doc(x):
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    assert lib().oracle_exp_doc(_ptr(x), _ptr(y), x.size) == 0
    return y


def exp_doc_constants():
    c = np.empty(17, dtype=np.float64)
    lib().oracle_exp_doc_constants(_ptr(c))
    return c


def tables():
    lut8 = np.empty(256, dtype=np.uint8)
    exp16 = np.empty(65536, dtype=np.uint16)
    rc = lib().oracle_tables(_ptr(lut8), _ptr(exp16))
    if rc != 0:
        raise RuntimeError("oracle table construction failed (%d)" % rc)
    return lut8, exp16


def scale(d):
    return lib().oracle_scale(d)


# ---------------------------------------------------------------- logits
def logits8(q, k, causal, window, row0, nrows, nthreads=0):
    """e4m3 codes of the 8-bit logits of rows [row0, row0+nrows): [B,Hq,nrows,N], 0xFF = invisible."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    out = np.empty((B, Hq, nrows, N), dtype=np.uint8)
    rc = lib().oracle_logits8(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window),
                              row0, nrows, _ptr(out), nthreads)
    assert rc == 0
    return out


def philox4x32_10(counter, key):
    """Philox4x32-10 (Salmon et al., SC 2011) of one counter (4 words) under key (2 words)."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    kk = np.ascontiguousarray(key, dtype=np.uint32)
    assert c.shape == (4,) and kk.shape == (2,)
    out = np.empty(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c), _ptr(kk), _ptr(out))
    return out


def sr_e4m3(t, r):
    """Stochastic rounding of values t to e4m3 with 16-bit random integers r (fp64 results)."""
    t = np.ascontiguousarray(t, dtype=np.float64)
    r = np.ascontiguousarray(np.broadcast_to(r, t.shape), dtype=np.uint32)
    y = np.empty_like(t)
    rc = lib().oracle_sr_e4m3(_ptr(t), _ptr(r), _ptr(y), t.size)
    if rc != 0:
        raise ValueError("random integers must lie in [0, 2^16)")
    return y


def logits8_sr(q, k, causal, window, row0, nrows, seed, nthreads=0):
    """e4m3 codes of the 8-bit logits with stochastic rounding, layout of logits8."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    out = np.empty((B, Hq, nrows, N), dtype=np.uint8)
    rc = lib().oracle_logits8_sr(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window),
                                 row0, nrows, int(seed), _ptr(out), nthreads)
    assert rc == 0
    return out


def logits16(q, k, causal, window, row0, nrows, nthreads=0):
    """e4m11 codes of the 16-bit logits, same layout; invisible entries hold 0xFFFF."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    out = np.empty((B, Hq, nrows, N), dtype=np.uint16)
    rc = lib().oracle_logits16(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window),
                               row0, nrows, _ptr(out), nthreads)
    assert rc == 0
    return out


def logits16_step(q, k, causal, window, row0, nrows, nthreads=0):
    """e4m11 codes of the 16-bit logits with e4m11 as the accumulator (rounded
    after every FMA), layout of logits16."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    out = np.empty((B, Hq, nrows, N), dtype=np.uint16)
    rc = lib().oracle_logits16_step(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window),
                                    row0, nrows, _ptr(out), nthreads)
    assert rc == 0
    return out


# ---------------------------------------------------------------- SIM profile
def round_sim(p, x):
    """Round doubles to p = 3 or 11 mantissa bits in FP32's exponent range (RNE, overflow to inf)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    assert lib().oracle_round_sim(p, _ptr(x), _ptr(y), x.size) == 0
    return y


def shift_sim(p, mu, y):
    """RN_p(max(0, mu - y)) of the exact difference."""
    mu = np.ascontiguousarray(mu, dtype=np.float64)
    y = np.ascontiguousarray(np.broadcast_to(y, mu.shape), dtype=np.float64)
    s = np.empty_like(mu)
    assert lib().oracle_shift_sim(p, _ptr(mu), _ptr(y), _ptr(s), mu.size) == 0
    return s


def sim_exp(p, s):
    """RN_p(exp(-s)), correctly rounded; raises if an enclosure cannot be certified."""
    s = np.ascontiguousarray(s, dtype=np.float64)
    e = np.empty_like(s)
    rc = lib().oracle_sim_exp(p, _ptr(s), _ptr(e), s.size)
    if rc != 0:
        raise RuntimeError("oracle_sim_exp: %d" % rc)
    return e


def trunc_sim3(x):
    return lib().oracle_trunc_sim3(float(x))


def logits_sim(q, k, causal, window, row0, nrows, high, nthreads=0):
    """SIM-profile logit values (high=0: 8-bit recursion, 1: 16-bit): [B,Hq,nrows,N], NaN = invisible."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    out = np.empty((B, Hq, nrows, N), dtype=np.float64)
    rc = lib().oracle_logits_sim(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window),
                                 row0, nrows, int(high), _ptr(out), nthreads)
    assert rc == 0
    return out


# ---------------------------------------------------------------- forward
STAGE1_OFF = 1   # the first stage disabled: mu_hat from the 8-bit maxima, stage 2 alone recomputes
MU_TRUNC = 2     # 8-bit shifts against mu_hat truncated to e4m3 (SIM: to 3 mantissa bits)
SIM = 4          # the "SIM" precision profile (FP32 range, 3/11-bit mantissas, no saturation)
SR8 = 8          # the 8-bit accumulation rounded stochastically (seeded Philox4x32-10 bits)
Y16_STEP = 16    # the 16-bit logits with e4m11 as the accumulator (rounded after every FMA; Sec. 3.3 literally)

STAT_NAMES = ("tiles", "stage1", "stage2", "inactive", "sat8", "sat16", "spec_unused", "late16")
STAT_HIST = len(STAT_NAMES)


def trunc_e4m3(x):
    return lib().oracle_trunc_e4m3(float(x))


def fwd(q, k, v, causal, window, bq, bk, nk, delta, tau, qblocks=None, nthreads=0, flags=0, seed=0,
        stats=False):
    """The LampAttention forward pass on the CPU.

    Returns (o [B,Hq,N,d] fp64, lse [B,Hq,N] fp64, mask [B,Hq,ceil(N/bq),
    ceil(N/(bk*nk))*nk] u8); N need not be a multiple of the block sizes.
    With `qblocks` (flat indices (b*Hq+h)*(N/bq)+qb) only those query blocks
    are computed; the other rows of o/lse hold NaN and their mask bytes 0xFE.
    `seed` keys the random numbers of flag 8 (stochastic rounding of the
    8-bit accumulation).  With `stats`, a fourth element: the statistics
    words (uint64 [8 + nk + 1], names STAT_NAMES then the histogram) of the
    computed query blocks.
    """
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    v = np.ascontiguousarray(v, dtype=np.uint16)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    o = np.full((B, Hq, N, d), np.nan, dtype=np.float64)
    lse = np.full((B, Hq, N), np.nan, dtype=np.float64)
    T = bk * nk
    mask = np.full((B, Hq, -(-N // bq), -(-N // T) * nk), 0xFE, dtype=np.uint8)
    if qblocks is not None:
        qbl = np.ascontiguousarray(qblocks, dtype=np.int64)
        qp, nq = _ptr(qbl), qbl.size
    else:
        qp, nq = None, 0
    st = np.zeros(STAT_HIST + nk + 1, dtype=np.uint64)
    rc = lib().lamp_oracle_fwd_ex(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, d, int(causal), int(window),
                                  bq, bk, nk, float(delta), float(tau), int(flags), int(seed),
                                  _ptr(o), _ptr(lse), _ptr(mask), qp, nq, nthreads, _ptr(st) if stats else None)
    if rc != 0:
        raise ValueError("lamp_oracle_fwd failed with %d" % rc)
    if stats:
        return o, lse, mask, st
    return o, lse, mask


def max_threads():
    return lib().oracle_max_threads()


def decode(q, k, v, causal, window, tk, delta, tau, rows=None, nthreads=0):
    """The vector-LAMP decode pass (Sec. 2, Eq. (6)) on the CPU.

    q [B,Hq,M,d]: M query rows at positions N-M .. N-1; k, v [B,Hkv,N,d].
    Returns (o [B,Hq,M,d] fp64, lse [B,Hq,M] fp64, mask [B,Hq,M,ceil(N/tk)*tk]
    u8 per key).  With `rows` (flat (b*Hq+h)*M+r) only those rows are computed
    (the others hold NaN and mask 0xFE)."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    v = np.ascontiguousarray(v, dtype=np.uint16)
    B, Hq, M, d = q.shape
    Hkv, N = k.shape[1], k.shape[2]
    o = np.full((B, Hq, M, d), np.nan, dtype=np.float64)
    lse = np.full((B, Hq, M), np.nan, dtype=np.float64)
    mask = np.full((B, Hq, M, -(-N // tk) * tk), 0xFE, dtype=np.uint8)
    if rows is not None:
        rl = np.ascontiguousarray(rows, dtype=np.int64)
        rp, nr = _ptr(rl), rl.size
    else:
        rp, nr = None, 0
    rc = lib().lamp_oracle_decode(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, M, N, d, int(causal), int(window), tk,
                                  float(delta), float(tau), 0, _ptr(o), _ptr(lse), _ptr(mask), rp, nr, nthreads)
    if rc != 0:
        raise ValueError("lamp_oracle_decode failed with %d" % rc)
    return o, lse, mask
