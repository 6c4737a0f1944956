"""Python binding of liblamp.so (the C ABI declared in include/lamp.h).

Argument marshalling only: every step of the forward pass runs in the HIP
kernels of the library.  PyTorch provides device memory and the stream.  The
library must have been built (python -m paper_2609_39361_amd.build); there is
no fallback path.
"""
import ctypes
import math
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# LAMP_LIBRARY may name the measurement build liblamp_phase.so (phase timer)
LIB_PATH = os.environ.get("LAMP_LIBRARY") or os.path.join(HERE, "liblamp.so")

LAMP_OK = 0
LAMP_ERR_NONFINITE_INPUT = 5
LAMP_ERR_WORKSPACE = 6
MASK_LOW, MASK_STAGE1, MASK_STAGE2, MASK_INACTIVE = 0, 1, 2, 3

# statistics words (include/lamp.h, LAMP_STAT_*)
STAT_NAMES = ("tiles", "stage1", "stage2", "inactive", "sat8", "sat16", "spec_unused", "late16")
STAT_HIST = len(STAT_NAMES)


def stats_words(nk):
    """Number of uint64 statistics words for nk sub-blocks per tile."""
    return STAT_HIST + nk + 1


class FwdExtra(ctypes.Structure):
    """struct lamp_fwd_extra (include/lamp.h)."""
    _fields_ = [("stats", ctypes.c_void_p), ("dbg_y8", ctypes.c_void_p), ("dbg_y16", ctypes.c_void_p),
                ("dbg_qb0", ctypes.c_int), ("dbg_nqb", ctypes.c_int), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t)]


class LampError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("lamp status %d: %s" % (status, msg))
        self.status = status


_lib = None


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("liblamp.so is not built; run `python -m paper_2609_39361_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, f64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_double, ctypes.c_size_t
        L.lamp_attn_fwd.argtypes = [P, P, P] + [i32] * 5 + [i32] * 5 + [f64, f64, ctypes.c_uint, P, P, P, P, P]
        L.lamp_attn_fwd.restype = i32
        L.lamp_attn_logits8.argtypes = [P, P] + [i32] * 9 + [P, P]
        L.lamp_attn_logits8.restype = i32
        L.lamp_attn_fwd_sr.argtypes = ([P, P, P] + [i32] * 5 + [i32] * 5 + [f64, f64, ctypes.c_uint, ctypes.c_uint64]
                                       + [P, P, P, P, P])
        L.lamp_attn_fwd_sr.restype = i32
        L.lamp_attn_fwd_noalloc.argtypes = [P, P, P] + [i32] * 5 + [i32] * 5 + [f64, f64, ctypes.c_uint, P, P, P, P, P]
        L.lamp_attn_fwd_noalloc.restype = i32
        L.lamp_attn_logits8_sr.argtypes = [P, P] + [i32] * 9 + [ctypes.c_uint64, P, P]
        L.lamp_attn_logits8_sr.restype = i32
        L.lamp_attn_logits16.argtypes = [P, P] + [i32] * 9 + [P, P]
        L.lamp_attn_logits16.restype = i32
        L.lamp_attn_decode.argtypes = [P, P, P] + [i32] * 9 + [f64, f64, ctypes.c_uint, P, P, P, P, P]
        L.lamp_attn_decode.restype = i32
        L.lamp_attn_logits_sim.argtypes = [P, P] + [i32] * 10 + [P, P]
        L.lamp_attn_logits_sim.restype = i32
        L.lamp_get_sim_tables.argtypes = [i32, P, P]
        L.lamp_get_sim_tables.restype = i32
        L.lamp_attn_fwd_workspace_size.argtypes = [i32] * 8
        L.lamp_attn_fwd_workspace_size.restype = sz
        L.lamp_attn_decode_workspace_size.argtypes = [i32] * 6
        L.lamp_attn_decode_workspace_size.restype = sz
        L.lamp_reserve.argtypes = [i32, sz]
        L.lamp_reserve.restype = i32
        L.lamp_init.argtypes = [i32]
        L.lamp_init.restype = i32
        L.lamp_shutdown.argtypes = []
        L.lamp_shutdown.restype = None
        L.lamp_selftest_e4m3.argtypes = [P, P, P, sz, P]
        L.lamp_selftest_e4m3.restype = i32
        L.lamp_selftest_exp_doc.argtypes = [P, P, sz, P]
        L.lamp_selftest_exp_doc.restype = i32
        L.lamp_get_tables.argtypes = [i32, P, P]
        L.lamp_get_tables.restype = i32
        L.lamp_get_exp16_parts.argtypes = [i32, P]
        L.lamp_get_exp16_parts.restype = i32
        L.lamp_issue_rates.argtypes = [P, P]
        L.lamp_issue_rates.restype = i32
        L.lamp_phase_read.argtypes = [P, i32]
        L.lamp_phase_read.restype = i32
        L.lamp_timing_enable.argtypes = [i32]
        L.lamp_timing_enable.restype = i32
        L.lamp_timing_read.argtypes = [P, P, P]
        L.lamp_timing_read.restype = i32
        L.lamp_status_str.argtypes = [i32]
        L.lamp_status_str.restype = ctypes.c_char_p
        L.lamp_last_error.argtypes = []
        L.lamp_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc):
    if rc != LAMP_OK:
        L = lib()
        raise LampError(rc, "%s: %s" % (L.lamp_status_str(rc).decode(), L.lamp_last_error().decode()))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check_inputs(q, k, v=None):
    for t in (q, k) + ((v,) if v is not None else ()):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
            raise ValueError("q, k, v must be contiguous 4-d bf16 CUDA tensors [B,H,N,d]")
    B, Hq, N, d = q.shape
    if k.shape[0] != B or k.shape[2] != N or k.shape[3] != d:
        raise ValueError("k shape %s does not match q %s" % (tuple(k.shape), tuple(q.shape)))
    if v is not None and v.shape != k.shape:
        raise ValueError("v shape %s differs from k %s" % (tuple(v.shape), tuple(k.shape)))
    if q.device != k.device or (v is not None and v.device != q.device):
        raise ValueError("q, k, v must be on one device")
    return B, Hq, k.shape[1], N, d


STAGE1_OFF = 1   # the first stage disabled: mu_hat from the 8-bit maxima, stage 2 alone recomputes
MU_TRUNC = 2     # 8-bit shifts against mu_hat truncated to e4m3 (SIM profile: to 3 mantissa bits)
SIM_PROFILE = 4  # the SIM precision profile (FP32 range, 3 / 11 mantissa bits, no saturation)
CHECK_FINITE = 8  # check q, k, v for NaN / infinity first (synchronous; LAMP_ERR_NONFINITE_INPUT)
COMPACT = 16     # the compact register layout of Sec. 3.3 as the kernel's schedule (same results)
# attn_decode flag: one key chunk and the passes one after another instead of the key-chunk
# pipeline (same masks and lse; O equal up to the order of its final sums)
DECODE_SERIAL = 256


def _check_out(t, name, shape, dtype, device):
    if (not isinstance(t, torch.Tensor) or tuple(t.shape) != tuple(shape) or t.dtype != dtype
            or t.device != device or not t.is_contiguous()):
        raise ValueError("%s must be a contiguous %s tensor of shape %s on %s" % (name, dtype, tuple(shape), device))


def _extra(stats=None, observe=None, workspace=None, device=None, nk=4):
    """(FwdExtra or None, tensors kept alive) from the optional arguments."""
    if stats is None and observe is None and workspace is None:
        return None, ()
    e = FwdExtra()
    keep = []
    if stats is not None:
        _check_out(stats, "stats", (stats_words(nk),), torch.int64, device)
        e.stats = stats.data_ptr()
        keep.append(stats)
    if observe is not None:
        qb0, nqb, y8, y16 = observe
        e.dbg_qb0, e.dbg_nqb = int(qb0), int(nqb)
        for t in (y8, y16):
            if t is not None:
                if not t.is_contiguous() or t.device != device:
                    raise ValueError("observable arrays must be contiguous tensors on the inputs' device")
                keep.append(t)
        e.dbg_y8 = y8.data_ptr() if y8 is not None else None
        e.dbg_y16 = y16.data_ptr() if y16 is not None else None
    if workspace is not None:
        if workspace.device != device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on the inputs' device")
        e.workspace = workspace.data_ptr()
        e.workspace_bytes = workspace.numel() * workspace.element_size()
        keep.append(workspace)
    return e, tuple(keep)


def attn_fwd(q, k, v, causal=True, window=0, bq=128, bk=16, nk=4, delta=2.0 ** -8, tau=0.5, out=None, flags=0,
             sr_seed=None, stats=None, observe=None, workspace=None):
    """LampAttention forward pass.  Returns (o fp32 [B,Hq,N,d], lse fp32
    [B,Hq,N], mask uint8 [B,Hq,ceil(N/bq),ceil(N/(bk*nk))*nk]); N need not be
    a multiple of the block sizes.  `out` may supply those three tensors to
    write into; `flags` selects the variants STAGE1_OFF, MU_TRUNC, the
    SIM_PROFILE numerics and the CHECK_FINITE input check.  With `sr_seed` (an
    int below 2^64) the 8-bit accumulation is rounded stochastically with that
    seed (lamp_attn_fwd_sr).

    Optional (struct lamp_fwd_extra): `stats`, an int64 tensor of
    stats_words(nk) elements on the device that the call adds the statistics
    words to; `observe` = (qb0, nqb, y8, y16), the forward kernel's 8-bit and
    16-bit logit codes of query blocks [qb0, qb0+nqb) (see observe_logits);
    `workspace`, a device tensor of at least fwd_workspace_size(...) bytes."""
    B, Hq, Hkv, N, d = _check_inputs(q, k, v)
    dev = q.device
    mshape = (B, Hq, -(-N // bq), -(-N // (bk * nk)) * nk)
    if out is None:
        o = torch.empty((B, Hq, N, d), dtype=torch.float32, device=dev)
        lse = torch.empty((B, Hq, N), dtype=torch.float32, device=dev)
        mask = torch.empty(mshape, dtype=torch.uint8, device=dev)
    else:
        o, lse, mask = out
        _check_out(o, "o", (B, Hq, N, d), torch.float32, dev)
        _check_out(lse, "lse", (B, Hq, N), torch.float32, dev)
        _check_out(mask, "mask", mshape, torch.uint8, dev)
    extra, keep = _extra(stats, observe, workspace, dev, nk)
    ep = ctypes.byref(extra) if extra is not None else None
    with torch.cuda.device(dev):
        if sr_seed is None:
            rc = lib().lamp_attn_fwd(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, d, int(causal), int(window),
                                     bq, bk, nk, float(delta), float(tau), int(flags), _ptr(o), _ptr(lse), _ptr(mask),
                                     ep, _stream(dev))
        else:
            rc = lib().lamp_attn_fwd_sr(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, d, int(causal), int(window),
                                        bq, bk, nk, float(delta), float(tau), int(flags), int(sr_seed),
                                        _ptr(o), _ptr(lse), _ptr(mask), ep, _stream(dev))
    del keep
    _check(rc)
    return o, lse, mask


NOALLOC_SCRATCH_BYTES = 256 << 20


def attn_fwd_noalloc(q, k, v, out, causal=True, window=0, bq=128, bk=16, nk=4, delta=2.0 ** -8, tau=0.5, flags=0,
                     stats=None):
    """attn_fwd through lamp_attn_fwd_noalloc: the library allocates nothing
    (its workspace is the device's fixed scratch of NOALLOC_SCRATCH_BYTES;
    init(device) must have been called).  `out` = (o, lse, mask) as for
    attn_fwd is required, so that nothing is allocated here either."""
    B, Hq, Hkv, N, d = _check_inputs(q, k, v)
    dev = q.device
    o, lse, mask = out
    _check_out(o, "o", (B, Hq, N, d), torch.float32, dev)
    _check_out(lse, "lse", (B, Hq, N), torch.float32, dev)
    _check_out(mask, "mask", (B, Hq, -(-N // bq), -(-N // (bk * nk)) * nk), torch.uint8, dev)
    extra, keep = _extra(stats=stats, device=dev, nk=nk)
    ep = ctypes.byref(extra) if extra is not None else None
    with torch.cuda.device(dev):
        rc = lib().lamp_attn_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, d, int(causal), int(window),
                                         bq, bk, nk, float(delta), float(tau), int(flags), _ptr(o), _ptr(lse),
                                         _ptr(mask), ep, _stream(dev))
    del keep
    _check(rc)
    return o, lse, mask


def observe_logits(q, k, v, qb0, nqb, causal=True, window=0, bq=128, bk=16, nk=4, delta=2.0 ** -8, tau=0.5,
                   flags=0, sr_seed=None, stats=None):
    """attn_fwd that also returns the forward kernel's own logit codes of the
    query blocks [qb0, qb0+nqb) of every (b, h): (o, lse, mask, y8, y16),
    y8 uint8 [B,Hq,nqb*bq,Nt] (e4m3 codes of visible pairs, 0xFF elsewhere)
    and y16 int16 bit patterns [B,Hq,nqb*bq,Nt] (e4m11 codes of visible pairs
    in 16-bit sub-blocks, 0xFFFF elsewhere), Nt = ceil(N/(bk*nk))*bk*nk."""
    B, Hq, Hkv, N, d = _check_inputs(q, k, v)
    Nt = -(-N // (bk * nk)) * bk * nk
    y8 = torch.empty((B, Hq, nqb * bq, Nt), dtype=torch.uint8, device=q.device)
    y16 = torch.empty((B, Hq, nqb * bq, Nt), dtype=torch.int16, device=q.device)
    o, lse, mask = attn_fwd(q, k, v, causal, window, bq, bk, nk, delta, tau, flags=flags, sr_seed=sr_seed,
                            stats=stats, observe=(qb0, nqb, y8, y16))
    return o, lse, mask, y8, y16


def fwd_workspace_size(B, Hq, Hkv, N, d, bq=128, bk=16, nk=4):
    """Bytes of workspace one attn_fwd call needs."""
    return int(lib().lamp_attn_fwd_workspace_size(B, Hq, Hkv, N, d, bq, bk, nk))


def decode_workspace_size(B, Hq, Hkv, M, N, d):
    return int(lib().lamp_attn_decode_workspace_size(B, Hq, Hkv, M, N, d))


def reserve(device, nbytes):
    """Grow the library's workspace of `device` to nbytes now (synchronous)."""
    _check(lib().lamp_reserve(int(device), int(nbytes)))


def stats_dict(stats, nk=4):
    """The statistics words as a dict (names of STAT_NAMES, 'hist' a list)."""
    w = [int(x) for x in stats.cpu().tolist()]
    r = dict(zip(STAT_NAMES, w[:STAT_HIST]))
    r["hist"] = w[STAT_HIST:STAT_HIST + nk + 1]
    return r


def attn_decode(q, k, v, causal=True, window=0, tk=64, delta=2.0 ** -8, tau=0.5, out=None, flags=0,
                workspace=None):
    """LampAttention in the vector form (Sec. 2, Eq. (6)) for M query rows per
    (b, h) at positions N-M .. N-1: q [B,Hq,M,d], k / v [B,Hkv,N,d] bf16.
    Returns (o fp32 [B,Hq,M,d], lse fp32 [B,Hq,M], mask uint8
    [B,Hq,M,ceil(N/tk)*tk] one code per key)."""
    if q.dim() != 4 or k.dim() != 4 or v.shape != k.shape:
        raise ValueError("q [B,Hq,M,d], k and v [B,Hkv,N,d] expected")
    B, Hq, M, d = q.shape
    Hkv, N = k.shape[1], k.shape[2]
    for t in (q, k, v):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous bf16 CUDA tensors")
    dev = q.device
    if q.device != k.device or v.device != k.device:
        raise ValueError("q, k, v must be on one device")
    mshape = (B, Hq, M, -(-N // tk) * tk)
    if out is None:
        o = torch.empty((B, Hq, M, d), dtype=torch.float32, device=dev)
        lse = torch.empty((B, Hq, M), dtype=torch.float32, device=dev)
        mask = torch.empty(mshape, dtype=torch.uint8, device=dev)
    else:
        o, lse, mask = out
        _check_out(o, "o", (B, Hq, M, d), torch.float32, dev)
        _check_out(lse, "lse", (B, Hq, M), torch.float32, dev)
        _check_out(mask, "mask", mshape, torch.uint8, dev)
    extra, keep = _extra(workspace=workspace, device=dev)
    ep = ctypes.byref(extra) if extra is not None else None
    with torch.cuda.device(dev):
        rc = lib().lamp_attn_decode(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, M, N, d, int(causal), int(window), tk,
                                    float(delta), float(tau), int(flags), _ptr(o), _ptr(lse), _ptr(mask),
                                    ep, _stream(dev))
    del keep
    _check(rc)
    return o, lse, mask


def logits8(q, k, causal=True, window=0, row0=0, nrows=None, sr_seed=None):
    """e4m3 codes of the 8-bit logits of rows [row0, row0+nrows): uint8 [B,Hq,nrows,N], 0xFF invisible;
    with `sr_seed`, stochastically rounded (lamp_attn_logits8_sr)."""
    B, Hq, Hkv, N, d = _check_inputs(q, k)
    nrows = N - row0 if nrows is None else nrows
    y = torch.empty((B, Hq, nrows, N), dtype=torch.uint8, device=q.device)
    with torch.cuda.device(q.device):
        if sr_seed is None:
            rc = lib().lamp_attn_logits8(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window), row0, nrows,
                                         _ptr(y), _stream(q.device))
        else:
            rc = lib().lamp_attn_logits8_sr(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window), row0,
                                            nrows, int(sr_seed), _ptr(y), _stream(q.device))
    _check(rc)
    return y


def logits16(q, k, causal=True, window=0, row0=0, nrows=None):
    """e4m11 codes of the 16-bit logits: int16 bit patterns [B,Hq,nrows,N] (0xFFFF invisible)."""
    B, Hq, Hkv, N, d = _check_inputs(q, k)
    nrows = N - row0 if nrows is None else nrows
    y = torch.empty((B, Hq, nrows, N), dtype=torch.int16, device=q.device)
    with torch.cuda.device(q.device):
        rc = lib().lamp_attn_logits16(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window), row0, nrows,
                                      _ptr(y), _stream(q.device))
    _check(rc)
    return y


def logits_sim(q, k, high, causal=True, window=0, row0=0, nrows=None):
    """SIM-profile logit values (high=False: 8-bit recursion, True: 16-bit):
    fp32 [B,Hq,nrows,N], NaN invisible."""
    B, Hq, Hkv, N, d = _check_inputs(q, k)
    nrows = N - row0 if nrows is None else nrows
    y = torch.empty((B, Hq, nrows, N), dtype=torch.float32, device=q.device)
    with torch.cuda.device(q.device):
        rc = lib().lamp_attn_logits_sim(_ptr(q), _ptr(k), B, Hq, Hkv, N, d, int(causal), int(window), row0, nrows,
                                        int(bool(high)), _ptr(y), _stream(q.device))
    _check(rc)
    return y


def selftest_e4m3(x):
    """(codes, raw codes) of fp32 CUDA tensor x by the device rounding sequence."""
    assert x.dtype == torch.float32 and x.is_cuda and x.is_contiguous()
    out = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    raw = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    with torch.cuda.device(x.device):
        _check(lib().lamp_selftest_e4m3(_ptr(x), _ptr(out), _ptr(raw), x.numel(), _stream(x.device)))
    return out, raw


def selftest_exp_doc(x):
    assert x.dtype == torch.float64 and x.is_cuda and x.is_contiguous()
    y = torch.empty_like(x)
    with torch.cuda.device(x.device):
        _check(lib().lamp_selftest_exp_doc(_ptr(x), _ptr(y), x.numel(), _stream(x.device)))
    return y


def get_tables(device=0):
    """(lut8 uint8[256], exp16 uint16[65536]) numpy copies of the device tables."""
    import numpy as np
    lut8 = np.empty(256, dtype=np.uint8)
    exp16 = np.empty(65536, dtype=np.uint16)
    _check(lib().lamp_get_tables(int(device), lut8.ctypes.data_as(ctypes.c_void_p),
                                 exp16.ctypes.data_as(ctypes.c_void_p)))
    return lut8, exp16


def get_exp16_parts(device=0):
    """uint32[65536]: the 16-bit exponentials as bf16 high (bits 15:0) and low
    (bits 31:16) parts."""
    import numpy as np
    parts = np.zeros(65536, dtype=np.uint32)
    _check(lib().lamp_get_exp16_parts(int(device), parts.ctypes.data_as(ctypes.c_void_p)))
    return parts


def get_sim_tables(device=0):
    """(sim8 uint16[112] bf16 bits, sim16 uint32[45056] FP32 patterns): the
    SIM profile's exponential tables, entry ((e - emin) << p) | m for the shift
    (2^p + m) 2^(e - p); p = 3, e in [-6, 7] and p = 11, e in [-14, 7]."""
    import numpy as np
    sim8 = np.zeros(112, dtype=np.uint16)
    sim16 = np.zeros(45056, dtype=np.uint32)
    _check(lib().lamp_get_sim_tables(int(device), sim8.ctypes.data_as(ctypes.c_void_p),
                                     sim16.ctypes.data_as(ctypes.c_void_p)))
    return sim8, sim16


def init(device=0):
    _check(lib().lamp_init(int(device)))


def shutdown():
    lib().lamp_shutdown()


def timing_enable(on=True):
    """Record HIP events around the prepass and forward kernel of each
    attn_fwd call (on the call's stream) until disabled."""
    _check(lib().lamp_timing_enable(1 if on else 0))


def timing_read():
    """(calls, forward-kernel ms summed, prepass ms summed) of the calls
    recorded since the previous read; waits for their events."""
    n, tf, tp = ctypes.c_int(0), ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(lib().lamp_timing_read(ctypes.byref(n), ctypes.byref(tf), ctypes.byref(tp)))
    return n.value, tf.value, tp.value


PHASE_NAMES = ("fused_pass", "emission", "barrier_B", "stage1", "exponentials", "barrier_E", "rescale_stage2",
               "pv_next_F0", "barrier_I", "prologue_epilogue")


def phase_read(reset=True):
    """Cycle sums per phase of the pipelined kernel and the wave count (a
    library built with the phase timer only; LampError otherwise)."""
    h = (ctypes.c_uint64 * (len(PHASE_NAMES) + 1))()
    _check(lib().lamp_phase_read(h, 1 if reset else 0))
    v = list(h)
    return dict(zip(PHASE_NAMES, v[:-1])), v[-1]


ISSUE_RATE_KINDS = ("fmac_f32", "fmac_f32_dpp", "cvt_pk_f32_fp8", "cvt_pk_fp8_f32", "emulated_step",
                    "emulated_step_sim")


def issue_rates():
    """Nanoseconds per wave-instruction per SIMD of the logit loops'
    instructions on the current device (dict keyed by ISSUE_RATE_KINDS;
    emulated_step is one step of the 8-bit loop, two multiply-adds per lane,
    emulated_step_sim one of the SIM profile's, one multiply-add)."""
    ns = (ctypes.c_double * len(ISSUE_RATE_KINDS))()
    _check(lib().lamp_issue_rates(ns, _stream(torch.device("cuda", torch.cuda.current_device()))))
    return dict(zip(ISSUE_RATE_KINDS, list(ns)))


def mask_stats(mask, nk):
    """Recompute statistics from a mask [B,Hq,nqb,ntiles*nk]: per key tile (nk
    sub-blocks, at least one active) the number of 16-bit sub-blocks, as a
    histogram 0..nk, plus counts per code.  Reporting only."""
    m = mask.reshape(-1, nk)
    active = (m != MASK_INACTIVE)
    tiles = active.any(dim=1)
    rec = ((m == MASK_STAGE1) | (m == MASK_STAGE2)).sum(dim=1)[tiles]
    hist = torch.bincount(rec.to(torch.int64), minlength=nk + 1).cpu().tolist()
    counts = torch.bincount(mask.reshape(-1).to(torch.int64), minlength=4).cpu().tolist()
    n_active = counts[0] + counts[1] + counts[2]
    return {
        "tile_hist": hist,
        "low": counts[0], "stage1": counts[1], "stage2": counts[2], "inactive": counts[3],
        "recompute_fraction": (counts[1] + counts[2]) / n_active if n_active else math.nan,
    }
