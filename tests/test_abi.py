"""The C-ABI library loads on the CPU and exports every function that
include/lamp.h declares (no compute calls: there is no GPU here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lamp.h")
LIB = os.path.join(ROOT, "paper_2609_39361_amd", "liblamp.so")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lamp_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("lamp_attn_fwd", "lamp_attn_logits8", "lamp_attn_logits16", "lamp_init", "lamp_shutdown",
              "lamp_status_str", "lamp_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings_without_gpu():
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    lib.lamp_status_str.restype = ctypes.c_char_p
    lib.lamp_status_str.argtypes = [ctypes.c_int]
    assert lib.lamp_status_str(0) == b"ok"
    assert lib.lamp_status_str(2) == b"unsupported configuration"


def test_binding_rejects_bad_arguments_without_gpu():
    """Host-side validation runs before any device call."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    lib.lamp_attn_fwd.restype = ctypes.c_int
    P = ctypes.c_void_p
    lib.lamp_attn_fwd.argtypes = [P, P, P] + [ctypes.c_int] * 10 + [ctypes.c_double] * 2 + [ctypes.c_uint] + [P, P, P, P, P]
    lib.lamp_last_error.restype = ctypes.c_char_p
    dummy = P(16)
    # Hq not a multiple of Hkv
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 3, 2, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 0,
                           dummy, dummy, dummy, None, None)
    assert rc == 1 and b"multiple" in lib.lamp_last_error()
    # unsupported head dimension
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 96, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 0,
                           dummy, dummy, dummy, None, None)
    assert rc == 2
    # window without causal
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 128, 0, 16, 128, 16, 4, 2 ** -8, 0.5, 0,
                           dummy, dummy, dummy, None, None)
    assert rc == 1
    # negative threshold
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, -1.0, 0,
                           dummy, dummy, dummy, None, None)
    assert rc == 1
    # unknown flag bits
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 32,
                           dummy, dummy, dummy, None, None)
    assert rc == 1 and b"flags" in lib.lamp_last_error()
    # the SIM profile is built for 16-key sub-blocks and d >= 128 only
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 128, 1, 0, 128, 64, 4, 2 ** -8, 0.5, 4,
                           dummy, dummy, dummy, None, None)
    assert rc == 2 and b"SIM" in lib.lamp_last_error()
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 64, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 4,
                           dummy, dummy, dummy, None, None)
    assert rc == 2 and b"SIM" in lib.lamp_last_error()
    # block sizes that are not built
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 128, 1, 0, 32, 16, 4, 2 ** -8, 0.5, 0,
                           dummy, dummy, dummy, None, None)
    assert rc == 2 and b"not built" in lib.lamp_last_error()
    rc = lib.lamp_attn_fwd(dummy, dummy, dummy, 1, 2, 1, 256, 128, 1, 0, 128, 32, 4, 2 ** -8, 0.5, 0,
                           dummy, dummy, dummy, None, None)
    assert rc == 2


def test_decode_rejects_bad_arguments_without_gpu():
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    lib.lamp_attn_decode.restype = ctypes.c_int
    lib.lamp_attn_decode.argtypes = [P, P, P] + [ctypes.c_int] * 9 + [ctypes.c_double] * 2 + [ctypes.c_uint] + [P] * 5
    lib.lamp_last_error.restype = ctypes.c_char_p
    d = P(16)
    # (B, Hq, Hkv, M, N, d, causal, window, tk)
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 128, 1, 0, 32, 2 ** -8, 0.5, 0, d, d, d, None, None) == 2
    assert b"tk" in lib.lamp_last_error()
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 128, 1, 0, 64, 2 ** -8, 0.5, 4, d, d, d, None, None) == 1
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 300, 256, 128, 1, 0, 64, 2 ** -8, 0.5, 0, d, d, d, None, None) == 1
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 96, 1, 0, 64, 2 ** -8, 0.5, 0, d, d, d, None, None) == 2
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 128, 1, 0, 64, 2 ** -8, -1.0, 0, d, d, d, None, None) == 1
    # flag bits other than LAMP_DECODE_SERIAL
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 128, 1, 0, 64, 2 ** -8, 0.5, 512, d, d, d, None, None) == 1
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 128, 1, 0, 64, 2 ** -8, 0.5, 257, d, d, d, None, None) == 1


def test_timing_read_without_calls():
    """Timing bookkeeping is host-only: nothing recorded reads as zero."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    from paper_2609_39361_amd import lamp
    lamp.timing_enable(True)
    lamp.timing_enable(False)
    assert lamp.timing_read() == (0, 0.0, 0.0)


def test_issue_rates_rejects_null_without_gpu():
    """lamp_issue_rates validates its output pointer before any device call."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    lib.lamp_issue_rates.restype = ctypes.c_int
    lib.lamp_issue_rates.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.lamp_last_error.restype = ctypes.c_char_p
    assert lib.lamp_issue_rates(None, None) == 1
    assert b"null" in lib.lamp_last_error()


def test_fwd_sr_rejects_bad_arguments_without_gpu():
    """lamp_attn_fwd_sr checks its arguments before any device call: unknown
    flags, the SIM profile (not built with stochastic rounding), block sizes."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    lib.lamp_attn_fwd_sr.restype = ctypes.c_int
    lib.lamp_attn_fwd_sr.argtypes = ([P, P, P] + [ctypes.c_int] * 10 + [ctypes.c_double] * 2 + [ctypes.c_uint]
                                     + [ctypes.c_uint64] + [P, P, P, P, P])
    lib.lamp_last_error.restype = ctypes.c_char_p
    d = ctypes.c_void_p(16)
    args = (d, d, d, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5)
    assert lib.lamp_attn_fwd_sr(*args, 32, 1, d, d, d, None, None) == 1
    assert lib.lamp_attn_fwd_sr(*args, 4, 1, d, d, d, None, None) == 2
    assert b"SIM" in lib.lamp_last_error()
    assert lib.lamp_attn_fwd_sr(d, d, d, 1, 2, 1, 256, 128, 1, 0, 128, 32, 4, 2 ** -8, 0.5, 0, 2 ** 64 - 1,
                                d, d, d, None, None) == 2


def test_length_limits_without_gpu():
    """N above 2^20, or B*Hq*N above 2^31, is LAMP_ERR_UNSUPPORTED before any
    device call; N = 2^20 itself passes the argument checks (the GPU tests run
    it)."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    lib.lamp_attn_fwd.restype = ctypes.c_int
    lib.lamp_attn_fwd.argtypes = [P, P, P] + [ctypes.c_int] * 10 + [ctypes.c_double] * 2 + [ctypes.c_uint] + [P, P, P, P, P]
    lib.lamp_last_error.restype = ctypes.c_char_p
    d = ctypes.c_void_p(16)
    assert lib.lamp_attn_fwd(d, d, d, 1, 1, 1, (1 << 20) + 1, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 0,
                             d, d, d, None, None) == 2
    assert b"2^20" in lib.lamp_last_error()
    assert lib.lamp_attn_fwd(d, d, d, 4096, 1024, 1, 1 << 20, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 0,
                             d, d, d, None, None) == 2
    assert b"2^31" in lib.lamp_last_error()


class _Extra(ctypes.Structure):
    _fields_ = [("stats", ctypes.c_void_p), ("dbg_y8", ctypes.c_void_p), ("dbg_y16", ctypes.c_void_p),
                ("dbg_qb0", ctypes.c_int), ("dbg_nqb", ctypes.c_int), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t)]


def test_extra_arguments_checked_without_gpu():
    """The optional arguments are validated before any device call: observed
    query blocks outside the range, observables with the SIM profile, and
    statistics or observables asked of the decode form."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    lib.lamp_attn_fwd.restype = ctypes.c_int
    lib.lamp_attn_fwd.argtypes = [P, P, P] + [ctypes.c_int] * 10 + [ctypes.c_double] * 2 + [ctypes.c_uint] + [P] * 5
    lib.lamp_attn_decode.restype = ctypes.c_int
    lib.lamp_attn_decode.argtypes = [P, P, P] + [ctypes.c_int] * 9 + [ctypes.c_double] * 2 + [ctypes.c_uint] + [P] * 5
    lib.lamp_last_error.restype = ctypes.c_char_p
    d = ctypes.c_void_p(16)
    e = _Extra()
    e.dbg_y8 = 16
    e.dbg_qb0, e.dbg_nqb = 1, 2          # N = 256, bq = 128: two query blocks, [1, 3) is outside
    assert lib.lamp_attn_fwd(d, d, d, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 0, d, d, d,
                             ctypes.byref(e), None) == 1
    assert b"observed" in lib.lamp_last_error()
    e.dbg_qb0, e.dbg_nqb = 0, 2
    assert lib.lamp_attn_fwd(d, d, d, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 4, d, d, d,
                             ctypes.byref(e), None) == 2
    e2 = _Extra()
    e2.stats = 16
    assert lib.lamp_attn_decode(d, d, d, 1, 4, 1, 1, 256, 128, 1, 0, 64, 2 ** -8, 0.5, 0, d, d, d,
                                ctypes.byref(e2), None) == 2
    # unknown flag bits beyond LAMP_COMPACT
    assert lib.lamp_attn_fwd(d, d, d, 1, 2, 1, 256, 128, 1, 0, 128, 16, 4, 2 ** -8, 0.5, 32, d, d, d,
                             None, None) == 1


def test_workspace_sizes_without_gpu():
    """Workspace sizes: a 256-byte header, the pre-scaled queries and the fp32
    keys of whole blocks and tiles, and V transposed (config 3: 176 MiB)."""
    if not os.path.exists(LIB):
        pytest.skip("liblamp.so not built")
    lib = ctypes.CDLL(LIB)
    lib.lamp_attn_fwd_workspace_size.restype = ctypes.c_size_t
    lib.lamp_attn_fwd_workspace_size.argtypes = [ctypes.c_int] * 8
    lib.lamp_attn_decode_workspace_size.restype = ctypes.c_size_t
    lib.lamp_attn_decode_workspace_size.argtypes = [ctypes.c_int] * 6
    n = lib.lamp_attn_fwd_workspace_size(1, 32, 8, 8192, 128, 128, 16, 4)
    assert n == 256 + 32 * 8192 * 128 * 4 + 8 * 8192 * 128 * 4 + 8 * 8192 * 128 * 2
    # ragged N: rows padded to whole query blocks, keys to whole tiles, each part 256-aligned
    def a256(x):
        return (x + 255) // 256 * 256
    assert lib.lamp_attn_fwd_workspace_size(1, 2, 1, 300, 128, 128, 16, 4) == \
        256 + a256(2 * 384 * 128 * 4) + a256(320 * 128 * 4) + a256(320 * 128 * 2)
    assert lib.lamp_attn_fwd_workspace_size(0, 2, 1, 300, 128, 128, 16, 4) == 0
    assert lib.lamp_attn_fwd_workspace_size(1, 2, 1, 300, 128, -1, 16, 4) == 0
    assert lib.lamp_attn_decode_workspace_size(32, 32, 8, 1, 8192, 128) > 0
    assert lib.lamp_attn_decode_workspace_size(1, 4, 1, 5, 4, 128) == 0    # M > N
    # sizes and block sizes the passes refuse need no workspace (and overflow nothing)
    assert lib.lamp_attn_fwd_workspace_size(1, 2, 1, 300, 128, 2 ** 31 - 1, 2 ** 31 - 1, 2 ** 31 - 1) == 0
    assert lib.lamp_attn_fwd_workspace_size(1, 2, 1, 300, 96, 128, 16, 4) == 0
    assert lib.lamp_attn_fwd_workspace_size(1, 1, 1, (1 << 20) + 1, 128, 128, 16, 4) == 0
    assert lib.lamp_attn_fwd_workspace_size(2 ** 31 - 1, 2 ** 31 - 1, 1, 1 << 20, 128, 128, 16, 4) == 0
    assert lib.lamp_attn_decode_workspace_size(1, 4, 1, 1, 2 ** 31 - 1, 128) == 0
    lib.lamp_status_str.restype = ctypes.c_char_p
    lib.lamp_status_str.argtypes = [ctypes.c_int]
    assert lib.lamp_status_str(5) == b"non-finite input"
    assert lib.lamp_status_str(6) == b"workspace too small"
