"""Pins of the oracle's exponential tables (paper Sec. 3.3: 8-bit LUT exp; Sec.
4.1: exponentials correctly rounded) and of exp_doc, the documented fp64
exponential of the rescale factor (Sec. 2.2: alpha_hat in high precision)."""

import mpmath as mp
import numpy as np
import pytest

from oracle import oracle as O
import fpmodel as M


@pytest.fixture(scope="session")
def mp_tables():
    return M.mp_exp_tables()


def test_lut8_every_entry_vs_mpmath(mp_tables):
    lut8, _ = O.tables()
    assert np.array_equal(lut8, mp_tables[0])
    assert lut8[0] == 0b11111000            # exp(-0) = 1.0
    assert np.all(np.diff(lut8.astype(int)) <= 0)   # exp(-s) is non-increasing


def test_exp16_every_entry_vs_mpmath(mp_tables):
    _, exp16 = O.tables()
    assert np.array_equal(exp16, mp_tables[1])
    assert exp16[0] == 0b11111 << 11
    assert np.all(np.diff(exp16.astype(int)) <= 0)


def test_exp_doc_constants_are_correctly_rounded():
    mp.mp.prec = 200
    c = O.exp_doc_constants()
    ln2 = mp.log(2)
    assert c[0] == float(1 / ln2)                        # LOG2E = RN64(1/ln 2)
    hi = mp.floor(ln2 * 2 ** 32) / 2 ** 32               # ln 2 truncated to 32 bits
    assert c[1] == float(hi) and mp.mpf(c[1]) == hi
    assert c[2] == float(ln2 - hi)                       # LN2_LO
    for k in range(14):
        assert c[3 + k] == float(1 / mp.factorial(k)), k


def test_exp_doc_accuracy_and_special_values():
    mp.mp.prec = 120
    rng = np.random.default_rng(0)
    x = np.concatenate([-rng.uniform(0, 700, 20000), -rng.uniform(0, 1, 5000),
                        -np.ldexp(1.0, -rng.integers(1, 60, 2000)), [0.0, -700.0]])
    y = O.exp_doc(x)
    ref = np.array([float(mp.exp(mp.mpf(v))) for v in x])
    ulp = np.spacing(ref)
    err = np.abs(y - ref) / ulp
    assert err.max() <= 2.0, err.max()
    assert O.exp_doc(np.array([0.0]))[0] == 1.0
    assert O.exp_doc(np.array([-700.5, -1e300]))[0] == 0.0
    assert np.all(np.diff(O.exp_doc(np.linspace(-50, 0, 10001))) >= 0)


def test_scale_constants():
    """s = RN32(1/sqrt(d)): exact powers of two for d = 64, 256; 0x3DB504F3 for 128."""
    import struct
    assert O.scale(64) == 0.125 and O.scale(256) == 0.0625
    assert struct.pack(">f", O.scale(128)).hex() == "3db504f3"
    mp.mp.prec = 100
    for d in (16, 32, 64, 96, 128, 160, 192, 256):
        exact = 1 / mp.sqrt(d)
        s = O.scale(d)
        # correctly rounded to fp32: |s - exact| <= half an fp32 ulp
        assert abs(mp.mpf(s) - exact) <= mp.mpf(float(np.spacing(np.float32(s)))) / 2
