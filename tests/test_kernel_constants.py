"""The numeric constants that the time-encoding kernels build their cosine and
sine from, read out of the HIP sources and checked on the CPU against the
mathematics they stand for (Sec. 6.1, the time encoder cos(omega dt + phi)
and its gradient), so that a mistyped digit fails here rather than as a
small error in a GPU sum.  No GPU and no library call."""
import math
import os
import re

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_05095_amd", "csrc")
HEX = r"(-?0x[0-9a-fA-F]\.[0-9a-fA-F]+p[-+]?\d+)"


def _src(name):
    with open(os.path.join(CSRC, name)) as f:
        return f.read()


def _body(src, head):
    i = src.index(head)
    return src[i:src.index("\n}\n", i)]


def _hex(s):
    return float.fromhex(s.rstrip("f"))


def test_backward_sine_polynomial_and_reduction():
    body = _body(_src("time_encode_bwd.hip"), "double sin_reduced(float xf)")
    init = re.search(r"double p = " + HEX + ";", body).group(1)
    steps = re.findall(r"p = fma\(p, r2, " + HEX + r"\);", body)
    coef = [_hex(init)] + [_hex(c) for c in steps]     # highest power of r^2 first
    assert len(coef) == 5
    r = np.linspace(0.0, math.pi / 2 + 1e-9, 400_001)
    r2 = r * r
    p = np.full_like(r, coef[0])
    for c in coef[1:]:
        p = p * r2 + c
    s = r + r * r2 * p
    rel = np.abs(s - np.sin(r))[1:] / np.sin(r[1:])
    assert rel.max() < 3e-11, rel.max()
    # the one-step reduction: k * (pi - PI_HI) over the in-line range
    pi_hi = _hex(re.search(r"PI_HI = " + HEX, body).group(1))
    assert pi_hi == math.pi                            # the fp64 rounding of pi
    pi_rest = 1.2246467991473532e-16                   # pi - fl64(pi)
    limit = _hex("0x1p0") * float(re.search(r"TB_ROW_LIMIT = ([0-9.e]+)f;",
                                            _src("time_encode_bwd.hip")).group(1))
    k_max = limit * (1 + 2.0 ** -22) / math.pi + 1
    assert limit * (1 + 2.0 ** -22) < 2.0 ** 20
    assert k_max * pi_rest < 4e-11
    inv_pi = _hex(re.search(r"INV_PI = " + HEX, body).group(1))
    assert inv_pi == 1 / math.pi


def test_forward_cosine_reduction_constants():
    body = _body(_src("time_encode.hip"), "float cos_rr(float x)")
    d1 = _hex(re.search(r"D1 = " + HEX, body).group(1))
    d2 = _hex(re.search(r"D2 = " + HEX, body).group(1))
    inv = _hex(re.search(r"INV_TWO_PI = " + HEX, body).group(1))
    # both parts are fp32 numbers and their sum is 2 pi to 2^-47 (each
    # reduction step is one fmaf, so k * D1 and k * D2 need not be exact)
    for v in (d1, d2, inv):
        assert float(np.float32(v)) == v
    two_pi_hi, two_pi_lo = 2 * math.pi, 2.4492935982947064e-16   # 2 pi = hi + lo
    assert abs((d1 - two_pi_hi) + d2 - two_pi_lo) < 2.0 ** -47
    assert inv == float(np.float32(1 / (2 * math.pi)))
