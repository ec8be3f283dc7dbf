"""The soft-cap polynomial of the max-folding kernels (softcap_poly.h).

C tanh(s / C) (Appendix A, "Softcap Attention") is evaluated on tiles whose
|y| = |scale dot / C| stays within a range R as dot (b0 + z (b1 + z b2)),
z = dot^2. These CPU tests read the fit table from the header and check,
against tanh in double precision: each fit's stated relative error, the
host's choice of R for caps up to the short form's limit (error bound within
1e-4 score units), and the kernel's float32 evaluation order at the chosen R.
"""
import math

import numpy as np
import pytest

from cap_poly import choose as _choose
from cap_poly import table

LOG2E = 1.4426950408889634
FITS, MAX_ERR = table()


def test_table_shape():
    assert len(FITS) >= 5
    rs = [r for r, _, _ in FITS]
    assert rs == sorted(rs, reverse=True) and rs[0] == 0.5


@pytest.mark.parametrize("i", range(7))
def test_fit_relative_error(i):
    r, a, e = FITS[i]
    y = np.linspace(1e-9, r, 200001)
    q = a[0] + a[1] * y * y + a[2] * y ** 4
    rel = np.abs(q - np.tanh(y) / y) / (np.tanh(y) / y)
    assert rel.max() <= e * 1.01
    # y -> 0: tanh(y)/y -> 1
    assert abs(a[0] - 1.0) <= e * 1.01


@pytest.mark.parametrize("cap", [1.0, 5.0, 20.0, 30.0, 50.0, 100.0, 256.0])
@pytest.mark.parametrize("d", [64, 128])
def test_chosen_range_error(cap, d):
    """float32 emulation of the kernel's evaluation at the host's coefficients:
    the soft-capped score (log2 units) errs by at most MAX_ERR plus float32
    rounding of a score of that size."""
    scale = 1.0 / math.sqrt(d)
    cu = cap * LOG2E
    r, a, e = _choose(cu)
    assert cu * r * e <= MAX_ERR
    sc = scale / cap
    b = [np.float32(cu * sc ** (2 * k + 1) * a[k]) for k in range(3)]
    zmax = r * r / (sc * sc)
    dot = np.linspace(-math.sqrt(zmax), math.sqrt(zmax), 100001).astype(np.float32)
    z = dot * dot
    assert float(z.max()) <= zmax * (1 + 1e-6)
    q = np.float32(b[2]) * z + b[1]
    q = q.astype(np.float32) * z + b[0]
    u = (dot * q.astype(np.float32)).astype(np.float64)
    ref = cu * np.tanh(sc * dot.astype(np.float64))
    err = np.abs(u - ref)
    bound = MAX_ERR + 4 * np.finfo(np.float32).eps * np.abs(ref)
    assert (err <= bound).all(), float((err - bound).max())


def test_workload_caps_stay_in_range():
    """The headline soft-cap workload (C = 50, D = 64, sigma 1.5 inputs) gets a
    range that its scores leave only beyond 7 standard deviations of q . k."""
    cu = 50.0 * LOG2E
    r, _, _ = _choose(cu)
    dot_limit = r * 50.0 * math.sqrt(64)  # |dot| <= R C / scale
    sd = 1.5 * 1.5 * math.sqrt(64)
    assert dot_limit / sd > 7.0
