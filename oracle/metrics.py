"""Error metrics of the paper's evaluation appendix (Appendix A.2), used to
summarise parity errors.  Test infrastructure only, like the rest of
``oracle``."""
from __future__ import annotations

import math

import numpy as np


def mape(pred, ref):
    """Mean absolute percentage error, Eq. 5: 100/n sum |(y_hat - y) / y|."""
    pred = np.asarray(pred, np.float64)
    ref = np.asarray(ref, np.float64)
    return 100.0 * float(np.mean(np.abs((pred - ref) / ref)))


def abs_pct_err(pred, ref):
    """Per-item absolute percent error, Eq. 6: 100 |y_hat - y| / y."""
    pred = np.asarray(pred, np.float64)
    ref = np.asarray(ref, np.float64)
    return 100.0 * np.abs(pred - ref) / ref


def percentile_nearest_rank(e, p):
    """Eq. 7: P_p = e_(k) with k = ceil(p/100 n) over the ascending e."""
    e = np.sort(np.asarray(e, np.float64).ravel())
    n = len(e)
    if n == 0:
        raise ValueError("empty sample")
    k = max(1, math.ceil(p / 100.0 * n))
    return float(e[k - 1])
