"""Error measures (fp64).

TEST INFRASTRUCTURE ONLY (see the package header).

snr_db: reconstruction SNR 10 log10(||x||^2 / ||x - x_hat||^2) as defined in
        Sec. 5.1, per signal along the last axis.
rel_l2: ||a - b|| / ||b|| per row along the last axis.
"""
from __future__ import annotations

import numpy as np


def snr_db(x, x_hat) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    e = x - np.asarray(x_hat, dtype=np.float64)
    num = np.sum(x * x, axis=-1)
    den = np.sum(e * e, axis=-1)
    with np.errstate(divide="ignore"):
        return 10.0 * np.log10(num / den)


def rel_l2(a, b) -> np.ndarray:
    a = np.asarray(a)
    b = np.asarray(b)
    num = np.sqrt(np.sum(np.abs(a.astype(np.complex128) - b) ** 2, axis=-1))
    den = np.sqrt(np.sum(np.abs(b.astype(np.complex128)) ** 2, axis=-1))
    return num / den
