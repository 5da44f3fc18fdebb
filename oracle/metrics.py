"""Error measures (fp64).

TEST INFRASTRUCTURE ONLY (see the package header).

snr_db: reconstruction SNR 10 log10(||x||^2 / ||x - x_hat||^2) as defined in
        Sec. 5.1, per signal along the last axis.
rel_l2: ||a - b|| / ||b|| per row along the last axis.
band_rel_l2: the same per band of a flat coefficient row, the bands starting
        at the given offsets (the last one running to the end of the row).
max_err_over_rms: max |a - b| / rms(b) per row, an element-wise bound.
band_max_err_over_rms: the same per band of a flat coefficient row.
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


def band_rel_l2(a, b, offsets) -> np.ndarray:
    """||a_band - b_band|| / ||b_band|| for every band, shape [..., n_bands];
    a band whose reference is all zero gives inf (or nan if a is zero too)."""
    a = np.asarray(a)
    b = np.asarray(b)
    off = np.asarray(offsets, dtype=np.int64)
    e2 = np.abs(a.astype(np.complex128) - b) ** 2
    r2 = np.abs(b.astype(np.complex128)) ** 2
    num = np.add.reduceat(e2, off, axis=-1)
    den = np.add.reduceat(r2, off, axis=-1)
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.sqrt(num / den)


def max_err_over_rms(a, b) -> np.ndarray:
    """max_i |a_i - b_i| / sqrt(mean_i |b_i|^2) per row along the last axis."""
    a = np.asarray(a)
    b = np.asarray(b)
    err = np.abs(a.astype(np.complex128) - b).max(axis=-1)
    rms = np.sqrt(np.mean(np.abs(b.astype(np.complex128)) ** 2, axis=-1))
    return err / rms


def band_max_err_over_rms(a, b, offsets) -> np.ndarray:
    """max over the band of |a - b| / rms of the band's reference, shape
    [..., n_bands]."""
    a = np.asarray(a)
    b = np.asarray(b)
    off = np.asarray(offsets, dtype=np.int64)
    n = b.shape[-1]
    cnt = np.diff(np.append(off, n))
    err = np.maximum.reduceat(np.abs(a.astype(np.complex128) - b), off, axis=-1)
    ms = np.add.reduceat(np.abs(b.astype(np.complex128)) ** 2, off, axis=-1) / cnt
    with np.errstate(divide="ignore", invalid="ignore"):
        return err / np.sqrt(ms)
