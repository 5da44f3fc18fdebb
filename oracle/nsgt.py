"""Analysis, synthesis and their real adjoints, from the plain definitions (fp64).

TEST INFRASTRUCTURE ONLY (see the package header).

The paper's packed factorisation reaches exactly the plain transform (Sec. 3,
eqs. 8 and 10), so this oracle evaluates the plain definitions and nothing of
the packed path: no packing, untangling, routing or retangling.

DFT convention (Sec. 2, eq. 1): [F_n]_{kj} = exp(-2 pi i k j / n) and
F_n^{-1} = F_n^H / n.

  analyse            c_lambda = F_M^{-1} E_lambda diag(g_lambda) F_N x        (eqs. 2-3)
  synthesise         x = F_N^{-1} sum_lambda diag(h_lambda) E_lambda^T F_M c_lambda,
                     bins 0..N/2 only, DC and Nyquist made real, negative
                     frequencies by conjugate symmetry                           (eq. 4)
  adjoint_analysis   T^dagger under <u, v> = Re(u^H v)                          (Sec. 3.2)
  adjoint_synthesis  S^dagger under the same inner product                      (Sec. 3.2)

The full-length F_N is numpy's FFT (a library routine). Each band transform is
a direct DFT: the twiddle for the product m*n is looked up by the exact integer
(m*n) mod M in an fp64 table of the M-th roots of unity, so no rounding of
the angle grows with the index. A ``mode="fft"`` switch replaces the direct
band DFT by numpy's FFT of the same length; it is cross-checked against the
direct form.

The adjoints are the transposes of the real-linear maps above, worked out
from the same definitions:
  T^dagger y = Re( F_N^H V ),  V_k = sum_lambda g_{lambda,k} [F_M y_lambda / M]_{slot(k)}
               for 0 <= k <= N/2 and V_k = 0 above N/2;
  (S^dagger x)_lambda = (M/N) F_M^{-1} E_lambda ( h_lambda * d * F_N x ),
               d_k = 1 at k = 0 and k = N/2, d_k = 2 in between.

Parity: pinned by tests (brute-force matrices at small N, closed forms for
cosines, constants and alternating signals, the energy identity, ST = I,
both adjoint identities, and the library FFT special case).
"""
from __future__ import annotations

import numpy as np

from .layout import Layout

_CHUNK_ELEMS = 1 << 22   # entries of a band DFT matrix block held at once


def _roots(M: int, sign: int) -> np.ndarray:
    """exp(sign * 2 pi i t / M) for t = 0..M-1 in fp64."""
    return np.exp(sign * 2j * np.pi * np.arange(M) / M)


def _direct(v: np.ndarray, sign: int) -> np.ndarray:
    """sum_m v[..., m] exp(sign 2 pi i (m n mod M) / M) for n = 0..M-1."""
    M = v.shape[-1]
    root = _roots(M, sign)
    m = np.arange(M, dtype=np.int64)
    out = np.empty(v.shape, dtype=np.complex128)
    step = max(1, _CHUNK_ELEMS // M)
    for n0 in range(0, M, step):
        n = np.arange(n0, min(M, n0 + step), dtype=np.int64)
        out[..., n0:n0 + len(n)] = v @ root[np.outer(m, n) % M]
    return out


def band_idft(u: np.ndarray, mode: str = "direct") -> np.ndarray:
    """F_M^{-1} u along the last axis (includes 1/M)."""
    if mode == "fft":
        return np.fft.ifft(u, axis=-1)
    return _direct(u, +1) / u.shape[-1]


def band_dft(c: np.ndarray, mode: str = "direct") -> np.ndarray:
    """F_M c along the last axis (no scaling)."""
    if mode == "fft":
        return np.fft.fft(c, axis=-1)
    return _direct(c, -1)


def split_bands(lay: Layout, c: np.ndarray) -> list:
    """Views of the flat [..., C] coefficients, one per band."""
    return [c[..., b.offset:b.offset + b.M] for b in lay.bands]


def _as_batch(a, n):
    a = np.asarray(a)
    if a.shape[-1] != n:
        raise ValueError(f"last axis must have length {n}")
    return a.reshape(-1, n), a.shape[:-1]


def analyse(lay: Layout, x, mode: str = "direct") -> np.ndarray:
    """Coefficients [..., C] (complex128) of real signals x [..., N]."""
    xb, lead = _as_batch(np.asarray(x, dtype=np.float64), lay.N)
    X = np.fft.fft(xb, axis=-1)                                  # F_N x
    c = np.empty((xb.shape[0], lay.n_coeffs), dtype=np.complex128)
    for b in lay.bands:
        u = np.zeros((xb.shape[0], b.M), dtype=np.complex128)
        u[:, b.slots] = b.g * X[:, b.k_lo:b.k_hi + 1]            # E diag(g) X
        c[:, b.offset:b.offset + b.M] = band_idft(u, mode)       # F_M^{-1} u
    return c.reshape(*lead, lay.n_coeffs)


def analyse_bands(lay: Layout, x, bands, mode: str = "direct") -> dict:
    """Coefficients of the listed bands only: {band index: [..., M]}.

    The same definition as ``analyse`` restricted to a subset of bands, for
    checking sampled outputs of large transforms one band at a time."""
    xb, lead = _as_batch(np.asarray(x, dtype=np.float64), lay.N)
    X = np.fft.fft(xb, axis=-1)
    out = {}
    for i in bands:
        b = lay.bands[i]
        u = np.zeros((xb.shape[0], b.M), dtype=np.complex128)
        u[:, b.slots] = b.g * X[:, b.k_lo:b.k_hi + 1]
        out[i] = band_idft(u, mode).reshape(*lead, b.M)
    return out


def _half_to_real(lay: Layout, Y: np.ndarray) -> np.ndarray:
    """Real signal whose spectrum is Y on 0..N/2 extended by conjugate symmetry."""
    N, half = lay.N, lay.half
    Y = Y.copy()
    Y[:, 0] = Y[:, 0].real
    Y[:, half] = Y[:, half].real
    full = np.empty((Y.shape[0], N), dtype=np.complex128)
    full[:, :half + 1] = Y
    full[:, half + 1:] = np.conj(Y[:, half - 1:0:-1])
    x = np.fft.ifft(full, axis=-1)                               # F_N^{-1}
    scale = max(1.0, float(np.max(np.abs(x.real))))
    assert np.max(np.abs(x.imag)) <= 1e-9 * scale
    return x.real


def synthesise(lay: Layout, c, mode: str = "direct") -> np.ndarray:
    """Real signals [..., N] from coefficients [..., C]."""
    cb, lead = _as_batch(np.asarray(c, dtype=np.complex128), lay.n_coeffs)
    Y = np.zeros((cb.shape[0], lay.half + 1), dtype=np.complex128)
    for b in lay.bands:
        U = band_dft(cb[:, b.offset:b.offset + b.M], mode)       # F_M c
        Y[:, b.k_lo:b.k_hi + 1] += b.h * U[:, b.slots]           # diag(h) E^T
    return _half_to_real(lay, Y).reshape(*lead, lay.N)


def adjoint_analysis(lay: Layout, y, mode: str = "direct") -> np.ndarray:
    """T^dagger y: coefficient cotangent [..., C] -> signal gradient [..., N]."""
    yb, lead = _as_batch(np.asarray(y, dtype=np.complex128), lay.n_coeffs)
    V = np.zeros((yb.shape[0], lay.N), dtype=np.complex128)
    for b in lay.bands:
        U = band_dft(yb[:, b.offset:b.offset + b.M], mode) / b.M
        V[:, b.k_lo:b.k_hi + 1] += b.g * U[:, b.slots]
    out = (np.conj(np.fft.fft(np.conj(V), axis=-1))).real       # Re(F_N^H V)
    return out.reshape(*lead, lay.N)


def adjoint_synthesis(lay: Layout, x, mode: str = "direct") -> np.ndarray:
    """S^dagger x: signal cotangent [..., N] -> coefficient gradient [..., C]."""
    xb, lead = _as_batch(np.asarray(x, dtype=np.float64), lay.N)
    X = np.fft.fft(xb, axis=-1)
    d = np.full(lay.half + 1, 2.0)
    d[0] = d[lay.half] = 1.0
    c = np.empty((xb.shape[0], lay.n_coeffs), dtype=np.complex128)
    for b in lay.bands:
        k = b.bins
        u = np.zeros((xb.shape[0], b.M), dtype=np.complex128)
        u[:, b.slots] = (b.h * d[k]) * X[:, k]
        c[:, b.offset:b.offset + b.M] = (b.M / lay.N) * band_idft(u, mode)
    return c.reshape(*lead, lay.n_coeffs)
