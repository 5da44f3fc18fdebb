"""Band layout, spectral windows and dual windows (fp64).

TEST INFRASTRUCTURE ONLY (see the package header).

The paper defines a band by a real spectral window g_lambda, a selection E_lambda
that places the window's support into local slots injectively, and a length
M_lambda (Sec. 2, eqs. 2-3). It restricts to the painless case: supports fit
without collisions and together cover every bin 0 <= k <= N/2. The aggregate
weight is a_k = sum_lambda M_lambda g_{lambda,k}^2 and the dual window is
h_{lambda,k} = M_lambda g_{lambda,k} / a_k, so that sum_lambda h g = 1 (Sec. 2).

The paper does not fix the window shapes for a general constant-Q layout; this
module implements the following reading (every choice is listed in the design
notes of the repository):

  * centres f_j = fmin * 2**(j/B) for j = 0, 1, ... while f_j <= fmax*(1+1e-12)
    and f_j < fs/2; Q = 1/(2**(1/B) - 1);
  * a positive band is a Hann window g(k) = cos^2(pi (k - xi)/(2 beta)) centred
    at xi = f N/fs bins with half-amplitude width beta = (f/Q) N/fs bins, on the
    integer bins with |k - xi| < beta, clipped to 0 <= k <= N/2;
  * a DC sideband on 0 <= k < xi_0 and a Nyquist sideband on xi_{K-1} < k <= N/2,
    each flat with a sin^2 taper complementary to the outer half of the
    neighbouring Hann window;
  * band length M = support width in bins; slot(k) = (k - k_c) mod M with the
    centre bin k_c = floor(xi + 1/2) (0 for DC, N/2 for Nyquist);
  * bands with empty support are dropped.

Parity: pinned by tests (closed-form windows, sum h g = 1, coverage bounds,
band counts, agreement with an independent integer layout).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

DC, POSITIVE, NYQUIST = 0, 1, 2


@dataclasses.dataclass
class Band:
    kind: int             # DC, POSITIVE or NYQUIST
    k_lo: int             # first support bin
    k_hi: int             # last support bin (inclusive)
    k_c: int              # bin placed in slot 0
    xi: float             # centre in bins (DC: xi_0, Nyquist: xi_{K-1})
    beta: float           # half-amplitude width in bins of the governing Hann
    centre_hz: float
    g: np.ndarray = None  # window on k_lo..k_hi (fp64)
    h: np.ndarray = None  # dual window on k_lo..k_hi (fp64)
    offset: int = 0       # first coefficient of this band in the flat layout

    @property
    def M(self) -> int:
        return self.k_hi - self.k_lo + 1

    @property
    def bins(self) -> np.ndarray:
        return np.arange(self.k_lo, self.k_hi + 1)

    @property
    def slots(self) -> np.ndarray:
        return (self.bins - self.k_c) % self.M


@dataclasses.dataclass
class Layout:
    fs: float
    fmin: float
    fmax: float
    bins_per_octave: int
    N: int
    bands: list
    a: np.ndarray         # aggregate weight a_k, 0 <= k <= N/2

    @property
    def half(self) -> int:
        return self.N // 2

    @property
    def n_coeffs(self) -> int:
        return sum(b.M for b in self.bands)

    def offsets(self) -> np.ndarray:
        return np.array([b.offset for b in self.bands], dtype=np.int64)


def _hann(k, xi, beta):
    return np.cos(np.pi * (k - xi) / (2.0 * beta)) ** 2


def build_layout(fs, fmin, fmax, bins_per_octave, N) -> Layout:
    """Constant-Q layout of the reading above for signals of N real samples."""
    N = int(N)
    B = int(bins_per_octave)
    if N % 2 or N < 4:
        raise ValueError("N must be even and >= 4")
    if not (fs > 0 and 0 < fmin < fs / 2 and fmax >= fmin and B >= 1):
        raise ValueError("invalid frequency parameters")
    half = N // 2
    Q = 1.0 / (2.0 ** (1.0 / B) - 1.0)

    centres = []
    j = 0
    while True:
        f = fmin * 2.0 ** (j / B)
        if not (f <= fmax * (1.0 + 1e-12) and f < fs / 2.0):
            break
        centres.append(f)
        j += 1
    xis = [f * N / fs for f in centres]
    betas = [(f / Q) * N / fs for f in centres]

    bands = []
    # DC sideband: bins 0 <= k < xi_0, flat then a sin^2 taper that complements
    # the lower half of the first Hann window.
    xi0, b0 = xis[0], betas[0]
    k = np.arange(0, math.ceil(xi0))
    g = np.where(k <= xi0 - b0, 1.0, np.sin(np.pi * (xi0 - k) / (2.0 * b0)) ** 2)
    bands.append(Band(DC, 0, int(math.ceil(xi0)) - 1, 0, xi0, b0, 0.0, g))

    for f, xi, beta in zip(centres, xis, betas):
        k_lo = max(0, math.floor(xi - beta) + 1)
        k_hi = min(half, math.ceil(xi + beta) - 1)
        if k_hi < k_lo:
            continue
        k = np.arange(k_lo, k_hi + 1)
        bands.append(Band(POSITIVE, k_lo, k_hi, math.floor(xi + 0.5), xi, beta, f,
                          _hann(k, xi, beta)))

    # Nyquist sideband: bins xi_{K-1} < k <= N/2, a taper that complements the
    # upper half of the last Hann window, then flat.
    xl, bl = xis[-1], betas[-1]
    k_lo = math.floor(xl) + 1
    k = np.arange(k_lo, half + 1)
    g = np.where(k >= xl + bl, 1.0, np.sin(np.pi * (k - xl) / (2.0 * bl)) ** 2)
    bands.append(Band(NYQUIST, k_lo, half, half, xl, bl, fs / 2.0, g))

    a = np.zeros(half + 1)
    off = 0
    for band in bands:
        band.offset = off
        off += band.M
        a[band.k_lo:band.k_hi + 1] += band.M * band.g ** 2
    if np.any(a <= 0.0):
        raise ValueError("layout leaves a bin uncovered (a_k = 0)")
    for band in bands:
        band.h = band.M * band.g / a[band.k_lo:band.k_hi + 1]
    return Layout(float(fs), float(fmin), float(fmax), B, N, bands, a)
