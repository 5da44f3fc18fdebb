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

An explicit band list (``build_band_layout``) uses the same window shapes at
given centres and widths with lengths M >= the support width: the slots past
the support hold zero, which is the band spectrum zero-padded to M (Sec. 2
only asks that E_lambda place the support injectively into M slots).
``table1_specs`` is the multi-resolution layout of Table 1 (Sec. 4) under the
reading stated in its docstring, and ``erb_specs`` an auditory layout on the
ERB-rate scale (another painless frame of the kind Sec. 6 says the
construction extends to).

Parity: pinned by tests (closed-form windows, sum h g = 1, coverage bounds,
band counts, agreement with an independent integer layout). Two conventions
are parity unpinned, since no passage fixes them: the phase of the slot map
(which bin goes to slot 0; every injective map gives a valid transform), and
the fan-out of the Table 1 reading, 6 against the paper's 7.
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
    length: int = 0       # band length M; 0 means the support width

    @property
    def width(self) -> int:
        return self.k_hi - self.k_lo + 1

    @property
    def M(self) -> int:
        return self.length or self.width

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

    a = _finish(bands, half)
    return Layout(float(fs), float(fmin), float(fmax), B, N, bands, a)


def _finish(bands, half):
    """Offsets, aggregate weight a_k = sum M g^2 and duals h = M g / a (Sec. 2)."""
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
    return a


def build_band_layout(fs, N, specs) -> Layout:
    """Layout of an explicit band list: tuples (kind, xi, beta, length[, centre_hz]).

    DC: bins 0 <= k < xi, flat up to xi - beta, then sin^2(pi (xi - k)/(2 beta)).
    POSITIVE: Hann cos^2(pi (k - xi)/(2 beta)) on |k - xi| < beta within 0..N/2,
    centre bin floor(xi + 1/2). NYQUIST: bins xi < k <= N/2, sin^2(pi (k - xi)/(2 beta))
    below xi + beta, then flat. length 0 means the support width; otherwise it
    must be at least the support width."""
    N = int(N)
    if N % 2 or N < 4:
        raise ValueError("N must be even and >= 4")
    half = N // 2
    bands = []
    for i, sp in enumerate(specs):
        kind, xi, beta, length = int(sp[0]), float(sp[1]), float(sp[2]), int(sp[3])
        f = float(sp[4]) if len(sp) > 4 else 0.0
        if not (beta > 0.0 and math.isfinite(xi) and math.isfinite(beta)) or length < 0:
            raise ValueError(f"band {i}: invalid width or length")
        if kind == DC:
            if i != 0:
                raise ValueError("a DC band must come first")
            k = np.arange(0, min(half, math.ceil(xi) - 1) + 1)
            g = np.where(k <= xi - beta, 1.0, np.sin(np.pi * (xi - k) / (2.0 * beta)) ** 2)
            k_c = 0
        elif kind == POSITIVE:
            k = np.arange(max(0, math.floor(xi - beta) + 1), min(half, math.ceil(xi + beta) - 1) + 1)
            g = _hann(k, xi, beta)
            k_c = math.floor(xi + 0.5)
        elif kind == NYQUIST:
            if i != len(specs) - 1:
                raise ValueError("a Nyquist band must come last")
            k = np.arange(max(0, math.floor(xi) + 1), half + 1)
            g = np.where(k >= xi + beta, 1.0, np.sin(np.pi * (k - xi) / (2.0 * beta)) ** 2)
            k_c = half
        else:
            raise ValueError(f"band {i}: unknown kind")
        if len(k) == 0:
            raise ValueError(f"band {i}: empty support")
        if length and length < len(k):
            raise ValueError(f"band {i}: length below the support width")
        bands.append(Band(kind, int(k[0]), int(k[-1]), k_c, xi, beta, f, g, length=length))
    a = _finish(bands, half)
    return Layout(float(fs), 0.0, 0.0, 0, N, bands, a)


def table1_specs():
    """(fs, N, band list) of the multi-resolution layout of Table 1 (Sec. 4).

    The paper fixes N = 65,536 at 44.1 kHz, three resolutions covering 3, 4
    and 2 octaves at 8, 16 and 32 bands per octave (152 positive bands),
    centres rounded to bins with the highest adjusted towards Nyquist, one
    length per octave from its widest support rounded up to a power of two,
    and sideband lengths 128 (DC) and 2048 (Nyquist). Reading of what it
    leaves open: the lowest centre is bin 64 (43.07 Hz, the table's 43 Hz);
    centre j of octave o (o = 0..8) is bin round(64 * 2^(o + j/B_o)); the
    highest centre is the table's 21,810 Hz rounded to a bin; each window is
    the Hann window of the constant-Q reading with Q = 1/(2^(1/B_o) - 1) and
    half-amplitude width xi/Q; the sidebands complement the outer halves of
    the lowest and highest windows."""
    fs, N = 44100.0, 65536
    half = N // 2
    per_octave = [8] * 3 + [16] * 4 + [32] * 2
    octave, xis = [], []
    for o, B in enumerate(per_octave):
        for j in range(B):
            octave.append(o)
            xis.append(float(round(64.0 * 2.0 ** (o + j / B))))
    xis[-1] = float(round(21810.0 * N / fs))
    betas = [xi / (1.0 / (2.0 ** (1.0 / per_octave[o]) - 1.0)) for xi, o in zip(xis, octave)]
    widest = [0] * len(per_octave)
    for xi, beta, o in zip(xis, betas, octave):
        lo = max(0, math.floor(xi - beta) + 1)
        hi = min(half, math.ceil(xi + beta) - 1)
        widest[o] = max(widest[o], hi - lo + 1)
    length = [1 << (w - 1).bit_length() for w in widest]
    specs = [(DC, xis[0], betas[0], 128, 0.0)]
    specs += [(POSITIVE, xi, beta, length[o], xi * fs / N) for xi, beta, o in zip(xis, betas, octave)]
    specs.append((NYQUIST, xis[-1], betas[-1], 2048, fs / 2.0))
    return fs, N, specs


def erb_hz(f):
    """Equivalent rectangular bandwidth (Glasberg and Moore, 1990) in Hz."""
    return 24.7 * (4.37 * f / 1000.0 + 1.0)


def erb_rate(f):
    """ERB-rate (number of ERBs below f) of the same model."""
    return 21.4 * math.log10(1.0 + 4.37 * f / 1000.0)


def erb_specs(fs, N, fmin, fmax, per_erb):
    """Auditory layout: centres one 1/per_erb apart on the ERB-rate scale from
    fmin (while <= fmax and below fs/2), Hann windows whose half-amplitude
    width is the centre spacing ERB(f)/per_erb, sidebands complementing the
    outer Hann halves, lengths equal to the support widths; bands without a
    bin inside their support are left out."""
    half = N // 2
    e0 = erb_rate(fmin)
    pos = []
    j = 0
    while True:
        f = (10.0 ** ((e0 + j / per_erb) / 21.4) - 1.0) * 1000.0 / 4.37
        if not (f <= fmax * (1.0 + 1e-12) and f < fs / 2.0):
            break
        xi = f * N / fs
        beta = erb_hz(f) / per_erb * N / fs
        if min(half, math.ceil(xi + beta) - 1) >= max(0, math.floor(xi - beta) + 1):
            pos.append((POSITIVE, xi, beta, 0, f))
        j += 1
    return [(DC, pos[0][1], pos[0][2], 0, 0.0)] + pos + [(NYQUIST, pos[-1][1], pos[-1][2], 0, fs / 2.0)]

