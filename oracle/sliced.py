"""Overlapping-slice (streaming) mode (fp64).

TEST INFRASTRUCTURE ONLY (see the package header).

Sec. 4 transforms long signals in independent slices of N_s samples with 50 %
overlap and a Tukey transition window, and recovers the signal by overlap-add.
The paper leaves the taper and the padding open; the reading implemented here
is:

  * hop H = N_s / 2 (N_s a multiple of 8); the signal is preceded by H zeros
    and followed by zeros; slice s covers padded samples [s H, s H + N_s),
    i.e. original samples [s H - H, s H + H), for s = 0 .. J-1 with
    J = ceil(n / H) + 1;
  * window w on 0 <= t < N_s: 0 below N_s/8, sin^2(pi (t - N_s/8)/(N_s/2)) up
    to 3N_s/8, 1 up to 5N_s/8, cos^2(pi (t - 5N_s/8)/(N_s/2)) up to 7N_s/8,
    0 above, so w(t) + w(t + H) = 1;
  * slice coefficients c_s = T(w * slice_s) with the layout built for N_s;
  * synthesis overlap-adds S c_s at the slice positions and crops to n.

Parity: pinned by tests (partition of unity in closed form, per-slice
coefficients equal T of the windowed slice, sliced round trip).
"""
from __future__ import annotations

import numpy as np

from .layout import Layout
from .nsgt import analyse, synthesise


def slice_window(Ns: int) -> np.ndarray:
    if Ns % 8:
        raise ValueError("slice length must be a multiple of 8")
    t = np.arange(Ns, dtype=np.float64)
    e, q = Ns // 8, Ns / 2.0
    w = np.zeros(Ns)
    up = (t >= e) & (t < 3 * e)
    w[up] = np.sin(np.pi * (t[up] - e) / q) ** 2
    w[(t >= 3 * e) & (t < 5 * e)] = 1.0
    dn = (t >= 5 * e) & (t < 7 * e)
    w[dn] = np.cos(np.pi * (t[dn] - 5 * e) / q) ** 2
    return w


def slice_count(n: int, Ns: int) -> int:
    H = Ns // 2
    return -(-n // H) + 1


def _padded(x: np.ndarray, Ns: int) -> np.ndarray:
    H = Ns // 2
    J = slice_count(x.shape[-1], Ns)
    xp = np.zeros(x.shape[:-1] + ((J + 1) * H,))
    xp[..., H:H + x.shape[-1]] = x
    return xp


def sliced_analyse(lay: Layout, x, mode: str = "direct") -> np.ndarray:
    """Coefficients [J, C_s] of one real signal x [n] in slices of lay.N."""
    x = np.asarray(x, dtype=np.float64)
    Ns, H = lay.N, lay.N // 2
    J = slice_count(x.shape[-1], Ns)
    xp = _padded(x, Ns)
    w = slice_window(Ns)
    segs = np.stack([w * xp[s * H:s * H + Ns] for s in range(J)])
    return analyse(lay, segs, mode)


def sliced_synthesise(lay: Layout, c, n: int, mode: str = "direct") -> np.ndarray:
    """Signal [n] overlap-added from slice coefficients [J, C_s]."""
    Ns, H = lay.N, lay.N // 2
    J = slice_count(n, Ns)
    y = synthesise(lay, np.asarray(c)[:J], mode)
    out = np.zeros((J + 1) * H)
    for s in range(J):
        out[s * H:s * H + Ns] += y[s]
    return out[H:H + n]
