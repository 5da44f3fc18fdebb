"""Seeded synthetic workloads for the constant-Q transform.

This module only draws input signals and cotangents; it contains none of the
transform's arithmetic, so both the fp64 oracle and the GPU path can consume
exactly the same fp32 arrays.

Five workloads are defined, each with its transform parameters and a signal
recipe (the evaluation in Sec. 5 uses fp32 signals resident on the device but
does not name their content, so these stand in for it):

  tiny    1 x 16,384 @ 22.05 kHz, N(0,1) noise; 110 Hz..fs/2, 12 bins/oct
  single  1 x 44,100 @ 44.1 kHz, 8 sinusoids + N(0, 0.01) noise;
          32.7 Hz..fs/2, 48 bins/oct
  train   16 x 220,500 @ 44.1 kHz, pink-ish noise (white shaped by
          1/sqrt(f)); 40 Hz..fs/2, 24 bins/oct; a complex N(0,1) cotangent
  long    1 x 2,880,000 @ 48 kHz, white noise; 20 Hz..fs/2, 96 bins/oct;
          sliced mode uses slices of 2**17 with 50 % overlap
  stress  128 x 88,200 @ 22.05 kHz, 8 sinusoids + Bernoulli(1e-3) +-1
          impulses + N(0, 0.05) noise; 55 Hz..fs/2, 36 bins/oct
  table1  128 x 65,536 @ 44.1 kHz, N(0,1) noise; the multi-resolution band
          list of the paper's Table 1 (the shape of its own measurements,
          whose signal content it does not state)

N(mu, v) is read with v the variance. Every signal of a batch gets its own
child generator from ``SeedSequence(seed).spawn(batch)``; values are drawn in
fp64 and rounded once to fp32.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    fs: float
    fmin: float
    fmax: float
    bins_per_octave: int
    n_samples: int
    batch: int
    seed: int
    cot_seed: int
    slice_len: int = 0          # 0: no sliced mode for this workload
    layout: str = "cq"          # "cq": constant-Q from (fs, fmin, fmax, B); "table1": Table 1 band list

    @property
    def plan_args(self):
        return (self.fs, self.fmin, self.fmax, self.bins_per_octave, self.n_samples)


WORKLOADS = {
    "tiny": Workload("tiny", 22050.0, 110.0, 11025.0, 12, 16384, 1, 1, 1001),
    "single": Workload("single", 44100.0, 32.7, 22050.0, 48, 44100, 1, 2, 1002),
    "train": Workload("train", 44100.0, 40.0, 22050.0, 24, 220500, 16, 3, 1003),
    "long": Workload("long", 48000.0, 20.0, 24000.0, 96, 2880000, 1, 4, 1004,
                     slice_len=131072),
    "stress": Workload("stress", 22050.0, 55.0, 11025.0, 36, 88200, 128, 5, 1005),
    "table1": Workload("table1", 44100.0, 0.0, 0.0, 0, 65536, 128, 6, 1006, layout="table1"),
}


def _children(seed: int, batch: int):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(batch)]


def _sinusoids(rng, n, fs, f_lo, f_hi, count=8):
    t = np.arange(n, dtype=np.float64) / fs
    f = np.exp(rng.uniform(np.log(f_lo), np.log(f_hi), size=count))
    a = rng.uniform(0.1, 1.0, size=count)
    ph = rng.uniform(0.0, 2.0 * np.pi, size=count)
    out = np.zeros(n)
    for fi, ai, pi in zip(f, a, ph):
        out += ai * np.sin(2.0 * np.pi * fi * t + pi)
    return out


def _pink(rng, n, fs):
    w = rng.standard_normal(n)
    spec = np.fft.rfft(w)
    f = np.fft.rfftfreq(n, d=1.0 / fs)
    f[0] = f[1]
    spec /= np.sqrt(f)
    y = np.fft.irfft(spec, n=n)
    return y / np.sqrt(np.mean(y * y))


def signal_row(w: Workload, rng, n=None):
    """One fp64 signal of the workload's recipe from one child generator."""
    n = w.n_samples if n is None else n
    if w.name in ("tiny", "long", "table1"):
        return rng.standard_normal(n)
    if w.name == "single":
        return _sinusoids(rng, n, w.fs, 30.0, 18000.0) + rng.normal(0.0, np.sqrt(0.01), n)
    if w.name == "train":
        return _pink(rng, n, w.fs)
    if w.name == "stress":
        s = _sinusoids(rng, n, w.fs, 55.0, 10000.0)
        hit = rng.random(n) < 1e-3
        sign = np.where(rng.random(n) < 0.5, -1.0, 1.0)
        return s + hit * sign + rng.normal(0.0, np.sqrt(0.05), n)
    raise KeyError(w.name)


def signals(w: Workload, batch=None, n=None) -> np.ndarray:
    """[batch][n] fp32 input signals (batch defaults to the workload's)."""
    b = w.batch if batch is None else batch
    rows = [signal_row(w, g, n) for g in _children(w.seed, b)]
    return np.ascontiguousarray(np.stack(rows).astype(np.float32))


def coeff_cotangent(seed: int, batch: int, n_coeffs: int) -> np.ndarray:
    """[batch][n_coeffs] complex64 cotangent with i.i.d. complex N(0,1) entries."""
    rows = []
    for g in _children(seed, batch):
        re = g.standard_normal(n_coeffs)
        im = g.standard_normal(n_coeffs)
        rows.append((re + 1j * im) / np.sqrt(2.0))
    return np.ascontiguousarray(np.stack(rows).astype(np.complex64))


def signal_cotangent(seed: int, batch: int, n: int) -> np.ndarray:
    """[batch][n] fp32 cotangent with i.i.d. N(0,1) entries."""
    rows = [g.standard_normal(n) for g in _children(seed, batch)]
    return np.ascontiguousarray(np.stack(rows).astype(np.float32))


def white(seed: int, batch: int, n: int) -> np.ndarray:
    """[batch][n] fp32 N(0,1) noise; used for small ad hoc shapes in tests."""
    return signal_cotangent(seed, batch, n)
