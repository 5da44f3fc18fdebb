"""Pins of the fp64 oracle to facts fixed by the paper and by the mathematics.

None of these re-evaluates the oracle's own formula: each checks a closed form,
an identity stated in the paper, a brute-force construction by explicit sums,
or a library routine for a special case. A plausible slip in the oracle (a
sign of the band DFT, the direction of the slot rotation, a missing 1/M, a
wrong dual window, a dropped conjugate or DC/Nyquist factor in an adjoint)
fails at least one test here.
"""
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from oracle.layout import DC, NYQUIST, POSITIVE


def small_layout(N=64, fs=64.0, fmin=3.0, fmax=32.0, B=3):
    return oracle.build_layout(fs, fmin, fmax, B, N)


# ----------------------------------------------------------------- layout pins

def test_band_count_closed_form():
    # Centres fmin 2^(j/B) <= fmax give floor(B log2(fmax/fmin)) + 1 positive
    # bands when fmax < fs/2; every band is non-empty at this size.
    fs, fmin, fmax, B, N = 22050.0, 110.0, 5000.0, 12, 16384
    lay = oracle.build_layout(fs, fmin, fmax, B, N)
    K = math.floor(B * math.log2(fmax / fmin)) + 1
    kinds = [b.kind for b in lay.bands]
    assert kinds[0] == DC and kinds[-1] == NYQUIST
    assert kinds.count(POSITIVE) == K


def test_hann_half_amplitude_points():
    # With fs = N every bin is 1 Hz wide. B = 1 gives Q = 1, so the band at
    # f = 64 has centre 64 and half-amplitude width 64 bins: the window is 1 at
    # the centre, 1/2 at +-32 bins and 3/4 at +-64/3 bins (cos^2 pi/6).
    lay = oracle.build_layout(1024.0, 64.0, 256.0, 1, 1024)
    b = [x for x in lay.bands if x.kind == POSITIVE and x.centre_hz == 64.0][0]
    g = dict(zip(b.bins.tolist(), b.g.tolist()))
    assert g[64] == pytest.approx(1.0, abs=1e-15)
    assert g[32] == pytest.approx(0.5, abs=1e-15)
    assert g[96] == pytest.approx(0.5, abs=1e-15)
    # support is |k - 64| < 64, i.e. bins 1..127
    assert (b.k_lo, b.k_hi) == (1, 127)
    assert b.k_c == 64 and b.M == 127


def test_sidebands_complement_outer_hann_halves():
    lay = oracle.build_layout(1024.0, 64.0, 256.0, 1, 1024)
    dc, first = lay.bands[0], lay.bands[1]
    assert (dc.k_lo, dc.k_hi) == (0, 63)
    for k in range(1, 64):
        gd = dc.g[k]
        gf = first.g[k - first.k_lo]
        assert gd + gf == pytest.approx(1.0, abs=1e-14)
    ny, last = lay.bands[-1], lay.bands[-2]
    assert last.centre_hz == 256.0 and (ny.k_lo, ny.k_hi) == (257, 512)
    for k in range(257, 512):
        assert ny.g[k - ny.k_lo] + last.g[k - last.k_lo] == pytest.approx(1.0, abs=1e-14)
    assert ny.g[-1] == 1.0 and dc.g[0] == 1.0


@pytest.mark.parametrize("name", ["tiny", "single", "stress"])
def test_layout_invariants(name):
    import workloads
    w = workloads.WORKLOADS[name]
    lay = oracle.build_layout(*w.plan_args)
    half = lay.half
    cov = np.zeros(half + 1)
    hg = np.zeros(half + 1)
    prev_lo = prev_hi = -1
    off = 0
    for b in lay.bands:
        assert b.M == b.k_hi - b.k_lo + 1 >= 1
        assert b.offset == off
        off += b.M
        assert sorted(b.slots.tolist()) == list(range(b.M))
        assert b.k_lo >= prev_lo and b.k_hi >= prev_hi
        prev_lo, prev_hi = b.k_lo, b.k_hi
        if b.kind == POSITIVE:
            k = b.bins
            assert np.all(np.abs(k - b.xi) < b.beta)
            assert b.k_lo == 0 or abs(b.k_lo - 1 - b.xi) >= b.beta
            assert b.k_hi == half or abs(b.k_hi + 1 - b.xi) >= b.beta
        cov[b.k_lo:b.k_hi + 1] += b.g ** 2
        hg[b.k_lo:b.k_hi + 1] += b.h * b.g
    # painless coverage (Sec. 2): a_k > 0, and the dual satisfies sum h g = 1
    assert np.all(lay.a > 0)
    np.testing.assert_allclose(hg, 1.0, atol=1e-13)
    # conditioning of the frame: neighbouring Hann windows nearly complement
    # each other (exactly so at the sidebands), so sum g^2 stays near [1/2, 1]
    assert cov.min() >= 0.45 and cov.max() <= 1.05


def test_invalid_parameters_rejected():
    with pytest.raises(ValueError):
        oracle.build_layout(22050.0, 110.0, 11025.0, 12, 16383)   # odd N
    with pytest.raises(ValueError):
        oracle.build_layout(22050.0, 0.0, 11025.0, 12, 16384)
    with pytest.raises(ValueError):
        oracle.build_layout(22050.0, 12000.0, 13000.0, 12, 16384)
    with pytest.raises(ValueError):
        oracle.build_layout(22050.0, 110.0, 100.0, 12, 16384)


# ------------------------------------------------------------ band DFT pins

@pytest.mark.parametrize("M", [1, 2, 7, 12, 97, 360, 1031])
def test_band_dft_matches_library_fft(M):
    rng = np.random.default_rng(M)
    u = rng.standard_normal((3, M)) + 1j * rng.standard_normal((3, M))
    np.testing.assert_allclose(oracle.band_idft(u), np.fft.ifft(u, axis=-1),
                               rtol=0, atol=1e-12 * np.abs(u).max())
    np.testing.assert_allclose(oracle.band_dft(u), np.fft.fft(u, axis=-1),
                               rtol=0, atol=1e-12 * M * np.abs(u).max())


def test_band_dft_against_definition_sums():
    # eq. (1) by explicit double sums with math.cos/math.sin
    M = 11
    rng = np.random.default_rng(3)
    c = rng.standard_normal(M) + 1j * rng.standard_normal(M)
    ref = [sum(c[j] * complex(math.cos(2 * math.pi * k * j / M),
                              -math.sin(2 * math.pi * k * j / M)) for j in range(M))
           for k in range(M)]
    np.testing.assert_allclose(oracle.band_dft(c), ref, atol=1e-13)


# ------------------------------------------------------------ analysis pins

@pytest.mark.parametrize("k0", [5, 11, 20, 27])
def test_cosine_closed_form(k0):
    # x_j = cos(2 pi k0 j / N + phi) has X_{k0} = (N/2) e^{i phi}; each band
    # holding k0 then has c[n] = g_{k0} (N/2) e^{i phi} e^{2 pi i slot(k0) n/M} / M
    # and every other band is zero.
    lay = small_layout()
    N, phi = lay.N, 0.7
    j = np.arange(N)
    x = np.cos(2 * np.pi * k0 * j / N + phi)
    c = oracle.analyse(lay, x)
    hit = 0
    for b, cb in zip(lay.bands, oracle.split_bands(lay, c)):
        if b.k_lo <= k0 <= b.k_hi:
            hit += 1
            g = b.g[k0 - b.k_lo]
            s = (k0 - b.k_c) % b.M
            n = np.arange(b.M)
            ref = g * (N / 2) * np.exp(1j * phi) * np.exp(2j * np.pi * s * n / b.M) / b.M
            np.testing.assert_allclose(cb, ref, atol=1e-12)
            assert np.allclose(np.abs(cb), N * g / (2 * b.M))
        else:
            assert np.abs(cb).max() < 1e-12
    assert hit >= 1


def test_constant_and_alternating_closed_forms():
    lay = small_layout()
    N = lay.N
    c = oracle.analyse(lay, np.ones(N))
    for b, cb in zip(lay.bands, oracle.split_bands(lay, c)):
        if b.kind == DC:
            np.testing.assert_allclose(cb, N / b.M * b.g[0], atol=1e-12)
        elif b.k_lo > 0:
            assert np.abs(cb).max() < 1e-12
    c = oracle.analyse(lay, (-1.0) ** np.arange(N))
    half = lay.half
    for b, cb in zip(lay.bands, oracle.split_bands(lay, c)):
        if b.k_hi == half:
            g = b.g[-1]
            assert np.allclose(np.abs(cb), N * g / b.M, atol=1e-12)
        else:
            assert np.abs(cb).max() < 1e-12


def test_energy_identity():
    # ||c_lambda||^2 = ||u_lambda||^2 / M_lambda (Parseval for F_M^{-1})
    lay = small_layout(N=250, fs=250.0, fmin=4.0, fmax=125.0, B=4)
    x = np.random.default_rng(0).standard_normal(lay.N)
    c = oracle.analyse(lay, x)
    X = np.fft.fft(x)
    lhs = sum(b.M * np.sum(np.abs(cb) ** 2) for b, cb in zip(lay.bands, oracle.split_bands(lay, c)))
    cov = np.zeros(lay.half + 1)
    for b in lay.bands:
        cov[b.k_lo:b.k_hi + 1] += b.g ** 2
    rhs = np.sum(cov * np.abs(X[:lay.half + 1]) ** 2)
    assert lhs == pytest.approx(rhs, rel=1e-12)


def _analysis_matrix_by_sums(lay):
    """T as a C x N complex matrix from explicit sums over the support."""
    N = lay.N
    rows = []
    for b in lay.bands:
        for n in range(b.M):
            row = np.zeros(N, dtype=complex)
            for k, g in zip(b.bins.tolist(), b.g.tolist()):
                s = (k - b.k_c) % b.M
                for j in range(N):
                    row[j] += g * complex(math.cos(2 * math.pi * (s * n / b.M - k * j / N)),
                                          math.sin(2 * math.pi * (s * n / b.M - k * j / N))) / b.M
            rows.append(row)
    return np.array(rows)


@pytest.mark.parametrize("N,fs,fmin,fmax,B", [(32, 32.0, 2.0, 16.0, 2), (50, 50.0, 3.0, 25.0, 3)])
def test_brute_force_matrices(N, fs, fmin, fmax, B):
    lay = oracle.build_layout(fs, fmin, fmax, B, N)
    T = _analysis_matrix_by_sums(lay)
    I = np.eye(N)
    To = oracle.analyse(lay, I).T          # column j = T e_j
    np.testing.assert_allclose(To, T, atol=1e-12)
    # S T = I as a matrix (Sec. 2)
    S_T = oracle.synthesise(lay, oracle.analyse(lay, I))
    np.testing.assert_allclose(S_T, I, atol=1e-12)
    # T^dagger is the transpose of T in the real representation:
    # <T e_j, y>_R = Re(conj(T_{:,j}) . y) = (T^dagger y)_j
    rng = np.random.default_rng(1)
    y = rng.standard_normal(T.shape[0]) + 1j * rng.standard_normal(T.shape[0])
    ref = np.real(np.conj(T).T @ y)
    np.testing.assert_allclose(oracle.adjoint_analysis(lay, y), ref, atol=1e-12)


# ----------------------------------------------- reconstruction and adjoints

@pytest.mark.parametrize("N,fs,fmin,fmax,B", [(64, 64.0, 3.0, 32.0, 3), (250, 250.0, 4.0, 125.0, 4),
                                              (16384, 22050.0, 110.0, 11025.0, 12)])
def test_perfect_reconstruction(N, fs, fmin, fmax, B):
    lay = oracle.build_layout(fs, fmin, fmax, B, N)
    x = np.random.default_rng(N).standard_normal((2, N))
    xr = oracle.synthesise(lay, oracle.analyse(lay, x))
    assert oracle.snr_db(x, xr).min() > 250.0


@pytest.mark.parametrize("N,fs,fmin,fmax,B", [(64, 64.0, 3.0, 32.0, 3), (250, 250.0, 4.0, 125.0, 4),
                                              (16384, 22050.0, 110.0, 11025.0, 12)])
def test_adjoint_identities(N, fs, fmin, fmax, B):
    lay = oracle.build_layout(fs, fmin, fmax, B, N)
    rng = np.random.default_rng(N + 1)
    x = rng.standard_normal((2, N))
    y = rng.standard_normal((2, lay.n_coeffs)) + 1j * rng.standard_normal((2, lay.n_coeffs))
    # <T x, y> = <x, T^dagger y>
    lhs = np.sum(np.real(np.conj(oracle.analyse(lay, x)) * y))
    rhs = np.sum(x * oracle.adjoint_analysis(lay, y))
    assert lhs == pytest.approx(rhs, rel=1e-12)
    # <S y, x> = <y, S^dagger x>
    lhs = np.sum(oracle.synthesise(lay, y) * x)
    rhs = np.sum(np.real(np.conj(y) * oracle.adjoint_synthesis(lay, x)))
    assert lhs == pytest.approx(rhs, rel=1e-12)


def test_synthesis_adjoint_by_sums():
    # S^dagger e_j computed column by column from S itself.
    lay = small_layout(N=32, fs=32.0, fmin=2.0, fmax=16.0, B=2)
    C = lay.n_coeffs
    # real representation of S: columns for Re and Im parts of each coefficient
    Sre = oracle.synthesise(lay, np.eye(C))
    Sim = oracle.synthesise(lay, 1j * np.eye(C))
    x = np.random.default_rng(5).standard_normal(lay.N)
    ref = Sre @ x + 1j * (Sim @ x)
    np.testing.assert_allclose(oracle.adjoint_synthesis(lay, x), ref, atol=1e-12)


def test_band_subset_matches_full_analysis():
    lay = small_layout(N=250, fs=250.0, fmin=4.0, fmax=125.0, B=4)
    x = np.random.default_rng(4).standard_normal((2, lay.N))
    full = oracle.split_bands(lay, oracle.analyse(lay, x))
    sub = oracle.analyse_bands(lay, x, [0, 3, len(lay.bands) - 1])
    for i, v in sub.items():
        np.testing.assert_allclose(v, full[i], atol=1e-13)


def test_direct_and_fft_modes_agree():
    lay = small_layout(N=250, fs=250.0, fmin=4.0, fmax=125.0, B=4)
    x = np.random.default_rng(2).standard_normal(lay.N)
    np.testing.assert_allclose(oracle.analyse(lay, x), oracle.analyse(lay, x, mode="fft"), atol=1e-12)


@settings(max_examples=25, deadline=None)
@given(N=st.integers(8, 200).map(lambda v: 2 * v),
       B=st.integers(1, 8),
       fmin_frac=st.floats(0.01, 0.2),
       fmax_frac=st.floats(0.3, 0.5))
def test_property_reconstruction_and_adjoints(N, B, fmin_frac, fmax_frac):
    fs = 1000.0
    try:
        lay = oracle.build_layout(fs, fmin_frac * fs, fmax_frac * fs, B, N)
    except ValueError:
        return     # an uncovered bin is a legitimate rejection
    rng = np.random.default_rng(N * 31 + B)
    x = rng.standard_normal(N)
    c = oracle.analyse(lay, x)
    assert oracle.snr_db(x, oracle.synthesise(lay, c)) > 200.0
    y = rng.standard_normal(lay.n_coeffs) + 1j * rng.standard_normal(lay.n_coeffs)
    lhs = np.sum(np.real(np.conj(c) * y))
    rhs = np.sum(x * oracle.adjoint_analysis(lay, y))
    assert abs(lhs - rhs) <= 1e-10 * (abs(lhs) + abs(rhs) + 1.0)
    hg = np.zeros(lay.half + 1)
    for b in lay.bands:
        hg[b.k_lo:b.k_hi + 1] += b.h * b.g
    np.testing.assert_allclose(hg, 1.0, atol=1e-12)


# --------------------------------------------------------- explicit band lists

def test_table1_layout_pins():
    # Table 1 and Sec. 4: N = 65,536 at 44.1 kHz, 152 positive bands (8, 8, 8,
    # 16, 16, 16, 16, 32, 32 per octave) plus DC and Nyquist sidebands of
    # lengths 128 and 2048, one length per octave (32 ... 2048) obtained by
    # rounding the octave's widest support up to a power of two, and 132,992
    # coefficients per slice. The lengths here come from that rounding rule
    # applied to the reading's window widths, so they pin the widths.
    fs, N, specs = oracle.table1_specs()
    assert (fs, N) == (44100.0, 65536)
    lay = oracle.build_band_layout(fs, N, specs)
    kinds = [b.kind for b in lay.bands]
    assert kinds == [DC] + [POSITIVE] * 152 + [NYQUIST]
    lengths = [b.M for b in lay.bands[1:-1]]
    table = [(8, 32), (8, 64), (8, 128), (16, 128), (16, 256), (16, 512), (16, 1024), (32, 1024), (32, 2048)]
    assert lengths == [M for n, M in table for _ in range(n)]
    assert (lay.bands[0].M, lay.bands[-1].M) == (128, 2048)
    assert lay.n_coeffs == 132992
    # painless: every support fits its length; every bin covered
    assert all(b.width <= b.M for b in lay.bands)
    assert np.all(lay.a > 0)
    # centres: the table's lowest (43 Hz) and highest (21,810 Hz) to a bin,
    # and each octave's printed range to within 7 % (the spacing inside the
    # resolutions is not stated)
    hz = [b.centre_hz for b in lay.bands[1:-1]]
    assert abs(hz[0] - 43.0) < 44100 / 65536 and abs(hz[-1] - 21810.0) < 44100 / 65536
    ranges = [(43, 81), (88, 165), (180, 337), (345, 666), (695, 1342), (1402, 2708), (2830, 5464),
              (5512, 10905), (11147, 21810)]
    i = 0
    for (n, _), (lo, hi) in zip(table, ranges):
        oc = hz[i:i + n]
        i += n
        assert abs(oc[0] / lo - 1) < 0.07 and abs(oc[-1] / hi - 1) < 0.07
    hg = np.zeros(lay.half + 1)
    for b in lay.bands:
        hg[b.k_lo:b.k_hi + 1] += b.h * b.g
    np.testing.assert_allclose(hg, 1.0, atol=1e-12)


def _padded_specs(N):
    # a small band list with lengths above the support widths, sidebands included
    half = N // 2
    xs = [3.0, 5.5, 8.0, 11.0, 14.5, 18.0]
    specs = [(DC, xs[0], 2.0, 7)]
    specs += [(POSITIVE, x, 3.1, L) for x, L in zip(xs, [0, 9, 8, 13, 8, 11])]
    specs.append((NYQUIST, xs[-1], 3.1, half - 14))
    return specs


def test_padded_band_list_brute_force():
    N = 40
    lay = oracle.build_band_layout(40.0, N, _padded_specs(N))
    assert any(b.M > b.width for b in lay.bands)
    T = _analysis_matrix_by_sums(lay)
    I = np.eye(N)
    np.testing.assert_allclose(oracle.analyse(lay, I).T, T, atol=1e-12)
    np.testing.assert_allclose(oracle.synthesise(lay, oracle.analyse(lay, I)), I, atol=1e-12)
    rng = np.random.default_rng(3)
    y = rng.standard_normal(T.shape[0]) + 1j * rng.standard_normal(T.shape[0])
    np.testing.assert_allclose(oracle.adjoint_analysis(lay, y), np.real(np.conj(T).T @ y), atol=1e-12)
    x = rng.standard_normal(N)
    lhs = np.sum(oracle.synthesise(lay, y) * x)
    rhs = np.sum(np.real(np.conj(y) * oracle.adjoint_synthesis(lay, x)))
    assert lhs == pytest.approx(rhs, rel=1e-12)


def test_zero_padding_doubles_time_resolution():
    # A band spectrum zero-padded from M to 2M slots, frequencies d = k - k_c
    # kept, gives c'[2n] = c[n] / 2: (1/2M) sum u_d e^{2 pi i d 2n / 2M}.
    N = 256
    base = [(DC, 6.0, 3.0, 0)] + [(POSITIVE, 6.0 * 1.5 ** j, 1.5 ** j * 3.0, 0) for j in range(7)]
    base.append((NYQUIST, base[-1][1], base[-1][2], 0))
    lay1 = oracle.build_band_layout(256.0, N, base)
    double = [(k, xi, be, 2 * b.M) for (k, xi, be, _), b in zip(base, lay1.bands)]
    lay2 = oracle.build_band_layout(256.0, N, double)
    x = np.random.default_rng(9).standard_normal(N)
    c1 = oracle.split_bands(lay1, oracle.analyse(lay1, x))
    c2 = oracle.split_bands(lay2, oracle.analyse(lay2, x))
    for a, b in zip(c1, c2):
        np.testing.assert_allclose(b[0::2], a / 2, atol=1e-13)
    # both are frames of the same signal
    assert oracle.snr_db(x, oracle.synthesise(lay2, oracle.analyse(lay2, x))) > 250


def test_table1_reconstruction_and_adjoint():
    fs, N, specs = oracle.table1_specs()
    lay = oracle.build_band_layout(fs, N, specs)
    rng = np.random.default_rng(12)
    x = rng.standard_normal(N)
    c = oracle.analyse(lay, x, mode="fft")
    assert oracle.snr_db(x, oracle.synthesise(lay, c, mode="fft")) > 250
    y = rng.standard_normal(lay.n_coeffs) + 1j * rng.standard_normal(lay.n_coeffs)
    lhs = np.sum(np.real(np.conj(c) * y))
    rhs = np.sum(x * oracle.adjoint_analysis(lay, y, mode="fft"))
    assert lhs == pytest.approx(rhs, rel=1e-11)


def test_band_list_rejections():
    N = 40
    good = _padded_specs(N)
    with pytest.raises(ValueError):          # length below the support width
        oracle.build_band_layout(40.0, N, [good[0], (POSITIVE, 8.0, 3.1, 4)] + good[2:])
    with pytest.raises(ValueError):          # DC not first
        oracle.build_band_layout(40.0, N, good[1:2] + good[0:1] + good[2:])
    with pytest.raises(ValueError):          # uncovered bins
        oracle.build_band_layout(40.0, N, good[:2])


def test_erb_scale_values():
    # Glasberg and Moore (1990): ERB(1 kHz) = 24.7 * 5.37 = 132.639 Hz and
    # 21.4 log10(5.37) = 15.621 ERBs below 1 kHz; ERB(0) = 24.7 Hz
    assert oracle.erb_hz(1000.0) == pytest.approx(132.639, abs=1e-9)
    assert oracle.erb_hz(0.0) == pytest.approx(24.7)
    assert oracle.erb_rate(1000.0) == pytest.approx(15.6214, abs=1e-4)
    # dE/df = 1.0032 / ERB(f) (the scale counts ERBs)
    f = 3000.0
    d = (oracle.erb_rate(f + 1e-3) - oracle.erb_rate(f - 1e-3)) / 2e-3
    assert d * oracle.erb_hz(f) == pytest.approx(21.4 * 4.37 / 1000 / math.log(10) * 24.7, rel=1e-6)


def test_erb_layout_spacing_and_frame():
    fs, N, v = 16000.0, 4000, 2.0
    specs = oracle.erb_specs(fs, N, 50.0, 8000.0, v)
    lay = oracle.build_band_layout(fs, N, specs)
    pos = [b for b in lay.bands if b.kind == POSITIVE]
    rates = np.array([oracle.erb_rate(b.centre_hz) for b in pos])
    # every kept centre sits on the 1/v grid of the ERB-rate scale
    steps = (rates - oracle.erb_rate(50.0)) * v
    np.testing.assert_allclose(steps, np.round(steps), atol=1e-9)
    # half-amplitude width = ERB / v; the next centre lies a fixed ratio of it
    # away: f' - f = (f + 1000/4.37)(10^(1/(21.4 v)) - 1) and
    # ERB(f) = 24.7 (4.37/1000)(f + 1000/4.37)
    for b in pos:
        assert b.beta == pytest.approx(oracle.erb_hz(b.centre_hz) / v * N / fs, rel=1e-12)
    sp = np.diff([b.xi for b in pos])
    w = np.array([b.beta for b in pos[:-1]])
    ratio = (10 ** (1 / (21.4 * v)) - 1) * v / (24.7 * 4.37 / 1000)
    np.testing.assert_allclose(sp / w, ratio, rtol=1e-9)
    assert abs(ratio - 1) < 0.03
    # a painless frame: S T = I, adjoint identity (library-FFT band mode)
    x = np.random.default_rng(21).standard_normal(N)
    c = oracle.analyse(lay, x)
    assert oracle.snr_db(x, oracle.synthesise(lay, c)) > 250
    y = np.random.default_rng(22).standard_normal(lay.n_coeffs) * (1 + 0j)
    assert np.sum(np.real(np.conj(c) * y)) == pytest.approx(np.sum(x * oracle.adjoint_analysis(lay, y)), rel=1e-11)


# ---------------------------------------------------------------- sliced mode

def test_slice_window_partition_of_unity():
    for Ns in (64, 1024, 131072):
        w = oracle.slice_window(Ns)
        H = Ns // 2
        np.testing.assert_allclose(w[:H] + w[H:], 1.0, atol=1e-15)
        assert w[: Ns // 8].max() == 0.0 and w[7 * Ns // 8:].max() == 0.0
        assert np.all(w[3 * Ns // 8:5 * Ns // 8] == 1.0)
        assert w[Ns // 4] == pytest.approx(0.5, abs=1e-15)


def test_sliced_round_trip_and_slices():
    Ns = 256
    lay = oracle.build_layout(1000.0, 20.0, 500.0, 6, Ns)
    n = 1000
    x = np.random.default_rng(9).standard_normal(n)
    c = oracle.sliced_analyse(lay, x)
    J = oracle.slice_count(n, Ns)
    assert c.shape == (J, lay.n_coeffs) and J == math.ceil(n / (Ns // 2)) + 1
    # each slice equals T of the windowed segment of the zero-padded signal
    H = Ns // 2
    xp = np.concatenate([np.zeros(H), x, np.zeros(2 * Ns)])
    w = oracle.slice_window(Ns)
    for s in (0, 3, J - 1):
        np.testing.assert_allclose(c[s], oracle.analyse(lay, w * xp[s * H:s * H + Ns]), atol=1e-12)
    xr = oracle.sliced_synthesise(lay, c, n)
    assert oracle.snr_db(x, xr) > 250.0


def test_metrics():
    x = np.ones(10)
    assert oracle.snr_db(x, x + 0.1) == pytest.approx(20.0)
    assert oracle.rel_l2(np.array([3.0, 4.0 + 1e-3]), np.array([3.0, 4.0])) == pytest.approx(2e-4)


def test_band_metrics():
    # two bands [0, 2) and [2, 5): errors 3e-3 on (3, 4) and 0 on the second
    ref = np.array([[3.0, 4.0, 1.0, 2.0, 2.0]], dtype=np.complex128)
    got = ref.copy()
    got[0, 1] += 5e-3
    got[0, 0] += 0.0
    rb = oracle.band_rel_l2(got, ref, [0, 2])
    assert rb.shape == (1, 2)
    assert rb[0, 0] == pytest.approx(1e-3) and rb[0, 1] == 0.0
    # rms of the row: sqrt((9 + 16 + 1 + 4 + 4) / 5)
    assert oracle.max_err_over_rms(got, ref)[0] == pytest.approx(5e-3 / np.sqrt(34.0 / 5.0))
    # per band: 5e-3 over the first band's rms sqrt(25 / 2); 0 in the second
    bm = oracle.band_max_err_over_rms(got, ref, [0, 2])
    assert bm[0, 0] == pytest.approx(5e-3 / np.sqrt(12.5)) and bm[0, 1] == 0.0
