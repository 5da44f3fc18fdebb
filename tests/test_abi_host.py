"""CPU checks of the C-ABI library: exports, layout, tables, error paths.

No compute call runs here (there is no GPU); plans are created host-only.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import workloads
from oracle.layout import DC, NYQUIST, POSITIVE

pn = pytest.importorskip("paper_2609_29119_amd")
from paper_2609_29119_amd import nsgcqt as nb  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(nb.LIB_PATH):
        pytest.fail("libnsgcqt.so is not built; run python -m paper_2609_29119_amd.build")
    return nb.lib()


def header_functions():
    text = open(os.path.join(ROOT, "include", "nsgcqt.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|int64_t|const char\*)\s+(nsgcqt_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(nb.EXPORTS) == names


def _host_plan(w, n=None, batch=None):
    return nb.Plan(w.fs, w.fmin, w.fmax, w.bins_per_octave, n or w.n_samples,
                   batch or w.batch, device=False)


LAYOUT_CASES = [(name, None) for name in ("tiny", "single", "train", "stress")] + [("long", 131072)]


@pytest.mark.parametrize("name,n", LAYOUT_CASES)
def test_integer_layout_identical_to_oracle(lib, name, n):
    w = workloads.WORKLOADS[name]
    N = n or w.n_samples
    lay = oracle.build_layout(w.fs, w.fmin, w.fmax, w.bins_per_octave, N)
    if n:
        p = nb.Plan.sliced(w.fs, w.fmin, w.fmax, w.bins_per_octave, N, 4, device=False)
    else:
        p = _host_plan(w)
    assert p.n_bands == len(lay.bands)
    assert p.n_coeffs == lay.n_coeffs
    assert p.info.packed_len == N // 2
    assert p.info.max_band_len == max(b.M for b in lay.bands)
    for i, (ob, cb) in enumerate(zip(lay.bands, p.bands())):
        assert (cb.kind, cb.k_lo, cb.k_hi, cb.k_centre, cb.length, cb.offset) == \
               (ob.kind, ob.k_lo, ob.k_hi, ob.k_c, ob.M, ob.offset), i
        assert cb.xi == ob.xi and cb.beta == ob.beta


@pytest.mark.parametrize("name", ["tiny", "single", "stress"])
def test_weight_tables_match_oracle(lib, name):
    w = workloads.WORKLOADS[name]
    lay = oracle.build_layout(*w.plan_args)
    p = _host_plan(w)
    N, half = lay.N, lay.half
    g = np.concatenate([b.g for b in lay.bands])
    h = np.concatenate([b.h for b in lay.bands])
    k = np.concatenate([b.bins for b in lay.bands])
    M = np.concatenate([np.full(b.M, b.M) for b in lay.bands])
    d = np.where((k == 0) | (k == half), 1.0, 2.0)
    ref = {nb.WEIGHT_G: g, nb.WEIGHT_H: h, nb.WEIGHT_ADJ_ANALYSIS: N / (d * M) * g,
           nb.WEIGHT_ADJ_SYNTHESIS: M * d / N * h}
    for which, r in ref.items():
        got = p.weights(which).astype(np.float64)
        np.testing.assert_allclose(got, r, rtol=1e-7, atol=1e-30)


def _packed_eval(p, lay, x):
    """Evaluate the packed factorisation (eqs. 5-10) in fp64 with the
    library's band records and weight tables."""
    N, L = lay.N, lay.N // 2
    z = x[0::2] + 1j * x[1::2]                 # eq. 5
    Z = np.fft.fft(z)
    om = np.exp(-2j * np.pi * np.arange(L + 1) / N)
    g = p.weights(nb.WEIGHT_G).astype(np.float64)
    hw = p.weights(nb.WEIGHT_H).astype(np.float64)
    C = p.n_coeffs
    c = np.zeros(C, complex)
    for b in p.bands():
        k = np.arange(b.k_lo, b.k_hi + 1)
        a = k % L
        W = b.k_hi - b.k_lo + 1                # support width (<= length)
        u = 0.5 * g[b.offset:b.offset + W] * ((1 - 1j * om[k]) * Z[a] + (1 + 1j * om[k]) * np.conj(Z[(-a) % L]))
        v = np.zeros(b.length, complex)
        v[(k - b.k_centre) % b.length] = u     # eq. 7 router, then eq. 8
        c[b.offset:b.offset + b.length] = np.fft.ifft(v)
    X = np.zeros(L + 1, complex)
    for b in p.bands():
        k = np.arange(b.k_lo, b.k_hi + 1)
        U = np.fft.fft(c[b.offset:b.offset + b.length])
        X[k] += hw[b.offset:b.offset + len(k)] * U[(k - b.k_centre) % b.length]
    X[0], X[L] = X[0].real, X[L].real
    q = np.arange(L)
    Zs = 0.5 * ((1 + 1j * np.conj(om[q])) * X[q] + (1 - 1j * np.conj(om[q])) * np.conj(X[L - q]))   # eq. 9
    zr = np.fft.ifft(Zs)
    xr = np.empty(N)
    xr[0::2], xr[1::2] = zr.real, zr.imag     # P^{-1}
    return c, xr


@pytest.mark.parametrize("N,fs,fmin,fmax,B", [(500, 250.0, 4.0, 125.0, 4), (16384, 22050.0, 110.0, 11025.0, 12)])
def test_library_tables_drive_packed_path(lib, N, fs, fmin, fmax, B):
    lay = oracle.build_layout(fs, fmin, fmax, B, N)
    p = nb.Plan(fs, fmin, fmax, B, N, 1, device=False)
    x = workloads.white(7, 1, N)[0].astype(np.float64)
    c, xr = _packed_eval(p, lay, x)
    # the fp32 tables limit agreement to about 1e-7
    assert oracle.rel_l2(c, oracle.analyse(lay, x)) < 3e-7
    assert oracle.snr_db(x, xr) > 130.0


def test_info_and_workspace(lib):
    w = workloads.WORKLOADS["stress"]
    p = _host_plan(w)
    i = p.info
    L, C, b = w.n_samples // 2, i.total_coeffs, w.batch
    assert i.ws_analyse >= 16 * L * b
    assert i.ws_synthesise >= 8 * C * b + 8 * L * b
    assert i.device_tables == 0 and i.table_bytes == 0
    assert i.max_overlap == 3 and i.max_fanout == 6
    names = [n for n, _ in p.stage_info(nb.OP_ANALYSE)]
    assert names[:2] == ["fft_fwd_a", "fft_fwd_b"] and all(n.startswith("band_analysis") for n in names[2:])
    tot = sum(b_ for _, b_ in p.stage_info(nb.OP_ANALYSE))
    assert tot == pytest.approx((16 + 16 + 8) * L * b + 8 * C * b)


def _status(fn, *args):
    h = ctypes.c_void_p()
    return fn(ctypes.byref(h), *args), h


@pytest.mark.parametrize("args", [
    (22050.0, 110.0, 11025.0, 12, 16383, 1),     # odd N
    (22050.0, 110.0, 11025.0, 12, 2, 1),         # N < 4
    (0.0, 110.0, 11025.0, 12, 16384, 1),         # fs
    (22050.0, 0.0, 11025.0, 12, 16384, 1),       # fmin <= 0
    (22050.0, 11025.0, 11025.0, 12, 16384, 1),   # fmin >= fs/2
    (22050.0, 110.0, 100.0, 12, 16384, 1),       # fmax < fmin
    (22050.0, 110.0, 11025.0, 0, 16384, 1),      # bins per octave
    (22050.0, 110.0, 11025.0, 12, 16384, 0),     # batch
])
def test_invalid_parameters(lib, args):
    st, h = _status(lib.nsgcqt_plan_create_host, *args)
    assert st == nb.EINVAL and not h.value
    assert lib.nsgcqt_last_error()


def test_empty_bands_dropped_identically(lib):
    # 48 bins per octave at N = 256 gives low bands narrower than one bin;
    # both implementations must drop the same empty bands and keep coverage
    args = (8000.0, 40.0, 4000.0, 48, 256)
    lay = oracle.build_layout(*args)
    p = nb.Plan(*args, 1, device=False)
    import math
    K = sum(1 for j in range(10000) if 40.0 * 2.0 ** (j / 48) < 4000.0)
    assert len(lay.bands) < K + 2            # some were dropped
    assert p.n_bands == len(lay.bands)
    assert [(b.k_lo, b.k_hi) for b in p.bands()] == [(b.k_lo, b.k_hi) for b in lay.bands]
    assert np.all(lay.a > 0)


def _prime_factors(n):
    out, m, d = [], n, 2
    while d * d <= m:
        while m % d == 0:
            out.append(d)
            m //= d
        d += 1
    if m > 1:
        out.append(m)
    return out


@pytest.mark.parametrize("name", ["stress", "train"])
def test_band_transform_choice(name):
    """Per band, a direct transform of length M (prime factors up to the
    largest Stockham radix, 257) or Bluestein over P >= 2M - 1 with prime
    factors up to 13; the choice does not depend on the batch size."""
    w = workloads.WORKLOADS[name]
    p1 = nb.Plan(*w.plan_args, batch=1, device=False)
    pb = nb.Plan(*w.plan_args, batch=w.batch, device=False)
    b1, bb = p1.bands(), pb.bands()
    assert [(b.fft_len, b.bluestein) for b in b1] == [(b.fft_len, b.bluestein) for b in bb]
    for b in bb:
        if b.bluestein:
            assert b.fft_len >= 2 * b.length - 1
            assert max(_prime_factors(b.fft_len)) <= 13
        else:
            assert b.fft_len == b.length
            assert max(_prime_factors(b.length) + [1]) <= 257
    assert all(b.bluestein for b in bb if max(_prime_factors(b.length) + [1]) > 257)
    assert any(b.bluestein for b in bb) and any(not b.bluestein for b in bb)


def test_size_limit(lib):
    # rows are addressed with 32-bit byte offsets: N below 2^29
    st, _ = _status(lib.nsgcqt_plan_create_host, 44100.0, 30.0, 22050.0, 12, 1 << 29, 1)
    assert st == nb.EUNSUPPORTED


def test_unsupported_packed_length(lib):
    # L = 2 * 263 has a prime factor above the largest Stockham radix (257)
    st, _ = _status(lib.nsgcqt_plan_create_host, 1052.0, 4.0, 526.0, 4, 1052, 1)
    assert st == nb.EUNSUPPORTED
    # L = 2 * 67 runs its prime factor as a matrix-core stage
    st, _ = _status(lib.nsgcqt_plan_create_host, 268.0, 4.0, 134.0, 4, 268, 1)
    assert st == nb.OK


def test_sliced_plan_rules(lib):
    st, _ = _status(lib.nsgcqt_sliced_plan_create_host, 48000.0, 20.0, 24000.0, 96, 131076, 4)
    assert st == nb.EINVAL     # not a multiple of 8
    p = nb.Plan.sliced(48000.0, 20.0, 24000.0, 96, 131072, 4, device=False)
    assert p.slice_count(2880000) == oracle.slice_count(2880000, 131072) == 45
    assert p.slice_count(1) == 2


def test_compute_calls_reject_bad_arguments(lib):
    w = workloads.WORKLOADS["tiny"]
    p = _host_plan(w)
    h = p._h
    buf = ctypes.c_void_p(16)      # never dereferenced: every call fails validation first
    need = p.info.ws_analyse
    assert lib.nsgcqt_analyse(None, buf, buf, buf, need, None) == nb.EINVAL
    assert lib.nsgcqt_analyse(h, None, buf, buf, need, None) == nb.EINVAL
    assert lib.nsgcqt_analyse(h, buf, buf, buf, need - 1, None) == nb.EWORKSPACE
    assert lib.nsgcqt_synthesise(h, buf, buf, buf, p.info.ws_synthesise - 1, None) == nb.EWORKSPACE
    assert lib.nsgcqt_adjoint(h, 7, buf, buf, buf, need, None) == nb.EINVAL
    assert lib.nsgcqt_sliced_analyse(h, buf, 100, buf, buf, need, None) == nb.EINVAL   # not sliced
    # a host-only plan with valid arguments has no device tables
    assert lib.nsgcqt_analyse(h, buf, buf, buf, need, None) == nb.EINVAL
    assert b"host-only" in lib.nsgcqt_last_error()
    # the allocation-free analysis: the same checks, and plans whose workspace
    # exceeds its device array are refused before any device call
    assert lib.nsgcqt_analyse_noalloc(None, buf, buf, None) == nb.EINVAL
    assert lib.nsgcqt_analyse_noalloc(h, buf, buf, None) == nb.EINVAL
    assert b"host-only" in lib.nsgcqt_last_error()
    big = _host_plan(workloads.WORKLOADS["stress"])
    assert big.info.ws_analyse > nb.NOALLOC_SCRATCH_BYTES
    assert lib.nsgcqt_analyse_noalloc(big._h, buf, buf, None) == nb.EWORKSPACE
    assert str(nb.NOALLOC_SCRATCH_BYTES).encode() in lib.nsgcqt_last_error()
    # complex64 data, pair-wise signals and the workspace need 8-byte alignment
    odd = ctypes.c_void_p(20)
    for args in ((odd, buf, buf), (buf, odd, buf), (buf, buf, odd)):
        assert lib.nsgcqt_analyse(h, *args, need, None) == nb.EINVAL
        assert b"aligned" in lib.nsgcqt_last_error()
    assert lib.nsgcqt_synthesise(h, odd, buf, buf, p.info.ws_synthesise, None) == nb.EINVAL
    assert b"aligned" in lib.nsgcqt_last_error()
    # the sliced calls read and write signals sample by sample: 4 bytes do
    sp = nb.Plan.sliced(22050.0, 110.0, 11025.0, 12, 4096, 2, device=False)
    sh, sneed = sp._h, max(sp.info.ws_analyse, sp.info.ws_synthesise)
    assert lib.nsgcqt_sliced_analyse(sh, odd, 100, buf, buf, sneed, None) == nb.EINVAL
    assert b"host-only" in lib.nsgcqt_last_error()
    assert lib.nsgcqt_sliced_synthesise(sh, buf, 100, odd, buf, sneed, None) == nb.EINVAL
    assert b"host-only" in lib.nsgcqt_last_error()
    assert lib.nsgcqt_sliced_analyse(sh, buf, 100, odd, buf, sneed, None) == nb.EINVAL
    assert b"aligned" in lib.nsgcqt_last_error()
    assert lib.nsgcqt_band_info(h, p.n_bands, ctypes.byref(nb.BandInfo())) == nb.EINVAL
    assert lib.nsgcqt_plan_weights(h, 9, buf, 1 << 20) == nb.EINVAL
    assert lib.nsgcqt_plan_destroy(None) == nb.OK


# ------------------------------------------------------ explicit band lists

def test_table1_preset_identical_to_oracle(lib):
    fs, N, specs = nb.table1_layout()
    ofs, oN, ospecs = oracle.table1_specs()
    assert (fs, N) == (ofs, oN)
    assert [tuple(b) for b in specs] == [tuple(b) for b in ospecs]
    p = nb.Plan.from_bands(fs, N, specs, batch=4, device=False)
    lay = oracle.build_band_layout(fs, N, ospecs)
    assert p.n_bands == 154 and p.n_coeffs == lay.n_coeffs == 132992
    for i, (ob, cb) in enumerate(zip(lay.bands, p.bands())):
        assert (cb.kind, cb.k_lo, cb.k_hi, cb.k_centre, cb.length, cb.offset) == \
               (ob.kind, ob.k_lo, ob.k_hi, ob.k_c, ob.M, ob.offset), i
    # power-of-two lengths: every band runs a direct transform
    assert not any(b.bluestein for b in p.bands())
    assert p.info.max_overlap == 3


def _band_list_case():
    # padded lengths, a length with a prime factor above 257 (Bluestein) and
    # a Nyquist band longer than N / 2
    N, fs = 1200, 1200.0
    xs = [8.0 * 1.35 ** j for j in range(12)]
    specs = [(nb.BAND_DC, xs[0], xs[0] * 0.35, 16)]
    lens = [0, 8, 0, 20, 0, 31, 40, 0, 67, 0, 2 * 263, 160]
    specs += [(nb.BAND_POSITIVE, x, x * 0.35, L, x) for x, L in zip(xs, lens)]
    specs.append((nb.BAND_NYQUIST, xs[-1], xs[-1] * 0.35, 1500))
    return fs, N, specs


def test_band_list_layout_and_weights_match_oracle(lib):
    fs, N, specs = _band_list_case()
    lay = oracle.build_band_layout(fs, N, specs)
    p = nb.Plan.from_bands(fs, N, specs, batch=2, device=False)
    assert p.n_coeffs == lay.n_coeffs
    for i, (ob, cb) in enumerate(zip(lay.bands, p.bands())):
        assert (cb.kind, cb.k_lo, cb.k_hi, cb.k_centre, cb.length, cb.offset) == \
               (ob.kind, ob.k_lo, ob.k_hi, ob.k_c, ob.M, ob.offset), i
    assert any(b.bluestein for b in p.bands())
    half = N // 2
    ref = {w: np.zeros(lay.n_coeffs) for w in (nb.WEIGHT_G, nb.WEIGHT_H, nb.WEIGHT_ADJ_ANALYSIS,
                                               nb.WEIGHT_ADJ_SYNTHESIS)}
    for b in lay.bands:
        k = b.bins
        d = np.where((k == 0) | (k == half), 1.0, 2.0)
        sl = slice(b.offset, b.offset + b.width)
        ref[nb.WEIGHT_G][sl] = b.g
        ref[nb.WEIGHT_H][sl] = b.h
        ref[nb.WEIGHT_ADJ_ANALYSIS][sl] = N / (d * b.M) * b.g
        ref[nb.WEIGHT_ADJ_SYNTHESIS][sl] = b.M * d / N * b.h
    for which, r in ref.items():
        np.testing.assert_allclose(p.weights(which).astype(np.float64), r, rtol=1e-7, atol=1e-30)
    # the library's tables drive the packed path (eqs. 5-10) to the oracle
    x = workloads.white(8, 1, N)[0].astype(np.float64)
    c, xr = _packed_eval(p, lay, x)
    assert oracle.rel_l2(c, oracle.analyse(lay, x)) < 3e-7
    assert oracle.snr_db(x, xr) > 130.0


def _spec_status(lib, fs, N, specs, batch=1):
    arr = (nb.BandSpec * max(1, len(specs)))(*[nb.BandSpec(*b) for b in specs])
    h = ctypes.c_void_p()
    st = lib.nsgcqt_plan_create_bands_host(ctypes.byref(h), fs, N, batch, len(specs), arr)
    if h.value:
        lib.nsgcqt_plan_destroy(h)
    return st, h


def test_band_list_rejections(lib):
    fs, N, specs = _band_list_case()
    assert _spec_status(lib, fs, N, specs)[0] == nb.OK
    bad = {
        "length below width": specs[:3] + [(nb.BAND_POSITIVE, specs[3][1], specs[3][2], 2)] + specs[4:],
        "DC not first": specs[1:2] + specs[0:1] + specs[2:],
        "Nyquist not last": specs[:-2] + specs[-1:] + specs[-2:-1],
        "beta <= 0": specs[:2] + [(nb.BAND_POSITIVE, specs[2][1], 0.0, 0)] + specs[3:],
        "kind": specs[:2] + [(5, specs[2][1], specs[2][2], 0)] + specs[3:],
        "empty support": specs[:2] + [(nb.BAND_POSITIVE, 10.5, 0.4, 0)] + specs[2:],
        "uncovered": specs[:3],
        "negative length": specs[:2] + [(nb.BAND_POSITIVE, specs[2][1], specs[2][2], -1)] + specs[3:],
        "nan centre": specs[:2] + [(nb.BAND_POSITIVE, float("nan"), specs[2][2], 0)] + specs[3:],
    }
    for what, sp in bad.items():
        st, h = _spec_status(lib, fs, N, sp)
        assert st == nb.EINVAL and not h.value, what
    assert _spec_status(lib, fs, N, [])[0] == nb.EINVAL
    assert _spec_status(lib, fs, N + 1, specs)[0] == nb.EINVAL
    assert _spec_status(lib, fs, N, specs, batch=0)[0] == nb.EINVAL
    # bands covering one bin that are not adjacent in the list
    swapped = specs[:4] + [specs[5], specs[4]] + specs[6:]
    assert _spec_status(lib, fs, N, swapped)[0] == nb.EUNSUPPORTED
    n = ctypes.c_int()
    assert lib.nsgcqt_layout_table1(None, 0, None, None, None) == nb.EINVAL
    assert lib.nsgcqt_layout_table1((nb.BandSpec * 10)(), 10, ctypes.byref(n), None, None) == nb.EINVAL
    assert n.value == 154


def test_erb_preset_identical_to_oracle(lib):
    args = (16000.0, 32000, 50.0, 8000.0, 2.0)
    specs = nb.erb_layout(*args)
    ospecs = oracle.erb_specs(*args)
    assert len(specs) == len(ospecs)
    for a, b in zip(specs, ospecs):
        assert a[0] == b[0] and a[3] == b[3]
        np.testing.assert_allclose(a[1:3] + a[4:], b[1:3] + b[4:], rtol=1e-13)
    p = nb.Plan.from_bands(16000.0, 32000, specs, batch=1, device=False)
    lay = oracle.build_band_layout(16000.0, 32000, ospecs)
    assert [(b.k_lo, b.k_hi, b.k_centre, b.length) for b in p.bands()] == \
           [(b.k_lo, b.k_hi, b.k_c, b.M) for b in lay.bands]
    n = ctypes.c_int()
    assert lib.nsgcqt_layout_erb(16000.0, 32000, 50.0, 8000.0, 0.0, None, 0, ctypes.byref(n)) == nb.EINVAL
    assert lib.nsgcqt_layout_erb(16000.0, 32000, 9000.0, 9500.0, 1.0, None, 0, ctypes.byref(n)) == nb.EINVAL


def test_sliced_band_list_plan(lib):
    fs, N, specs = nb.table1_layout()
    p = nb.Plan.sliced_from_bands(fs, N, specs, 8, device=False)
    assert p.info.sliced == 1 and p.n_coeffs == 132992
    assert p.slice_count(2646000) == oracle.slice_count(2646000, N)
    arr = (nb.BandSpec * len(specs))(*[nb.BandSpec(*b) for b in specs])
    h = ctypes.c_void_p()
    # a slice length that is not a multiple of 8
    assert lib.nsgcqt_sliced_plan_create_bands_host(ctypes.byref(h), fs, N + 2, 8, len(specs), arr) == nb.EINVAL
    assert not h.value


def test_coarse_layouts_of_long_signals_build(lib):
    # bands of a coarse layout over a long signal overlap by more than 2^15
    # coefficients; the plan switches to wide overlap-add records
    for args in [(48000.0, 20.0, 24000.0, 12, 2880000), (44100.0, 30.0, 22050.0, 12, 1323000)]:
        lay = oracle.build_layout(*args)
        p = nb.Plan(*args, 1, device=False)
        assert p.n_coeffs == lay.n_coeffs



def test_stage_order_follows_the_launch_schedule(lib):
    # band phases that fill the GPU launch by bucket in ascending transform
    # size; phases of small launches with enough work fan out and are
    # enqueued longest first
    stress = [n for n, _ in _host_plan(workloads.WORKLOADS["stress"]).stage_info(nb.OP_ANALYSE)]
    assert stress[2:] == ["band_analysis_64x8", "band_analysis_256x8", "band_analysis_256x16"]
    train = _host_plan(workloads.WORKLOADS["train"])
    an = [n for n, _ in train.stage_info(nb.OP_ANALYSE)]
    assert an[2:] == ["band_analysis_1024x16", "band_analysis_512x16", "band_analysis_256x16",
                      "band_analysis_256x8", "band_analysis_64x8"]
    syn = [n for n, _ in train.stage_info(nb.OP_SYNTHESISE)]
    assert syn == [n.replace("analysis", "synthesis") for n in an[2:]] + ["fft_inv_a_overlap_add", "fft_inv_b"]


def test_sliced_stage_info_lists_one_chunk(lib):
    # a sliced plan reports the kernels of one chunk of slices: the analysis
    # chain, and the synthesis chain followed by the overlap-add
    w = workloads.WORKLOADS["long"]
    sp = nb.Plan.sliced(w.fs, w.fmin, w.fmax, w.bins_per_octave, w.slice_len, 16, device=False)
    plain = nb.Plan(w.fs, w.fmin, w.fmax, w.bins_per_octave, w.slice_len, 16, device=False)
    an, syn = sp.stage_info(nb.OP_ANALYSE), sp.stage_info(nb.OP_SYNTHESISE)
    assert an == plain.stage_info(nb.OP_ANALYSE)
    assert syn[:-1] == plain.stage_info(nb.OP_SYNTHESISE)
    assert syn[-1] == ("sliced_overlap_add", 6.0 * w.slice_len * 16)
    for op in (nb.OP_ADJ_ANALYSIS, nb.OP_ADJ_SYNTHESIS):
        assert lib.nsgcqt_stage_info(sp._h, op, -1, None, 0, None) == nb.EINVAL


def test_missing_library_fails_loudly():
    # without the built library there is no fallback: loading it and making a
    # plan both raise (run in a child so this process keeps its handle)
    import subprocess
    import sys
    code = (
        "import paper_2609_29119_amd.nsgcqt as nb\n"
        "nb.LIB_PATH = '/nonexistent/libnsgcqt.so'\n"
        "for f in (nb.lib, lambda: nb.Plan(22050.0, 110.0, 11025.0, 12, 16384, 1, device=False)):\n"
        "    try:\n"
        "        f()\n"
        "    except RuntimeError as e:\n"
        "        assert 'missing' in str(e)\n"
        "    else:\n"
        "        raise SystemExit('no error')\n"
        "print('raised')\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120, cwd=root)
    assert r.returncode == 0 and "raised" in r.stdout, (r.stdout, r.stderr)
