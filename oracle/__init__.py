"""fp64 CPU oracle for the invertible nonstationary-Gabor constant-Q transform.

TEST INFRASTRUCTURE ONLY. This package is the slow, plain reference against
which the GPU library is checked. Only the test suite, the smoke check and the
CPU-baseline leg of the benchmark may import it; the library itself never
does, and nothing here is shared with the GPU path (no kernels, tables,
helpers or constants).

Everything follows the plain definitions of Sec. 2 of the paper:
  * ``layout``  - band layout, spectral windows g, aggregate weight a and dual
                  windows h (Sec. 2, painless case);
  * ``nsgt``    - analysis T (eqs. 2-3), synthesis S (eq. 4) and the real
                  adjoints of both (Sec. 3.2), each built from a full-length
                  DFT, selection/windowing/reordering and a direct DFT per band;
  * ``sliced``  - the overlapping-slice mode of Sec. 4;
  * ``metrics`` - reconstruction SNR (Sec. 5.1), relative L2 error (per
                  signal and per band) and an element-wise error bound.

Parity status of each function is stated in its module header.
"""
from .layout import (Band, Layout, build_layout, build_band_layout, table1_specs, erb_specs, erb_hz,
                     erb_rate)
from .nsgt import (analyse, analyse_bands, synthesise, adjoint_analysis, adjoint_synthesis,
                   band_idft, band_dft, split_bands)
from .sliced import slice_window, slice_count, sliced_analyse, sliced_synthesise
from .metrics import snr_db, rel_l2, band_rel_l2, max_err_over_rms, band_max_err_over_rms

__all__ = [
    "Band", "Layout", "build_layout", "build_band_layout", "table1_specs", "erb_specs", "erb_hz", "erb_rate",
    "analyse", "analyse_bands", "synthesise", "adjoint_analysis", "adjoint_synthesis",
    "band_idft", "band_dft", "split_bands",
    "slice_window", "slice_count", "sliced_analyse", "sliced_synthesise",
    "snr_db", "rel_l2", "band_rel_l2", "max_err_over_rms", "band_max_err_over_rms",
]
