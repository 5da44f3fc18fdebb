"""Exactly invertible nonstationary-Gabor constant-Q transform for AMD MI355X.

The transform runs in hand-written HIP kernels behind the C ABI declared in
include/nsgcqt.h (libnsgcqt.so, built in-tree by ``build.py``); this package
is its Python binding. ``paper_2609_29119_amd.autograd`` makes analysis and
synthesis differentiable through their explicit adjoints.
"""
from .nsgcqt import (Plan, NsgcqtError, Info, BandInfo, BandSpec, lib, LIB_PATH, table1_layout, erb_layout,
                     BAND_DC, BAND_POSITIVE, BAND_NYQUIST,
                     OP_ANALYSE, OP_SYNTHESISE, OP_ADJ_ANALYSIS, OP_ADJ_SYNTHESIS,
                     WEIGHT_G, WEIGHT_H, WEIGHT_ADJ_ANALYSIS, WEIGHT_ADJ_SYNTHESIS,
                     OK, EINVAL, ENOMEM, EDEVICE, EWORKSPACE, EUNSUPPORTED)

__all__ = ["Plan", "NsgcqtError", "Info", "BandInfo", "BandSpec", "lib", "LIB_PATH", "table1_layout", "erb_layout",
           "BAND_DC", "BAND_POSITIVE", "BAND_NYQUIST",
           "OP_ANALYSE", "OP_SYNTHESISE", "OP_ADJ_ANALYSIS", "OP_ADJ_SYNTHESIS",
           "WEIGHT_G", "WEIGHT_H", "WEIGHT_ADJ_ANALYSIS", "WEIGHT_ADJ_SYNTHESIS",
           "OK", "EINVAL", "ENOMEM", "EDEVICE", "EWORKSPACE", "EUNSUPPORTED"]
