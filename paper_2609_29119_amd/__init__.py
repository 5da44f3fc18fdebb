"""Exactly invertible nonstationary-Gabor constant-Q transform for AMD MI355X.

The transform runs in hand-written HIP kernels behind the C ABI declared in
include/nsgcqt.h (libnsgcqt.so, built in-tree by ``build.py``); this package
is its Python binding.
"""
from .nsgcqt import (Plan, NsgcqtError, Info, BandInfo, lib, LIB_PATH,
                     OP_ANALYSE, OP_SYNTHESISE, OP_ADJ_ANALYSIS, OP_ADJ_SYNTHESIS,
                     WEIGHT_G, WEIGHT_H, WEIGHT_ADJ_ANALYSIS, WEIGHT_ADJ_SYNTHESIS,
                     OK, EINVAL, ENOMEM, EDEVICE, EWORKSPACE, EUNSUPPORTED)

__all__ = ["Plan", "NsgcqtError", "Info", "BandInfo", "lib", "LIB_PATH",
           "OP_ANALYSE", "OP_SYNTHESISE", "OP_ADJ_ANALYSIS", "OP_ADJ_SYNTHESIS",
           "WEIGHT_G", "WEIGHT_H", "WEIGHT_ADJ_ANALYSIS", "WEIGHT_ADJ_SYNTHESIS",
           "OK", "EINVAL", "ENOMEM", "EDEVICE", "EWORKSPACE", "EUNSUPPORTED"]
