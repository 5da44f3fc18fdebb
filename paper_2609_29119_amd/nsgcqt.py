"""ctypes binding of libnsgcqt.so.

Argument marshalling only: every step of the transform runs in the library's
HIP kernels. torch is used for device memory and streams. The library must be
built first (``python -m paper_2609_29119_amd.build``); importing the binding
does not build or fall back to anything.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnsgcqt.so")

OK, EINVAL, ENOMEM, EDEVICE, EWORKSPACE, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
OP_ANALYSE, OP_SYNTHESISE, OP_ADJ_ANALYSIS, OP_ADJ_SYNTHESIS = 0, 1, 2, 3
BAND_DC, BAND_POSITIVE, BAND_NYQUIST = 0, 1, 2
WEIGHT_G, WEIGHT_H, WEIGHT_ADJ_ANALYSIS, WEIGHT_ADJ_SYNTHESIS = 0, 1, 2, 3

_STATUS = {OK: "OK", EINVAL: "EINVAL", ENOMEM: "ENOMEM", EDEVICE: "EDEVICE",
           EWORKSPACE: "EWORKSPACE", EUNSUPPORTED: "EUNSUPPORTED"}

EXPORTS = [
    "nsgcqt_plan_create", "nsgcqt_plan_create_host", "nsgcqt_sliced_plan_create",
    "nsgcqt_sliced_plan_create_host", "nsgcqt_plan_destroy", "nsgcqt_plan_info",
    "nsgcqt_band_info", "nsgcqt_plan_weights", "nsgcqt_analyse", "nsgcqt_synthesise",
    "nsgcqt_adjoint", "nsgcqt_sliced_count", "nsgcqt_sliced_analyse",
    "nsgcqt_sliced_synthesise", "nsgcqt_set_stage_events", "nsgcqt_stage_info",
    "nsgcqt_last_error", "nsgcqt_plan_create_bands", "nsgcqt_plan_create_bands_host",
    "nsgcqt_layout_table1", "nsgcqt_layout_erb", "nsgcqt_sliced_plan_create_bands",
    "nsgcqt_sliced_plan_create_bands_host", "nsgcqt_analyse_noalloc",
]
NOALLOC_SCRATCH_BYTES = 64 << 20     # NSGCQT_NOALLOC_SCRATCH_BYTES


class NsgcqtError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class Info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "n_bands", "batch", "n_samples", "packed_len", "total_coeffs", "max_band_len",
        "max_fanout", "max_overlap", "sliced", "ws_analyse", "ws_synthesise",
        "ws_adjoint_analysis", "ws_adjoint_synthesis", "table_bytes", "device_tables")]


class BandInfo(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int64), ("k_lo", ctypes.c_int64), ("k_hi", ctypes.c_int64),
                ("k_centre", ctypes.c_int64), ("length", ctypes.c_int64), ("offset", ctypes.c_int64),
                ("centre_hz", ctypes.c_double), ("xi", ctypes.c_double), ("beta", ctypes.c_double),
                ("fft_len", ctypes.c_int64), ("bluestein", ctypes.c_int64)]


class BandSpec(ctypes.Structure):
    """One band of an explicit layout: kind, centre xi and half-width beta in
    bins, length M (0: the support width), centre in Hz (reported only)."""
    _fields_ = [("kind", ctypes.c_int32), ("xi", ctypes.c_double), ("beta", ctypes.c_double),
                ("length", ctypes.c_int64), ("centre_hz", ctypes.c_double)]

    def as_tuple(self):
        return (int(self.kind), float(self.xi), float(self.beta), int(self.length), float(self.centre_hz))


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_29119_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, D, I, V = ctypes.c_void_p, ctypes.c_int64, ctypes.c_double, ctypes.c_int, ctypes.c_void_p
    pp = ctypes.POINTER(ctypes.c_void_p)
    sig = {
        "nsgcqt_plan_create": [pp, D, D, D, I, I64, I],
        "nsgcqt_plan_create_host": [pp, D, D, D, I, I64, I],
        "nsgcqt_sliced_plan_create": [pp, D, D, D, I, I64, I],
        "nsgcqt_sliced_plan_create_host": [pp, D, D, D, I, I64, I],
        "nsgcqt_plan_destroy": [P],
        "nsgcqt_plan_info": [P, ctypes.POINTER(Info)],
        "nsgcqt_band_info": [P, I, ctypes.POINTER(BandInfo)],
        "nsgcqt_plan_weights": [P, I, V, ctypes.c_size_t],
        "nsgcqt_analyse": [P, V, V, V, ctypes.c_size_t, V],
        "nsgcqt_analyse_noalloc": [P, V, V, V],
        "nsgcqt_synthesise": [P, V, V, V, ctypes.c_size_t, V],
        "nsgcqt_adjoint": [P, I, V, V, V, ctypes.c_size_t, V],
        "nsgcqt_sliced_count": [P, I64],
        "nsgcqt_sliced_analyse": [P, V, I64, V, V, ctypes.c_size_t, V],
        "nsgcqt_sliced_synthesise": [P, V, I64, V, V, ctypes.c_size_t, V],
        "nsgcqt_set_stage_events": [P, ctypes.POINTER(ctypes.c_void_p), I],
        "nsgcqt_stage_info": [P, I, I, ctypes.c_char_p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_double)],
        "nsgcqt_last_error": [],
        "nsgcqt_plan_create_bands": [pp, D, I64, I, I, ctypes.POINTER(BandSpec)],
        "nsgcqt_plan_create_bands_host": [pp, D, I64, I, I, ctypes.POINTER(BandSpec)],
        "nsgcqt_sliced_plan_create_bands": [pp, D, I64, I, I, ctypes.POINTER(BandSpec)],
        "nsgcqt_sliced_plan_create_bands_host": [pp, D, I64, I, I, ctypes.POINTER(BandSpec)],
        "nsgcqt_layout_table1": [ctypes.POINTER(BandSpec), I, ctypes.POINTER(ctypes.c_int),
                                 ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)],
        "nsgcqt_layout_erb": [D, I64, D, D, D, ctypes.POINTER(BandSpec), I, ctypes.POINTER(ctypes.c_int)],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    L.nsgcqt_sliced_count.restype = ctypes.c_int64
    L.nsgcqt_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status):
    if status != OK:
        raise NsgcqtError(status, lib().nsgcqt_last_error().decode())
    return status


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


class Plan:
    """A transform plan: layout, device tables and workspace sizes.

    Plan(fs, fmin, fmax, bins_per_octave, n_samples, batch) transforms
    [batch][n_samples] float32 signals; Plan.sliced(...) builds a sliced
    (streaming) plan. device=False builds the host tables only.
    """

    def __init__(self, fs, fmin, fmax, bins_per_octave, n_samples, batch=1, device=True, _sliced=False,
                 _bands=None):
        L = lib()
        h = ctypes.c_void_p()
        if _bands is not None:
            arr = (BandSpec * len(_bands))(*[BandSpec(*b) for b in _bands])
            if _sliced:
                fn = L.nsgcqt_sliced_plan_create_bands if device else L.nsgcqt_sliced_plan_create_bands_host
            else:
                fn = L.nsgcqt_plan_create_bands if device else L.nsgcqt_plan_create_bands_host
            _check(fn(ctypes.byref(h), float(fs), int(n_samples), int(batch), len(_bands), arr))
        else:
            if _sliced:
                fn = L.nsgcqt_sliced_plan_create if device else L.nsgcqt_sliced_plan_create_host
            else:
                fn = L.nsgcqt_plan_create if device else L.nsgcqt_plan_create_host
            _check(fn(ctypes.byref(h), float(fs), float(fmin), float(fmax), int(bins_per_octave),
                      int(n_samples), int(batch)))
        self._h = h
        self.info = Info()
        _check(L.nsgcqt_plan_info(self._h, ctypes.byref(self.info)))
        self.device = bool(self.info.device_tables)
        self._ws = {}
        i = self.info
        self._ws_need = {OP_ANALYSE: max(1, i.ws_analyse), OP_SYNTHESISE: max(1, i.ws_synthesise),
                         OP_ADJ_ANALYSIS: max(1, i.ws_adjoint_analysis),
                         OP_ADJ_SYNTHESIS: max(1, i.ws_adjoint_synthesis)}

    @classmethod
    def sliced(cls, fs, fmin, fmax, bins_per_octave, slice_len, slices_per_chunk=16, device=True):
        return cls(fs, fmin, fmax, bins_per_octave, slice_len, slices_per_chunk, device, _sliced=True)

    @classmethod
    def from_bands(cls, fs, n_samples, bands, batch=1, device=True):
        """Plan of an explicit band list: tuples (kind, xi, beta, length[, centre_hz])
        as nsgcqt_band_spec, in coefficient order."""
        return cls(fs, 0.0, 0.0, 0, n_samples, batch, device, _bands=[tuple(b) for b in bands])

    @classmethod
    def sliced_from_bands(cls, fs, slice_len, bands, slices_per_chunk=16, device=True):
        """Sliced (streaming) plan of an explicit band list for slices of slice_len."""
        return cls(fs, 0.0, 0.0, 0, slice_len, slices_per_chunk, device, _sliced=True,
                   _bands=[tuple(b) for b in bands])

    def close(self):
        if getattr(self, "_h", None):
            lib().nsgcqt_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- queries
    @property
    def n_bands(self):
        return self.info.n_bands

    @property
    def n_coeffs(self):
        return self.info.total_coeffs

    @property
    def n_samples(self):
        return self.info.n_samples

    @property
    def batch(self):
        return self.info.batch

    def band(self, i) -> BandInfo:
        b = BandInfo()
        _check(lib().nsgcqt_band_info(self._h, int(i), ctypes.byref(b)))
        return b

    def bands(self):
        return [self.band(i) for i in range(self.n_bands)]

    def weights(self, which):
        import numpy as np
        out = np.empty(self.n_coeffs, dtype=np.float32)
        _check(lib().nsgcqt_plan_weights(self._h, int(which), out.ctypes.data_as(ctypes.c_void_p), out.nbytes))
        return out

    def workspace_bytes(self, op):
        i = self.info
        return {OP_ANALYSE: i.ws_analyse, OP_SYNTHESISE: i.ws_synthesise,
                OP_ADJ_ANALYSIS: i.ws_adjoint_analysis, OP_ADJ_SYNTHESIS: i.ws_adjoint_synthesis}[op]

    def workspace(self, op, device=None, stream=None):
        """A cached uint8 device buffer big enough for `op`, one per (op,
        stream): calls on different streams that use the default workspace
        never share it. It is allocated on that stream (the stream's current
        one if None), so the caching allocator ties it to the stream that
        uses it."""
        import torch
        dev = torch.device(device or "cuda")
        return self._ws_on(op, dev, torch.cuda.current_stream(dev) if stream is None else stream)

    def _ws_on(self, op, dev, s):
        ws = self._ws.get((op, s.cuda_stream))
        need = self._ws_need[op]
        if ws is None or ws.numel() < need:
            import torch
            with torch.cuda.stream(s):
                ws = torch.empty(need, dtype=torch.uint8, device=dev)
            self._ws[(op, s.cuda_stream)] = ws
        return ws

    @staticmethod
    def _on(t, stream):
        """The stream of a call on tensor t (t's device's current stream if
        None) and its raw handle."""
        import torch
        s = torch.cuda.current_stream(t.device) if stream is None else stream
        return s, ctypes.c_void_p(s.cuda_stream)

    def stage_info(self, op):
        """[(kernel name, algorithmic bytes per launch)] of one call of `op`."""
        L = lib()
        n = L.nsgcqt_stage_info(self._h, int(op), -1, None, 0, None)
        if n < 0:
            _check(n)
        out = []
        for i in range(n):
            name = ctypes.create_string_buffer(64)
            b = ctypes.c_double()
            _check(min(0, L.nsgcqt_stage_info(self._h, int(op), i, name, 64, ctypes.byref(b))))
            out.append((name.value.decode(), b.value))
        return out

    def set_stage_events(self, handles):
        """Bracket kernel i of each call with handles[2i], handles[2i+1]
        (see nsgcqt_set_stage_events); None stops. `handles` is a sequence
        of event handles (None entries allowed) or a ctypes c_void_p array."""
        if handles is None or len(handles) == 0:
            _check(lib().nsgcqt_set_stage_events(self._h, None, 0))
            return
        arr = handles if isinstance(handles, ctypes.Array) else (ctypes.c_void_p * len(handles))(*handles)
        _check(lib().nsgcqt_set_stage_events(self._h, arr, len(arr)))

    # ---------------------------------------------------------------- compute
    def _new(self, shape, dtype, like):
        import torch
        return torch.empty(shape, dtype=dtype, device=like.device)

    def analyse(self, x, out=None, ws=None, stream=None):
        """x [batch][N] float32 (cuda) -> coefficients [batch][C] complex64."""
        import torch
        self._expect(x, torch.float32, (self.batch, self.n_samples))
        out = self._new((self.batch, self.n_coeffs), torch.complex64, x) if out is None else out
        self._expect(out, torch.complex64, (self.batch, self.n_coeffs))
        st, sh = self._on(x, stream)
        ws = self._ws_on(OP_ANALYSE, x.device, st) if ws is None else ws
        _check(lib().nsgcqt_analyse(self._h, _ptr(x), _ptr(out), _ptr(ws), ws.numel(), sh))
        return out

    def analyse_noalloc(self, x, out, stream=None):
        """As analyse, through nsgcqt_analyse_noalloc: the workspace is the
        library's device array (no allocation); `out` must be given."""
        import torch
        self._expect(x, torch.float32, (self.batch, self.n_samples))
        self._expect(out, torch.complex64, (self.batch, self.n_coeffs))
        _check(lib().nsgcqt_analyse_noalloc(self._h, _ptr(x), _ptr(out), self._on(x, stream)[1]))
        return out

    def synthesise(self, c, out=None, ws=None, stream=None):
        """coefficients [batch][C] complex64 -> signals [batch][N] float32."""
        import torch
        self._expect(c, torch.complex64, (self.batch, self.n_coeffs))
        out = self._new((self.batch, self.n_samples), torch.float32, c) if out is None else out
        self._expect(out, torch.float32, (self.batch, self.n_samples))
        st, sh = self._on(c, stream)
        ws = self._ws_on(OP_SYNTHESISE, c.device, st) if ws is None else ws
        _check(lib().nsgcqt_synthesise(self._h, _ptr(c), _ptr(out), _ptr(ws), ws.numel(), sh))
        return out

    def adjoint(self, op, inp, out=None, ws=None, stream=None):
        """OP_ADJ_ANALYSIS: [b][C] c64 -> [b][N] f32; OP_ADJ_SYNTHESIS: [b][N] f32 -> [b][C] c64."""
        import torch
        if op == OP_ADJ_ANALYSIS:
            self._expect(inp, torch.complex64, (self.batch, self.n_coeffs))
            shape, dt = (self.batch, self.n_samples), torch.float32
        elif op == OP_ADJ_SYNTHESIS:
            self._expect(inp, torch.float32, (self.batch, self.n_samples))
            shape, dt = (self.batch, self.n_coeffs), torch.complex64
        else:
            raise ValueError("op must be OP_ADJ_ANALYSIS or OP_ADJ_SYNTHESIS")
        out = self._new(shape, dt, inp) if out is None else out
        self._expect(out, dt, shape)
        st, sh = self._on(inp, stream)
        ws = self._ws_on(op, inp.device, st) if ws is None else ws
        _check(lib().nsgcqt_adjoint(self._h, int(op), _ptr(inp), _ptr(out), _ptr(ws), ws.numel(), sh))
        return out

    def slice_count(self, n):
        r = lib().nsgcqt_sliced_count(self._h, int(n))
        if r < 0:
            _check(int(r))
        return int(r)

    def sliced_analyse(self, x, out=None, ws=None, stream=None):
        """One signal x [n] float32 -> slice coefficients [J][C] complex64."""
        import torch
        n = x.numel()
        J = self.slice_count(n)
        self._expect(x, torch.float32, (n,))
        out = self._new((J, self.n_coeffs), torch.complex64, x) if out is None else out
        self._expect(out, torch.complex64, (J, self.n_coeffs))
        st, sh = self._on(x, stream)
        ws = self._ws_on(OP_ANALYSE, x.device, st) if ws is None else ws
        _check(lib().nsgcqt_sliced_analyse(self._h, _ptr(x), n, _ptr(out), _ptr(ws), ws.numel(), sh))
        return out

    def sliced_synthesise(self, c, n, out=None, ws=None, stream=None):
        """Slice coefficients [J][C] complex64 -> signal [n] float32."""
        import torch
        J = self.slice_count(n)
        self._expect(c, torch.complex64, (J, self.n_coeffs))
        out = self._new((n,), torch.float32, c) if out is None else out
        self._expect(out, torch.float32, (n,))
        st, sh = self._on(c, stream)
        ws = self._ws_on(OP_SYNTHESISE, c.device, st) if ws is None else ws
        _check(lib().nsgcqt_sliced_synthesise(self._h, _ptr(c), int(n), _ptr(out), _ptr(ws), ws.numel(), sh))
        return out

    @staticmethod
    def _expect(t, dtype, shape):
        if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"expected a contiguous cuda {dtype} tensor of shape {tuple(shape)}, "
                             f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def table1_layout():
    """The Table-1 multi-resolution layout: (fs, n_samples, band tuples)."""
    L = lib()
    n = ctypes.c_int()
    fs = ctypes.c_double()
    N = ctypes.c_int64()
    _check(L.nsgcqt_layout_table1(None, 0, ctypes.byref(n), ctypes.byref(fs), ctypes.byref(N)))
    arr = (BandSpec * n.value)()
    _check(L.nsgcqt_layout_table1(arr, n.value, ctypes.byref(n), None, None))
    return fs.value, N.value, [b.as_tuple() for b in arr]


def erb_layout(fs, n_samples, fmin, fmax, bands_per_erb=1.0):
    """The auditory (ERB-rate) layout of nsgcqt_layout_erb as band tuples."""
    L = lib()
    n = ctypes.c_int()
    args = (float(fs), int(n_samples), float(fmin), float(fmax), float(bands_per_erb))
    _check(L.nsgcqt_layout_erb(*args, None, 0, ctypes.byref(n)))
    arr = (BandSpec * n.value)()
    _check(L.nsgcqt_layout_erb(*args, arr, n.value, ctypes.byref(n)))
    return [b.as_tuple() for b in arr]

