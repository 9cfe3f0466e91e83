"""ctypes binding of libblconv.so (the band-limited FFT convolution library).

Argument marshalling only: every compute step runs in the HIP kernels of the
library.  Torch tensors supply device pointers and the current HIP stream.
If the library is missing the import still works, but every entry point
raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libblconv.so")

BL_REUSE_X = 0x1
BL_REUSE_W = 0x2
BL_REUSE_DY = 0x4

BL_DESC_BF16_SPECTRA = 0x1
BL_DESC_FUSED_FORWARD = 0x2

BL_SPEC_X = 0
BL_SPEC_W = 1

STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported configuration", 3: "workspace too small",
          4: "HIP error", 5: "out of host memory"}

EXPORTED = (
    "bl_conv_plan_create", "bl_conv_plan_destroy", "bl_conv_plan_info", "bl_conv_plan_get_mask",
    "bl_conv_plan_get_bins", "bl_conv_workspace_size", "bl_conv_workspace_layout", "bl_conv_forward",
    "bl_conv_backward_input", "bl_conv_backward_weight", "bl_status_string", "bl_profile_begin",
    "bl_profile_end", "bl_profile_count", "bl_profile_get", "bl_profile_release", "bl_conv_input_energy",
    "bl_conv_rate_for_energy", "bl_conv_zero_smallest", "bl_conv_fine_band_for_energy", "bl_conv_zero_bins",
    "bl_conv_forward_noalloc", "bl_conv_backward",
)


class BlError(RuntimeError):
    def __init__(self, call, code):
        super().__init__(f"{call} failed: {STATUS.get(code, code)} ({code})")
        self.code = code


class Desc(ctypes.Structure):
    _fields_ = [
        ("ndim", ctypes.c_int), ("N", ctypes.c_int), ("C_in", ctypes.c_int), ("C_out", ctypes.c_int),
        ("H", ctypes.c_int), ("W", ctypes.c_int), ("K", ctypes.c_int),
        ("pad_lo", ctypes.c_int * 2), ("pad_hi", ctypes.c_int * 2), ("c", ctypes.c_double),
        ("fft_h", ctypes.c_int), ("fft_w", ctypes.c_int), ("flags", ctypes.c_uint),
    ]


_lib = None


def load():
    """Load libblconv.so once (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_1911_09287_amd.build`")
    try:
        import torch  # noqa: F401  -- loads torch's HIP runtime first
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P, I, U, L, D, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint, ctypes.c_long, ctypes.c_double, ctypes.c_size_t
    lib.bl_conv_plan_create.argtypes = [ctypes.POINTER(P), ctypes.POINTER(Desc)]
    lib.bl_conv_plan_destroy.argtypes = [P]
    lib.bl_conv_plan_info.argtypes = [P, ctypes.POINTER(I), ctypes.POINTER(I), ctypes.POINTER(I),
                                      ctypes.POINTER(I), ctypes.POINTER(L), ctypes.POINTER(L), ctypes.POINTER(D)]
    lib.bl_conv_plan_get_mask.argtypes = [P, P, S]
    lib.bl_conv_plan_get_bins.argtypes = [P, P, P, S]
    lib.bl_conv_workspace_size.argtypes = [P, ctypes.POINTER(S)]
    lib.bl_conv_workspace_layout.argtypes = [P, ctypes.POINTER(S), ctypes.POINTER(S), ctypes.POINTER(S)]
    for name in ("bl_conv_forward", "bl_conv_backward_input", "bl_conv_backward_weight"):
        getattr(lib, name).argtypes = [P, P, P, P, P, U, P]
    lib.bl_conv_forward_noalloc.argtypes = [P, P, P, P, P]
    lib.bl_conv_backward.argtypes = [P, P, P, P, P, P, P, U, P]
    lib.bl_conv_input_energy.argtypes = [P, P, P, U, P, P]
    lib.bl_conv_rate_for_energy.argtypes = [P, P, S, D, ctypes.POINTER(I), ctypes.POINTER(D), ctypes.POINTER(D)]
    lib.bl_conv_zero_smallest.argtypes = [P, P, P, U, ctypes.c_longlong, U, P]
    lib.bl_conv_fine_band_for_energy.argtypes = [P, P, S, D, ctypes.POINTER(I), ctypes.POINTER(D), ctypes.POINTER(D),
                                                 P, S, ctypes.POINTER(S)]
    lib.bl_conv_zero_bins.argtypes = [P, P, U, P, P]
    lib.bl_status_string.argtypes = [I]
    lib.bl_status_string.restype = ctypes.c_char_p
    lib.bl_profile_begin.argtypes = [I]
    lib.bl_profile_count.restype = I
    lib.bl_profile_get.argtypes = [I, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_float),
                                   ctypes.POINTER(D), ctypes.POINTER(D)]
    for name in EXPORTED:
        getattr(lib, name)  # every declared symbol must be exported
    _lib = lib
    return lib


def _check(call, code):
    if code != 0:
        raise BlError(call, code)


class Plan:
    """A band-limited convolution plan (host only until a compute call).

    2-D: ``Plan(2, N, C_in, C_out, (H, W), K, pad=(top, bottom, left, right), c=...)``.
    1-D: ``Plan(1, N, C_in, C_out, (L,), K, pad=(lo, hi), c=...)``.
    ``desc_flags``: 0, or BL_DESC_BF16_SPECTRA (spectra stored in bfloat16,
    contracted with fp32 sums) and/or BL_DESC_FUSED_FORWARD (fused small-map
    forward kernel where it applies).
    """

    def __init__(self, ndim, N, C_in, C_out, spatial, K, pad, c, fft=None, desc_flags=0):
        lib = load()
        d = Desc()
        d.ndim, d.N, d.C_in, d.C_out, d.K = ndim, N, C_in, C_out, K
        if ndim == 2:
            d.H, d.W = spatial
            pt, pb, pl, pr = pad
            d.pad_lo[0], d.pad_hi[0], d.pad_lo[1], d.pad_hi[1] = pt, pb, pl, pr
            if fft is not None:
                d.fft_h, d.fft_w = fft
        else:
            d.H, d.W = spatial[0], 1
            d.pad_lo[0], d.pad_hi[0] = pad
            if fft is not None:
                d.fft_h = fft
        d.c = float(c)
        d.flags = int(desc_flags)
        self.desc = d
        self.desc_flags = int(desc_flags)
        self.ndim, self.N, self.C_in, self.C_out, self.K = ndim, N, C_in, C_out, K
        self.spatial = tuple(spatial)
        self.pad = tuple(pad)
        h = ctypes.c_void_p()
        _check("bl_conv_plan_create", lib.bl_conv_plan_create(ctypes.byref(h), ctypes.byref(d)))
        self._h = h
        self._lib = lib
        fh, fw, rh, rw = (ctypes.c_int() for _ in range(4))
        kept, total = ctypes.c_long(), ctypes.c_long()
        ceff = ctypes.c_double()
        _check("bl_conv_plan_info", lib.bl_conv_plan_info(h, ctypes.byref(fh), ctypes.byref(fw), ctypes.byref(rh),
                                                          ctypes.byref(rw), ctypes.byref(kept),
                                                          ctypes.byref(total), ctypes.byref(ceff)))
        self.fft = (fh.value, fw.value)
        self.r_h, self.r_w = rh.value, rw.value
        self.kept, self.total, self.c_eff = kept.value, total.value, ceff.value
        sz = ctypes.c_size_t()
        _check("bl_conv_workspace_size", lib.bl_conv_workspace_size(h, ctypes.byref(sz)))
        self.workspace_bytes = sz.value
        ox, ow, od = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        _check("bl_conv_workspace_layout",
               lib.bl_conv_workspace_layout(h, ctypes.byref(ox), ctypes.byref(ow), ctypes.byref(od)))
        self.offsets = {"X": ox.value, "W": ow.value, "DY": od.value}

    # -- shapes ---------------------------------------------------------------
    @property
    def out_spatial(self):
        if self.ndim == 1:
            lo, hi = self.pad
            return (self.spatial[0] + lo + hi - self.K + 1,)
        pt, pb, pl, pr = self.pad
        H, W = self.spatial
        return (H + pt + pb - self.K + 1, W + pl + pr - self.K + 1)

    def x_shape(self):
        return (self.N, self.C_in) + self.spatial

    def w_shape(self):
        return (self.C_out, self.C_in) + (self.K,) * self.ndim

    def y_shape(self):
        return (self.N, self.C_out) + self.out_spatial

    # -- host queries -----------------------------------------------------------
    def mask(self):
        m = np.zeros(self.total, dtype=np.uint8)
        _check("bl_conv_plan_get_mask", self._lib.bl_conv_plan_get_mask(self._h, m.ctypes.data, m.size))
        if self.ndim == 1:
            return m
        return m.reshape(self.fft[0], self.fft[1] // 2 + 1)

    def bins(self):
        u = np.zeros(self.kept, dtype=np.int32)
        v = np.zeros(self.kept, dtype=np.int32)
        _check("bl_conv_plan_get_bins", self._lib.bl_conv_plan_get_bins(self._h, u.ctypes.data, v.ctypes.data,
                                                                        self.kept))
        return u, v

    # -- device calls ----------------------------------------------------------
    def workspace(self, device="cuda"):
        import torch
        return torch.empty(self.workspace_bytes, dtype=torch.uint8, device=device)

    @staticmethod
    def _ptr(t, shape, name):
        if t is None:
            return None
        import torch
        if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous float32 tensor on the GPU")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
        return t.data_ptr()

    @staticmethod
    def _stream(stream):
        import torch
        s = torch.cuda.current_stream() if stream is None else stream
        return s.cuda_stream

    def _ws(self, ws):
        if ws is None or ws.numel() < self.workspace_bytes or not ws.is_cuda:
            raise ValueError("workspace must be a GPU tensor of at least workspace_bytes bytes")
        return ws.data_ptr()

    def forward(self, x, w, y, ws, flags=0, stream=None):
        _check("bl_conv_forward", self._lib.bl_conv_forward(
            self._h, self._ptr(x, self.x_shape(), "x"), self._ptr(w, self.w_shape(), "w"),
            self._ptr(y, self.y_shape(), "y"), self._ws(ws), flags, self._stream(stream)))

    def forward_noalloc(self, x, w, y, stream=None):
        """Forward pass on the library's static device array (no workspace, no
        allocation); calls on one GPU must not overlap."""
        _check("bl_conv_forward_noalloc", self._lib.bl_conv_forward_noalloc(
            self._h, self._ptr(x, self.x_shape(), "x"), self._ptr(w, self.w_shape(), "w"),
            self._ptr(y, self.y_shape(), "y"), self._stream(stream)))

    def backward_input(self, dy, w, dx, ws, flags=0, stream=None):
        _check("bl_conv_backward_input", self._lib.bl_conv_backward_input(
            self._h, self._ptr(dy, self.y_shape(), "dy"), self._ptr(w, self.w_shape(), "w"),
            self._ptr(dx, self.x_shape(), "dx"), self._ws(ws), flags, self._stream(stream)))

    def backward_weight(self, x, dy, dw, ws, flags=0, stream=None):
        _check("bl_conv_backward_weight", self._lib.bl_conv_backward_weight(
            self._h, self._ptr(x, self.x_shape(), "x"), self._ptr(dy, self.y_shape(), "dy"),
            self._ptr(dw, self.w_shape(), "dw"), self._ws(ws), flags, self._stream(stream)))

    def backward(self, dy, w, x, dx, dw, ws, flags=0, stream=None):
        """Both gradients (bl_conv_backward)."""
        _check("bl_conv_backward", self._lib.bl_conv_backward(
            self._h, self._ptr(dy, self.y_shape(), "dy"), self._ptr(w, self.w_shape(), "w"),
            self._ptr(x, self.x_shape(), "x"), self._ptr(dx, self.x_shape(), "dx"),
            self._ptr(dw, self.w_shape(), "dw"), self._ws(ws), flags, self._stream(stream)))

    def input_energy(self, x, ws, energy=None, flags=0, stream=None):
        """Per kept bin h_v * sum |X|^2 of the input spectrum (fp64, on the GPU);
        `energy` (float64 GPU tensor of kept elements) is allocated if None."""
        import torch
        if energy is None:
            energy = torch.empty(self.kept, dtype=torch.float64, device=ws.device)
        if not (energy.is_cuda and energy.dtype == torch.float64 and energy.is_contiguous()
                and energy.numel() == self.kept):
            raise ValueError("energy must be a contiguous float64 GPU tensor of kept elements")
        _check("bl_conv_input_energy", self._lib.bl_conv_input_energy(
            self._h, self._ptr(x, self.x_shape(), "x"), self._ws(ws), flags, energy.data_ptr(),
            self._stream(stream)))
        return energy

    def rate_for_energy(self, energy, fraction):
        """(t, c, preserved) of the band keeping at least `fraction` of the bin
        energies (host array in the plan's bin order)."""
        e = np.ascontiguousarray(np.asarray(energy, dtype=np.float64))
        t, c, f = ctypes.c_int(), ctypes.c_double(), ctypes.c_double()
        _check("bl_conv_rate_for_energy", self._lib.bl_conv_rate_for_energy(
            self._h, e.ctypes.data, e.size, float(fraction), ctypes.byref(t), ctypes.byref(c), ctypes.byref(f)))
        return t.value, c.value, f.value

    def fine_band_for_energy(self, energy, fraction):
        """(t, c, preserved, keep) of the fine-grained band: keep is a uint8 array
        over the bins of the coarse band (rate c), 1 kept, 0 dropped."""
        e = np.ascontiguousarray(np.asarray(energy, dtype=np.float64))
        t, c, f, n = ctypes.c_int(), ctypes.c_double(), ctypes.c_double(), ctypes.c_size_t()
        _check("bl_conv_fine_band_for_energy", self._lib.bl_conv_fine_band_for_energy(
            self._h, e.ctypes.data, e.size, float(fraction), ctypes.byref(t), ctypes.byref(c), ctypes.byref(f),
            None, 0, ctypes.byref(n)))
        keep = np.zeros(n.value, dtype=np.uint8)
        _check("bl_conv_fine_band_for_energy", self._lib.bl_conv_fine_band_for_energy(
            self._h, e.ctypes.data, e.size, float(fraction), ctypes.byref(t), ctypes.byref(c), ctypes.byref(f),
            keep.ctypes.data, keep.size, ctypes.byref(n)))
        return t.value, c.value, f.value, keep

    def zero_bins(self, ws, which, keep, stream=None):
        """Zero the stored spectrum ("X" or "W") at the bins where `keep` (a
        uint8 GPU tensor of kept elements) is 0."""
        import torch
        if not (keep.is_cuda and keep.dtype == torch.uint8 and keep.is_contiguous() and keep.numel() == self.kept):
            raise ValueError("keep must be a contiguous uint8 GPU tensor of kept elements")
        code = {"X": BL_SPEC_X, "W": BL_SPEC_W}[which]
        _check("bl_conv_zero_bins", self._lib.bl_conv_zero_bins(self._h, self._ws(ws), code, keep.data_ptr(),
                                                                self._stream(stream)))

    def zero_smallest(self, src, ws, which, k, flags=0, stream=None):
        """Zero the k smallest-magnitude coefficients of each sample's ("X") or
        each filter's ("W") stored spectrum (see bl_conv_zero_smallest); `src`
        is x or w, or None with the matching reuse flag."""
        code = {"X": BL_SPEC_X, "W": BL_SPEC_W}[which]
        shape, name = (self.x_shape(), "x") if which == "X" else (self.w_shape(), "w")
        _check("bl_conv_zero_smallest", self._lib.bl_conv_zero_smallest(
            self._h, self._ptr(src, shape, name), self._ws(ws), code, int(k), flags, self._stream(stream)))

    def spectrum(self, ws, which):
        """View of a stored spectrum in the workspace, [kept][rows][cols]: complex64,
        or with BL_DESC_BF16_SPECTRA int32 words each holding a bfloat16 pair
        (real part in the low 16 bits, imaginary part in the high 16 bits)."""
        import torch
        rows, cols = {"X": (self.N, self.C_in), "W": (self.C_in, self.C_out), "DY": (self.N, self.C_out)}[which]
        off = self.offsets[which]
        bf16 = bool(self.desc_flags & BL_DESC_BF16_SPECTRA)
        n = self.kept * rows * cols * (4 if bf16 else 8)
        return ws[off:off + n].view(torch.int32 if bf16 else torch.complex64).view(self.kept, rows, cols)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.bl_conv_plan_destroy(h)
            self._h = None


def plan_for_layer(layer, c, fft=None, desc_flags=0):
    """Plan for a layer description with fields ndim, N, C_in, C_out, H, W, K, pad."""
    spatial = (layer.H,) if layer.ndim == 1 else (layer.H, layer.W)
    return Plan(layer.ndim, layer.N, layer.C_in, layer.C_out, spatial, layer.K, layer.pad, c, fft, desc_flags)


class Profile:
    """Per-kernel HIP-event timing of the library's launches (see bl_profile_*)."""

    def __init__(self, capacity=4096):
        self.lib = load()
        self.capacity = capacity

    def __enter__(self):
        _check("bl_profile_begin", self.lib.bl_profile_begin(self.capacity))
        return self

    def __exit__(self, *exc):
        self.lib.bl_profile_end()
        return False

    def records(self):
        """[(kernel name, ms, algorithmic bytes, algorithmic flops)] for every
        timed launch; call after synchronising the stream."""
        out = []
        name = ctypes.c_char_p()
        ms = ctypes.c_float()
        nb, nf = ctypes.c_double(), ctypes.c_double()
        for i in range(self.lib.bl_profile_count()):
            _check("bl_profile_get", self.lib.bl_profile_get(i, ctypes.byref(name), ctypes.byref(ms),
                                                             ctypes.byref(nb), ctypes.byref(nf)))
            out.append((name.value.decode(), ms.value, nb.value, nf.value))
        return out

    def release(self):
        self.lib.bl_profile_release()
