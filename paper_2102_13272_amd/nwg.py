"""ctypes binding of the C ABI in include/nwg.h (argument marshalling only).

Every function of the header is exposed under the same name on the loaded
library object; ``Plan`` wraps a plan handle for torch tensors (device
pointers from ``tensor.data_ptr()``, streams from
``torch.cuda.current_stream().cuda_stream``).  There is no fallback: if
``libnwg.so`` is missing or cannot be loaded, every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnwg.so")

NWG_TILE_F2X2_3X3 = 0
NWG_TILE_F3X3_3X3 = 1
NWG_TILE_LD_F2X2_3X3 = 2
NWG_TILE_MIX_F23_F33 = 3
NWG_TILE_AUTO = -1
NWG_PRECISION_FP32 = 0
NWG_PRECISION_BF16_SPLIT = 1
NWG_OK, NWG_EINVAL, NWG_ENOMEM, NWG_EHIP, NWG_EUNSUPPORTED = 0, -1, -2, -3, -4
NWG_MAX_DEPTH = 4


class nwg_plan_info(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int), ("M", ctypes.c_int), ("N", ctypes.c_int), ("H", ctypes.c_int),
        ("W", ctypes.c_int), ("r", ctypes.c_int), ("pad", ctypes.c_int), ("tile", ctypes.c_int),
        ("Ho", ctypes.c_int), ("Wo", ctypes.c_int), ("n", ctypes.c_int),
        ("m", ctypes.c_int), ("rb", ctypes.c_int), ("l", ctypes.c_int),
        ("strides", ctypes.c_int * NWG_MAX_DEPTH),
        ("Mn", ctypes.c_int), ("Kn", ctypes.c_int), ("Ln", ctypes.c_int),
        ("th", ctypes.c_int), ("tw", ctypes.c_int),
        ("T", ctypes.c_longlong), ("P", ctypes.c_longlong),
        ("u_bytes", ctypes.c_size_t), ("v_bytes", ctypes.c_size_t),
        ("yhat_bytes", ctypes.c_size_t), ("workspace_bytes", ctypes.c_size_t),
        ("ewmm_mults", ctypes.c_longlong), ("direct_flop", ctypes.c_double),
        ("contract_flop", ctypes.c_double), ("fused_input", ctypes.c_int),
        ("depthwise", ctypes.c_int), ("fused_conv", ctypes.c_int),
        ("pipeline_parts", ctypes.c_int), ("precision", ctypes.c_int), ("ld_c", ctypes.c_int),
        ("fused_output", ctypes.c_int), ("outer33", ctypes.c_int),
        ("live_np", ctypes.c_int), ("live_prefix", ctypes.c_ulonglong * 2),
        ("live_groups", ctypes.c_longlong), ("level1_live", ctypes.c_int),
        ("mix_planar", ctypes.c_int),
    ]

    def as_dict(self):
        d = {name: getattr(self, name) for name, _ in self._fields_}
        d["strides"] = list(self.strides)[: self.n]
        d["live_prefix"] = list(self.live_prefix)
        return d


_P = ctypes.c_void_p
_I = ctypes.c_int
# (name, restype, argtypes) for every symbol declared in include/nwg.h
SIGNATURES = [
    ("nwg_plan_geometry", _I, [_I] * 8 + [ctypes.POINTER(nwg_plan_info)]),
    ("nwg_plan_create", _P, [_I] * 7),
    ("nwg_plan_create_pad", _P, [_I] * 8),
    ("nwg_plan_geometry_depthwise", _I, [_I] * 7 + [ctypes.POINTER(nwg_plan_info)]),
    ("nwg_plan_create_depthwise", _P, [_I] * 7),
    ("nwg_plan_destroy", None, [_P]),
    ("nwg_plan_query", _I, [_P, ctypes.POINTER(nwg_plan_info)]),
    ("nwg_conv2d", _I, [_P, _P, _P, _P, _P]),
    ("nwg_plan_set_weights", _I, [_P, _P, _P]),
    ("nwg_kernel_transform", _I, [_P, _P, _P, _P]),
    ("nwg_input_transform", _I, [_P, _P, _P, _P]),
    ("nwg_contract", _I, [_P, _P, _P, _P, _P]),
    ("nwg_input_contract", _I, [_P, _P, _P, _P, _P]),
    ("nwg_output_transform", _I, [_P, _P, _P, _P]),
    ("nwg_plan_set_pipeline", _I, [_P, _I]),
    ("nwg_plan_set_precision", _I, [_P, _I]),
    ("nwg_plan_set_timing", _I, [_P, _I]),
    ("nwg_plan_get_timing", _I, [_P, ctypes.POINTER(ctypes.c_double),
                                 ctypes.POINTER(ctypes.c_longlong)]),
    ("nwg_conv2d_noalloc", _I, [_I] * 8 + [_P] * 4),
    ("nwg_last_error", ctypes.c_char_p, []),
    ("nwg_last_status", _I, []),
    ("nwg_version", ctypes.c_char_p, []),
]

_lib: Optional[ctypes.CDLL] = None


class NwgError(RuntimeError):
    pass


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libnwg.so (once) and declare every entry point; raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise NwgError(f"{path} is missing: build it with `python -c 'import __graft_entry__ as g; "
                       f"g.build()'` (no CPU fallback exists)")
    lib = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def last_error() -> str:
    return load_library().nwg_last_error().decode()


def _check(rc: int, what: str):
    if rc != NWG_OK:
        raise NwgError(f"{what} failed ({rc}): {last_error()}")


def plan_geometry(B, M, N, H, W, r, pad=0, tile=NWG_TILE_F2X2_3X3) -> dict:
    """Host-only geometry of a convolution (no device is touched)."""
    info = nwg_plan_info()
    _check(load_library().nwg_plan_geometry(B, M, N, H, W, r, pad, tile, ctypes.byref(info)),
           "nwg_plan_geometry")
    return info.as_dict()


def plan_geometry_depthwise(B, C, H, W, r, pad=0, tile=NWG_TILE_F2X2_3X3) -> dict:
    """Host-only geometry of a depthwise convolution (no device is touched)."""
    info = nwg_plan_info()
    _check(load_library().nwg_plan_geometry_depthwise(B, C, H, W, r, pad, tile,
                                                      ctypes.byref(info)),
           "nwg_plan_geometry_depthwise")
    return info.as_dict()


def _ptr(t, numel: int, what: str) -> int:
    """Device pointer of a tensor the library will read or write: a
    contiguous float32 GPU tensor of at least `numel` elements, 16-byte
    aligned.  Raises NwgError before any call into the library otherwise
    (an undersized buffer would be read or written past its end)."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise NwgError(f"{what}: expected a torch tensor, got {type(t).__name__}")
    if t.dtype != torch.float32:
        raise NwgError(f"{what}: dtype {t.dtype}, the library computes in float32")
    if not t.is_contiguous():
        raise NwgError(f"{what}: not contiguous")
    if t.numel() < numel:
        raise NwgError(f"{what}: {t.numel()} elements, the plan needs {numel}")
    if not t.is_cuda:
        raise NwgError(f"{what}: a {t.device} tensor, the library takes GPU memory")
    p = int(t.data_ptr())
    if p % 16:
        raise NwgError(f"{what}: address not 16-byte aligned")
    return p


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    return int(getattr(stream, "cuda_stream", stream))


NWG_NOALLOC_SCRATCH_BYTES = 64 << 20


def conv2d_noalloc(x, w, y, pad=0, tile=NWG_TILE_F2X2_3X3, stream=None):
    """y = conv(x, w) through nwg_conv2d_noalloc: no plan, no device allocation
    (the library's static per-GPU scratch holds the workspace; see nwg.h)."""
    B, M, H, W = x.shape
    N, _, r, _ = w.shape
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    _check(load_library().nwg_conv2d_noalloc(
        B, M, N, H, W, r, pad, tile, _ptr(x, B * M * H * W, "x"), _ptr(w, N * M * r * r, "w"),
        _ptr(y, B * N * max(Ho, 0) * max(Wo, 0), "y"), _stream(stream)), "nwg_conv2d_noalloc")


class Plan:
    """A plan handle; tensors are torch float32 CUDA (HIP) tensors, contiguous."""

    def __init__(self, B, M, N, H, W, r, pad=0, tile=NWG_TILE_F2X2_3X3, depthwise=False):
        """Dense plan (M -> N channels), or with depthwise=True a depthwise plan
        over M = N channels (nwg_plan_create_depthwise)."""
        lib = load_library()
        self._lib = lib
        self._w, self._w_version = None, None
        if depthwise:
            if M != N:
                raise ValueError("a depthwise plan has M == N channels")
            self.handle = lib.nwg_plan_create_depthwise(B, M, H, W, r, pad, tile)
        else:
            self.handle = lib.nwg_plan_create_pad(B, M, N, H, W, r, pad, tile)
        if not self.handle:
            raise NwgError(f"plan creation failed: {last_error()}")
        info = nwg_plan_info()
        _check(lib.nwg_plan_query(self.handle, ctypes.byref(info)), "nwg_plan_query")
        self.info = info.as_dict()

    def close(self):
        if getattr(self, "handle", None):
            self._lib.nwg_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # shapes of the Winograd-domain buffers (F(2x2,3x3): quad-interleaved;
    # F(3x3,3x3): plain; see include/nwg.h)
    @property
    def _f33(self):
        return self.info["tile"] == NWG_TILE_F3X3_3X3 and self.info["n"] > 0

    @property
    def _mv(self):
        """channels of V (and of the contraction): M, or M c^2 for the linear decomposition"""
        i = self.info
        return i["M"] * i["ld_c"] ** 2 if i["ld_c"] else i["M"]

    @property
    def u_shape(self):
        i = self.info
        mk = 1 if i["depthwise"] else self._mv
        if not i["n"]:
            return (mk, i["N"])
        if i["mix_planar"]:
            return (i["live_groups"], 9, mk, i["N"])
        return (i["P"], mk, i["N"]) if self._f33 else (i["P"] // 4, mk, i["N"], 4)

    @property
    def v_shape(self):
        i = self.info
        if i["mix_planar"]:
            return (i["live_groups"], 9, i["M"], i["T"])
        return (i["P"], i["M"], i["T"]) if self._f33 else (i["P"] // 4, self._mv, i["T"], 4)

    @property
    def z_shape(self):
        i = self.info
        if self._f33:
            return (i["P"] // 25, 5, 3, i["N"], i["T"])
        return (i["P"] // 16, i["N"], i["T"], 4)

    @property
    def y_shape(self):
        i = self.info
        return (i["B"], i["N"], i["Ho"], i["Wo"])

    # element counts of the tensors the calls take
    @property
    def _x_numel(self):
        i = self.info
        return i["B"] * i["M"] * i["H"] * i["W"]

    @property
    def _w_numel(self):
        i = self.info
        return i["N"] * (1 if i["depthwise"] else i["M"]) * i["r"] * i["r"]

    @property
    def _y_numel(self):
        i = self.info
        return i["B"] * i["N"] * i["Ho"] * i["Wo"]

    def _buf_numel(self, which):
        """U, V or Z of the stage calls (depth 0: V is x and Z is y)."""
        i = self.info
        if not i["n"] and which in ("V", "Z"):
            return self._x_numel if which == "V" else self._y_numel
        return i[{"U": "u_bytes", "V": "v_bytes", "Z": "yhat_bytes"}[which]] // 4

    def conv2d(self, x, w, y, stream=None):
        """y = conv(x, w).  The transformed weights are cached by the library
        under w's address; the plan also keeps w itself (so that its memory
        cannot be freed and handed to another weight tensor while cached) and
        w's version counter, and transforms w again when either changes."""
        xp = _ptr(x, self._x_numel, "x")
        wp = _ptr(w, self._w_numel, "w")
        yp = _ptr(y, self._y_numel, "y")
        if self._w is not w or self._w_version != w._version:
            self.set_weights(w, stream)
        _check(self._lib.nwg_conv2d(self.handle, xp, wp, yp, _stream(stream)), "nwg_conv2d")

    def set_weights(self, w, stream=None):
        self._w, self._w_version = None, None
        _check(self._lib.nwg_plan_set_weights(self.handle, _ptr(w, self._w_numel, "w"),
                                              _stream(stream)), "nwg_plan_set_weights")
        self._w, self._w_version = w, w._version

    def kernel_transform(self, w, U, stream=None):
        _check(self._lib.nwg_kernel_transform(self.handle, _ptr(w, self._w_numel, "w"),
                                              _ptr(U, self._buf_numel("U"), "U"),
                                              _stream(stream)), "nwg_kernel_transform")

    def input_transform(self, x, V, stream=None):
        _check(self._lib.nwg_input_transform(self.handle, _ptr(x, self._x_numel, "x"),
                                             _ptr(V, self._buf_numel("V"), "V"),
                                             _stream(stream)), "nwg_input_transform")

    def contract(self, U, V, Z, stream=None):
        _check(self._lib.nwg_contract(self.handle, _ptr(U, self._buf_numel("U"), "U"),
                                      _ptr(V, self._buf_numel("V"), "V"),
                                      _ptr(Z, self._buf_numel("Z"), "Z"), _stream(stream)),
               "nwg_contract")

    def input_contract(self, x, U, Z, stream=None):
        _check(self._lib.nwg_input_contract(self.handle, _ptr(x, self._x_numel, "x"),
                                            _ptr(U, self._buf_numel("U"), "U"),
                                            _ptr(Z, self._buf_numel("Z"), "Z"),
                                            _stream(stream)), "nwg_input_contract")

    def output_transform(self, Z, y, stream=None):
        _check(self._lib.nwg_output_transform(self.handle, _ptr(Z, self._buf_numel("Z"), "Z"),
                                              _ptr(y, self._y_numel, "y"), _stream(stream)),
               "nwg_output_transform")

    def set_pipeline(self, parts: int):
        _check(self._lib.nwg_plan_set_pipeline(self.handle, int(parts)), "nwg_plan_set_pipeline")
        info = nwg_plan_info()
        _check(self._lib.nwg_plan_query(self.handle, ctypes.byref(info)), "nwg_plan_query")
        self.info = info.as_dict()

    def set_precision(self, precision: int):
        _check(self._lib.nwg_plan_set_precision(self.handle, int(precision)),
               "nwg_plan_set_precision")
        self._w, self._w_version = None, None
        info = nwg_plan_info()
        _check(self._lib.nwg_plan_query(self.handle, ctypes.byref(info)), "nwg_plan_query")
        self.info = info.as_dict()

    def set_timing(self, enable: bool):
        _check(self._lib.nwg_plan_set_timing(self.handle, int(bool(enable))), "nwg_plan_set_timing")

    def get_timing(self):
        """Wait for recorded stages; returns (ms[4], count[4]) summed since the last call."""
        ms = (ctypes.c_double * 4)()
        cnt = (ctypes.c_longlong * 4)()
        _check(self._lib.nwg_plan_get_timing(self.handle, ms, cnt), "nwg_plan_get_timing")
        return list(ms), list(cnt)
