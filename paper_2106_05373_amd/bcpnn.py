"""Python binding of libbcpnn (include/bcpnn.h): argument marshalling only.

Every computation runs in the library's HIP kernels.  PyTorch provides device memory (tensors
whose data pointers are passed through) and the stream the layer enqueues on.  Importing this
module loads the library; if it is missing the import fails (build it with
``python -m paper_2106_05373_amd.build`` or ``__graft_entry__.build()``).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
# torch ships its own HIP runtime (libamdhip64.so.7); it must be loaded before this library so
# that the library's dependency on that soname resolves to the same runtime.  Loading the
# system copy first would put two HIP runtimes in the process.
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbcpnn.so")

STORAGE = {"f32": 0, "bf16": 1, "m10": 2}
KERNELS = {"sweep": 0, "support": 1, "active": 2, "weights": 3, "structural": 4}
STATUS = {0: "BCPNN_OK", -1: "BCPNN_EINVAL", -2: "BCPNN_ENOMEM", -3: "BCPNN_EDEVICE",
          -4: "BCPNN_ESTATE", -5: "BCPNN_EINPUT"}

EXPORTS = [
    "bcpnn_config_default", "bcpnn_layer_create", "bcpnn_layer_destroy", "bcpnn_forward",
    "bcpnn_train_batch", "bcpnn_recompute_weights", "bcpnn_structural_update",
    "bcpnn_structural_update_static", "bcpnn_readout", "bcpnn_flush", "bcpnn_get_state",
    "bcpnn_set_state", "bcpnn_get_mi", "bcpnn_profile_enable", "bcpnn_profile_read",
    "bcpnn_profile_read_kernel", "bcpnn_last_error",
]


class Config(ctypes.Structure):
    """Mirror of bcpnn_config."""
    _fields_ = [
        ("in_hcu", ctypes.c_int32), ("in_mcu", ctypes.c_int32),
        ("out_hcu", ctypes.c_int32), ("out_mcu", ctypes.c_int32),
        ("max_batch", ctypes.c_int32), ("alpha", ctypes.c_float),
        ("n_cycles", ctypes.c_int32), ("gain", ctypes.c_float),
        ("bias_gain", ctypes.c_float), ("eps", ctypes.c_float),
        ("pi_init", ctypes.c_float), ("pj_init", ctypes.c_float),
        ("init_noise", ctypes.c_float), ("seed", ctypes.c_uint64),
        ("n_swaps", ctypes.c_int32), ("storage", ctypes.c_int32),
        ("complement_pairs", ctypes.c_int32),
    ]


class StateView(ctypes.Structure):
    _fields_ = [("pi", ctypes.c_void_p), ("pj", ctypes.c_void_p), ("pij", ctypes.c_void_p),
                ("w", ctypes.c_void_p), ("b", ctypes.c_void_p), ("mask", ctypes.c_void_p)]


class BcpnnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2106_05373_amd/build.py")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    sig = {
        "bcpnn_config_default": (None, [ctypes.POINTER(Config), i32, i32, i32, i32, i32]),
        "bcpnn_layer_create": (i32, [ctypes.POINTER(Config), vp, vp, ctypes.POINTER(vp)]),
        "bcpnn_layer_destroy": (None, [vp]),
        "bcpnn_forward": (i32, [vp, vp, i32, vp, vp]),
        "bcpnn_train_batch": (i32, [vp, vp, i32, vp, vp]),
        "bcpnn_recompute_weights": (i32, [vp]),
        "bcpnn_structural_update": (i32, [vp, ctypes.POINTER(i32)]),
        "bcpnn_readout": (i32, [vp, vp, i32, vp]),
        "bcpnn_flush": (i32, [vp]),
        "bcpnn_structural_update_static": (i32, [vp, vp]),
        "bcpnn_get_state": (i32, [vp, ctypes.POINTER(StateView)]),
        "bcpnn_set_state": (i32, [vp, ctypes.POINTER(StateView)]),
        "bcpnn_get_mi": (i32, [vp, vp]),
        "bcpnn_profile_enable": (i32, [vp, i32]),
        "bcpnn_profile_read": (i32, [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]),
        "bcpnn_profile_read_kernel": (i32, [vp, i32, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(i32)]),
        "bcpnn_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


lib = _load()


def last_error() -> str:
    return lib.bcpnn_last_error().decode()


def _check(status: int):
    if status != 0:
        raise BcpnnError(status, last_error())


def default_config(in_hcu, in_mcu, out_hcu, out_mcu, max_batch, **overrides) -> Config:
    """bcpnn_config_default, then the given fields (storage may be "f32"/"bf16"/"m10")."""
    c = Config()
    lib.bcpnn_config_default(ctypes.byref(c), in_hcu, in_mcu, out_hcu, out_mcu, max_batch)
    for k, v in overrides.items():
        if k == "storage" and isinstance(v, str):
            v = STORAGE[v]
        if not hasattr(c, k):
            raise AttributeError(f"bcpnn_config has no field {k!r}")
        setattr(c, k, v)
    return c


def _dev_ptr(t, name, dtype=None, shape=None):
    """Data pointer of a contiguous CUDA tensor (checked), or None."""
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _host(a: np.ndarray, dtype, shape):
    a = np.ascontiguousarray(a, dtype=dtype)
    if a.size != int(np.prod(shape)):
        raise ValueError(f"host array of size {a.size}, expected shape {shape}")
    return a.reshape(shape)


class Layer:
    """A BCPNN hidden layer held on the GPU (one bcpnn_layer)."""

    def __init__(self, cfg: Config, mask: Optional[np.ndarray] = None, stream=None):
        import torch
        self.cfg = cfg
        self.n_in = cfg.in_hcu * cfg.in_mcu
        self.n_out = cfg.out_hcu * cfg.out_mcu
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        self._mask_keep = None
        mp = None
        if mask is not None:
            self._mask_keep = _host(mask, np.uint8, (cfg.in_hcu, cfg.out_hcu))
            mp = self._mask_keep.ctypes.data_as(ctypes.c_void_p)
        h = ctypes.c_void_p()
        _check(lib.bcpnn_layer_create(ctypes.byref(cfg), mp, ctypes.c_void_p(stream.cuda_stream),
                                      ctypes.byref(h)))
        self._h = h

    # -- lifetime --------------------------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None):
            lib.bcpnn_layer_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- compute ---------------------------------------------------------------------------
    def forward(self, x, y, s=None):
        import torch
        B = x.shape[0]
        _check(lib.bcpnn_forward(self._h, _dev_ptr(x, "x", torch.float32, (B, self.n_in)), B,
                                 _dev_ptr(y, "y", torch.float32, (B, self.n_out)),
                                 _dev_ptr(s, "s", torch.float32, (B, self.n_out))))

    def train_batch(self, x, target=None, y=None):
        import torch
        B = x.shape[0]
        _check(lib.bcpnn_train_batch(self._h, _dev_ptr(x, "x", torch.float32, (B, self.n_in)), B,
                                     _dev_ptr(target, "target", torch.float32, (B, self.n_out)),
                                     _dev_ptr(y, "y", torch.float32, (B, self.n_out))))

    def recompute_weights(self):
        _check(lib.bcpnn_recompute_weights(self._h))

    def structural_update(self, count: bool = True) -> Optional[int]:
        if not count:
            _check(lib.bcpnn_structural_update(self._h, None))
            return None
        n = ctypes.c_int32()
        _check(lib.bcpnn_structural_update(self._h, ctypes.byref(n)))
        return int(n.value)

    def structural_update_static(self, n_swapped=None):
        """bcpnn_structural_update_static: the swap count goes to n_swapped (a CUDA int32
        tensor of one element, or None); no allocation, no host wait."""
        import torch
        _check(lib.bcpnn_structural_update_static(
            self._h, _dev_ptr(n_swapped, "n_swapped", torch.int32, (1,))))

    def readout(self, x, winner):
        import torch
        B = x.shape[0]
        _check(lib.bcpnn_readout(self._h, _dev_ptr(x, "x", torch.float32, (B, self.n_in)), B,
                                 _dev_ptr(winner, "winner", torch.int32, (B, self.cfg.out_hcu))))

    def flush(self):
        """Applies the queued silent-block updates of Pij on the layer's stream (no host wait)."""
        _check(lib.bcpnn_flush(self._h))

    # -- state -----------------------------------------------------------------------------
    def get_state(self, which=("pi", "pj", "pij", "w", "b", "mask")) -> dict:
        shapes = dict(pi=(self.n_in,), pj=(self.n_out,), pij=(self.n_in, self.n_out),
                      w=(self.n_in, self.n_out), b=(self.n_out,),
                      mask=(self.cfg.in_hcu, self.cfg.out_hcu))
        out = {k: np.empty(shapes[k], np.uint8 if k == "mask" else np.float32) for k in which}
        v = StateView(*[out[k].ctypes.data if k in out else None
                        for k in ("pi", "pj", "pij", "w", "b", "mask")])
        _check(lib.bcpnn_get_state(self._h, ctypes.byref(v)))
        return out

    def set_state(self, st: dict):
        arrs = dict(pi=_host(st["pi"], np.float32, (self.n_in,)),
                    pj=_host(st["pj"], np.float32, (self.n_out,)),
                    pij=_host(st["pij"], np.float32, (self.n_in, self.n_out)),
                    w=_host(st["w"], np.float32, (self.n_in, self.n_out)),
                    b=_host(st["b"], np.float32, (self.n_out,)),
                    mask=_host(st["mask"], np.uint8, (self.cfg.in_hcu, self.cfg.out_hcu)))
        v = StateView(*[arrs[k].ctypes.data for k in ("pi", "pj", "pij", "w", "b", "mask")])
        _check(lib.bcpnn_set_state(self._h, ctypes.byref(v)))

    def get_mi(self) -> np.ndarray:
        mi = np.empty((self.cfg.in_hcu, self.cfg.out_hcu), np.float64)
        _check(lib.bcpnn_get_mi(self._h, mi.ctypes.data_as(ctypes.c_void_p)))
        return mi

    # -- measurement -----------------------------------------------------------------------
    def profile_enable(self, period: int = 1):
        """Time every period-th launch of each train_batch kernel with dispatch-stamped events
        (0 = off)."""
        _check(lib.bcpnn_profile_enable(self._h, int(period)))

    def profile_read(self):
        """(total ms, launches) of the silent-block sweep (the active-block kernel when the mask
        has no silent block) since the last read."""
        ms = ctypes.c_double()
        n = ctypes.c_int32()
        _check(lib.bcpnn_profile_read(self._h, ctypes.byref(ms), ctypes.byref(n)))
        return float(ms.value), int(n.value)

    def profile_read_kernel(self, kernel: str):
        """(total ms, launches) of one kernel: "sweep", "support", "active" (train_batch),
        "weights" (recompute_weights) or "structural" (MI + swap of structural_update)."""
        ms = ctypes.c_double()
        n = ctypes.c_int32()
        _check(lib.bcpnn_profile_read_kernel(self._h, KERNELS[kernel], ctypes.byref(ms),
                                             ctypes.byref(n)))
        return float(ms.value), int(n.value)
