"""Python driver of the CPU oracle (``bcpnn_oracle.c``).

TEST INFRASTRUCTURE: only the tests, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package.  The product path (``paper_2106_05373_amd``)
never imports it, and it imports nothing from the product except the seeded input
generators, which live in a module of their own.

The C library computes in fp64 from fp32 state; this module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "bcpnn_oracle.c")
# a test may point this at another build of the same source (planted-mistake checks)
LIB = os.environ.get("BCPNN_ORACLE_LIB", os.path.join(_HERE, "liboracle.so"))

STORAGE = {"f32": 0, "bf16": 1, "m10": 2}


def build(out: str = LIB) -> str:
    """Compile the oracle with gcc (IEEE fp64, no contraction, OpenMP)."""
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", out, SRC, "-lm"]
    subprocess.run(cmd, check=True, cwd=_HERE)
    return out


class Params(ctypes.Structure):
    _fields_ = [
        ("in_hcu", ctypes.c_int32), ("in_mcu", ctypes.c_int32),
        ("out_hcu", ctypes.c_int32), ("out_mcu", ctypes.c_int32),
        ("alpha", ctypes.c_float), ("n_cycles", ctypes.c_int32),
        ("gain", ctypes.c_float), ("bias_gain", ctypes.c_float), ("eps", ctypes.c_float),
        ("pi_init", ctypes.c_float), ("pj_init", ctypes.c_float),
        ("init_noise", ctypes.c_float), ("seed", ctypes.c_uint64),
        ("n_swaps", ctypes.c_int32), ("storage", ctypes.c_int32),
    ]


_lib_handle = None


def lib() -> ctypes.CDLL:
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        P = ctypes.POINTER(Params)
        f32 = ctypes.POINTER(ctypes.c_float)
        f64 = ctypes.POINTER(ctypes.c_double)
        u8 = ctypes.POINTER(ctypes.c_uint8)
        i32p = ctypes.POINTER(ctypes.c_int32)
        i32 = ctypes.c_int32
        sig = {
            "oracle_threads": (ctypes.c_int, []),
            "oracle_set_threads": (None, [ctypes.c_int]),
            "oracle_round_storage": (ctypes.c_float, [ctypes.c_float, i32]),
            "oracle_splitmix_uniform": (ctypes.c_double, [ctypes.c_uint64, ctypes.c_uint64]),
            "oracle_init_state": (None, [P, u8, f32, f32, f32, f32, f32]),
            "oracle_support": (None, [P, i32, f32, f32, f32, f32]),
            "oracle_softmax": (None, [P, i32, f32, f32]),
            "oracle_update_traces": (None, [P, i32, f32, f32, f32, f32, f32]),
            "oracle_update_weights": (None, [P, u8, f32, f32, f32, f32, f32]),
            "oracle_mutual_information": (None, [P, f32, f32, f32, f64]),
            "oracle_plasticity_swap": (i32, [P, f64, u8, i32p]),
            "oracle_structural_update": (i32, [P, f32, f32, f32, u8, f32, f64, i32p]),
            "oracle_readout": (None, [P, i32, f32, i32p]),
            "oracle_train_batch": (None, [P, i32, f32, f32, f32, f32, f32, f32, f32, f32, f32,
                                          u8]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib_handle = L
    return _lib_handle


def _ptr(a: Optional[np.ndarray], ctype):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _f32(a):
    return _ptr(a, ctypes.c_float)


def _f64(a):
    return _ptr(a, ctypes.c_double)


def _u8(a):
    return _ptr(a, ctypes.c_uint8)


def _i32(a):
    return _ptr(a, ctypes.c_int32)


def threads() -> int:
    return int(lib().oracle_threads())


def set_threads(n: int) -> None:
    """OpenMP threads of the oracle's loops from now on (results do not depend on it)."""
    lib().oracle_set_threads(int(n))


def splitmix_uniform(seed: int, idx: int) -> float:
    return float(lib().oracle_splitmix_uniform(seed, idx))


def round_storage(v: float, storage: str) -> float:
    return float(lib().oracle_round_storage(ctypes.c_float(v), STORAGE[storage]))


def make_params(in_hcu, in_mcu, out_hcu, out_mcu, alpha=1e-3, n_cycles=1, gain=1.0,
                bias_gain=1.0, eps=1e-8, pi_init=0.0, pj_init=0.0, init_noise=0.1, seed=0,
                n_swaps=1, storage="f32") -> Params:
    return Params(in_hcu, in_mcu, out_hcu, out_mcu, alpha, n_cycles, gain, bias_gain, eps,
                  pi_init, pj_init, init_noise, seed, n_swaps,
                  STORAGE[storage] if isinstance(storage, str) else storage)


def _c(a, dtype=np.float32):
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------------------------------
# Function-level wrappers (each returns new arrays; inputs are not modified)
# ------------------------------------------------------------------------------------------
def dims(p: Params):
    return p.in_hcu * p.in_mcu, p.out_hcu * p.out_mcu


def init_state(p: Params, mask: np.ndarray):
    n_in, n_out = dims(p)
    pi = np.empty(n_in, np.float32)
    pj = np.empty(n_out, np.float32)
    pij = np.empty((n_in, n_out), np.float32)
    w = np.empty((n_in, n_out), np.float32)
    b = np.empty(n_out, np.float32)
    mask = _c(mask, np.uint8)
    lib().oracle_init_state(ctypes.byref(p), _u8(mask), _f32(pi), _f32(pj), _f32(pij), _f32(w),
                            _f32(b))
    return dict(pi=pi, pj=pj, pij=pij, w=w, b=b, mask=mask.copy())


def support(p: Params, x, w, b):
    n_in, n_out = dims(p)
    x, w, b = _c(x), _c(w), _c(b)
    s = np.empty((x.shape[0], n_out), np.float32)
    lib().oracle_support(ctypes.byref(p), x.shape[0], _f32(x), _f32(w), _f32(b), _f32(s))
    return s


def softmax(p: Params, s):
    s = _c(s)
    y = np.empty_like(s)
    lib().oracle_softmax(ctypes.byref(p), s.shape[0], _f32(s), _f32(y))
    return y


def update_traces(p: Params, x, y, pi, pj, pij):
    x, y = _c(x), _c(y)
    pi, pj, pij = _c(pi).copy(), _c(pj).copy(), _c(pij).copy()
    lib().oracle_update_traces(ctypes.byref(p), x.shape[0], _f32(x), _f32(y), _f32(pi), _f32(pj),
                               _f32(pij))
    return pi, pj, pij


def update_weights(p: Params, mask, pi, pj, pij):
    n_in, n_out = dims(p)
    w = np.empty((n_in, n_out), np.float32)
    b = np.empty(n_out, np.float32)
    lib().oracle_update_weights(ctypes.byref(p), _u8(_c(mask, np.uint8)), _f32(_c(pi)),
                                _f32(_c(pj)), _f32(_c(pij)), _f32(w), _f32(b))
    return w, b


def mutual_information(p: Params, pi, pj, pij):
    mi = np.empty((p.in_hcu, p.out_hcu), np.float64)
    lib().oracle_mutual_information(ctypes.byref(p), _f32(_c(pi)), _f32(_c(pj)), _f32(_c(pij)),
                                    _f64(mi))
    return mi


def plasticity_swap(p: Params, mi, mask):
    mask = _c(mask, np.uint8).copy()
    swaps = np.empty((p.out_hcu, p.n_swaps, 2), np.int32)
    n = lib().oracle_plasticity_swap(ctypes.byref(p), _f64(_c(mi, np.float64)), _u8(mask),
                                     _i32(swaps))
    return int(n), mask, swaps


def readout(p: Params, s):
    s = _c(s)
    win = np.empty((s.shape[0], p.out_hcu), np.int32)
    lib().oracle_readout(ctypes.byref(p), s.shape[0], _f32(s), _i32(win))
    return win


# ------------------------------------------------------------------------------------------
# Stateful layer with the same calls as the GPU library
# ------------------------------------------------------------------------------------------
class OracleLayer:
    """A BCPNN hidden layer held on the host, stepped by the oracle."""

    def __init__(self, params: Params, mask: Optional[np.ndarray] = None):
        self.p = params
        if mask is None:
            mask = np.ones((params.in_hcu, params.out_hcu), np.uint8)
        assert mask.shape == (params.in_hcu, params.out_hcu)
        st = init_state(params, mask)
        self.pi, self.pj, self.pij, self.w, self.b, self.mask = (
            st["pi"], st["pj"], st["pij"], st["w"], st["b"], st["mask"])

    @property
    def n_in(self):
        return self.p.in_hcu * self.p.in_mcu

    @property
    def n_out(self):
        return self.p.out_hcu * self.p.out_mcu

    def get_state(self):
        return dict(pi=self.pi.copy(), pj=self.pj.copy(), pij=self.pij.copy(), w=self.w.copy(),
                    b=self.b.copy(), mask=self.mask.copy())

    def set_state(self, st):
        self.pi = _c(st["pi"]).copy()
        self.pj = _c(st["pj"]).copy()
        self.pij = _c(st["pij"]).reshape(self.n_in, self.n_out).copy()
        self.w = _c(st["w"]).reshape(self.n_in, self.n_out).copy()
        self.b = _c(st["b"]).copy()
        self.mask = _c(st["mask"], np.uint8).reshape(self.p.in_hcu, self.p.out_hcu).copy()

    def forward(self, x):
        s = support(self.p, x, self.w, self.b)
        return s, softmax(self.p, s)

    def train_batch(self, x, target=None):
        x = _c(x)
        B = x.shape[0]
        s = np.empty((B, self.n_out), np.float32)
        y = np.empty((B, self.n_out), np.float32)
        t = None if target is None else _c(target)
        lib().oracle_train_batch(ctypes.byref(self.p), B, _f32(x), _f32(t), _f32(s), _f32(y),
                                 _f32(self.pi), _f32(self.pj), _f32(self.pij), _f32(self.w),
                                 _f32(self.b), _u8(self.mask))
        return s, y

    def recompute_weights(self):
        self.w, self.b = update_weights(self.p, self.mask, self.pi, self.pj, self.pij)

    def structural_update(self):
        mi = np.empty((self.p.in_hcu, self.p.out_hcu), np.float64)
        swaps = np.empty((self.p.out_hcu, self.p.n_swaps, 2), np.int32)
        n = lib().oracle_structural_update(ctypes.byref(self.p), _f32(self.pi), _f32(self.pj),
                                           _f32(self.pij), _u8(self.mask), _f32(self.w),
                                           _f64(mi), _i32(swaps))
        return int(n), mi, swaps

    def readout(self, x):
        s = support(self.p, x, self.w, self.b)
        return readout(self.p, s)
