"""The C-ABI library without a GPU: it loads, exports every function include/bcpnn.h declares,
and rejects invalid arguments on the host before any device work."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bcpnn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bcpnn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def b():
    from paper_2106_05373_amd import bcpnn
    return bcpnn


def test_header_declares_the_expected_entry_points():
    names = declared_functions()
    for must in ("bcpnn_layer_create", "bcpnn_forward", "bcpnn_train_batch",
                 "bcpnn_recompute_weights", "bcpnn_structural_update", "bcpnn_readout"):
        assert must in names


def test_library_exports_every_declared_function(b):
    for name in declared_functions():
        assert hasattr(b.lib, name), name
    assert set(declared_functions()) == set(b.EXPORTS)


def test_default_config(b):
    c = b.default_config(784, 2, 30, 100, 128)
    assert (c.in_hcu, c.in_mcu, c.out_hcu, c.out_mcu, c.max_batch) == (784, 2, 30, 100, 128)
    assert c.alpha == pytest.approx(1e-3) and c.n_cycles == 1 and c.gain == 1.0
    assert c.eps == pytest.approx(1e-8) and c.n_swaps == 1 and c.storage == 0
    assert c.complement_pairs == 0


BAD = {
    "zero hcu": dict(in_hcu=0),
    "negative mcu": dict(out_mcu=-2),
    "out_mcu too large": dict(out_mcu=1025),
    "alpha 0": dict(alpha=0.0),
    "alpha above 1": dict(alpha=1.5),
    "alpha nan": dict(alpha=float("nan")),
    "cycles 0": dict(n_cycles=0),
    "negative gain": dict(gain=-1.0),
    "eps 0": dict(eps=0.0),
    "eps subnormal": dict(eps=1e-40),
    "max_batch 0": dict(max_batch=0),
    "max_batch above 2^20": dict(max_batch=(1 << 20) + 1),
    "N_out above 2^22": dict(out_hcu=(1 << 22) // 1024 + 1, out_mcu=1024),
    "HCU pairs above 2^26": dict(in_hcu=40000, out_hcu=2000, out_mcu=1),
    "row tiles x hidden HCUs above 2^23": dict(max_batch=1 << 20, out_hcu=200, out_mcu=1),
    "swaps negative": dict(n_swaps=-1),
    "swaps too many": dict(n_swaps=257),
    "storage unknown": dict(storage=7),
    "pi_init above 1": dict(pi_init=2.0),
    "noise negative": dict(init_noise=-0.1),
    "complement pairs of 3 MCUs": dict(in_mcu=3, complement_pairs=1),
    "complement pairs flag 2": dict(complement_pairs=2),
}


@pytest.mark.parametrize("case", list(BAD))
def test_invalid_config_rejected_on_host(b, case):
    c = b.default_config(8, 2, 3, 4, 16)
    for k, v in BAD[case].items():
        setattr(c, k, v)
    h = ctypes.c_void_p()
    st = b.lib.bcpnn_layer_create(ctypes.byref(c), None, None, ctypes.byref(h))
    assert st == -1, (case, b.last_error())
    assert not h.value
    assert b.last_error()


@pytest.mark.parametrize("bad", ["empty column", "value 2"])
def test_invalid_mask_rejected_on_host(b, bad):
    c = b.default_config(8, 2, 3, 4, 16)
    m = np.ones((8, 3), np.uint8)
    if bad == "empty column":
        m[:, 1] = 0
    else:
        m[2, 2] = 2
    h = ctypes.c_void_p()
    st = b.lib.bcpnn_layer_create(ctypes.byref(c), m.ctypes.data_as(ctypes.c_void_p), None,
                                  ctypes.byref(h))
    assert st == -1
    assert "mask" in b.last_error() or "active" in b.last_error()


def test_null_layer_calls_are_rejected(b):
    L = b.lib
    assert L.bcpnn_forward(None, None, 1, None, None) == -1
    assert L.bcpnn_train_batch(None, None, 1, None, None) == -1
    assert L.bcpnn_recompute_weights(None) == -1
    assert L.bcpnn_structural_update(None, None) == -1
    assert L.bcpnn_readout(None, None, 1, None) == -1
    assert L.bcpnn_get_mi(None, None) == -1
    assert L.bcpnn_flush(None) == -1
    assert L.bcpnn_layer_create(None, None, None, None) == -1
    L.bcpnn_layer_destroy(None)
