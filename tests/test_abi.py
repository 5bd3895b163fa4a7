"""The C-ABI library loads here (no GPU) and exports every symbol that
include/gm.h declares; the host-side checks of gm_model_create reject bad
configurations before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2509_16248_amd import gm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "gm.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(gm_[a-z0-9_]+)\s*\(", src)
    return sorted(set(n for n in names if not n.endswith("_cb")))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(gm.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = gm.lib()
    for name in declared_functions():
        assert hasattr(L, name), name


def test_strerror_and_null_checks_without_device():
    assert gm.gm_strerror(gm.GM_E_INVAL) == "invalid argument"
    L = gm.lib()
    out = ctypes.c_void_p()
    assert L.gm_model_create(None, None, ctypes.byref(out)) == gm.GM_E_INVAL
    assert out.value is None
    cfg = gm.gm_config(abi_version=99)
    assert L.gm_model_create(ctypes.byref(cfg), None, ctypes.byref(out)) == gm.GM_E_INVAL
    assert b"abi" in L.gm_last_error()


@pytest.mark.parametrize("field,value,msg", [
    ("n_heads", 5, b"multiple of n_heads"),
    ("d_ff", 100, b"multiples of 64"),
    ("max_batch", 2000, b"max_batch"),
    ("fp16_clamp", 1, b"fp16_clamp"),
])
def test_config_validation(field, value, msg):
    import synth
    from paper_2509_16248_amd.model import make_config
    c = make_config(synth.preset("causal_lm_768"))
    setattr(c, field, value)
    w = gm.gm_weights()
    out = ctypes.c_void_p()
    assert gm.lib().gm_model_create(ctypes.byref(c), ctypes.byref(w), ctypes.byref(out)) == gm.GM_E_INVAL
    assert msg in gm.lib().gm_last_error()
