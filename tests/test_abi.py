"""The C-ABI library: it loads, exports every entry point include/*.h
declares, and rejects bad arguments on the host (no GPU work is issued)."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

from paper_2609_16874_amd import native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(cpe_\w+)\s*\(", text))
    return names


def test_header_declares_the_binding_exports():
    assert declared_functions() == set(native.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = native.library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_null_handles():
    lib = native.library()
    assert native.status_string(0) == "ok"
    assert "invalid" in native.status_string(1)
    assert lib.cpe_decode_destroy(None) == 0
    assert lib.cpe_decode(None, None, None, None, 4, 4, 0.5, 0.0, None, None, None, None) == native.CPE_ERR_INVALID_ARG
    assert lib.cpe_decode_get_tables(None, None, None, None, None) == native.CPE_ERR_INVALID_ARG
    assert lib.cpe_decode_get_histogram(None, None, None) == native.CPE_ERR_INVALID_ARG
    assert lib.cpe_decode_workspace_bytes(None) == 0
    assert lib.cpe_decode_launch_count(None) == 0
    opt = native.DecodeOptions(0.5, 0, 0.0, float("inf"))
    assert lib.cpe_decode_ex(None, None, None, None, 4, 4, ctypes.byref(opt), None, None, None, None) == \
        native.CPE_ERR_INVALID_ARG
    assert lib.cpe_decode_masks(None, None, None, 4, 4, 0, 1, None) == native.CPE_ERR_INVALID_ARG


def test_options_struct_layout():
    """cpe_decode_options: float, int32, double, double -- 24 bytes, the
    doubles at offsets 8 and 16."""
    assert ctypes.sizeof(native.DecodeOptions) == 24
    assert native.DecodeOptions.peak_threshold.offset == 8 and native.DecodeOptions.tau.offset == 16
    text = open(os.path.join(ROOT, "include", "cpe_decode.h")).read()
    body = re.search(r"typedef struct \{([^{}]*)\} cpe_decode_options;", text).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"(\w+)\s+(\w+);", body)
    assert fields == [("float", "fg_threshold"), ("int32_t", "reserved"), ("double", "peak_threshold"),
                      ("double", "tau")]


@pytest.mark.parametrize("kw", [dict(H=0), dict(W=-1), dict(D=17), dict(n_freq=0), dict(n_freq=17, D=68),
                                dict(dtype=7), dict(bins_w=0), dict(bins_h=129), dict(cap=0), dict(cap=10 ** 6),
                                dict(H=65536, W=65536), dict(H=32768, W=65281), dict(freq_nan=True)])
def test_create_rejects_bad_arguments(kw):
    lib = native.library()
    a = dict(H=16, W=16, D=16, dtype=0, n_freq=4, bins_w=8, bins_h=8, cap=16)
    a.update({k: v for k, v in kw.items() if k != "freq_nan"})
    fx = np.ones(max(a["n_freq"], 1))
    if kw.get("freq_nan"):
        fx[0] = np.nan
    h = ctypes.c_void_p(123)
    st = lib.cpe_decode_create(ctypes.byref(h), a["H"], a["W"], a["D"], a["dtype"], fx.ctypes.data, fx.ctypes.data,
                               a["n_freq"], a["bins_w"], a["bins_h"], a["cap"])
    assert st == native.CPE_ERR_INVALID_ARG
    assert h.value is None


@pytest.mark.parametrize("D,dtype,n_freq,expect", [
    (12, 0, 4, "invalid"),        # fewer channels than 4 n_freq
    (18, 0, 4, "unsupported"),    # f32, 72-byte rows: the y block starts 36 bytes in
    (20, 1, 4, "unsupported"),    # f16, 40-byte rows: the y block starts 20 bytes in
    (35, 0, 4, "invalid"),        # odd channel count
])
def test_create_rejects_unaligned_longer_encodings(D, dtype, n_freq, expect):
    """A longer encoding (D > 4 n_freq, low harmonics only) must split into
    two 16-byte aligned axis blocks; these checks run before any device call."""
    lib = native.library()
    fx = np.ones(n_freq)
    h = ctypes.c_void_p(123)
    st = lib.cpe_decode_create(ctypes.byref(h), 16, 16, D, dtype, fx.ctypes.data, fx.ctypes.data, n_freq, 8, 8, 16)
    want = native.CPE_ERR_INVALID_ARG if expect == "invalid" else native.CPE_ERR_UNSUPPORTED
    assert st == want
    assert h.value is None
