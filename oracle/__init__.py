"""Python access to the CPU oracle (``oracle/cpe_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
benchmark's CPU-baseline leg.  The product path never imports this package.

``build()`` compiles ``libcpe_oracle.so`` with gcc (no fast-math, no FMA
contraction); ``decode()`` / ``decode_real()`` run the canonical and the
real-valued decoders on host numpy arrays.
"""
from __future__ import annotations

import contextlib
import ctypes
import math
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "cpe_oracle.c")
LIB = os.path.join(HERE, "libcpe_oracle.so")

CENTROID_DTYPE = np.dtype([("bin_x", "<i4"), ("bin_y", "<i4"), ("x", "<f4"), ("y", "<f4"),
                           ("score", "<f8"), ("npix", "<i4"), ("reserved", "<i4")])
assert CENTROID_DTYPE.itemsize == 32

W_KEYS = 8192          # weight buckets: 32 binades x 2^8 mantissa steps of fl32(S+1)

_lib = None


def build(verbose: bool = False, src: str = SRC, out: str = LIB) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
           "-Wall", "-Wextra", "-I", HERE, "-o", out, src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    global _lib
    if out == LIB:
        _lib = None
    return out


@contextlib.contextmanager
def using_library(path: str):
    """Temporarily route decode()/decode_real() through another build of the
    oracle source (used by the tests that plant mistakes in a copy)."""
    global _lib
    saved = _lib
    _lib = _bind(ctypes.CDLL(path))
    try:
        yield
    finally:
        _lib = saved


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = _bind(ctypes.CDLL(LIB))
    return _lib


def _bind(lib):
    P = ctypes.c_void_p
    i32 = ctypes.c_int32
    lib.cpe_oracle_decode.restype = i32
    lib.cpe_oracle_decode.argtypes = [i32, i32, i32, i32, P, P, P, P, i32, i32, i32, i32,
                                      ctypes.c_float, ctypes.c_double, P, P, P, P, P, P, P, P]
    lib.cpe_oracle_decode_ex.restype = i32
    lib.cpe_oracle_decode_ex.argtypes = [i32, i32, i32, i32, P, P, P, P, i32, i32, i32, i32,
                                         ctypes.c_float, ctypes.c_double, ctypes.c_double,
                                         P, P, P, P, P, P, P, P]
    lib.cpe_oracle_decode_real.restype = i32
    lib.cpe_oracle_decode_real.argtypes = [i32, i32, i32, i32, P, P, P, P, i32, i32, i32, i32,
                                           ctypes.c_float, ctypes.c_double, P, P, P, P]
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.float16:
        return 1
    raise TypeError(f"unsupported dtype {a.dtype}")


def decode(emb, fg, freq_x, freq_y, bins_w=32, bins_h=32, capacity=None,
           fg_threshold=0.5, peak_threshold=0.0, *, tau=math.inf, want_score=True, check=True):
    """Canonical decode.  Returns a dict with centroids (structured array of
    length min(K, capacity)), K, labels [H][W] int32, score_map, hist
    [bins_h][bins_w] uint64, pal_x, pal_y, weights (the weight buckets).
    fg=None: every pixel participates; tau: the Eq8 mask threshold in
    distance units (inf: none)."""
    lib = _load()
    emb = np.ascontiguousarray(emb)
    fg = None if fg is None else np.ascontiguousarray(fg, dtype=emb.dtype)
    H, W, D = emb.shape
    fx = np.ascontiguousarray(freq_x, dtype=np.float64)
    fy = np.ascontiguousarray(freq_y, dtype=np.float64)
    F = len(fx)
    if capacity is None:
        capacity = ((bins_w + 1) // 2) * ((bins_h + 1) // 2)
    cents = np.zeros(capacity, dtype=CENTROID_DTYPE)
    K = np.zeros(1, dtype=np.int32)
    labels = np.empty((H, W), dtype=np.int32)
    score = np.empty((H, W), dtype=np.float32) if want_score else None
    hist = np.empty((bins_h, bins_w), dtype=np.uint64)
    pal_x = np.empty((bins_w, 2 * F), dtype=np.int16)
    pal_y = np.empty((bins_h, 2 * F), dtype=np.int16)
    wt = np.empty(W_KEYS, dtype=np.uint16)
    rc = lib.cpe_oracle_decode_ex(H, W, D, _dtype_code(emb), _ptr(emb), _ptr(fg), _ptr(fx), _ptr(fy), F,
                                  bins_w, bins_h, capacity, float(fg_threshold), float(peak_threshold),
                                  float(tau), _ptr(cents), _ptr(K), _ptr(labels), _ptr(score), _ptr(hist),
                                  _ptr(pal_x), _ptr(pal_y), _ptr(wt))
    if rc != 0:
        if check:
            raise ValueError(f"oracle rejected the arguments (code {rc})")
        return {"rc": rc}
    k = int(K[0])
    return {"rc": 0, "K": k, "centroids": cents[:min(k, capacity)].copy(), "labels": labels,
            "score_map": score, "hist": hist, "pal_x": pal_x, "pal_y": pal_y, "weights": wt}


def decode_real(emb, fg, freq_x, freq_y, bins_w=32, bins_h=32, capacity=None,
                fg_threshold=0.5, peak_threshold=0.0):
    """Real-valued fp64 decode (diagnostic).  Returns hist (fp64), peaks (bin
    indices), K and labels."""
    lib = _load()
    emb = np.ascontiguousarray(emb)
    fg = np.ascontiguousarray(fg, dtype=emb.dtype)
    H, W, D = emb.shape
    fx = np.ascontiguousarray(freq_x, dtype=np.float64)
    fy = np.ascontiguousarray(freq_y, dtype=np.float64)
    if capacity is None:
        capacity = bins_w * bins_h
    hist = np.empty((bins_h, bins_w), dtype=np.float64)
    peaks = np.zeros(capacity, dtype=np.int32)
    K = np.zeros(1, dtype=np.int32)
    labels = np.empty((H, W), dtype=np.int32)
    rc = lib.cpe_oracle_decode_real(H, W, D, _dtype_code(emb), _ptr(emb), _ptr(fg), _ptr(fx), _ptr(fy),
                                    len(fx), bins_w, bins_h, capacity, float(fg_threshold),
                                    float(peak_threshold), _ptr(hist), _ptr(peaks), _ptr(K), _ptr(labels))
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (code {rc})")
    k = int(K[0])
    return {"K": k, "hist": hist, "peaks": peaks[:min(k, capacity)].copy(), "labels": labels}


def decode_frame(frame, bins=None, peak_threshold=0.0, capacity=None, **kw):
    """Convenience: decode a ``synth.Frame`` with its spec's frequencies."""
    spec = frame.spec
    fx, fy = spec.freqs()
    b = bins or spec.bins
    return decode(frame.emb, frame.fg, fx, fy, b, b, capacity, spec.fg_threshold, peak_threshold, **kw)
