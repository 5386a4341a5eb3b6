"""ctypes binding of ``libcpe_decode.so`` (the gfx950 decoder's C ABI).

Argument marshalling only: every step of the decode runs in the HIP kernels
behind the C ABI.  Device buffers are torch tensors on the GPU; their raw
pointers and torch's current HIP stream are passed through unchanged.  If
the library has not been built this module raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcpe_decode.so")

CPE_OK, CPE_ERR_INVALID_ARG, CPE_ERR_UNSUPPORTED, CPE_ERR_OUT_OF_MEMORY, CPE_ERR_HIP = range(5)
CPE_F32, CPE_F16 = 0, 1
W_KEYS = 8192

CENTROID_DTYPE = np.dtype([("bin_x", "<i4"), ("bin_y", "<i4"), ("x", "<f4"), ("y", "<f4"),
                           ("score", "<f8"), ("npix", "<i4"), ("reserved", "<i4")])

# Every entry point declared in include/cpe_decode.h.
EXPORTS = ("cpe_decode_create", "cpe_decode", "cpe_decode_ex", "cpe_decode_masks", "cpe_decode_destroy",
           "cpe_status_string", "cpe_decode_get_tables", "cpe_decode_get_histogram", "cpe_decode_workspace_bytes",
           "cpe_decode_set_stage_events", "cpe_decode_naive", "cpe_check_sqrt",
           "cpe_decode_test_fail_launch", "cpe_decode_noalloc", "cpe_decode_launch_count",
           "cpe_decode_test_search_mode")
STAGE_EVENTS = 6
MFMA_BINS = 32


def stage_layout(dec):
    """The stages of one frame of decoder dec as (name, launch index i):
    stage events 2i and 2i+1 bracket it."""
    if dec.launch_count() == 2:
        return (("compact_vote", 1), ("assign_label", 2))
    if dec.bins_w <= MFMA_BINS and dec.bins_h <= MFMA_BINS:
        return (("compact", 0), ("recover_vote", 1), ("assign_label", 2))
    return (("compact", 0), ("recover_vote", 1), ("peaks_assign_label", 2))

_lib = None


class DecodeOptions(ctypes.Structure):
    """cpe_decode_options (include/cpe_decode.h)."""
    _fields_ = [("fg_threshold", ctypes.c_float), ("reserved", ctypes.c_int32),
                ("peak_threshold", ctypes.c_double), ("tau", ctypes.c_double)]


class CpeError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


def library():
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(LIB_PATH)
        P, i32 = ctypes.c_void_p, ctypes.c_int32
        lib.cpe_decode_create.restype = i32
        lib.cpe_decode_create.argtypes = [ctypes.POINTER(P), i32, i32, i32, i32, P, P, i32, i32, i32, i32]
        lib.cpe_decode.restype = i32
        lib.cpe_decode.argtypes = [P, P, P, P, i32, i32, ctypes.c_float, ctypes.c_double, P, P, P, P]
        lib.cpe_decode_ex.restype = i32
        lib.cpe_decode_ex.argtypes = [P, P, P, P, i32, i32, ctypes.POINTER(DecodeOptions), P, P, P, P]
        lib.cpe_decode_masks.restype = i32
        lib.cpe_decode_masks.argtypes = [P, P, P, i32, i32, i32, i32, P]
        lib.cpe_decode_destroy.restype = i32
        lib.cpe_decode_destroy.argtypes = [P]
        lib.cpe_status_string.restype = ctypes.c_char_p
        lib.cpe_status_string.argtypes = [i32]
        lib.cpe_decode_get_tables.restype = i32
        lib.cpe_decode_get_tables.argtypes = [P, P, P, P]
        lib.cpe_decode_get_histogram.restype = i32
        lib.cpe_decode_get_histogram.argtypes = [P, P, P]
        lib.cpe_decode_workspace_bytes.restype = ctypes.c_size_t
        lib.cpe_decode_workspace_bytes.argtypes = [P]
        lib.cpe_decode_launch_count.restype = i32
        lib.cpe_decode_launch_count.argtypes = [P]
        lib.cpe_decode_set_stage_events.restype = i32
        lib.cpe_decode_set_stage_events.argtypes = [P, P, i32]
        lib.cpe_decode_naive.restype = i32
        lib.cpe_decode_naive.argtypes = [P, P, P, P, i32, i32, ctypes.c_float, ctypes.c_double, P, P, P, P]
        lib.cpe_decode_noalloc.restype = i32
        lib.cpe_decode_noalloc.argtypes = [P, P, P, P, i32, i32, ctypes.POINTER(DecodeOptions), P, P, P, P]
        lib.cpe_decode_test_fail_launch.restype = i32
        lib.cpe_decode_test_fail_launch.argtypes = [P, i32]
        lib.cpe_decode_test_search_mode.restype = i32
        lib.cpe_decode_test_search_mode.argtypes = [P, i32]
        lib.cpe_check_sqrt.restype = i32
        lib.cpe_check_sqrt.argtypes = [P, P]
        _lib = lib
    return _lib


def status_string(status: int) -> str:
    return library().cpe_status_string(int(status)).decode()


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(int(s.cuda_stream))


class Decoder:
    """Handle of one decoder (fixed frame size, dtype, frequencies, bins)."""

    def __init__(self, H: int, W: int, n_freq: int, dtype: str, freq_x, freq_y,
                 bins_w: int = 32, bins_h: int = 32, capacity: Optional[int] = None, D: Optional[int] = None):
        lib = library()
        self.H, self.W, self.F = int(H), int(W), int(n_freq)
        self.D = 4 * self.F if D is None else int(D)
        self.dtype = dtype
        self.bins_w, self.bins_h = int(bins_w), int(bins_h)
        self.capacity = int(capacity if capacity is not None else ((bins_w + 1) // 2) * ((bins_h + 1) // 2))
        fx = np.ascontiguousarray(freq_x, dtype=np.float64)
        fy = np.ascontiguousarray(freq_y, dtype=np.float64)
        code = {"f32": CPE_F32, "f16": CPE_F16}[dtype]
        h = ctypes.c_void_p()
        st = lib.cpe_decode_create(ctypes.byref(h), self.H, self.W, self.D, code, fx.ctypes.data, fy.ctypes.data,
                                   len(fx), self.bins_w, self.bins_h, self.capacity)
        if st != CPE_OK:
            raise CpeError(st, "cpe_decode_create")
        self._h = h

    # -- the C ABI, one call each ------------------------------------------------
    def decode(self, emb, fg, fg_threshold: float, peak_threshold: float, centroids, num_centroids, labels,
               score_map=None, stream=None, H: Optional[int] = None, W: Optional[int] = None) -> int:
        """Enqueue one frame.  ``centroids`` is a device uint8 tensor of
        capacity*32 bytes, ``num_centroids`` a device int32 tensor, ``labels``
        device int32 [H][W], ``score_map`` device float32 [H][W] or None."""
        st = library().cpe_decode(self._h, _stream_ptr(stream), _ptr(emb), _ptr(fg),
                                  self.H if H is None else H, self.W if W is None else W,
                                  float(fg_threshold), float(peak_threshold), _ptr(centroids), _ptr(num_centroids),
                                  _ptr(labels), _ptr(score_map))
        return st

    def decode_ex(self, emb, fg, fg_threshold: float, peak_threshold: float, tau: float, centroids, num_centroids,
                  labels, score_map=None, stream=None, reserved: int = 0) -> int:
        """cpe_decode_ex: ``fg`` may be None (every pixel participates);
        ``tau`` is the Eq8 mask threshold (math.inf: none)."""
        opt = DecodeOptions(float(fg_threshold), int(reserved), float(peak_threshold), float(tau))
        return library().cpe_decode_ex(self._h, _stream_ptr(stream), _ptr(emb), _ptr(fg), self.H, self.W,
                                       ctypes.byref(opt), _ptr(centroids), _ptr(num_centroids), _ptr(labels),
                                       _ptr(score_map))

    def decode_noalloc(self, emb, fg, fg_threshold: float, peak_threshold: float, tau: float, centroids,
                       num_centroids, labels, score_map=None, stream=None, reserved: int = 0) -> int:
        """cpe_decode_noalloc: cpe_decode_ex with the library's static per-device
        scratch instead of the handle's."""
        opt = DecodeOptions(float(fg_threshold), int(reserved), float(peak_threshold), float(tau))
        return library().cpe_decode_noalloc(self._h, _stream_ptr(stream), _ptr(emb), _ptr(fg), self.H, self.W,
                                            ctypes.byref(opt), _ptr(centroids), _ptr(num_centroids), _ptr(labels),
                                            _ptr(score_map))

    def masks(self, labels, first: int, count: int, masks, stream=None, H: Optional[int] = None,
              W: Optional[int] = None) -> int:
        """cpe_decode_masks: ``masks`` is a device uint8 tensor of count*H*W bytes."""
        return library().cpe_decode_masks(self._h, _stream_ptr(stream), _ptr(labels),
                                          self.H if H is None else H, self.W if W is None else W,
                                          int(first), int(count), _ptr(masks))

    def decode_naive(self, emb, fg, fg_threshold: float, peak_threshold: float, centroids, num_centroids, labels,
                     hist=None, stream=None) -> int:
        """cpe_decode_naive (the per-tuple ablation): ``hist`` is a device
        float32 [bins_h][bins_w] tensor or None."""
        return library().cpe_decode_naive(self._h, _stream_ptr(stream), _ptr(emb), _ptr(fg), self.H, self.W,
                                          float(fg_threshold), float(peak_threshold), _ptr(centroids),
                                          _ptr(num_centroids), _ptr(labels), _ptr(hist))

    def test_fail_launch(self, launch: int) -> int:
        """cpe_decode_test_fail_launch: the next decode stops before launch
        ``launch`` and reports CPE_ERR_HIP."""
        return library().cpe_decode_test_fail_launch(self._h, int(launch))

    def test_search_mode(self, mode: int) -> int:
        """cpe_decode_test_search_mode: 0 default (fast search on frames of
        2^20 pixels or more), 1 every tile recomputed exactly, 2 the fast
        search at any size."""
        return library().cpe_decode_test_search_mode(self._h, int(mode))

    def histogram(self, out, stream=None) -> int:
        return library().cpe_decode_get_histogram(self._h, _stream_ptr(stream), _ptr(out))

    def tables(self):
        pal_x = np.empty((self.bins_w, 2 * self.F), np.int16)
        pal_y = np.empty((self.bins_h, 2 * self.F), np.int16)
        wt = np.empty(W_KEYS, np.uint16)
        st = library().cpe_decode_get_tables(self._h, pal_x.ctypes.data, pal_y.ctypes.data, wt.ctypes.data)
        if st != CPE_OK:
            raise CpeError(st, "cpe_decode_get_tables")
        return pal_x, pal_y, wt

    def set_stage_events(self, events) -> int:
        """``events``: a ctypes array of CPE_STAGE_EVENTS hipEvent_t handles, or
        None; events 2i and 2i+1 bracket launch i of every later decode."""
        if events is None:
            return library().cpe_decode_set_stage_events(self._h, None, 0)
        return library().cpe_decode_set_stage_events(self._h, ctypes.cast(events, ctypes.c_void_p), len(events))

    def workspace_bytes(self) -> int:
        return int(library().cpe_decode_workspace_bytes(self._h))

    def launch_count(self) -> int:
        return int(library().cpe_decode_launch_count(self._h))

    def close(self):
        if getattr(self, "_h", None):
            library().cpe_decode_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- convenience (allocation happens here, outside the C ABI) ----------------
    def new_outputs(self, device="cuda", score=False):
        import torch
        out = {
            "centroids": torch.zeros(self.capacity * 32, dtype=torch.uint8, device=device),
            "num_centroids": torch.zeros(1, dtype=torch.int32, device=device),
            "labels": torch.empty((self.H, self.W), dtype=torch.int32, device=device),
            "score_map": torch.empty((self.H, self.W), dtype=torch.float32, device=device) if score else None,
        }
        return out

    def run(self, emb, fg, fg_threshold, peak_threshold, score=True, stream=None, outputs=None, tau=None):
        """Decode one frame, synchronise, and return host numpy results
        (cpe_decode_ex when ``tau`` is given or ``fg`` is None)."""
        import torch
        out = outputs or self.new_outputs(emb.device, score)
        if tau is None and fg is not None:
            st = self.decode(emb, fg, fg_threshold, peak_threshold, out["centroids"], out["num_centroids"],
                             out["labels"], out["score_map"], stream)
        else:
            st = self.decode_ex(emb, fg, fg_threshold, peak_threshold, math.inf if tau is None else tau,
                                out["centroids"], out["num_centroids"], out["labels"], out["score_map"], stream)
        if st != CPE_OK:
            raise CpeError(st, "cpe_decode")
        torch.cuda.synchronize()
        K = int(out["num_centroids"].item())
        cents = out["centroids"].cpu().numpy().view(CENTROID_DTYPE)[:min(K, self.capacity)].copy()
        res = {"K": K, "centroids": cents, "labels": out["labels"].cpu().numpy()}
        if out["score_map"] is not None:
            res["score_map"] = out["score_map"].cpu().numpy()
        return res


def check_sqrt(stream=None) -> int:
    """cpe_check_sqrt: the number of binary32 inputs on which the library's
    square root differs from the correctly rounded one (synchronises)."""
    import torch
    out = torch.empty(1, dtype=torch.int64, device="cuda")
    st = library().cpe_check_sqrt(_stream_ptr(stream), _ptr(out))
    if st != CPE_OK:
        raise CpeError(st, "cpe_check_sqrt")
    torch.cuda.synchronize()
    return int(out.item())


def torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "f16": torch.float16}[dtype]
