"""ctypes binding of synth/libturnkl_synth.so (seeded logits generator)."""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libturnkl_synth.so")


class SynthParams(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("vocab", ctypes.c_int64),
        ("ld", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("n_peaks", ctypes.c_int32),
        ("student_sigma", ctypes.c_float),
        ("peak_boost", ctypes.c_float),
        ("shift_threshold", ctypes.c_uint32),
        ("reserved", ctypes.c_uint32),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python synth/build.py`")
        l = ctypes.CDLL(LIB_PATH)
        l.synth_fill_device.restype = ctypes.c_int
        l.synth_fill_device.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p]
        l.synth_fill_host.restype = ctypes.c_int
        l.synth_fill_host.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_void_p,
                                      ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_int]
        l.synth_fill_host_rows.restype = ctypes.c_int
        l.synth_fill_host_rows.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int]
        _lib = l
    return _lib


def fill_host(params: SynthParams, teacher_sigma: np.ndarray, r0: int, r1: int,
              zs: np.ndarray | None, zt: np.ndarray | None, n_threads: int = 0) -> None:
    """Write rows [r0, r1) into host arrays whose first row is row r0."""
    if n_threads <= 0:
        n_threads = min(16, os.cpu_count() or 1)
    ts = np.ascontiguousarray(teacher_sigma, dtype=np.float32)
    rc = lib().synth_fill_host(ctypes.byref(params), ts.ctypes.data, r0, r1,
                               None if zs is None else zs.ctypes.data,
                               None if zt is None else zt.ctypes.data, n_threads)
    if rc != 0:
        raise RuntimeError(f"synth_fill_host failed ({rc})")


def fill_host_rows(params: SynthParams, teacher_sigma: np.ndarray, rows: np.ndarray,
                   zs: np.ndarray | None, zt: np.ndarray | None, n_threads: int = 0) -> None:
    """Write the listed rows (absolute indices) into consecutive rows of host arrays."""
    if n_threads <= 0:
        n_threads = min(16, os.cpu_count() or 1)
    ts = np.ascontiguousarray(teacher_sigma, dtype=np.float32)
    r = np.ascontiguousarray(rows, dtype=np.int64)
    rc = lib().synth_fill_host_rows(ctypes.byref(params), ts.ctypes.data, r.ctypes.data, r.shape[0],
                                    None if zs is None else zs.ctypes.data,
                                    None if zt is None else zt.ctypes.data, n_threads)
    if rc != 0:
        raise RuntimeError(f"synth_fill_host_rows failed ({rc})")


def fill_device(params: SynthParams, teacher_sigma_ptr: int, r0: int, r1: int,
                zs_ptr: int | None, zt_ptr: int | None, stream: int) -> None:
    """Write rows [r0, r1) into device buffers whose first row is row r0."""
    rc = lib().synth_fill_device(ctypes.byref(params), teacher_sigma_ptr, r0, r1,
                                 zs_ptr, zt_ptr, stream)
    if rc != 0:
        raise RuntimeError(f"synth_fill_device failed ({rc})")
