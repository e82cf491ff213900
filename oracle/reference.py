"""ctypes wrapper around the plain C oracle in ``ref.c``.

TEST INFRASTRUCTURE ONLY: see the package docstring.  Every function here takes and
returns numpy arrays of plain integers; nothing here touches a GPU.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ref.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_i64 = ctypes.c_int64
_p = ctypes.c_void_p


def build(force: bool = True) -> str:
    """Compile ref.c into liboracle.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               "-Wall", "-Werror", _SRC, "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        build(force=False)
        L = ctypes.CDLL(_LIB_PATH)
        L.orc_row_words.restype = _i64
        L.orc_row_words.argtypes = [_i64, ctypes.c_int]
        L.orc_pack.restype = _i64
        L.orc_pack.argtypes = [_p, _i64, _i64, ctypes.c_int, ctypes.c_int, _p]
        L.orc_unpack.restype = None
        L.orc_unpack.argtypes = [_p, _i64, _i64, ctypes.c_int, ctypes.c_int, _p]
        L.orc_conv1d.restype = None
        L.orc_conv1d.argtypes = [_p, _i64, _p, ctypes.c_int, _p]
        L.orc_conv2d.restype = None
        L.orc_conv2d.argtypes = [_p, _p, _p, _p]
        L.orc_conv2d_point.restype = _i64
        L.orc_conv2d_point.argtypes = [_p, _p, _p, _i64, _i64, _i64, _i64]
        L.orc_requant_shift.restype = ctypes.c_int
        L.orc_requant_shift.argtypes = [_p, _i64, ctypes.c_int]
        L.orc_relu_requant.restype = None
        L.orc_relu_requant.argtypes = [_p, _i64, ctypes.c_int, ctypes.c_int, _p]
        L.orc_threads.restype = ctypes.c_int
        L.orc_threads.argtypes = []
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def threads() -> int:
    return lib().orc_threads()


def row_words(length: int, bits: int) -> int:
    return int(lib().orc_row_words(length, bits))


def pack(vals: np.ndarray, bits: int, signed: bool) -> Tuple[np.ndarray, int]:
    """Pack the last axis of ``vals`` into the library's storage format.

    Returns (uint32 words shaped vals.shape[:-1] + (row_words,), out-of-range count)."""
    v = np.ascontiguousarray(vals, dtype=np.int32)
    length = v.shape[-1]
    rows = v.size // length if length else 0
    out = np.zeros(v.shape[:-1] + (row_words(length, bits),), dtype=np.uint32)
    bad = lib().orc_pack(_ptr(v), rows, length, bits, int(signed), _ptr(out))
    return out, int(bad)


def unpack(words: np.ndarray, length: int, bits: int, signed: bool) -> np.ndarray:
    w = np.ascontiguousarray(words, dtype=np.uint32)
    rows = w.size // w.shape[-1] if w.shape[-1] else 0
    out = np.zeros(w.shape[:-1] + (length,), dtype=np.int32)
    lib().orc_unpack(_ptr(w), rows, length, bits, int(signed), _ptr(out))
    return out


def conv1d(x: np.ndarray, k: np.ndarray) -> np.ndarray:
    """Valid-mode true convolution: y[i] = sum_t k[t] x[i+K-1-t]."""
    xx = np.ascontiguousarray(x, dtype=np.int64)
    kk = np.ascontiguousarray(k, dtype=np.int64)
    n, K = xx.size, kk.size
    y = np.zeros(max(n - K + 1, 0), dtype=np.int64)
    lib().orc_conv1d(_ptr(xx), n, _ptr(kk), K, _ptr(y))
    return y


def out_hw(shape: Sequence[int]) -> Tuple[int, int]:
    N, C, H, W, M, KH, KW, sh, sw, ph, pw = shape
    return (H + 2 * ph - KH) // sh + 1, (W + 2 * pw - KW) // sw + 1


def conv2d(x: np.ndarray, w: np.ndarray, shape: Sequence[int]) -> np.ndarray:
    """Cross-correlation with zero padding, summed over channels, int64 result."""
    shape = tuple(int(s) for s in shape)
    N, C, H, W, M, KH, KW = shape[:7]
    assert x.shape == (N, C, H, W) and w.shape == (M, C, KH, KW)
    Ho, Wo = out_hw(shape)
    xx = np.ascontiguousarray(x, dtype=np.int32)
    ww = np.ascontiguousarray(w, dtype=np.int32)
    d = np.array(shape, dtype=np.int32)
    y = np.zeros((N, M, Ho, Wo), dtype=np.int64)
    lib().orc_conv2d(_ptr(xx), _ptr(ww), _ptr(d), _ptr(y))
    return y


def conv2d_points(x: np.ndarray, w: np.ndarray, shape: Sequence[int], idx: np.ndarray) -> np.ndarray:
    """Outputs at the (n, m, ho, wo) rows of ``idx``, each computed on its own."""
    xx = np.ascontiguousarray(x, dtype=np.int32)
    ww = np.ascontiguousarray(w, dtype=np.int32)
    d = np.array([int(s) for s in shape], dtype=np.int32)
    L = lib()
    return np.array([L.orc_conv2d_point(_ptr(xx), _ptr(ww), _ptr(d), int(a), int(b), int(c), int(e))
                     for a, b, c, e in idx], dtype=np.int64)


def requant_shift(acc: np.ndarray, bits: int) -> int:
    a = np.ascontiguousarray(acc, dtype=np.int64)
    return int(lib().orc_requant_shift(_ptr(a), a.size, bits))


def relu_requant(acc: np.ndarray, shift: int, bits: int) -> np.ndarray:
    a = np.ascontiguousarray(acc, dtype=np.int64)
    q = np.zeros(a.shape, dtype=np.int32)
    lib().orc_relu_requant(_ptr(a), a.size, shift, bits, _ptr(q))
    return q


def stack(x: np.ndarray, ws: List[np.ndarray], shapes: List[Sequence[int]], bits: int):
    """The AlexNet-shaped stack: conv, then ReLU + requantisation to unsigned b bits
    between layers (none after the last).

    Returns (accs, acts, shifts): accs[l] is layer l's int64 output, acts[l] the
    unsigned b-bit activation entering layer l (acts[0] = x), shifts[l] the shift
    applied after layer l (len(shifts) = layers - 1)."""
    acts, accs, shifts = [np.asarray(x, dtype=np.int32)], [], []
    for li, (w, shp) in enumerate(zip(ws, shapes)):
        y = conv2d(acts[-1], w, shp)
        accs.append(y)
        if li + 1 < len(ws):
            s = requant_shift(y, bits)
            shifts.append(s)
            acts.append(relu_requant(y, s, bits))
    return accs, acts, shifts
