"""Loader for the C oracle of Eq. (1) (``conv_ref.c``) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check and the benchmark's cpu_baseline leg may use
this module.  It builds ``liboracle_conv.so`` from ``conv_ref.c`` with the host
C compiler (gcc, -O2, no fast-math, OpenMP) and calls it through ctypes.

All inputs are float32 numpy arrays (bf16 inputs are passed as their exact
float32 widening); all outputs are float64.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "conv_ref.c")
_LIB = os.path.join(_HERE, "liboracle_conv.so")
_lib = None


def build(force=True):
    """Compile the oracle library (host C only)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Werror",
           _SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build(force=False)
        lib = ctypes.CDLL(_LIB)
        i32, i64 = ctypes.c_int, ctypes.c_int64
        fp, dp, lp = (ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double),
                      ctypes.POINTER(ctypes.c_int64))
        lib.oracle_conv_fwd.argtypes = [i32] * 7 + [fp, fp, dp]
        lib.oracle_conv_fwd.restype = i32
        lib.oracle_conv_fwd_points.argtypes = [i32] * 7 + [fp, fp, lp, i64, dp]
        lib.oracle_conv_fwd_points.restype = i32
        lib.oracle_conv_fwd_ex.argtypes = [i32] * 11 + [fp, fp, dp]
        lib.oracle_conv_fwd_ex.restype = i32
        lib.oracle_conv_fwd_ex_points.argtypes = [i32] * 11 + [fp, fp, lp, i64, dp]
        lib.oracle_conv_fwd_ex_points.restype = i32
        lib.oracle_set_num_threads.argtypes = [i32]
        lib.oracle_set_num_threads.restype = i32
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = i32
        _lib = lib
    return _lib


def _f32(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    return x, x.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def conv_fwd(In, Ker):
    """Out = Eq. (1) of In [N,C,H,W] and Ker [K,C,R,S], as float64 [N,K,P,Q]."""
    In, pin = _f32(In)
    Ker, pker = _f32(Ker)
    N, C, H, W = In.shape
    K, C2, R, S = Ker.shape
    if C2 != C:
        raise ValueError("channel mismatch")
    if R > H or S > W:
        raise ValueError("kernel larger than input")
    out = np.empty((N, K, H - R + 1, W - S + 1), dtype=np.float64)
    rc = _load().oracle_conv_fwd(N, C, K, H, W, R, S, pin, pker,
                                 out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError(f"oracle_conv_fwd returned {rc}")
    return out


def conv_fwd_points(In, Ker, flat_idx):
    """Selected outputs of Eq. (1): ``flat_idx`` indexes the flattened [N,K,P,Q]."""
    In, pin = _f32(In)
    Ker, pker = _f32(Ker)
    N, C, H, W = In.shape
    K, C2, R, S = Ker.shape
    if C2 != C:
        raise ValueError("channel mismatch")
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.empty(idx.shape, dtype=np.float64)
    rc = _load().oracle_conv_fwd_points(
        N, C, K, H, W, R, S, pin, pker, idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
        idx.size, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError(f"oracle_conv_fwd_points returned {rc}")
    return out


def num_threads():
    return int(_load().oracle_num_threads())


def set_num_threads(n):
    """Threads of the oracle's later OpenMP regions; returns the previous count."""
    return int(_load().oracle_set_num_threads(int(n)))


def ex_extents(H, W, R, S, stride, pad):
    """Output extents P, Q of the strided, padded form (None if undefined)."""
    sh, sw = stride
    ph, pw = pad
    if sh <= 0 or sw <= 0 or ph < 0 or pw < 0 or H + 2 * ph < R or W + 2 * pw < S:
        return None
    return (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1


def conv_fwd_ex(In, Ker, stride=(1, 1), pad=(0, 0)):
    """Strided, zero-padded correlation (see ``conv_ref.c``), float64 [N,K,P,Q]."""
    In, pin = _f32(In)
    Ker, pker = _f32(Ker)
    N, C, H, W = In.shape
    K, C2, R, S = Ker.shape
    if C2 != C:
        raise ValueError("channel mismatch")
    ext = ex_extents(H, W, R, S, stride, pad)
    if ext is None:
        raise ValueError("undefined strided shape")
    out = np.empty((N, K) + ext, dtype=np.float64)
    rc = _load().oracle_conv_fwd_ex(N, C, K, H, W, R, S, stride[0], stride[1], pad[0], pad[1], pin, pker,
                                    out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError(f"oracle_conv_fwd_ex returned {rc}")
    return out


def conv_fwd_ex_points(In, Ker, flat_idx, stride=(1, 1), pad=(0, 0)):
    """Selected outputs of the strided, padded form (flat [N,K,P,Q] indices)."""
    In, pin = _f32(In)
    Ker, pker = _f32(Ker)
    N, C, H, W = In.shape
    K, C2, R, S = Ker.shape
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.float64)
    rc = _load().oracle_conv_fwd_ex_points(
        N, C, K, H, W, R, S, stride[0], stride[1], pad[0], pad[1], pin, pker,
        idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), idx.size,
        out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError(f"oracle_conv_fwd_ex_points returned {rc}")
    return out
