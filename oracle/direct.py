"""ctypes wrapper around the plain C direct convolution (``direct_conv.c``).  Oracle code.

``direct_conv(x, w)`` is Eq. 1 of the paper (Sec. 2.1): 3x3 cross-correlation,
stride 1, zero padding 1, fp32 inputs promoted to fp64, fp64 result.
"""

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "direct_conv.c")
_BUILD_DIR = os.path.join(_HERE, "_build")
_LIB = os.path.join(_BUILD_DIR, "liboracle_direct.so")

_lib = None


def build(force=False, sanitize=False, out=None):
    """Compile ``direct_conv.c`` with gcc/OpenMP into ``oracle/_build`` (or `out`).
    sanitize: with AddressSanitizer and UndefinedBehaviorSanitizer (for the
    sanitizer run of the oracle pins; preload libasan when loading it)."""
    os.makedirs(_BUILD_DIR, exist_ok=True)
    target = out or _LIB
    if (not force and not sanitize and os.path.exists(target)
            and os.path.getmtime(target) >= os.path.getmtime(_SRC)):
        return target
    tmp = target + ".tmp%d" % os.getpid()
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-g"] if sanitize else []
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Werror"] + san + [
        _SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, target)
    return target


def _load():
    global _lib
    if _lib is None:
        # ORACLE_DIRECT_LIB selects another build (the sanitizer run's)
        path = os.environ.get("ORACLE_DIRECT_LIB") or build()
        lib = ctypes.CDLL(path)
        i64 = ctypes.c_int64
        fp = ctypes.POINTER(ctypes.c_float)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int64)
        lib.oracle_direct_conv_f64.argtypes = [fp, fp, dp, i64, i64, i64, i64, i64]
        lib.oracle_direct_conv_f64.restype = ctypes.c_int
        lib.oracle_direct_conv_planes_f64.argtypes = [fp, fp, dp, i64, i64, i64, i64, i64,
                                                      ip, ip, i64]
        lib.oracle_direct_conv_planes_f64.restype = ctypes.c_int
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _check(x, w):
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.float32)
    if x.ndim != 4 or w.ndim != 4 or w.shape[2:] != (3, 3) or w.shape[1] != x.shape[1]:
        raise ValueError(f"expected x NCHW and w KCRS with 3x3 kernels, got {x.shape}, {w.shape}")
    return x, w


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def direct_conv(x, w):
    """y[n,k,h,v] = sum_{c,r,s} x[n,c,h+r-1,v+s-1] w[k,c,r,s] in fp64 (Eq. 1, pad 1)."""
    x, w = _check(x, w)
    N, C, H, W = x.shape
    K = w.shape[0]
    y = np.empty((N, K, H, W), dtype=np.float64)
    rc = _load().oracle_direct_conv_f64(_ptr(x, ctypes.c_float), _ptr(w, ctypes.c_float),
                                        _ptr(y, ctypes.c_double), N, C, K, H, W)
    if rc != 0:
        raise RuntimeError("oracle_direct_conv_f64 failed")
    return y


def direct_conv_planes(x, w, planes):
    """Output planes y[n, k, :, :] for each (n, k) in ``planes``, stacked (fp64)."""
    x, w = _check(x, w)
    N, C, H, W = x.shape
    K = w.shape[0]
    planes = list(planes)
    n_idx = np.array([p[0] for p in planes], dtype=np.int64)
    k_idx = np.array([p[1] for p in planes], dtype=np.int64)
    y = np.empty((len(planes), H, W), dtype=np.float64)
    rc = _load().oracle_direct_conv_planes_f64(
        _ptr(x, ctypes.c_float), _ptr(w, ctypes.c_float), _ptr(y, ctypes.c_double),
        N, C, K, H, W, _ptr(n_idx, ctypes.c_int64), _ptr(k_idx, ctypes.c_int64), len(planes))
    if rc != 0:
        raise RuntimeError("oracle_direct_conv_planes_f64: bad plane index or size")
    return y


def num_threads():
    """OpenMP threads the oracle runs on."""
    return int(_load().oracle_num_threads())
