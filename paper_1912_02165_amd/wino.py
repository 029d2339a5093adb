"""Python binding of ``include/wino_conv.h`` and ``include/wino_tune.h`` (ctypes;
argument marshalling only).

The functions keep the C names.  Every computation runs in the HIP library
``libwino_conv.so``; if it is not built, the first call raises ``ImportError``
(there is no fallback).  Tensors may be passed as torch CUDA tensors (checked for
dtype float32, device and contiguity) or as raw device addresses (int).
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# WINO_LIB selects another build of the same library (the sanitizer test's)
LIB_PATH = os.environ.get("WINO_LIB") or os.path.join(HERE, "libwino_conv.so")

WINO_OK, WINO_EINVAL, WINO_EUNSUPPORTED, WINO_ENOMEM, WINO_EHIP, WINO_EKERNEL = 0, -1, -2, -3, -4, -5
WINO_ALGO_FUSED, WINO_ALGO_THREE_STAGE, WINO_ALGO_FFT = 0, 1, 2
WINO_BUF_WEIGHTS, WINO_BUF_INPUT, WINO_BUF_PRODUCT = 0, 1, 2

ALGOS = {"fused": WINO_ALGO_FUSED, "three_stage": WINO_ALGO_THREE_STAGE, "fft": WINO_ALGO_FFT}
ALGO_NAMES = {v: k for k, v in ALGOS.items()}

# Every symbol the header declares, with (restype, argtypes).
_vp = ctypes.c_void_p
_i = ctypes.c_int
SIGNATURES = {
    "wino_conv_plan": (_vp, [_i, _i, _i, _i, _i, _i]),
    "wino_conv_plan_ex": (_vp, [_i, _i, _i, _i, _i, _i, _i, _vp]),
    "wino_conv_run": (_i, [_vp, _vp, _vp, _vp, _vp]),
    "wino_conv_set_weights": (_i, [_vp, _vp, _vp]),
    "wino_conv_run_pretransformed": (_i, [_vp, _vp, _vp, _vp]),
    "wino_conv_run_noalloc": (_i, [_i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp]),
    "wino_conv_destroy": (None, [_vp]),
    "wino_conv_workspace_bytes": (ctypes.c_size_t, [_vp]),
    "wino_conv_info": (_i, [_vp, ctypes.POINTER(ctypes.c_longlong),
                            ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "wino_conv_intermediate_dims": (_i, [_vp, _i, ctypes.POINTER(ctypes.c_longlong)]),
    "wino_conv_copy_intermediate": (_i, [_vp, _i, ctypes.POINTER(ctypes.c_float), ctypes.c_size_t]),
    "wino_conv_status": (_i, [_vp]),
    "wino_conv_debug_set_status": (_i, [_vp, ctypes.c_uint]),
    "wino_conv_describe": (_i, [_vp, ctypes.c_char_p, ctypes.c_size_t]),
    "wino_last_error": (ctypes.c_char_p, []),
    # wino_tune.h
    "wino_conv_plan_tuned": (_vp, [_i, _i, _i, _i, _i, ctypes.c_uint, ctypes.POINTER(_i),
                                   ctypes.POINTER(_i), ctypes.POINTER(ctypes.c_double)]),
    "wino_conv_plan_params": (_i, [_vp, ctypes.POINTER(_i), ctypes.POINTER(_i), ctypes.POINTER(_i),
                                   ctypes.POINTER(_i)]),
    "wino_fused_blockings": (_i, [ctypes.POINTER(_i), ctypes.POINTER(_i), ctypes.POINTER(_i), _i]),
    "wino_wisdom_lookup": (_i, [ctypes.c_char_p, _i, _i, _i, _i, _i, _i, ctypes.c_uint,
                                ctypes.POINTER(_i), ctypes.POINTER(_i), ctypes.POINTER(_i),
                                ctypes.POINTER(_i), ctypes.POINTER(_i)]),
    "wino_wisdom_save": (_i, [ctypes.c_char_p]),
    "wino_wisdom_load": (_i, [ctypes.c_char_p]),
    "wino_wisdom_clear": (None, []),
    "wino_wisdom_size": (_i, []),
}

WINO_TUNE_M2, WINO_TUNE_M4, WINO_TUNE_M5, WINO_TUNE_M6 = 1 << 2, 1 << 4, 1 << 5, 1 << 6
WINO_TUNE_M7 = 1 << 7  # three-stage only: with WINO_TUNE_THREE_STAGE
WINO_TUNE_THREE_STAGE = 1 << 8
WINO_TUNE_FFT = 1 << 9
WINO_TUNE_ALL_M = WINO_TUNE_M2 | WINO_TUNE_M4 | WINO_TUNE_M5 | WINO_TUNE_M6 | WINO_TUNE_M7

WINO_MAX_CHANNEL_SPLITS = 64


class WinoTuning(ctypes.Structure):
    _fields_ = [("tiles_per_wg", ctypes.c_int), ("k_per_wg", ctypes.c_int),
                ("c_chunk", ctypes.c_int), ("channel_splits", ctypes.c_int)]


class WinoError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"wino status {status}: {msg}")
        self.status = status


_lib = None


def lib():
    """The loaded library; raises ImportError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_1912_02165_amd.build` (hipcc, gfx950)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(l, name)
            fn.restype = res
            fn.argtypes = args
        _lib = l
    return _lib


def wino_last_error():
    msg = lib().wino_last_error()
    return msg.decode() if msg else ""


def _check(status):
    if status != WINO_OK:
        raise WinoError(status, wino_last_error())
    return status


def _ptr(t, name):
    """Device address of a float32 contiguous CUDA tensor, or an int address."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor or an int address")
    if t.dtype != torch.float32:
        raise TypeError(f"{name}: expected float32, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name}: expected a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def wino_conv_plan(N, C, K, H, W, m):
    p = lib().wino_conv_plan(N, C, K, H, W, m)
    if not p:
        raise WinoError(WINO_EINVAL, wino_last_error())
    return p


def wino_conv_plan_ex(N, C, K, H, W, m, algo=WINO_ALGO_FUSED, tuning=None):
    if isinstance(algo, str):
        algo = ALGOS[algo]
    t = None
    if tuning is not None:
        t = ctypes.byref(tuning if isinstance(tuning, WinoTuning) else WinoTuning(**tuning))
    p = lib().wino_conv_plan_ex(N, C, K, H, W, m, algo, t)
    if not p:
        raise WinoError(WINO_EINVAL, wino_last_error())
    return p


def wino_conv_run(plan, x, w, y, stream=None):
    return _check(lib().wino_conv_run(plan, _ptr(x, "x"), _ptr(w, "w"), _ptr(y, "y"),
                                      _stream(stream)))


def wino_conv_set_weights(plan, w, stream=None):
    return _check(lib().wino_conv_set_weights(plan, _ptr(w, "w"), _stream(stream)))


def wino_conv_run_pretransformed(plan, x, y, stream=None):
    return _check(lib().wino_conv_run_pretransformed(plan, _ptr(x, "x"), _ptr(y, "y"),
                                                     _stream(stream)))


def wino_conv_run_noalloc(N, C, K, H, W, m, x, w, y, status=None, stream=None):
    """y = conv(x, w) through the fused path without a plan and without allocating
    (scratch in a fixed device array per GPU; calls overlapping on one GPU race).
    status: None or a device int32/uint32 word the kernels OR their give-up bits into."""
    st = None
    if status is not None:
        st = status if isinstance(status, int) else status.data_ptr()
    return _check(lib().wino_conv_run_noalloc(N, C, K, H, W, m, _ptr(x, "x"), _ptr(w, "w"),
                                              _ptr(y, "y"), st, _stream(stream)))


def wino_conv_destroy(plan):
    lib().wino_conv_destroy(plan)


def wino_conv_workspace_bytes(plan):
    return int(lib().wino_conv_workspace_bytes(plan))


def wino_conv_info(plan):
    """(n_tiles, direct_flops, tdomain_flops)."""
    nt, df, tf = ctypes.c_longlong(), ctypes.c_double(), ctypes.c_double()
    _check(lib().wino_conv_info(plan, ctypes.byref(nt), ctypes.byref(df), ctypes.byref(tf)))
    return nt.value, df.value, tf.value


def wino_conv_intermediate_dims(plan, which):
    dims = (ctypes.c_longlong * 4)()
    _check(lib().wino_conv_intermediate_dims(plan, which, dims))
    return tuple(int(d) for d in dims)


def wino_conv_copy_intermediate(plan, which):
    """Copy an intermediate buffer to a new float32 NumPy array shaped by its dims."""
    import numpy as np
    dims = wino_conv_intermediate_dims(plan, which)
    out = np.empty(dims, dtype=np.float32)
    _check(lib().wino_conv_copy_intermediate(
        plan, which, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), out.size))
    return out


def wino_conv_plan_tuned(N, C, K, H, W, candidates=WINO_TUNE_ALL_M):
    """(plan handle, m, algo, microseconds per call) of the fastest candidate."""
    m, algo, us = ctypes.c_int(), ctypes.c_int(), ctypes.c_double()
    p = lib().wino_conv_plan_tuned(N, C, K, H, W, candidates, ctypes.byref(m), ctypes.byref(algo),
                                   ctypes.byref(us))
    if not p:
        raise WinoError(WINO_EINVAL, wino_last_error())
    return p, m.value, algo.value, us.value


def wino_conv_plan_params(plan):
    """(m, algo, tiles_per_wg, k_per_wg) of a plan (the last two 0 unless fused)."""
    m, algo, R, kit = ctypes.c_int(), ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(lib().wino_conv_plan_params(plan, ctypes.byref(m), ctypes.byref(algo), ctypes.byref(R),
                                       ctypes.byref(kit)))
    return m.value, algo.value, R.value, kit.value


def wino_fused_blockings():
    """[(m, tiles_per_wg, k_per_wg), ...] the fused kernel is built for."""
    n = lib().wino_fused_blockings(None, None, None, 0)
    m, R, kit = (ctypes.c_int * n)(), (ctypes.c_int * n)(), (ctypes.c_int * n)()
    lib().wino_fused_blockings(m, R, kit, n)
    return [(m[i], R[i], kit[i]) for i in range(n)]


def wino_conv_status(plan):
    """Raises WinoError (status WINO_EKERNEL) if a kernel wait of a call since the
    last check gave up (synchronises the device)."""
    return _check(lib().wino_conv_status(plan))


def wino_conv_debug_set_status(plan, word):
    return _check(lib().wino_conv_debug_set_status(plan, word))


def wino_conv_describe(plan):
    buf = ctypes.create_string_buffer(512)
    _check(lib().wino_conv_describe(plan, buf, len(buf)))
    return buf.value.decode()


def wino_wisdom_lookup(arch, cus, N, C, K, H, W, candidates):
    """(m, algo, tiles_per_wg, k_per_wg) of a wisdom entry, or None."""
    found, m, algo = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    R, kit = ctypes.c_int(), ctypes.c_int()
    _check(lib().wino_wisdom_lookup(arch.encode(), cus, N, C, K, H, W, candidates,
                                    ctypes.byref(found), ctypes.byref(m), ctypes.byref(algo),
                                    ctypes.byref(R), ctypes.byref(kit)))
    return (m.value, algo.value, R.value, kit.value) if found.value else None


def wino_wisdom_save(path):
    return _check(lib().wino_wisdom_save(os.fsencode(path)))


def wino_wisdom_load(path):
    return _check(lib().wino_wisdom_load(os.fsencode(path)))


def wino_wisdom_clear():
    lib().wino_wisdom_clear()


def wino_wisdom_size():
    return int(lib().wino_wisdom_size())


class Plan:
    """Owning wrapper of a plan handle (``with Plan(...) as p: p.run(x, w, y)``)."""

    def __init__(self, N, C, K, H, W, m, algo="fused", tuning=None, _handle=None):
        self.shape = (N, C, K, H, W)
        self.m = m
        self.algo = algo
        self.handle = _handle if _handle is not None else wino_conv_plan_ex(N, C, K, H, W, m, algo,
                                                                           tuning)

    @classmethod
    def tuned(cls, N, C, K, H, W, candidates=WINO_TUNE_ALL_M):
        """The fastest plan among the candidates (timed now, or from the wisdom table);
        its m, algorithm and measured call time are attributes."""
        h, m, algo, us = wino_conv_plan_tuned(N, C, K, H, W, candidates)
        p = cls(N, C, K, H, W, m, ALGO_NAMES[algo], _handle=h)
        p.call_us = us
        return p

    def _shape(self, t, shape, name):
        """A tensor argument must hold exactly the plan's tensor (raw addresses are
        passed through; the library checks their allocation's extent)."""
        if t is None or isinstance(t, int):
            return
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name}: expected shape {tuple(shape)} for this plan, got {tuple(t.shape)}")

    def _check_xy(self, x, y):
        N, C, K, H, W = self.shape
        self._shape(x, (N, C, H, W), "x")
        self._shape(y, (N, K, H, W), "y")

    def run(self, x, w, y, stream=None):
        N, C, K, H, W = self.shape
        self._check_xy(x, y)
        self._shape(w, (K, C, 3, 3), "w")
        wino_conv_run(self.handle, x, w, y, stream)

    def set_weights(self, w, stream=None):
        N, C, K, H, W = self.shape
        self._shape(w, (K, C, 3, 3), "w")
        wino_conv_set_weights(self.handle, w, stream)

    def run_pretransformed(self, x, y, stream=None):
        self._check_xy(x, y)
        wino_conv_run_pretransformed(self.handle, x, y, stream)

    def status(self):
        """Raises WinoError if a kernel wait of a call since the last check gave up."""
        wino_conv_status(self.handle)

    def describe(self):
        return wino_conv_describe(self.handle)

    def params(self):
        """(m, algo, tiles_per_wg, k_per_wg)."""
        return wino_conv_plan_params(self.handle)

    def info(self):
        return wino_conv_info(self.handle)

    def workspace_bytes(self):
        return wino_conv_workspace_bytes(self.handle)

    def intermediate(self, which):
        return wino_conv_copy_intermediate(self.handle, which)

    def close(self):
        if self.handle:
            wino_conv_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def conv2d(x, w, m=4, algo="fused", stream=None):
    """y = 3x3 conv of x (N,C,H,W) with w (K,C,3,3), stride 1, pad 1, via the library."""
    import torch
    N, C, H, W = x.shape
    K = w.shape[0]
    y = torch.empty((N, K, H, W), dtype=torch.float32, device=x.device)
    with Plan(N, C, K, H, W, m, algo) as p:
        p.run(x, w, y, stream)
        # the plan's workspace must outlive the queued work
        (torch.cuda.current_stream() if stream is None else stream).synchronize()
    return y
