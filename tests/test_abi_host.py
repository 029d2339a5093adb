"""The C-ABI library loads and exports every symbol of include/wino_conv.h, and its
host-side argument checks fail cleanly.  No GPU is touched: every case here is
rejected before any HIP call is made."""

import ctypes
import os
import re

import pytest

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import wino

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wino_conv.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wino_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(wino.LIB_PATH):
        from paper_1912_02165_amd import build
        build.build()
    return wc.lib()


def test_header_declares_the_abi():
    names = declared_functions()
    for n in ("wino_conv_plan", "wino_conv_plan_ex", "wino_conv_run", "wino_conv_destroy",
              "wino_conv_workspace_bytes", "wino_conv_info", "wino_last_error"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_covers_every_declared_symbol():
    assert sorted(wino.SIGNATURES) == declared_functions()


def _plan_fails(lib, *args):
    p = lib.wino_conv_plan_ex(*args)
    assert not p
    return wc.wino_last_error()


@pytest.mark.parametrize("args", [
    (0, 64, 64, 56, 56, 4), (1, 0, 64, 56, 56, 4), (1, 64, -1, 56, 56, 4),
    (1, 64, 64, 0, 56, 4), (1, 64, 64, 56, 0, 4)])
def test_bad_sizes(lib, args):
    msg = _plan_fails(lib, *args, wino.WINO_ALGO_FUSED, None)
    assert "sizes must be >= 1" in msg


@pytest.mark.parametrize("m", [0, 1, 3, 5, 7, 8])
def test_bad_m(lib, m):
    assert "only F(2x2" in _plan_fails(lib, 1, 4, 4, 8, 8, m, wino.WINO_ALGO_FUSED, None)


def test_too_large(lib):
    assert "2^31" in _plan_fails(lib, 64, 512, 512, 224, 224, 4, wino.WINO_ALGO_FUSED, None)


def test_bad_algo(lib):
    assert "unknown algorithm" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, 7, None)


def test_bad_tuning(lib):
    t = wino.WinoTuning(schedule=wino.WINO_SCHED_PER_WAVE, k_blocks_per_wave=3)
    assert "not built" in _plan_fails(lib, 1, 4, 4, 8, 8, 6, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    t = wino.WinoTuning(schedule=wino.WINO_SCHED_SHARED, tile_blocks=2)
    assert "not built" in _plan_fails(lib, 1, 4, 4, 8, 8, 6, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    t = wino.WinoTuning(schedule=5)
    assert "not built" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    t = wino.WinoTuning(waves_per_group=-1)
    assert ">= 0" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, wino.WINO_ALGO_FUSED, ctypes.byref(t))


def test_forced_allocation_failure(lib, monkeypatch):
    monkeypatch.setenv("WINO_TEST_FAIL_ALLOC", "1")
    msg = _plan_fails(lib, 1, 4, 4, 8, 8, 4, wino.WINO_ALGO_THREE_STAGE, None)
    assert "allocation" in msg


def test_null_plan_calls(lib):
    assert lib.wino_conv_run(None, None, None, None, None) == wino.WINO_EINVAL
    assert "NULL" in wc.wino_last_error()
    assert lib.wino_conv_set_weights(None, None, None) == wino.WINO_EINVAL
    assert lib.wino_conv_run_pretransformed(None, None, None, None) == wino.WINO_EINVAL
    assert lib.wino_conv_info(None, None, None, None) == wino.WINO_EINVAL
    assert lib.wino_conv_workspace_bytes(None) == 0
    dims = (ctypes.c_longlong * 4)()
    assert lib.wino_conv_intermediate_dims(None, 0, dims) == wino.WINO_EINVAL
    lib.wino_conv_destroy(None)


def test_python_errors_raise(lib):
    with pytest.raises(wc.WinoError):
        wc.wino_conv_plan(1, 4, 4, 8, 8, 3)
