"""The C-ABI library loads and exports every symbol of include/*.h, and its
host-side argument checks fail cleanly; the wisdom table's file format round-trips.
No GPU is touched: every case here is rejected before any HIP call is made."""

import ctypes
import glob
import os
import re

import pytest

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import wino

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"\b(wino_\w+)\s*\(", text))
    return sorted(names)


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


@pytest.mark.parametrize("m", [0, 1, 3, 8])
def test_bad_m(lib, m):
    assert "only F(2x2" in _plan_fails(lib, 1, 4, 4, 8, 8, m, wino.WINO_ALGO_FUSED, None)


def test_m7_is_three_stage_only(lib):
    """F(7x7,3x3) is refused by the fused algorithm (before any HIP call) and by the
    no-allocation entry point, which runs the fused kernel."""
    assert "three-stage algorithm only" in _plan_fails(lib, 1, 4, 4, 8, 8, 7, wino.WINO_ALGO_FUSED, None)
    assert "m = 14" in _plan_fails(lib, 1, 4, 4, 8, 8, 7, wino.WINO_ALGO_FFT, None)
    assert lib.wino_conv_run_noalloc(1, 4, 4, 8, 8, 7, None, None, None, None, None) == wino.WINO_EUNSUPPORTED
    assert "three-stage algorithm only" in wc.wino_last_error()


@pytest.mark.parametrize("m", [2, 4, 6, 13, 16])
def test_fft_needs_m14(lib, m):
    assert "m = 14" in _plan_fails(lib, 1, 4, 4, 8, 8, m, wino.WINO_ALGO_FFT, None)


def test_m14_is_fft_only(lib):
    for algo in (wino.WINO_ALGO_FUSED, wino.WINO_ALGO_THREE_STAGE):
        assert "only F(2x2" in _plan_fails(lib, 1, 4, 4, 8, 8, 14, algo, None)


def test_fft_refuses_channel_splits(lib):
    t = wino.WinoTuning(channel_splits=2)
    assert "fused algorithm only" in _plan_fails(lib, 1, 8, 4, 8, 8, 14, wino.WINO_ALGO_FFT, ctypes.byref(t))


def test_algorithm_names():
    assert wino.ALGOS == {"fused": 0, "three_stage": 1, "fft": 2}
    with open(os.path.join(ROOT, "include", "wino_conv.h")) as f:
        hdr = f.read()
    for name, value in (("WINO_ALGO_FUSED", 0), ("WINO_ALGO_THREE_STAGE", 1), ("WINO_ALGO_FFT", 2)):
        assert re.search(r"%s = %d\b" % (name, value), hdr)


def test_blockings_listed_match_header(lib):
    """wino_fused_blockings lists the blockings the header documents as built."""
    got = wc.wino_fused_blockings()
    assert got == [(2, 32, 64), (2, 16, 64), (2, 32, 32), (2, 16, 32), (2, 16, 16),
                   (4, 16, 64), (4, 16, 32), (5, 16, 32), (5, 16, 16), (6, 16, 32), (6, 16, 16)]
    with open(os.path.join(ROOT, "include", "wino_conv.h")) as f:
        hdr = f.read()
    for m, R, k in got:
        assert f"({R}, {k})" in hdr


def test_too_large(lib):
    assert "2^31" in _plan_fails(lib, 64, 512, 512, 224, 224, 4, wino.WINO_ALGO_FUSED, None)


def test_transformed_kernels_too_large(lib):
    """The kernels address the transformed kernels with 32-bit byte offsets: a layer
    whose W' reaches 2^32 bytes (C = K = 4096 at F(6): 4096 * 4096 * 64 * 4 bytes) is
    refused before any allocation instead of wrapping the offsets."""
    assert "2^32" in _plan_fails(lib, 1, 4096, 4096, 14, 14, 6, wino.WINO_ALGO_FUSED, None)
    assert "2^32" in _plan_fails(lib, 1, 4096, 4096, 14, 14, 6, wino.WINO_ALGO_THREE_STAGE, None)


def test_bad_algo(lib):
    assert "unknown algorithm" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, 7, None)


@pytest.mark.parametrize("m, fields", [
    (6, dict(tiles_per_wg=32)),                 # F(6) holds 16 tiles per task
    (6, dict(k_per_wg=64)),                     # 16 x 64 x 64 results do not fit registers
    (4, dict(k_per_wg=16)),
    (4, dict(tiles_per_wg=32, k_per_wg=64)),
    (2, dict(tiles_per_wg=8)),
    (5, dict(k_per_wg=48)),
])
def test_bad_tuning(lib, m, fields):
    t = wino.WinoTuning(**fields)
    assert "not built" in _plan_fails(lib, 1, 4, 4, 8, 8, m, wino.WINO_ALGO_FUSED, ctypes.byref(t))


def test_bad_tuning_fields(lib):
    t = wino.WinoTuning(k_per_wg=-1)
    assert ">= 0" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    # a stage holds 256 / R input channels
    t = wino.WinoTuning(c_chunk=8)
    assert "256 / tiles_per_wg" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    t = wino.WinoTuning(tiles_per_wg=32, c_chunk=16)
    assert "256 / tiles_per_wg" in _plan_fails(lib, 1, 4, 4, 8, 8, 2, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    # blocking overrides are for the fused algorithm
    t = wino.WinoTuning(k_per_wg=32)
    assert "fused algorithm only" in _plan_fails(lib, 1, 4, 4, 8, 8, 4, wino.WINO_ALGO_THREE_STAGE,
                                                 ctypes.byref(t))


def test_tuning_struct_matches_header():
    """The binding's wino_tuning has the header's fields, in order."""
    with open(os.path.join(ROOT, "include", "wino_conv.h")) as f:
        hdr = f.read()
    body = re.search(r"typedef struct \{([^}]*)\} wino_tuning;", hdr).group(1)
    fields = re.findall(r"int (\w+);", body)
    assert fields == [f for f, _ in wino.WinoTuning._fields_]
    limit = int(re.search(r"#define WINO_MAX_CHANNEL_SPLITS (\d+)", hdr).group(1))
    assert limit == wino.WINO_MAX_CHANNEL_SPLITS


def test_bad_channel_splits(lib):
    """Channel splitting is checked before any device work: a negative count, a
    count above the limit, another schedule or the three-stage algorithm."""
    t = wino.WinoTuning(channel_splits=-2)
    assert ">= 0" in _plan_fails(lib, 1, 64, 16, 8, 8, 4, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    t = wino.WinoTuning(channel_splits=wino.WINO_MAX_CHANNEL_SPLITS + 1)
    assert "exceeds" in _plan_fails(lib, 1, 64, 16, 8, 8, 4, wino.WINO_ALGO_FUSED, ctypes.byref(t))
    t = wino.WinoTuning(channel_splits=2)
    assert "fused algorithm only" in _plan_fails(lib, 1, 64, 16, 8, 8, 4, wino.WINO_ALGO_THREE_STAGE,
                                                 ctypes.byref(t))


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
    assert lib.wino_conv_status(None) == wino.WINO_EINVAL
    assert lib.wino_conv_debug_set_status(None, 1) == wino.WINO_EINVAL
    buf = ctypes.create_string_buffer(64)
    assert lib.wino_conv_describe(None, buf, 64) == wino.WINO_EINVAL
    lib.wino_conv_destroy(None)


def test_python_errors_raise(lib):
    with pytest.raises(wc.WinoError):
        wc.wino_conv_plan(1, 4, 4, 8, 8, 3)


# ---- wisdom table (include/wino_tune.h), host only --------------------------

WISDOM = """# winograd wisdom: arch cus N C K H W candidates m algo tiles_per_wg k_per_wg microseconds
gfx950 256 32 64 64 224 224 0x54 4 0 16 64 417.900
gfx950 256 64 512 512 14 14 0x154 6 1 0 0 12.500
gfx950 256 64 128 128 28 28 0x210 14 2 0 0 321.000
gfx950 256 64 128 128 28 28 0x14 4 0 16 32 57.000
gfx950 256 64 512 512 14 14 0x1f4 7 1 0 0 140.000
"""


def test_wisdom_roundtrip(lib, tmp_path):
    wc.wino_wisdom_clear()
    assert wc.wino_wisdom_size() == 0
    src = tmp_path / "in.txt"
    src.write_text(WISDOM)
    wc.wino_wisdom_load(str(src))
    assert wc.wino_wisdom_size() == 5
    assert wc.wino_wisdom_lookup("gfx950", 256, 32, 64, 64, 224, 224, 0x54) == (4, 0, 16, 64)
    assert wc.wino_wisdom_lookup("gfx950", 256, 64, 128, 128, 28, 28, 0x210) == (14, 2, 0, 0)
    assert wc.wino_wisdom_lookup("gfx950", 256, 64, 512, 512, 14, 14, 0x154) == (6, 1, 0, 0)
    assert wc.wino_wisdom_lookup("gfx950", 256, 64, 128, 128, 28, 28, 0x14) == (4, 0, 16, 32)
    assert wc.wino_wisdom_lookup("gfx950", 256, 64, 512, 512, 14, 14, 0x1f4) == (7, 1, 0, 0)
    # every key field matters
    assert wc.wino_wisdom_lookup("gfx942", 256, 32, 64, 64, 224, 224, 0x54) is None
    assert wc.wino_wisdom_lookup("gfx950", 304, 32, 64, 64, 224, 224, 0x54) is None
    assert wc.wino_wisdom_lookup("gfx950", 256, 32, 64, 64, 224, 224, 0x14) is None
    out = tmp_path / "out.txt"
    wc.wino_wisdom_save(str(out))
    wc.wino_wisdom_clear()
    wc.wino_wisdom_load(str(out))
    assert wc.wino_wisdom_size() == 5
    assert wc.wino_wisdom_lookup("gfx950", 256, 64, 512, 512, 14, 14, 0x154) == (6, 1, 0, 0)
    lines = [l for l in out.read_text().splitlines() if not l.startswith("#")]
    assert sorted(lines) == sorted(l for l in WISDOM.splitlines() if not l.startswith("#"))
    # a later entry with the same key replaces the earlier one
    upd = tmp_path / "upd.txt"
    upd.write_text("gfx950 256 32 64 64 224 224 0x54 2 0 32 32 500\n")
    wc.wino_wisdom_load(str(upd))
    assert wc.wino_wisdom_size() == 5
    assert wc.wino_wisdom_lookup("gfx950", 256, 32, 64, 64, 224, 224, 0x54) == (2, 0, 32, 32)
    wc.wino_wisdom_clear()


@pytest.mark.parametrize("line", [
    "gfx950 256 32 64 64 224 224 0x54 4 0 16 64",             # missing field
    "gfx950 256 32 64 64 224 224 0x54 4 0 16 64 1.0 extra",   # extra field
    "gfx950 256 32 64 64 224 224 0x54 4 0 1.0",               # old format without the blocking
    "gfx950 256 32 64 64 224 224 0x54 3 0 16 64 1.0",         # m not a tile size
    "gfx950 256 32 64 64 224 224 0x14 6 0 16 32 1.0",         # m not among the candidates
    "gfx950 256 32 64 64 224 224 0x54 4 1 0 0 1.0",           # three-stage not a candidate
    "gfx950 256 32 64 64 224 224 0x154 4 1 16 64 1.0",        # three-stage with a blocking
    "gfx950 256 32 64 64 224 224 0x54 4 0 32 64 1.0",         # blocking not built for m = 4
    "gfx950 256 32 64 64 224 224 0x54 6 0 16 64 1.0",         # blocking not built for m = 6
    "gfx950 256 32 64 64 224 224 0x1d4 7 0 16 32 1.0",        # m = 7 is three-stage only
    "gfx950 256 32 64 64 224 224 0x154 7 1 0 0 1.0",          # m = 7 not a candidate
    "gfx950 256 32 64 64 224 224 0x2 2 0 32 64 1.0",          # mask without a tile-size bit
    "gfx950 256 32 64 64 224 224 0x10 14 2 0 0 1.0",          # FFT not a candidate
    "gfx950 256 32 64 64 224 224 0x210 4 2 0 0 1.0",          # FFT with m other than 14
    "gfx950 256 32 64 64 224 224 0x210 14 0 0 0 1.0",         # m = 14 is FFT only
    "gfx950 256 32 0 64 224 224 0x54 4 0 16 64 1.0",          # size < 1
    "gfx950 256 32 64 64 224 224 0x54 4 0 16 64 -1",          # negative time
])
def test_wisdom_rejects_malformed_and_keeps_table(lib, tmp_path, line):
    wc.wino_wisdom_clear()
    good = tmp_path / "good.txt"
    good.write_text(WISDOM)
    wc.wino_wisdom_load(str(good))
    bad = tmp_path / "bad.txt"
    bad.write_text("gfx950 256 1 1 1 1 1 0x4 2 0 32 64 1.0\n" + line + "\n")
    with pytest.raises(wc.WinoError, match=r"bad.txt:2: malformed"):
        wc.wino_wisdom_load(str(bad))
    assert wc.wino_wisdom_size() == 5          # nothing of the bad file was merged
    assert wc.wino_wisdom_lookup("gfx950", 256, 1, 1, 1, 1, 1, 0x4) is None
    wc.wino_wisdom_clear()


def test_wisdom_file_errors(lib, tmp_path):
    with pytest.raises(wc.WinoError, match="cannot read"):
        wc.wino_wisdom_load(str(tmp_path / "missing.txt"))
    with pytest.raises(wc.WinoError, match="cannot write"):
        wc.wino_wisdom_save(str(tmp_path / "no_such_dir" / "w.txt"))


@pytest.mark.parametrize("mask", [0, wc.WINO_TUNE_THREE_STAGE, 1 << 3, wc.WINO_TUNE_M4 | (1 << 10),
                                  wc.WINO_TUNE_M7])
def test_plan_tuned_bad_mask(lib, mask):
    assert not lib.wino_conv_plan_tuned(1, 4, 4, 8, 8, mask, None, None, None)
    assert "candidate mask" in wc.wino_last_error()


def test_plan_tuned_bad_sizes(lib):
    assert not lib.wino_conv_plan_tuned(1, 0, 4, 8, 8, wc.WINO_TUNE_ALL_M, None, None, None)
    assert "sizes must be >= 1" in wc.wino_last_error()


def test_plan_params_null(lib):
    assert lib.wino_conv_plan_params(None, None, None, None, None) == wino.WINO_EINVAL


def test_noalloc_checks_before_any_hip_call(lib):
    """wino_conv_run_noalloc refuses a bad tile size and a layer whose transformed
    kernels exceed its scratch array (C = K = 512 at F(6x6,3x3): 67 MB) before any
    HIP call."""
    assert lib.wino_conv_run_noalloc(1, 4, 4, 8, 8, 3, None, None, None, None, None) == wino.WINO_EINVAL
    assert "only F(2x2" in wc.wino_last_error()
    rc = lib.wino_conv_run_noalloc(64, 512, 512, 14, 14, 6, None, None, None, None, None)
    assert rc == wino.WINO_EUNSUPPORTED
    assert "scratch" in wc.wino_last_error()
    with open(os.path.join(ROOT, "include", "wino_conv.h")) as f:
        assert re.search(r"#define WINO_NOALLOC_SCRATCH_BYTES \(16u << 20\)", f.read())
