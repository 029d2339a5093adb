"""GPU parity: the HIP library (through the C ABI) against the CPU oracle.

* small and ragged shapes (several tiles and workgroups, C and K not multiples of
  4 or 16, images smaller than a tile) against the full fp64 direct convolution,
  for the default plan and for every fused blocking the library is built for (the
  candidates the tuner picks from);
* the 56x56 layer (N=1, C=K=64) in full at every m it runs with;
* the full-size VGG/ResNet-shaped layers, whole outputs, in the launch
  configuration the benchmark times (the oracle is computed once per layer), for
  both algorithms, every tile size including F(2) and F(5) (whose outputs of 128
  MB or more are stored with the streaming cache policy), and each layer's other
  fused blockings; the benchmark's timed path (kernels transformed ahead, then
  run_pretransformed) bitwise equal to run;
* NaN inputs reaching exactly the outputs the transforms connect them to;
* the plan's status word (bounded waits) after every call, and its plumbing.
"""

import re

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads
from oracle.direct import direct_conv
from parity import assert_close

pytestmark = pytest.mark.gpu

ALGOS = ("fused", "three_stage")

SMALL = [
    (1, 1, 1, 1, 1), (1, 2, 3, 2, 5), (1, 3, 4, 1, 9), (1, 3, 5, 7, 9), (2, 4, 16, 8, 8),
    (1, 5, 17, 13, 11), (3, 8, 20, 17, 23), (2, 37, 45, 29, 35), (2, 16, 33, 30, 31),
    (1, 64, 64, 20, 20), (4, 12, 40, 6, 6), (1, 130, 18, 9, 10),
    # more output channels than one group and kernels outweighing the input: items
    # numbered tile-group fastest
    (1, 32, 128, 8, 8), (2, 20, 96, 13, 6), (1, 9, 200, 5, 5),
    # few items of 16 channel stages (the last ragged): the last round's items are
    # split into pieces whose partial outputs are added
    (1, 250, 40, 9, 10), (2, 256, 96, 7, 6),
]


def run_gpu(x, w, m, algo, tuning=None):
    N, C, H, W = x.shape
    K = w.shape[0]
    xd = torch.from_numpy(x).cuda()
    wd = torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), dtype=torch.float32, device="cuda")
    with wc.Plan(N, C, K, H, W, m, algo, tuning) as p:
        p.run(xd, wd, y)
        p.status()  # synchronises; raises if a bounded wait gave up
    return y


def rand(shape, seed):
    return np.random.default_rng(seed).uniform(-1, 1, size=shape).astype(np.float32)


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("m", (2, 4, 5, 6))
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_small_shapes(algo, m, shape):
    N, C, K, H, W = shape
    x, w = workloads.random_inputs(N, C, K, H, W, seed=sum(shape) + m)
    print(f"\n[gpu] small {algo} m={m} shape={shape}", flush=True)
    y = run_gpu(x, w, m, algo).cpu().numpy()
    assert_close(y, direct_conv(x, w), m, f"{algo} F({m}) {shape}")


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_small_shapes_f7_three_stage(shape):
    """F(7x7,3x3), three-stage only (T = 9: tiles wider than the row-vector loader
    and the fused kernel's stage ring take)."""
    N, C, K, H, W = shape
    x, w = workloads.random_inputs(N, C, K, H, W, seed=sum(shape) + 7)
    print(f"\n[gpu] small three_stage m=7 shape={shape}", flush=True)
    y = run_gpu(x, w, 7, "three_stage").cpu().numpy()
    assert_close(y, direct_conv(x, w), 7, f"three_stage F(7) {shape}")


BLOCKINGS = wc.wino_fused_blockings()
BLOCKING_SHAPES = [(1, 1, 1, 1, 1), (1, 3, 5, 7, 9), (2, 37, 45, 29, 35), (2, 16, 33, 30, 31),
                   (1, 130, 18, 9, 10), (1, 32, 128, 8, 8), (3, 8, 20, 17, 23), (1, 64, 64, 20, 20)]


@pytest.mark.parametrize("blocking", BLOCKINGS, ids=lambda b: "m%d-R%d-K%d" % b)
@pytest.mark.parametrize("shape", BLOCKING_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_blocking_small(blocking, shape):
    """Every (m, tiles per task, output channels per task) the tuner may pick."""
    m, R, kit = blocking
    N, C, K, H, W = shape
    x, w = workloads.random_inputs(N, C, K, H, W, seed=sum(shape) + 3 * m + R + kit)
    print(f"\n[gpu] blocking m={m} R={R} Kit={kit} shape={shape}", flush=True)
    y = run_gpu(x, w, m, "fused", {"tiles_per_wg": R, "k_per_wg": kit}).cpu().numpy()
    assert_close(y, direct_conv(x, w), m, f"F({m}) R={R} Kit={kit} {shape}")


@pytest.mark.parametrize("algo,m", [(a, m) for a in ALGOS for m in (2, 4, 5)] + [("three_stage", 7)])
def test_layer1_full(algo, m):
    layer = workloads.LAYER_BY_ID[1]
    x, w = workloads.layer_inputs(layer)
    print(f"\n[gpu] {layer.tag(m)} {algo}", flush=True)
    y = run_gpu(x, w, m, algo).cpu().numpy()
    rel, mx = assert_close(y, direct_conv(x, w), m, f"{layer.tag(m)} {algo}")
    print(f"rel_l2={rel:.3e} max={mx:.3e}")


_REF = {}


def layer_ref(layer):
    """(x, w, fp64 oracle output) of a full layer, computed once per layer."""
    if layer.id not in _REF:
        x, w = workloads.layer_inputs(layer)
        _REF[layer.id] = (x, w, direct_conv(x, w))
    return _REF[layer.id]


# (layer, m, blocking or None for the default): the configured pairs, the 14x14
# C=K=512 layer at F(4) (the tile size the tuner picks there), F(2) and F(5) on
# every full layer (F(2) and F(5) outputs of 128 MB or more take the streaming
# stores), and each configured pair's other built blockings.  Grouped by layer
# so the oracle output is computed once per layer.
def _full_cases():
    cases = []
    for layer in workloads.LAYERS:
        if layer.id == 1:
            continue
        ms = sorted(set(layer.ms) | {2, 4, 5} | ({6} if layer.id in (3, 5) else set()))
        for m in ms:
            cases.append((layer, m, None))
            if m in layer.ms or (layer.id == 5 and m == 4):
                for (bm, R, kit) in BLOCKINGS:
                    if bm == m:
                        cases.append((layer, m, (R, kit)))
    return cases


FULL_CASES = _full_cases()


def _case_id(c):
    layer, m, b = c
    return layer.tag(m) + ("" if b is None else "-R%d-K%d" % b)


@pytest.mark.parametrize("case", FULL_CASES, ids=_case_id)
def test_full_layers_fused(case):
    """Whole output of a full-size layer against the oracle; the benchmark's timed
    path (kernels set ahead, then run_pretransformed) gives the same bits as run."""
    layer, m, blocking = case
    x, w, ref = layer_ref(layer)
    tuning = None if blocking is None else {"tiles_per_wg": blocking[0], "k_per_wg": blocking[1]}
    N, C, K, H, W = layer.N, layer.C, layer.K, layer.H, layer.W
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    with wc.Plan(N, C, K, H, W, m, "fused", tuning) as p:
        print(f"\n[gpu] {_case_id(case)} fused full size: {p.describe()}", flush=True)
        p.run(xd, wd, y)
        p.status()
        y2 = torch.full_like(y, float("nan"))
        p.set_weights(wd)
        p.run_pretransformed(xd, y2)
        p.status()
    assert torch.equal(y, y2), "run_pretransformed differs from run"
    del y2
    rel, mx = assert_close(y.cpu().numpy(), ref, m, f"{_case_id(case)} fused")
    print(f"rel_l2={rel:.3e} max={mx:.3e} (whole output)")


# the three-stage path also at F(7) (every configured image side is a multiple of 7)
THREE_STAGE_FULL = [c for c in FULL_CASES if c[2] is None] + [
    (layer, 7, None) for layer in workloads.LAYERS if layer.id != 1]


@pytest.mark.parametrize("case", THREE_STAGE_FULL, ids=_case_id)
def test_full_layers_three_stage(case):
    layer, m, _ = case
    x, w, ref = layer_ref(layer)
    print(f"\n[gpu] {_case_id(case)} three_stage full size", flush=True)
    y = run_gpu(x, w, m, "three_stage")
    rel, mx = assert_close(y.cpu().numpy(), ref, m, f"{_case_id(case)} three_stage")
    print(f"rel_l2={rel:.3e} max={mx:.3e} (whole output)")


@pytest.mark.parametrize("m", (2, 4, 5, 6, 7))
def test_three_stage_intermediates(m):
    """Each unfused stage against the fp64 CPU Winograd's matching intermediate."""
    from oracle import winograd
    N, C, K, H, W = 2, 6, 20, 11, 13
    x, w = workloads.random_inputs(N, C, K, H, W, seed=70 + m)
    T2 = (m + 2) ** 2
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.empty((N, K, H, W), device="cuda")
    with wc.Plan(N, C, K, H, W, m, "three_stage") as p:
        p.run(xd, wd, y)
        torch.cuda.synchronize()
        wt = p.intermediate(wc.WINO_BUF_WEIGHTS)       # (Kb, Cs, T2P, 64) operand order
        U = p.intermediate(wc.WINO_BUF_INPUT)          # (F4, TB, Cs, 256) operand order
        Mf = p.intermediate(wc.WINO_BUF_PRODUCT)       # (F4, TB, Kb, 1024) accumulator order
    Wt_ref = winograd.weight_transform(w, m)             # (T2, C, K)
    U_ref = winograd.input_transform(x, m)               # (T2, C, ntiles)
    M_ref = winograd.frequency_gemm(U_ref, Wt_ref)       # (T2, K, ntiles)
    ntiles = U_ref.shape[2]
    # undo the operand order: [kb][cs][f/4][lane][f%4], lane = (c%4)*16 + k%16; the
    # frequency dim is padded to whole float4s (F(5): 49 -> 52) with zeros
    Kb, Cs, T2P = wt.shape[:3]
    assert T2P == (T2 + 3) // 4 * 4
    flat = wt.reshape(Kb, Cs, T2P // 4, 64, 4)
    for f in range(T2, T2P):
        assert not flat[:, :, f // 4, :, f % 4].any()
    wt_fck = np.empty((T2, Cs * 4, Kb * 16), np.float32)
    for f in range(T2):
        blk = flat[:, :, f // 4, :, f % 4].reshape(Kb, Cs, 4, 16)   # kb, cs, c%4, k%16
        wt_fck[f] = blk.transpose(1, 2, 0, 3).reshape(Cs * 4, Kb * 16)
    np.testing.assert_allclose(wt_fck[:, :C, :K], Wt_ref, rtol=1e-6, atol=1e-7)
    assert not wt_fck[:, C:, :].any() and not wt_fck[:, :, K:].any()
    # U: [f4][tb][cs][lane][f%4], lane = (c%4)*16 + t%16 -> (f, c, t)
    F4, TB, UCs = U.shape[:3]
    u = U.reshape(F4, TB, UCs, 4, 16, 4)                     # f4, tb, cs, c%4, t%16, f%4
    u_fct = u.transpose(0, 5, 2, 3, 1, 4).reshape(F4 * 4, UCs * 4, TB * 16)
    assert not u_fct[T2:].any()
    u_fct = u_fct[:T2]
    scale = np.abs(U_ref).max()
    np.testing.assert_allclose(u_fct[:, :C, :ntiles], U_ref, rtol=0, atol=1e-6 * scale)
    assert not u_fct[:, C:, :].any() and not u_fct[:, :, ntiles:].any()
    # M: [f4][tb][kb][v][lane][f%4], lane = ((k%16)/4)*16 + t%16, v = k%4 -> (f, k, t)
    F4, TB, MKb = Mf.shape[:3]
    mm = Mf.reshape(F4, TB, MKb, 4, 4, 16, 4)                # f4, tb, kb, v, k%16/4, t%16, f%4
    m_fkt = mm.transpose(0, 6, 2, 4, 3, 1, 5).reshape(F4 * 4, MKb * 16, TB * 16)
    assert not m_fkt[T2:].any()
    m_fkt = m_fkt[:T2]
    scale = np.abs(M_ref).max()
    np.testing.assert_allclose(m_fkt[:, :K, :ntiles], M_ref, rtol=0, atol=1e-5 * scale)
    assert not m_fkt[:, K:, :].any() and not m_fkt[:, :, ntiles:].any()
    assert_close(y.cpu().numpy(), direct_conv(x, w), m, "three-stage end to end")


def split_items(plan):
    """Items of the plan's last round split into pieces (from its description)."""
    found = re.search(r"split items (\d+) x (\d+) pieces", plan.describe())
    return int(found.group(1)) if found else 0


@pytest.mark.parametrize("m", (2, 4, 5, 6))
def test_plan_reused_across_calls(m):
    """One plan, several calls: split items' arrival counters are back at zero after
    every call, so each call is correct and bitwise equal to the first."""
    N, C, K, H, W = 2, 256, 80, 14, 15
    x, w = workloads.random_inputs(N, C, K, H, W, seed=40 + m)
    ref = direct_conv(x, w)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    ys = []
    with wc.Plan(N, C, K, H, W, m) as p:
        assert split_items(p) > 0, p.describe()
        for _ in range(3):
            y = torch.full((N, K, H, W), float("nan"), device="cuda")
            p.run(xd, wd, y)
            ys.append(y)
        torch.cuda.synchronize()
    for y in ys:
        assert torch.equal(y, ys[0])
    assert_close(ys[0].cpu().numpy(), ref, m, f"reused plan F({m})")


@pytest.mark.parametrize("algo", ALGOS)
def test_deterministic(algo):
    x, w = workloads.random_inputs(3, 40, 48, 30, 26, seed=5)
    a = run_gpu(x, w, 4, algo)
    b = run_gpu(x, w, 4, algo)
    assert torch.equal(a, b)


@pytest.mark.parametrize("algo", ALGOS)
def test_guard_regions_untouched(algo):
    N, C, K, H, W = 2, 8, 24, 9, 14
    x, w = workloads.random_inputs(N, C, K, H, W, seed=6)
    n = N * K * H * W
    buf = torch.full((n + 2 * 1024,), float("nan"), device="cuda")
    y = buf[1024:1024 + n].view(N, K, H, W)
    with wc.Plan(N, C, K, H, W, 4, algo) as p:
        p.run(torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(), y)
        torch.cuda.synchronize()
    assert torch.isnan(buf[:1024]).all() and torch.isnan(buf[1024 + n:]).all()
    assert_close(y.cpu().numpy(), direct_conv(x, w), 4, "guarded")


@pytest.mark.parametrize("algo,m", [(a, m) for a in ALGOS for m in (2, 4, 5, 6)] + [("three_stage", 7)])
def test_pretransformed_matches_run(algo, m):
    """Kernels transformed ahead (set_weights) then run_pretransformed: the same bits
    as run, and within tolerance of the oracle."""
    N, C, K, H, W = 2, 20, 36, 15, 16
    x, w = workloads.random_inputs(N, C, K, H, W, seed=7 + m)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y1 = torch.full((N, K, H, W), float("nan"), device="cuda")
    y2 = torch.full_like(y1, float("nan"))
    with wc.Plan(N, C, K, H, W, m, algo) as p:
        with pytest.raises(wc.WinoError):
            p.run_pretransformed(xd, y2)       # no kernels set yet
        p.set_weights(wd)
        p.run_pretransformed(xd, y2)
        p.status()
        p.run(xd, wd, y1)
        p.status()
    assert torch.equal(y1, y2)
    assert_close(y2.cpu().numpy(), direct_conv(x, w), m, f"pretransformed {algo} F({m})")


CSPLIT_SHAPES = [(1, 1, 1, 1, 1), (3, 8, 20, 17, 23), (2, 37, 45, 29, 35), (1, 64, 64, 20, 20),
                 (1, 130, 18, 9, 10), (1, 32, 128, 8, 8)]


@pytest.mark.parametrize("csplit", (2, 3, 64))
@pytest.mark.parametrize("m", (2, 4, 5, 6))
@pytest.mark.parametrize("shape", CSPLIT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_channel_split_small(shape, m, csplit):
    """Every work item cut into channel pieces whose partial outputs are added:
    one-stage layers (nothing to split), ragged channel tails, more pieces asked
    for than there are stages."""
    N, C, K, H, W = shape
    x, w = workloads.random_inputs(N, C, K, H, W, seed=sum(shape) + 7 * m + csplit)
    print(f"\n[gpu] channel split {csplit} m={m} shape={shape}", flush=True)
    y = run_gpu(x, w, m, "fused", {"channel_splits": csplit}).cpu().numpy()
    assert_close(y, direct_conv(x, w), m, f"F({m}) {shape} channel_splits={csplit}")


CSPLIT_FULL = [(5, 6, 2), (5, 6, 4), (5, 4, 3), (4, 4, 2)]


@pytest.mark.parametrize("case", CSPLIT_FULL, ids=lambda c: f"layer{c[0]}-F{c[1]}-split{c[2]}")
def test_channel_split_full_layers(case):
    lid, m, csplit = case
    layer = workloads.LAYER_BY_ID[lid]
    x, w, ref = layer_ref(layer)
    print(f"\n[gpu] {layer.tag(m)} channel split {csplit} full size", flush=True)
    y = run_gpu(x, w, m, "fused", {"channel_splits": csplit})
    rel, mx = assert_close(y.cpu().numpy(), ref, m, f"{layer.tag(m)} channel_splits={csplit}")
    print(f"rel_l2={rel:.3e} max={mx:.3e} (whole output)")


def test_channel_split_reproducible():
    """Partial outputs are added in channel order whatever order the pieces
    finish in, and the arrival counters are left at zero: repeated calls on one
    plan give identical bits."""
    N, C, K, H, W = 2, 96, 80, 18, 22
    x, w = workloads.random_inputs(N, C, K, H, W, seed=9)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    ys = []
    with wc.Plan(N, C, K, H, W, 4, "fused", {"channel_splits": 3}) as p:
        for _ in range(3):
            y = torch.full((N, K, H, W), float("nan"), device="cuda")
            p.run(xd, wd, y)
            ys.append(y)
        torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1]) and torch.equal(ys[0], ys[2])
    assert_close(ys[0].cpu().numpy(), direct_conv(x, w), 4, "channel_splits=3 repeated")


def test_bad_pointers_rejected():
    N, C, K, H, W = 1, 4, 4, 8, 8
    xd = torch.zeros((N, C, H, W), device="cuda")
    wd = torch.zeros((K, C, 3, 3), device="cuda")
    with wc.Plan(N, C, K, H, W, 4) as p:
        with pytest.raises(wc.WinoError, match="overlaps"):
            p.run(xd, wd, xd)
        host = np.zeros(N * K * H * W, np.float32)
        with pytest.raises(wc.WinoError, match="device"):
            p.run(xd, wd, host.ctypes.data)
        with pytest.raises(wc.WinoError, match="aligned"):
            p.run(xd, wd, xd.data_ptr() + 2)
    # an allocation too small for the tensor
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    ptr = ctypes.c_void_p()
    assert hip.hipMalloc(ctypes.byref(ptr), ctypes.c_size_t(1024)) == 0
    try:
        with wc.Plan(1, 4, 4, 64, 64, 4) as p:
            with pytest.raises(wc.WinoError, match="allocation holds"):
                p.run(torch.zeros((1, 4, 64, 64), device="cuda"), torch.zeros((4, 4, 3, 3), device="cuda"),
                      ptr.value)
    finally:
        hip.hipFree(ptr)


@pytest.mark.parametrize("m", (2, 4, 5, 6))
def test_unaligned_input_pointer(m):
    """x starting 4 bytes past an aligned address takes the per-element load path."""
    N, C, K, H, W = 2, 9, 20, 16, 24
    x, w = workloads.random_inputs(N, C, K, H, W, seed=9 + m)
    buf = torch.zeros(x.size + 1, device="cuda")
    buf[1:] = torch.from_numpy(x.reshape(-1)).cuda()
    xd = buf[1:].view(N, C, H, W)
    assert xd.data_ptr() % 16 == 4
    y = torch.empty((N, K, H, W), device="cuda")
    with wc.Plan(N, C, K, H, W, m) as p:
        p.run(xd, torch.from_numpy(w).cuda(), y)
        torch.cuda.synchronize()
    assert_close(y.cpu().numpy(), direct_conv(x, w), m, f"unaligned x F({m})")


# ---- tuned plans (include/wino_tune.h) --------------------------------------

def _device_key():
    prop = torch.cuda.get_device_properties(0)
    return prop.gcnArchName.split(":")[0], prop.multi_processor_count


@pytest.mark.parametrize("mask", [wc.WINO_TUNE_ALL_M | wc.WINO_TUNE_THREE_STAGE, wc.WINO_TUNE_M4,
                                  wc.WINO_TUNE_M2 | wc.WINO_TUNE_M6, wc.WINO_TUNE_FFT,
                                  wc.WINO_TUNE_M6 | wc.WINO_TUNE_FFT,
                                  wc.WINO_TUNE_M7 | wc.WINO_TUNE_THREE_STAGE])
def test_plan_tuned(mask, tmp_path):
    """The tuned plan is one of the candidates, matches the oracle at its m, and is
    remembered: the second request, and one after a save / clear / load of the
    wisdom table, return the same choice without timing again."""
    N, C, K, H, W = 2, 37, 45, 29, 35
    x, w = workloads.random_inputs(N, C, K, H, W, seed=95)
    print(f"\n[gpu] tuned plan mask={mask:#x}", flush=True)
    wc.wino_wisdom_clear()
    p = wc.Plan.tuned(N, C, K, H, W, mask)
    if p.algo == "fft":
        assert p.m == 14 and mask & wc.WINO_TUNE_FFT
    else:
        assert mask & (1 << p.m)
        assert p.algo == "fused" or mask & wc.WINO_TUNE_THREE_STAGE
    pm, palgo, R, kit = wc.wino_conv_plan_params(p.handle)
    assert (pm, palgo) == (p.m, wc.ALGOS[p.algo])
    assert (R, kit) == ((0, 0) if p.algo != "fused" else (R, kit))
    if p.algo == "fused":
        assert (p.m, R, kit) in BLOCKINGS
    assert p.call_us > 0
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    p.run(xd, wd, y)
    torch.cuda.synchronize()
    assert_close(y.cpu().numpy(), direct_conv(x, w), p.m, f"tuned F({p.m}) {p.algo}")
    arch, cus = _device_key()
    assert wc.wino_wisdom_lookup(arch, cus, N, C, K, H, W, mask) == (p.m, wc.ALGOS[p.algo], R, kit)
    p2 = wc.Plan.tuned(N, C, K, H, W, mask)
    assert (p2.m, p2.algo, p2.call_us) == (p.m, p.algo, p.call_us)
    assert p2.params() == p.params()
    f = tmp_path / "wisdom.txt"
    wc.wino_wisdom_save(str(f))
    wc.wino_wisdom_clear()
    wc.wino_wisdom_load(str(f))
    p3 = wc.Plan.tuned(N, C, K, H, W, mask)
    assert (p3.m, p3.algo) == (p.m, p.algo) and abs(p3.call_us - p.call_us) < 1e-3
    assert p3.params() == p.params()
    for q in (p, p2, p3):
        q.close()
    wc.wino_wisdom_clear()


# ---- status word, shape checks ---------------------------------------------

def test_status_word_plumbing():
    """A bit set in the plan's status word (as a kernel wait that gave up would set
    it) is reported once by wino_conv_status and then cleared; the plan still
    computes correct results afterwards.  No kernel is made to give up."""
    N, C, K, H, W = 1, 40, 48, 17, 19
    x, w = workloads.random_inputs(N, C, K, H, W, seed=11)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    with wc.Plan(N, C, K, H, W, 4) as p:
        p.status()
        wc.wino_conv_debug_set_status(p.handle, 1)
        with pytest.raises(wc.WinoError, match="gave up") as e:
            p.status()
        assert e.value.status == wc.WINO_EKERNEL
        p.status()  # cleared
        p.run(xd, wd, y)
        p.status()
    assert_close(y.cpu().numpy(), direct_conv(x, w), 4, "after a status reset")


def test_wrong_shapes_refused():
    """Tensors that do not hold the plan's tensors are refused before any launch."""
    N, C, K, H, W = 2, 8, 24, 9, 14
    x = torch.zeros((N, C, H, W), device="cuda")
    w = torch.zeros((K, C, 3, 3), device="cuda")
    y = torch.full((N, K, H, W), 7.0, device="cuda")
    with wc.Plan(N, C, K, H, W, 4) as p:
        with pytest.raises(ValueError, match="y: expected shape"):
            p.run(x, w, torch.zeros((N, K - 1, H, W), device="cuda"))
        with pytest.raises(ValueError, match="x: expected shape"):
            p.run(torch.zeros((N, C, H + 1, W), device="cuda"), w, y)
        with pytest.raises(ValueError, match="w: expected shape"):
            p.set_weights(torch.zeros((K, C + 1, 3, 3), device="cuda"))
        with pytest.raises(ValueError, match="y: expected shape"):
            p.run_pretransformed(x, torch.zeros((N, K, H, W - 1), device="cuda"))
        torch.cuda.synchronize()
    assert bool((y == 7.0).all())


# ---- non-finite inputs -----------------------------------------------------

def _nan_mask(N, K, H, W, m, nan_pixels):
    """Outputs that a NaN input reaches: output (i, j) of a tile depends on window
    element (a, b) when the transforms connect them structurally, i.e. (|A^T| |B^T|)
    is nonzero at (i, a) and at (j, b), from the oracle's exact matrices (for FFT
    tiles every output of the tile depends on every window element).  The kernels
    skip structurally zero coefficients, so exactly these outputs become NaN."""
    from oracle import toom_cook
    if m == 14:
        T = 16
        dep = np.ones((m, T), dtype=bool)
    else:
        AT, _, BT = toom_cook.matrices_f64(m)
        T = m + 2
        dep = (np.abs(np.array(AT, dtype=np.float64)) @ np.abs(np.array(BT, dtype=np.float64))) > 0
    mask = np.zeros((N, K, H, W), dtype=bool)
    for (n, c, h, v) in nan_pixels:
        for ty in range((H + m - 1) // m):
            a = h - (ty * m - 1)
            if not 0 <= a < T:
                continue
            for tx in range((W + m - 1) // m):
                b = v - (tx * m - 1)
                if not 0 <= b < T:
                    continue
                for i in range(m):
                    for j in range(m):
                        hh, vv = ty * m + i, tx * m + j
                        if hh < H and vv < W and dep[i, a] and dep[j, b]:
                            mask[n, :, hh, vv] = True
    return mask


NAN_CASES = [(m, algo) for m in (2, 4, 5, 6) for algo in ALGOS] + [(7, "three_stage"), (14, "fft")]


@pytest.mark.parametrize("case", NAN_CASES, ids=lambda c: f"m{c[0]}-{c[1]}")
def test_nan_reaches_exactly_its_tiles(case):
    """NaNs in x (Sec. 2.1's overlapping windows): one where a 16-tile lane row of the
    producers wraps from one tile row to the next (the halo exchange between lanes
    must not carry it into the previous row's last tile), one on the right and
    bottom image edges, one on an inner tile boundary.  NaN appears exactly in the
    outputs the transforms connect it to; every other output is finite and matches
    the oracle."""
    m, algo = case
    N, C, K, H, W = 2, 20, 24, 31, 30
    x, w = workloads.random_inputs(N, C, K, H, W, seed=31 + m)
    TW = (W + m - 1) // m
    row2 = 2 * m + 1                           # a row of the third tile row
    pixels = [(0, 3, min(row2, H - 1), 0),      # first column: left halo of tile column 0 only
              (1, C - 1, H - 1, W - 1),         # bottom-right corner
              (1, 0, 5, min(W - 1, (TW // 2) * m - 1))]  # last own column of an inner tile column
    for (n, c, h, v) in pixels:
        x[n, c, h, v] = np.nan
    mask = _nan_mask(N, K, H, W, m, pixels)
    print(f"\n[gpu] NaN injection {algo} m={m}: {int(mask.sum())} NaN outputs expected", flush=True)
    y = run_gpu(x, w, m, algo).cpu().numpy()
    got = np.isnan(y)
    assert np.array_equal(got, mask), (f"NaN outputs: {int(got.sum())} got, {int(mask.sum())} expected, "
                                       f"{int((got & ~mask).sum())} unexpected, {int((mask & ~got).sum())} missing")
    assert np.isfinite(y[~mask]).all()
    ref = direct_conv(np.nan_to_num(x, nan=0.0), w)
    tol_m = m if m != 14 else 14
    rel, mx = __import__("parity").errors(y[~mask], ref[~mask])
    from parity import REL_L2, MAX_ERR
    assert rel <= REL_L2[tol_m] and mx <= MAX_ERR, (rel, mx)
