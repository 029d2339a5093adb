"""GPU parity: the HIP library (through the C ABI) against the CPU oracle.

* small and ragged shapes (several tiles and workgroups, C and K not multiples of
  4 or 16, images smaller than a tile) against the full fp64 direct convolution;
* the 56x56 layer (N=1, C=K=64) in full at every m it runs with;
* the full-size VGG/ResNet-shaped layers in the launch configuration the
  benchmark times, on sampled output planes the oracle computes one by one;
* both algorithms (fused and three-stage) everywhere.
"""

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads
from oracle.direct import direct_conv, direct_conv_planes
from parity import assert_close

pytestmark = pytest.mark.gpu

ALGOS = ("fused", "three_stage")

SMALL = [
    (1, 1, 1, 1, 1), (1, 2, 3, 2, 5), (1, 3, 4, 1, 9), (1, 3, 5, 7, 9), (2, 4, 16, 8, 8),
    (1, 5, 17, 13, 11), (3, 8, 20, 17, 23), (2, 37, 45, 29, 35), (2, 16, 33, 30, 31),
    (1, 64, 64, 20, 20), (4, 12, 40, 6, 6), (1, 130, 18, 9, 10),
    # more output channels than one group and kernels outweighing the input: items
    # numbered tile-group fastest, most of them split into pieces
    (1, 32, 128, 8, 8), (2, 20, 96, 13, 6), (1, 9, 200, 5, 5),
]


def run_gpu(x, w, m, algo, tuning=None):
    N, C, H, W = x.shape
    K = w.shape[0]
    xd = torch.from_numpy(x).cuda()
    wd = torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), dtype=torch.float32, device="cuda")
    with wc.Plan(N, C, K, H, W, m, algo, tuning) as p:
        p.run(xd, wd, y)
        torch.cuda.synchronize()
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


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("m", (2, 4, 5))
def test_layer1_full(algo, m):
    layer = workloads.LAYER_BY_ID[1]
    x, w = workloads.layer_inputs(layer)
    print(f"\n[gpu] {layer.tag(m)} {algo}", flush=True)
    y = run_gpu(x, w, m, algo).cpu().numpy()
    rel, mx = assert_close(y, direct_conv(x, w), m, f"{layer.tag(m)} {algo}")
    print(f"rel_l2={rel:.3e} max={mx:.3e}")


def sample_planes(N, K, seed, count=8):
    rng = np.random.default_rng(seed)
    planes = {(0, 0), (N - 1, K - 1), (N // 2, K // 3), (min(1, N - 1), K - 1), (N - 1, 0)}
    while len(planes) < count:
        planes.add((int(rng.integers(N)), int(rng.integers(K))))
    return sorted(planes)


# the configured pairs, plus the 14x14 C=K=512 layer at F(4) (the tile size a
# tuned plan picks there; 4.5 rounds of work items, the last split into pieces)
FULL_PAIRS = [(l, m) for (l, m) in workloads.PAIRS if l.id != 1] + [(workloads.LAYER_BY_ID[5], 4)]


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("pair", FULL_PAIRS, ids=lambda p: p[0].tag(p[1]))
def test_full_layers_sampled(algo, pair):
    layer, m = pair
    x, w = workloads.layer_inputs(layer)
    print(f"\n[gpu] {layer.tag(m)} {algo} full size", flush=True)
    y = run_gpu(x, w, m, algo)
    assert bool(torch.isfinite(y).all()), "non-finite output"
    planes = sample_planes(layer.N, layer.K, seed=layer.id * 10 + m)
    n_idx = torch.tensor([p[0] for p in planes], device="cuda")
    k_idx = torch.tensor([p[1] for p in planes], device="cuda")
    got = y[n_idx, k_idx].cpu().numpy()
    ref = direct_conv_planes(x, w, planes)
    rel, mx = assert_close(got, ref, m, f"{layer.tag(m)} {algo} planes {planes}")
    print(f"rel_l2={rel:.3e} max={mx:.3e} over {len(planes)} planes")


@pytest.mark.parametrize("m", (2, 4, 5, 6))
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
        wt = p.intermediate(wc.WINO_BUF_WEIGHTS)       # (Kb, Cs, T2, 64) operand order
        U = p.intermediate(wc.WINO_BUF_INPUT)          # (T2, Cp, tiles_p, 1)
        Mf = p.intermediate(wc.WINO_BUF_PRODUCT)       # (T2, Kp, tiles_p, 1)
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
    U = U[..., 0]
    scale = np.abs(U_ref).max()
    np.testing.assert_allclose(U[:, :C, :ntiles], U_ref, rtol=0, atol=1e-6 * scale)
    assert not U[:, C:, :].any() and not U[:, :, ntiles:].any()
    Mf = Mf[..., 0]
    scale = np.abs(M_ref).max()
    np.testing.assert_allclose(Mf[:, :K, :ntiles], M_ref, rtol=0, atol=1e-5 * scale)
    assert_close(y.cpu().numpy(), direct_conv(x, w), m, "three-stage end to end")


@pytest.mark.parametrize("m", (2, 4, 5, 6))
def test_plan_reused_across_calls(m):
    """One plan, several calls: split items' arrival counters are back at zero after
    every call, so each call is correct and bitwise equal to the first."""
    N, C, K, H, W = 2, 24, 80, 14, 15
    x, w = workloads.random_inputs(N, C, K, H, W, seed=40 + m)
    ref = direct_conv(x, w)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    ys = []
    with wc.Plan(N, C, K, H, W, m) as p:
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


@pytest.mark.parametrize("algo", ALGOS)
def test_pretransformed_matches_run(algo):
    N, C, K, H, W = 2, 20, 36, 15, 16
    x, w = workloads.random_inputs(N, C, K, H, W, seed=7)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y1 = torch.empty((N, K, H, W), device="cuda")
    y2 = torch.empty_like(y1)
    with wc.Plan(N, C, K, H, W, 6, algo) as p:
        with pytest.raises(wc.WinoError):
            p.run_pretransformed(xd, y2)       # no kernels set yet
        p.run(xd, wd, y1)
        p.set_weights(wd)
        p.run_pretransformed(xd, y2)
        torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_tuning_overrides_agree():
    x, w = workloads.random_inputs(2, 24, 64, 21, 19, seed=8)
    ref = direct_conv(x, w)
    for m, nkbs in ((2, (1, 2, 4)), (4, (1, 2)), (6, (1,))):
        for nkb in nkbs:
            for waves in (1, 2, 4):
                t = {"schedule": wc.WINO_SCHED_PER_WAVE, "k_blocks_per_wave": nkb,
                     "waves_per_group": waves}
                y = run_gpu(x, w, m, "fused", t)
                assert_close(y.cpu().numpy(), ref, m, f"per-wave F({m}) nkb={nkb} waves={waves}")
        for tb in ((1, 2) if m <= 4 else (1,)):
            t = {"schedule": wc.WINO_SCHED_SHARED, "tile_blocks": tb}
            y = run_gpu(x, w, m, "fused", t)
            assert_close(y.cpu().numpy(), ref, m, f"shared F({m}) tile_blocks={tb}")


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
def test_channel_split_full_layers_sampled(case):
    lid, m, csplit = case
    layer = workloads.LAYER_BY_ID[lid]
    x, w = workloads.layer_inputs(layer)
    print(f"\n[gpu] {layer.tag(m)} channel split {csplit} full size", flush=True)
    y = run_gpu(x, w, m, "fused", {"channel_splits": csplit})
    assert bool(torch.isfinite(y).all()), "non-finite output"
    planes = sample_planes(layer.N, layer.K, seed=layer.id * 10 + m + 100 * csplit)
    n_idx = torch.tensor([p[0] for p in planes], device="cuda")
    k_idx = torch.tensor([p[1] for p in planes], device="cuda")
    got = y[n_idx, k_idx].cpu().numpy()
    ref = direct_conv_planes(x, w, planes)
    rel, mx = assert_close(got, ref, m, f"{layer.tag(m)} channel_splits={csplit} planes {planes}")
    print(f"rel_l2={rel:.3e} max={mx:.3e} over {len(planes)} planes")


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
                                  wc.WINO_TUNE_M6 | wc.WINO_TUNE_FFT])
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
    assert wc.wino_conv_plan_params(p.handle) == (p.m, wc.ALGOS[p.algo])
    assert p.call_us > 0
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    p.run(xd, wd, y)
    torch.cuda.synchronize()
    assert_close(y.cpu().numpy(), direct_conv(x, w), p.m, f"tuned F({p.m}) {p.algo}")
    arch, cus = _device_key()
    assert wc.wino_wisdom_lookup(arch, cus, N, C, K, H, W, mask) == (p.m, wc.ALGOS[p.algo])
    p2 = wc.Plan.tuned(N, C, K, H, W, mask)
    assert (p2.m, p2.algo, p2.call_us) == (p.m, p.algo, p.call_us)
    f = tmp_path / "wisdom.txt"
    wc.wino_wisdom_save(str(f))
    wc.wino_wisdom_clear()
    wc.wino_wisdom_load(str(f))
    p3 = wc.Plan.tuned(N, C, K, H, W, mask)
    assert (p3.m, p3.algo) == (p.m, p.algo) and abs(p3.call_us - p.call_us) < 1e-3
    for q in (p, p2, p3):
        q.close()
    wc.wino_wisdom_clear()
