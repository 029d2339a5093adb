"""Small drivers for profiling runs (rocprofv3) of the library.

    python -m paper_1912_02165_amd.profile_run layer ID M ALGO [REPS]
        REPS calls of the fused or three-stage path on a seeded layer, after one
        kernel transform (so the transform-domain kernels run REPS times).
    python -m paper_1912_02165_amd.profile_run copy MIB [REPS]
        REPS device-to-device copies of MIB MiB: a plain copy kernel of known
        size, the reference that scales the FETCH_SIZE / WRITE_SIZE counters.
"""

import sys


def run_layer(layer_id, m, algo, reps):
    import torch
    from . import wino, workloads
    layer = workloads.LAYER_BY_ID[layer_id]
    x, w = workloads.layer_inputs(layer)
    x, w = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.empty((layer.N, layer.K, layer.H, layer.W), device="cuda")
    with wino.Plan(layer.N, layer.C, layer.K, layer.H, layer.W, m, algo) as p:
        p.set_weights(w)
        for _ in range(reps):
            p.run_pretransformed(x, y)
        torch.cuda.synchronize()
    print(f"ran {layer.tag(m)} {algo} x{reps}", flush=True)


def run_copy(mib, reps):
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x{reps}", flush=True)


def main(argv):
    if len(argv) >= 4 and argv[0] == "layer":
        run_layer(int(argv[1]), int(argv[2]), argv[3], int(argv[4]) if len(argv) > 4 else 3)
    elif len(argv) >= 2 and argv[0] == "copy":
        run_copy(int(argv[1]), int(argv[2]) if len(argv) > 2 else 3)
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
