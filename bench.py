"""Benchmark: one SPVConv block (Sec. 3.3, Fig. 2) on a ~120k-point synthetic 64-beam
LiDAR sweep at C=96 in bf16 with fp32 accumulation, on one MI355X.

A step = one spv_block call: voxelize (Eq. 1-2, hash) -> submanifold kernel map ->
2 x (3x3x3 sparse conv 96->96 + folded BN + ReLU) -> trilinear devoxelize + point
MLP 96->96 + BN + ReLU + add.  Inputs are resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu]

Prints ONE JSON line.  `value` is the sparse-conv throughput in TFLOP/s on its
effective FLOPs (2 * Cin * Cout * sum_k |map_k|, MACs over active synapses only),
measured with HIP events around each conv launch inside the timed steps;
`ms_per_step` is the whole block.  The oracle leg times the plain CPU oracle on
one full conv layer of the same workload (single thread).
"""
from __future__ import annotations

import argparse
import ctypes as ct
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E

# Sources of the dominant kernel (the 3x3x3 neighbour-table conv); the committed
# FETCH_SIZE / WRITE_SIZE summary applies only while their hash is unchanged.
CONV_SOURCES = ("paper_2007_16100_amd/csrc/conv_union.hip", "paper_2007_16100_amd/csrc/conv_common.hpp")
CONV_TRAFFIC = "profiles/conv_union_c96_traffic.txt"


def conv_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in CONV_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def conv_traffic_bytes():
    """HBM bytes per conv launch from the committed rocprofv3 counter summary, each
    counter scaled by what it reads for a plain copy of known size; None when the
    summary is missing or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, CONV_TRAFFIC)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != conv_source_hash():
        return None
    cb = float(kv["copy_bytes"])
    fetch = float(kv["fetch_kib_per_dispatch"]) * cb / float(kv["copy_fetch_kib"])
    write = float(kv["write_kib_per_dispatch"]) * cb / float(kv["copy_write_kib"])
    return fetch + write


class HipEvents:
    """hipEvent_t handles through the HIP runtime (recorded by libspv on the bench stream)."""

    def __init__(self, n):
        self.hip = ct.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ct.POINTER(ct.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ct.POINTER(ct.c_float), ct.c_void_p, ct.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ct.c_void_p]
        self.ev = []
        for _ in range(n):
            e = ct.c_void_p()
            assert self.hip.hipEventCreate(ct.byref(e)) == 0
            self.ev.append(e)
        self.arr = (ct.c_void_p * n)(*[e.value for e in self.ev])

    def ms(self, a, b):
        t = ct.c_float()
        assert self.hip.hipEventSynchronize(self.ev[b]) == 0
        assert self.hip.hipEventElapsedTime(ct.byref(t), self.ev[a], self.ev[b]) == 0
        return float(t.value)


def make_workload(seed=1004, C=96):
    from paper_2007_16100_amd import synth
    xyz = synth.lidar_sweep(seed)
    feat = synth.normal((len(xyz), C), seed + 1, dtype="bf16")
    convs = []
    for l in range(2):
        sc, sh = synth.folded_bn(C, seed + 6 + l)
        convs.append((synth.conv_weight(27, C, C, seed + 2 + l, "bf16"), sc, sh, True))
    Wp = synth.linear_weight(C, C, seed + 4, "bf16")
    scp, shp = synth.folded_bn(C, seed + 5)
    return xyz, feat, convs, Wp, scp, shp


def cpu_baseline(xyz, convs, C, v=0.05):
    """The oracle, as it stands, on one full 96->96 conv layer of the workload (one thread)."""
    import oracle
    from paper_2007_16100_amd import synth
    oracle.build(force=False)
    coords, _, _, _ = oracle.voxelize(xyz, v)
    _, off, pairs = oracle.kernel_map(coords)
    x = synth.normal((len(coords), C), 7, dtype="bf16")
    W, sc, sh, r = convs[0]
    t0 = time.perf_counter()
    oracle.sparse_conv(x, off, pairs, W, len(coords), "bf16", sc, sh, r)
    dt = time.perf_counter() - t0
    flops = 2.0 * C * C * int(off[-1])
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": 1, "kind": "oracle",
            "sample": f"one submanifold 3x3x3 conv {C}->{C} (bf16 storage, fp64 accumulation) over the full "
                      f"{len(coords)}-voxel sweep, {int(off[-1])} kernel-map pairs; {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline leg")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy three times (the reference for scaling "
                         "the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        nbytes = 256 << 20
        x = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": nbytes, "repeats": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the SPVConv hot path here runs on a single MI355X); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2007_16100_amd import spv

    C, v = 96, 0.05
    xyz, feat, convs, Wp, scp, shp = make_workload(C=C)
    n = len(xyz)
    dev = torch.device("cuda:0")

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    d_xyz = torch.from_numpy(xyz).to(dev)
    d_feat = bf(feat)
    d_convs = [(bf(W), torch.from_numpy(sc).to(dev), torch.from_numpy(sh).to(dev), r) for W, sc, sh, r in convs]
    d_Wp, d_scp, d_shp = bf(Wp), torch.from_numpy(scp).to(dev), torch.from_numpy(shp).to(dev)
    params = spv.make_block_params(C, torch.bfloat16, v, d_convs, d_Wp, d_scp, d_shp, relu_p=True)
    ws = spv.Workspace.for_block(n, C)
    out = torch.empty((n, C), dtype=torch.bfloat16, device=dev)

    # sizes of this workload (m voxels, kernel-map pairs) from the library itself
    ws2 = spv.Workspace.for_ops(n, C)
    vox = spv.spv_voxelize(ws2, d_xyz, v)
    km = spv.spv_kernel_map(ws2, vox.coords[:vox.m].contiguous())
    m, pairs_total = vox.m, km.total
    del ws2, vox, km

    n_ev = 7
    steps, warm = args.steps, args.warmup
    evs = [HipEvents(n_ev) for _ in range(steps)]
    params_plain = params
    for _ in range(warm):
        spv.spv_block(ws, params_plain, d_xyz, d_feat, out=out)
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for s in range(steps):
        params.events = ct.cast(evs[s].arr, ct.POINTER(ct.c_void_p))
        params.n_events = n_ev
        spv.spv_block(ws, params, d_xyz, d_feat, out=out)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    params.events = None
    params.n_events = 0

    phase_names = ["voxelize", "kernel_map", "conv_plan", "conv1", "conv2", "devox_mlp_add"]
    ph = {k: [] for k in phase_names}
    block_ms = []
    for e in evs:
        for i, k in enumerate(phase_names):
            ph[k].append(e.ms(i, i + 1))
        block_ms.append(e.ms(0, 6))
    med = {k: float(np.median(vv)) for k, vv in ph.items()}
    conv_ms = [a for k in ("conv1", "conv2") for a in ph[k]]
    conv_avg_ms = float(np.mean(conv_ms))
    F_conv = 2.0 * C * C * pairs_total
    conv_tflops = F_conv / (conv_avg_ms * 1e-3) / 1e12
    # algorithmic bytes of one conv launch: input rows + output rows (bf16) + kernel map + weights
    B_conv = m * C * 2 + m * C * 2 + pairs_total * 8 + 27 * C * C * 2
    conv_gbps = B_conv / (conv_avg_ms * 1e-3) / 1e9
    t_mfma = F_conv / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = B_conv / (PEAK_HBM_GBPS * 1e9)
    if t_hbm >= t_mfma:
        roof = {"bound": "hbm", "achieved": conv_gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": conv_gbps / PEAK_HBM_GBPS}
    else:
        roof = {"bound": "mfma", "achieved": conv_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": conv_tflops / PEAK_BF16_TFLOPS}
    roof.update({"traffic": conv_traffic_bytes(), "kernel": "k_conv_union (3x3x3 submanifold, 96->96, bf16)",
                 "alg_bytes_per_launch": B_conv, "eff_flops_per_launch": F_conv,
                 "mfma_frac_eff": conv_tflops / PEAK_BF16_TFLOPS, "avg_launch_us": conv_avg_ms * 1e3})

    res = {
        "metric": "SPVConv block ms & sparse-conv TFLOP/s at 120k pts; % of MFMA/HBM roofline",
        "value": conv_tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": wall * 1e3 / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "SPVConv block C=96 (2 submanifold 3x3x3 convs + folded BN + ReLU, point MLP "
                               "96->96 + BN + ReLU, trilinear devox, add) on a synthetic 64-beam LiDAR sweep, "
                               "voxel 0.05 m, bf16 storage / fp32 accumulation",
                   "points": n, "voxels": m, "kernel_map_pairs": pairs_total, "C": C, "seed": 1004},
        "block_ms_median": float(np.median(block_ms)),
        "phases_ms_median": med,
        "roofline": roof,
    }
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(xyz, convs, C)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
