"""Benchmark: one SPVConv block (Sec. 3.3, Fig. 2) on a ~120k-point synthetic 64-beam
LiDAR sweep at C=96 in bf16 with fp32 accumulation, on one MI355X.

A step = one spv_block call: voxelize (Eq. 1-2, hash) -> submanifold kernel map ->
2 x (3x3x3 sparse conv 96->96 + folded BN + ReLU) -> trilinear devoxelize + point
MLP 96->96 + BN + ReLU + add.  Inputs are resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu]
    python bench.py --sizes      # block phases on batches of 1, 4, 16, 64 sweeps (GB/s vs n)
    python bench.py --configs    # map build and conv alone: 32->32 k3, 64->128 k2s2, 128->64 transposed

Prints ONE JSON line.  `ms_per_step` is the whole block, timed over K calls with
no events inside them.  A second run of K calls records HIP events between the
phases (the phase breakdown) and around each conv launch: `value` is the
sparse-conv throughput in TFLOP/s on its effective FLOPs (2 * Cin * Cout *
sum_k |map_k|, MACs over active synapses only) from those conv launch times.
The oracle leg times the plain CPU oracle on one full conv layer of the same
workload (single thread).
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


def table_slots(n):
    """Hash-table capacity the library uses for n keys (power of two >= 2n, at least 1024)."""
    c = 1024
    while c < 2 * n:
        c <<= 1
    return c


def phase_bytes(n, m, pairs, C, nconv=2):
    """Algorithmic bytes per phase of the block: compulsory reads of inputs plus writes of
    outputs, each gathered row counted once.  The hash table has 16 B per slot (64-byte
    buckets of 4 keys and 4 values); clearing it writes the 8-byte keys of every slot."""
    S = table_slots(n)
    return {
        # xyz + features in; coords, counts, pt2vox, voxel features out; the table's keys
        # cleared and one key + value written per voxel
        "voxelize": 12 * n + 2 * C * n + 16 * m + 4 * m + 4 * n + 2 * C * m + 8 * S + 12 * m,
        # coords in, table read once, 27-entry neighbour table out
        "kernel_map": 16 * m + 16 * S + 108 * m,
        # input rows + output rows + the map (8 B per pair) + weights, per conv
        "conv": 2 * C * m + 2 * C * m + 8 * pairs + 27 * C * C * 2,
        # xyz + point features + pt2vox + neighbour rows + voxel features + output
        "devox_mlp_add": 12 * n + 2 * C * n + 4 * n + 108 * m + 2 * C * m + 2 * C * n,
    }


def phase_roofline(n, m, pairs, C, med):
    """Each phase's algorithmic bytes over its median event time, against 8 TB/s."""
    pb = phase_bytes(n, m, pairs, C)
    res = {}
    for k, key in (("voxelize", "voxelize"), ("kernel_map", "kernel_map"), ("conv1", "conv"),
                   ("conv2", "conv"), ("devox_mlp_add", "devox_mlp_add")):
        gbps = pb[key] / (med[k] * 1e-3) / 1e9
        res[k] = {"bound": "hbm", "alg_bytes": pb[key], "ms": med[k], "achieved": gbps, "peak": PEAK_HBM_GBPS,
                  "unit": "GB/s", "frac": gbps / PEAK_HBM_GBPS}
    return res


def time_block(spv, ws, params, d_xyz, d_feat, out, steps, warm, batch=None):
    """Per-phase HIP-event times (ms) of `steps` block calls after `warm` untimed ones."""
    n_ev = 7
    evs = [HipEvents(n_ev) for _ in range(steps)]
    for _ in range(warm):
        spv.spv_block(ws, params, d_xyz, d_feat, batch=batch, out=out)
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        params.events = ct.cast(evs[s].arr, ct.POINTER(ct.c_void_p))
        params.n_events = n_ev
        spv.spv_block(ws, params, d_xyz, d_feat, batch=batch, out=out)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    params.events = None
    params.n_events = 0
    names = ["voxelize", "kernel_map", "conv_plan", "conv1", "conv2", "devox_mlp_add"]
    ph = {k: [e.ms(i, i + 1) for e in evs] for i, k in enumerate(names)}
    ph["block"] = [e.ms(0, 6) for e in evs]
    return ph, wall


def block_graph_ms(spv, ws, params, d_xyz, d_feat, out, steps):
    """Mean time (ms) of one block call captured into a graph and replayed `steps` times."""
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        spv.spv_block(ws, params, d_xyz, d_feat, out=out)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    ga, gb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ga.record()
    for _ in range(steps):
        g.replay()
    gb.record()
    torch.cuda.synchronize()
    return ga.elapsed_time(gb) / steps


def sizes_mode(args):
    """The block on batches of 1, 4, 16 and 64 independent sweeps (batch index in the key),
    one JSON line per batch: per-phase median time and GB/s of algorithmic bytes."""
    import torch
    from paper_2007_16100_amd import spv, synth
    C, v = 96, 0.05
    dev = torch.device("cuda:0")
    batches = [int(b) for b in args.batches.split(",")]
    sweeps = []
    for i in range(max(batches)):
        sweeps.append(synth.lidar_sweep(2000 + i))
        if (i + 1) % 8 == 0:
            print(f"# generated {i + 1} sweeps", file=sys.stderr, flush=True)
    _, _, convs, Wp, scp, shp = make_workload(C=C)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    d_convs = [(bf(W), torch.from_numpy(sc).to(dev), torch.from_numpy(sh).to(dev), r) for W, sc, sh, r in convs]
    params = spv.make_block_params(C, torch.bfloat16, v, d_convs, bf(Wp), torch.from_numpy(scp).to(dev),
                                   torch.from_numpy(shp).to(dev), relu_p=True)
    for B in batches:
        xyz = np.concatenate(sweeps[:B])
        bt = np.concatenate([np.full(len(sweeps[i]), i, np.int32) for i in range(B)])
        n = len(xyz)
        feat = synth.normal((n, C), 2100 + B, dtype="bf16")
        d_xyz, d_bt, d_feat = torch.from_numpy(xyz).to(dev), torch.from_numpy(bt).to(dev), bf(feat)
        ws2 = spv.Workspace.for_ops(n, C)
        vox = spv.spv_voxelize(ws2, d_xyz, v, batch=d_bt)
        km = spv.spv_kernel_map(ws2, vox.coords[:vox.m].contiguous())
        m, pairs = vox.m, km.total
        del ws2, vox, km
        ws = spv.Workspace.for_block(n, C)
        out = torch.empty((n, C), dtype=torch.bfloat16, device=dev)
        ph, _ = time_block(spv, ws, params, d_xyz, d_feat, out, args.steps, args.warmup, batch=d_bt)
        pb = phase_bytes(n, m, pairs, C)
        med = {k: float(np.median(x)) for k, x in ph.items()}
        conv_ms = float(np.median(ph["conv1"] + ph["conv2"]))
        gbps = {k: pb[k] / (med[k] * 1e-3) / 1e9 for k in ("voxelize", "kernel_map", "devox_mlp_add")}
        gbps["conv"] = pb["conv"] / (conv_ms * 1e-3) / 1e9
        print(json.dumps({"sweeps": B, "points": n, "voxels": m, "kernel_map_pairs": pairs, "C": C,
                          "phases_ms_median": med, "alg_bytes": pb, "GBps": gbps,
                          "hbm_frac": {k: x / PEAK_HBM_GBPS for k, x in gbps.items()},
                          "conv_TFLOPs": 2.0 * C * C * pairs / (conv_ms * 1e-3) / 1e12}), flush=True)
        del ws, out, d_xyz, d_bt, d_feat
        torch.cuda.empty_cache()


def configs_mode(args):
    """Map build and conv alone on the sweep: a submanifold 3x3x3 conv 32->32 (seed 1002), and
    the stride-2 maps (K = 2 and K = 3) with a strided conv 64->128 and its transposed 128->64
    on each (seed 1003).  One JSON
    line per op: median HIP-event time, algorithmic bytes / FLOPs and both roofline fractions."""
    import torch
    from paper_2007_16100_amd import spv, synth
    dev = torch.device("cuda:0")

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(args.steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            ts.append((a, b))
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ts]))

    def report(op, ms, nbytes, flops=0.0, **kw):
        gbps = nbytes / (ms * 1e-3) / 1e9
        tf = flops / (ms * 1e-3) / 1e12
        print(json.dumps({"op": op, "ms_median": ms, "alg_bytes": nbytes, "GBps": gbps,
                          "hbm_frac": gbps / PEAK_HBM_GBPS, "eff_flops": flops, "TFLOPs": tf,
                          "mfma_frac": tf / PEAK_BF16_TFLOPS, **kw}), flush=True)

    for seed in (1002, 1003):
        xyz = synth.lidar_sweep(seed)
        d_xyz = torch.from_numpy(xyz).to(dev)
        ws = spv.Workspace.for_ops(len(xyz), 128)
        vox = spv.spv_voxelize(ws, d_xyz, 0.05)
        m = vox.m
        coords = vox.coords[:m].contiguous()
        wsm = spv.Workspace.for_ops(len(xyz), 128)
        if seed == 1002:
            km = spv.spv_kernel_map(wsm, coords)
            P = km.total
            # Sec. 4.3's resource model on this scan: |map_k| per offset and the MACs
            # of the block's two 96->96 convs and of a 32->32 conv
            from paper_2007_16100_amd import mapstats
            ms = mapstats.MapStats()
            sizes = ms.add("s1k3", km.off)
            total_macs, per_layer = mapstats.conv_macs([("s1k3", 96, 96), ("s1k3", 96, 96), ("s1k3", 32, 32)], ms)
            print(json.dumps({"op": "kernel_map k3 s1 statistics", "map_sizes": [int(x) for x in sizes],
                              "macs_layers": ["96->96", "96->96", "32->32"], "macs": per_layer,
                              "macs_total": total_macs}), flush=True)
            ms = timed(lambda: spv.spv_kernel_map(wsm, coords, sync=False))
            report("kernel_map k3 s1", ms, 16 * m + 12 * table_slots(m) + 8 * P + 4 * 28, voxels=m, pairs=P)
            C = 32
            x = bf(synth.normal((m, C), seed + 1, dtype="bf16"))
            W = bf(synth.conv_weight(27, C, C, seed + 2, "bf16"))
            out = torch.empty((m, C), dtype=torch.bfloat16, device=dev)
            ms = timed(lambda: spv.spv_sparse_conv(wsm, x, km.off, km.pairs, W, m, out=out))
            report("conv k3 32->32", ms, 2 * C * m * 2 + 8 * P + 27 * C * C * 2, 2.0 * C * C * P, voxels=m, pairs=P)
            # the neighbour-table route: the map as a [m][27] table, and the conv on it
            # with weights packed once (no per-call plan)
            nbr = torch.empty((m, 27), dtype=torch.int32, device=dev)
            ms = timed(lambda: spv.spv_kernel_map_nbr(wsm, coords, out=nbr))
            report("kernel_map_nbr k3 s1", ms, 16 * m + 12 * table_slots(m) + 108 * m, voxels=m, pairs=P)
            Wp = spv.spv_pack_weights(W)
            ms = timed(lambda: spv.spv_sparse_conv_nbr_packed(wsm, x, nbr, Wp, C, m, out=out))
            report("conv k3 32->32 on the neighbour table", ms, 2 * C * m * 2 + 108 * m + 27 * C * C * 2,
                   2.0 * C * C * P, voxels=m, pairs=P)
        else:
            km = spv.spv_kernel_map(wsm, coords, K=2, stride=2)
            mc = int(km.m_out_dev.item())
            P = km.total
            from paper_2007_16100_amd import mapstats
            print(json.dumps({"op": "kernel_map k2 s2 statistics",
                              "map_sizes": [int(x) for x in mapstats.map_sizes(km.off)]}), flush=True)
            ms = timed(lambda: spv.spv_kernel_map(wsm, coords, K=2, stride=2, sync=False))
            report("kernel_map k2 s2", ms, 16 * m + 16 * mc + 12 * table_slots(m) + 8 * P + 4 * 9,
                   voxels=m, coarse_voxels=mc, pairs=P)
            x = bf(synth.normal((m, 64), seed + 1, dtype="bf16"))
            W = bf(synth.conv_weight(8, 64, 128, seed + 2, "bf16"))
            WT = bf(synth.conv_weight(8, 128, 64, seed + 3, "bf16"))
            y = torch.empty((mc, 128), dtype=torch.bfloat16, device=dev)
            z = torch.empty((m, 64), dtype=torch.bfloat16, device=dev)
            ms = timed(lambda: spv.spv_sparse_conv(wsm, x, km.off, km.pairs, W, mc, m_out_dev=km.m_out_dev, out=y))
            report("conv k2s2 64->128", ms, 2 * 64 * m + 2 * 128 * mc + 8 * P + 8 * 64 * 128 * 2,
                   2.0 * 64 * 128 * P, voxels=m, coarse_voxels=mc, pairs=P)
            ms = timed(lambda: spv.spv_sparse_conv(wsm, y, km.off, km.pairs, WT, m, transposed=True, out=z))
            report("conv k2s2 transposed 128->64", ms, 2 * 128 * mc + 2 * 64 * m + 8 * P + 8 * 64 * 128 * 2,
                   2.0 * 64 * 128 * P, voxels=m, coarse_voxels=mc, pairs=P)
            # the 3x3x3 stride-2 map (same coarse voxels; probes of the fine table) and its convs
            km3 = spv.spv_kernel_map(wsm, coords, K=3, stride=2)
            P3 = km3.total
            print(json.dumps({"op": "kernel_map k3 s2 statistics",
                              "map_sizes": [int(x) for x in mapstats.map_sizes(km3.off)]}), flush=True)
            ms = timed(lambda: spv.spv_kernel_map(wsm, coords, K=3, stride=2, sync=False))
            report("kernel_map k3 s2", ms, 16 * m + 16 * mc + 24 * table_slots(m) + 8 * P3 + 4 * 28,
                   voxels=m, coarse_voxels=mc, pairs=P3)
            W3 = bf(synth.conv_weight(27, 64, 128, seed + 4, "bf16"))
            W3T = bf(synth.conv_weight(27, 128, 64, seed + 5, "bf16"))
            ms = timed(lambda: spv.spv_sparse_conv(wsm, x, km3.off, km3.pairs, W3, mc, m_out_dev=km3.m_out_dev,
                                                   out=y))
            report("conv k3s2 64->128", ms, 2 * 64 * m + 2 * 128 * mc + 8 * P3 + 27 * 64 * 128 * 2,
                   2.0 * 64 * 128 * P3, voxels=m, coarse_voxels=mc, pairs=P3)
            ms = timed(lambda: spv.spv_sparse_conv(wsm, y, km3.off, km3.pairs, W3T, m, transposed=True, out=z))
            report("conv k3s2 transposed 128->64", ms, 2 * 128 * mc + 2 * 64 * m + 8 * P3 + 27 * 64 * 128 * 2,
                   2.0 * 64 * 128 * P3, voxels=m, coarse_voxels=mc, pairs=P3)
        del ws, wsm
        torch.cuda.empty_cache()


def spvcnn_flops(P, plan, n):
    """Effective FLOPs of one network forward (Sec. 4.3: active synapses only): per layer
    2 * C_in * C_out times its kernel-map pairs (convs) or rows (1x1 shortcuts, point MLPs,
    head)."""
    pairs = lambda km: int(km.off[-1].item())
    subm = [int((plan.nbr[s][: plan.m[s]] > 0).sum().item()) for s in range(5)]  # nonzero table entries
    units = {}
    for name in P:
        parts = name.split(".")
        if parts[0] == "stem":
            units[name] = subm[0]
        elif parts[0] == "down":
            units[name] = pairs(plan.down[int(parts[1])])
        elif parts[0] == "up":
            units[name] = pairs(plan.down[5 - int(parts[1])])
        elif parts[0] in ("enc", "dec"):
            s = int(parts[1]) if parts[0] == "enc" else 4 - int(parts[1])
            units[name] = plan.m[s] if parts[3] == "sc" else subm[s]
        else:  # point MLPs and the head run on every point
            units[name] = n
    return sum(2.0 * P[k][0].shape[-2] * P[k][0].shape[-1] * u for k, u in units.items())


def spvcnn_mode(args):
    """The SPVCNN-style encoder-decoder forward on a batch of 4 sweeps (seeds 1005-1008, batch
    index in the key), bf16: wall-clock per forward (synchronized, the plan's per-stride count
    read-backs included) and effective conv + linear TFLOP/s."""
    import torch
    from paper_2007_16100_amd import synth
    from paper_2007_16100_amd.spvcnn import SPVCNN
    sw = [synth.lidar_sweep(1005 + i) for i in range(4)]
    xyz = np.concatenate(sw)
    batch = np.concatenate([np.full(len(a), i, np.int32) for i, a in enumerate(sw)])
    feat = synth.point_features(xyz, 9001, "bf16")
    P = synth.spvcnn_params(9002, "bf16")
    net = SPVCNN(P, "bf16", 0.05)
    d_xyz = torch.from_numpy(xyz).cuda()
    d_b = torch.from_numpy(batch).cuda()
    d_f = torch.from_numpy(feat.view(np.int16)).view(torch.bfloat16).cuda()
    tr = {}
    net.forward(d_xyz, d_f, d_b, trace=tr)
    torch.cuda.synchronize()
    F = spvcnn_flops(P, tr["plan"], len(xyz))
    for _ in range(args.warmup):
        net.forward(d_xyz, d_f, d_b)
    torch.cuda.synchronize()
    ts = []
    for _ in range(args.steps):
        t0 = time.perf_counter()
        net.forward(d_xyz, d_f, d_b)
        torch.cuda.synchronize()
        ts.append(time.perf_counter() - t0)
    ms = float(np.median(ts)) * 1e3
    print(json.dumps({"op": "spvcnn forward, 4 sweeps", "points": int(len(xyz)), "voxels_per_stride": tr["plan"].m,
                      "ms_median": ms, "ms_p10": float(np.percentile(ts, 10)) * 1e3,
                      "ms_p90": float(np.percentile(ts, 90)) * 1e3, "points_per_s": len(xyz) / (ms * 1e-3),
                      "eff_flops": F, "TFLOPs": F / (ms * 1e-3) / 1e12, "steps": args.steps}), flush=True)


def backward_mode(args):
    """The backward passes at the block's shape (sweep 1004, C = 96, bf16): conv input and
    weight gradients on the submanifold map, scatter-mean and devoxelization backward.  One
    JSON line per op: median HIP-event time, effective TFLOP/s or algorithmic GB/s."""
    import torch
    from paper_2007_16100_amd import spv, synth
    dev = torch.device("cuda:0")
    C = 96

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(args.steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            ts.append((a, b))
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ts]))

    xyz = synth.lidar_sweep(1004)
    n = len(xyz)
    d_xyz = torch.from_numpy(xyz).to(dev)
    ws = spv.Workspace.for_ops(n, C)
    vox = spv.spv_voxelize(ws, d_xyz, 0.05, bf(synth.normal((n, C), 1, dtype="bf16")))
    m = vox.m
    coords = vox.coords[:m].contiguous()
    km = spv.spv_kernel_map(ws, coords)
    P = km.total
    x = bf(synth.normal((m, C), 2, dtype="bf16"))
    dy = bf(synth.normal((m, C), 3, dtype="bf16"))
    W = bf(synth.conv_weight(27, C, C, 4, "bf16"))
    dx = torch.empty((m, C), dtype=torch.bfloat16, device=dev)
    F = 2.0 * C * C * P

    def line(op, ms, flops=0.0, nbytes=0.0):
        print(json.dumps({"op": op, "ms_median": ms, "eff_flops": flops, "TFLOPs": flops / (ms * 1e-3) / 1e12,
                          "alg_bytes": nbytes, "GBps": nbytes / (ms * 1e-3) / 1e9, "voxels": m, "pairs": P,
                          "points": n}), flush=True)

    ms = timed(lambda: spv.spv_sparse_conv_dgrad(ws, dy, km.off, km.pairs, W, m, out=dx))
    line("conv dgrad 96->96 (plan included)", ms, F, 2 * 2 * C * m + 8 * P + 27 * C * C * 2)
    nbr = spv.spv_kernel_map_nbr(ws, coords)
    ms = timed(lambda: spv.spv_sparse_conv_dgrad_nbr(ws, dy, nbr, W, out=dx))
    line("conv dgrad 96->96 on the neighbour table", ms, F, 2 * 2 * C * m + 108 * m + 27 * C * C * 2)
    wsw = spv.Workspace.for_wgrad(27, C, C)
    dW = torch.empty((27, C, C), dtype=torch.float32, device=dev)
    ms = timed(lambda: spv.spv_sparse_conv_wgrad(wsw, x, dy, km.off, km.pairs, 27, out=dW))
    line("conv wgrad 96->96", ms, F, 2 * 2 * C * m + 8 * P + 27 * C * C * 4)
    dvf = bf(synth.normal((m, C), 5, dtype="bf16"))
    dfeat = torch.empty((n, C), dtype=torch.bfloat16, device=dev)
    ms = timed(lambda: spv.spv_voxelize_backward(dvf, vox.counts, vox.pt2vox, m, out=dfeat))
    line("voxelize backward C=96", ms, 0.0, 2 * C * m + 4 * m + 4 * n + 2 * C * n)
    _, ci, cw = spv.spv_devoxelize(ws, coords, x, d_xyz, 0.05, want_corners=True)
    dout = bf(synth.normal((n, C), 6, dtype="bf16"))
    dv = torch.empty((m, C), dtype=torch.float32, device=dev)
    wsd = spv.Workspace.for_devox_backward(n, m)
    ms = timed(lambda: spv.spv_devoxelize_backward(wsd, ci, cw, dout, m, out=dv))
    line("devoxelize backward C=96", ms, 0.0, 64 * n + 2 * C * n + 4 * C * m)
    # the same at stride 16 (the network's second devoxelization: 0.8 m voxels, thousands of corner
    # entries on the densest)
    cs = coords
    for _ in range(4):
        k2 = spv.spv_kernel_map(ws, cs, K=2, stride=2)
        cs = k2.out_coords[: int(k2.m_out_dev.item())].contiguous()
    m16 = cs.shape[0]
    v16 = bf(synth.normal((m16, C), 11, dtype="bf16"))
    _, ci16, cw16 = spv.spv_devoxelize(ws, cs, v16, d_xyz, 0.05, stride_log2=4, want_corners=True)
    dv16 = torch.empty((m16, C), dtype=torch.float32, device=dev)
    wsd16 = spv.Workspace.for_devox_backward(n, m16)
    ms = timed(lambda: spv.spv_devoxelize_backward(wsd16, ci16, cw16, dout, m16, out=dv16))
    line("devoxelize backward C=96, stride 16", ms, 0.0, 64 * n + 2 * C * n + 4 * C * m16)
    # the point branch's layer ReLU(scale * (x @ W) + shift) + res over the n points
    pf = bf(synth.normal((n, C), 7, dtype="bf16"))
    Wl = bf(synth.linear_weight(C, C, 8, "bf16"))
    wsl = spv.Workspace.for_ops(n, C)
    a = spv.spv_linear(wsl, pf, Wl)
    sc = torch.from_numpy(0.5 + synth.uniform_cube(C, 1.0, 9)[:, 0] ** 2).to(dev)  # seeded, in [0.5, 1.5)
    sh = torch.from_numpy(synth.normal((C,), 10, std=0.1)).to(dev)
    wse = spv.Workspace.for_epilogue_backward(n, C)
    ms = timed(lambda: spv.spv_epilogue_backward(wse, dout, a, sc, sh, True, dout, True))
    line("epilogue backward C=96 (BN + ReLU + residual, n points)", ms, 0.0, 2 * C * n * 4)
    wlb = spv.Workspace.for_linear_backward(C, C)
    da = spv.spv_epilogue_backward(wse, dout, a, sc, sh, True)[0]
    ms = timed(lambda: spv.spv_linear_backward(wlb, pf, Wl, da))
    line("linear backward 96->96 (dx and dW, n points)", ms, 2 * 2.0 * n * C * C, 2 * C * n * 3 + 4 * C * C)


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
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": 1, "kind": "oracle",
            "nproc": os.cpu_count(), "cpu_model": model,
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
    ap.add_argument("--no-graph", action="store_true", help="skip the graph-replay timing of the block")
    ap.add_argument("--sizes", action="store_true", help="block phases on batches of sweeps (GB/s against n)")
    ap.add_argument("--batches", default="1,4,16,64", help="sweeps per batch for --sizes")
    ap.add_argument("--configs", action="store_true",
                    help="map build and conv alone at the 32->32 and 64<->128 (k2s2, transposed) shapes")
    ap.add_argument("--spvcnn", action="store_true",
                    help="the SPVCNN-style encoder-decoder forward on a batch of 4 sweeps")
    ap.add_argument("--backward", action="store_true",
                    help="the backward passes (conv input / weight gradients, scatter-mean and devox backward)")
    args = ap.parse_args()
    if args.backward:
        backward_mode(args)
        return
    if args.spvcnn:
        spvcnn_mode(args)
        return
    if args.sizes:
        sizes_mode(args)
        return
    if args.configs:
        configs_mode(args)
        return
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

    steps, warm = args.steps, args.warmup
    # the timed steps: block calls with no events inside, bracketed by a sync
    for _ in range(warm):
        spv.spv_block(ws, params, d_xyz, d_feat, out=out)
    torch.cuda.synchronize()
    ta, tb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ta.record()
    for _ in range(steps):
        spv.spv_block(ws, params, d_xyz, d_feat, out=out)
    tb.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    block_ms_mean = ta.elapsed_time(tb) / steps
    # the same number of calls again with HIP events between the phases (the
    # phase breakdown and the conv launch times; the events add a little time)
    ph, _ = time_block(spv, ws, params, d_xyz, d_feat, out, steps, 0)
    block_ms = ph.pop("block")
    med = {k: float(np.median(vv)) for k, vv in ph.items()}
    p10 = {k: float(np.percentile(vv, 10)) for k, vv in ph.items()}
    p90 = {k: float(np.percentile(vv, 90)) for k, vv in ph.items()}

    # the same block captured once into a graph and replayed (no events inside)
    graph_ms = None if args.no_graph else block_graph_ms(spv, ws, params, d_xyz, d_feat, out, steps)
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
        "block_ms_mean": block_ms_mean,
        "block_ms_median_with_phase_events": float(np.median(block_ms)),
        "block_ms_p10_with_phase_events": float(np.percentile(block_ms, 10)),
        "block_ms_p90_with_phase_events": float(np.percentile(block_ms, 90)),
        "block_ms_graph_replay": graph_ms,
        "phases_ms_median": med,
        "phases_ms_p10": p10,
        "phases_ms_p90": p90,
        "roofline": roof,
        "phase_roofline": phase_roofline(n, m, pairs_total, C, med),
    }
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(xyz, convs, C)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
