"""Writes spvcnn_4sweeps.txt: the oracle's reference for the SPVCNN-style forward on the
benchmarked batch of four full synthetic sweeps (seeds 1005-1008, batch index in the key,
point features seed 9001, parameters seed 9002, bf16 storage).

Only the oracle (oracle/) and the seeded input generators run here.  The full logits are
too large to keep, so the file holds:
* per stride 1, 2, 4, 8, 16: the voxel count and the SHA-256 of the int32 (b, x, y, z)
  coordinate array (canonical order) -- the GPU's coordinate sets must hash the same;
* the SHA-256 and the largest magnitude of the oracle's full logit array;
* the oracle's logits (bf16 bit patterns, hex) at 1024 points drawn without replacement
  with numpy default_rng(4242).

    python tests/golden/make_spvcnn_4sweeps.py      # about 20 minutes on one core
"""
import hashlib
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle import spvcnn as ospvcnn  # noqa: E402
from paper_2007_16100_amd import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "spvcnn_4sweeps.txt")
SAMPLES, SAMPLE_SEED = 1024, 4242


def inputs():
    """The benchmarked workload: four sweeps, their batch indices, features and parameters."""
    sw = [synth.lidar_sweep(1005 + i) for i in range(4)]
    xyz = np.concatenate(sw)
    batch = np.concatenate([np.full(len(a), i, np.int32) for i, a in enumerate(sw)])
    feat = synth.point_features(xyz, 9001, "bf16")
    P = synth.spvcnn_params(9002, "bf16")
    return xyz, batch, feat, P


def sample_points(n):
    return np.sort(np.random.default_rng(SAMPLE_SEED).choice(n, SAMPLES, replace=False))


def coords_sha(c):
    return hashlib.sha256(np.ascontiguousarray(c, dtype="<i4").tobytes()).hexdigest()


def main():
    oracle.build(force=False)
    xyz, batch, feat, P = inputs()
    t0 = time.time()
    c, _, _, _ = oracle.voxelize(xyz, 0.05, batch=batch)
    sets = [c]
    for _ in range(4):
        c, _, _ = oracle.kernel_map(c, 2, 2)
        sets.append(c)
    ref = ospvcnn.spvcnn_forward(xyz, feat, P, 0.05, "bf16", batch)
    r = synth.from_storage(ref, "bf16").astype(np.float64)
    idx = sample_points(len(xyz))
    with open(OUT, "w") as f:
        f.write("# oracle reference of the SPVCNN-style forward, 4 full sweeps (written by make_spvcnn_4sweeps.py)\n")
        f.write(f"points {len(xyz)}\n")
        for s, cs in enumerate(sets):
            f.write(f"stride {2 ** s} voxels {len(cs)} coords_sha256 {coords_sha(cs)}\n")
        f.write(f"logits_sha256 {hashlib.sha256(np.ascontiguousarray(ref).tobytes()).hexdigest()}\n")
        f.write(f"logits_maxabs {float(np.abs(r).max())!r}\n")
        f.write(f"samples {SAMPLES} seed {SAMPLE_SEED} classes {ref.shape[1]}\n")
        for k in idx:
            f.write(f"{k} " + " ".join(f"{int(v):04x}" for v in ref[k]) + "\n")
    print(f"wrote {OUT} in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()
