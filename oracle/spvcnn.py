"""Oracle forward of an SPVCNN-style encoder-decoder -- TEST INFRASTRUCTURE ONLY.

The backbone of the paper's appendix A.1 ("SPVCNN: Backbone Network"): a
MinkowskiNet-style U-Net of residual sparse-conv blocks wrapped by four SPVConv
point branches.  The first module voxelizes the input points and devoxelizes
after the stem; the second voxelizes again and devoxelizes after the four
downsampling stages; the last two each wrap two upsampling stages.  Every
devoxelization is fused with the point branch's MLP by addition (Sec. 3.3).

This is a plain composition of the oracle's own operations (voxelize, kernel
map, sparse conv, devoxelize, linear), in the order written, with the skip
connections as explicit concatenations.  Layer names and widths follow
``synth.spvcnn_params``; the readings that the paper leaves open (block counts,
the decoder widths, where the skips come from, the BN placement) are listed
beside the HIP implementation's description of the same network.
"""
from __future__ import annotations

import numpy as np

from . import OracleError, ERR_INVALID_ARG, devoxelize, kernel_map, linear, sparse_conv, voxelize


def voxel_size_at(v: float, s: int) -> float:
    """Voxel size of stride 2^s: the float32 voxel size scaled by 2^s (exact in float32)."""
    return float(np.float32(v) * np.float32(2.0 ** s))


def spvcnn_forward(xyz, feat, P, v, dtype="f32", batch=None, mode="center", trace=None):
    """Per-point logits [n][classes].  trace (a dict or None) receives the voxel counts per
    stride, the point features after each fusion and the encoder / decoder outputs."""
    xyz = np.asarray(xyz, np.float32)

    def conv(x, name, mp, m_out, relu=True, transposed=False, res=None):
        W, sc, sh = P[name]
        _, off, pairs = mp
        return sparse_conv(x, off, pairs, W, m_out, dtype, sc, sh, relu, transposed, res)

    def resblock(x, name, mp):
        m = len(x)
        h = conv(x, name + ".a", mp, m)
        if name + ".sc" in P:
            W, sc, sh = P[name + ".sc"]
            s = linear(x, W, dtype, sc, sh, False)
        else:
            s = x
        return conv(h, name + ".b", mp, m, res=s)

    def revoxelize(z, s, coords):
        c, vf, _, _ = voxelize(xyz, voxel_size_at(v, s), z, dtype, batch)
        if not np.array_equal(c, coords):
            raise OracleError(ERR_INVALID_ARG, f"re-voxelized coordinates at stride {2 ** s} differ")
        return vf

    def fuse(coords, vfeat, s, z_prev, name):
        W, sc, sh = P[name]
        return devoxelize(coords, vfeat, xyz, v, s, mode, batch, z_prev, W, sc, sh, True, dtype)

    # coordinate sets per stride and their maps
    c0, x, _, _ = voxelize(xyz, voxel_size_at(v, 0), feat, dtype, batch)
    coords = [c0]
    down = [None]
    for s in range(1, 5):
        down.append(kernel_map(coords[s - 1], 2, 2))
        coords.append(down[s][0])
    subm = [kernel_map(c) for c in coords]
    m = [len(c) for c in coords]
    if trace is not None:
        trace["m"] = m

    # SPVConv 1: stem, then devoxelize + point MLP
    x = conv(x, "stem.0", subm[0], m[0])
    x = conv(x, "stem.1", subm[0], m[0])
    skips = [x]
    z = fuse(coords[0], x, 0, feat, "point.0")

    # SPVConv 2: voxelize, four downsampling stages, devoxelize + point MLP
    x = revoxelize(z, 0, coords[0])
    for s in range(1, 5):
        x = conv(x, f"down.{s}", down[s], m[s])
        x = resblock(x, f"enc.{s}.0", subm[s])
        x = resblock(x, f"enc.{s}.1", subm[s])
        skips.append(x)
    z = fuse(coords[4], x, 4, z, "point.1")
    if trace is not None:
        trace["z1"], trace["x"] = z, skips

    def up(y, u):
        t = conv(y, f"up.{u}", down[5 - u], m[4 - u], transposed=True)
        y = np.concatenate([t, skips[4 - u]], axis=1)
        y = resblock(y, f"dec.{u}.0", subm[4 - u])
        return resblock(y, f"dec.{u}.1", subm[4 - u])

    # SPVConv 3: voxelize, two upsampling stages, devoxelize + point MLP
    y = revoxelize(z, 4, coords[4])
    y = up(y, 1)
    y = up(y, 2)
    z = fuse(coords[2], y, 2, z, "point.2")
    if trace is not None:
        trace["z2"], trace["y2"] = z, y

    # SPVConv 4: voxelize, two upsampling stages, devoxelize + point MLP
    y = revoxelize(z, 2, coords[2])
    y = up(y, 3)
    y = up(y, 4)
    z = fuse(coords[0], y, 0, z, "point.3")
    if trace is not None:
        trace["z3"], trace["y4"] = z, y

    W, _, bias = P["head"]
    return linear(z, W, dtype, None, bias, False)
