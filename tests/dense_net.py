"""The SPVCNN-style network evaluated densely in float64, to pin the oracle's
composition (tests only; nothing here calls the oracle or the HIP library).

Every operation is the dense formulation of ``dense_ref``: Eq. 1-2 as an
indicator matrix (voxelization at each stride is the points quantized with the
stride's voxel size), convolutions as torch conv3d / conv_transpose3d on the
zero-filled grid, devoxelization as grid_sample over features and occupancy.
Single scene (one batch index).  The layer list is the one
``synth.spvcnn_params`` names.
"""
import numpy as np

from tests import dense_ref


def _bn(y, sc, sh):
    return y * np.asarray(sc, np.float64) + np.asarray(sh, np.float64)


def dense_spvcnn(xyz, feat64, P64, v, mode="center"):
    """P64: the parameter dict with float64 arrays.  Returns (logits [n][classes], voxel counts)."""
    def vs(s):
        return float(np.float32(v) * np.float32(2.0 ** s))

    coords = []
    for s in range(5):
        c, _, _ = dense_ref.eq2_literal(xyz, np.zeros((len(xyz), 1)), vs(s))
        coords.append(c)
    _, x, _ = dense_ref.eq2_literal(xyz, feat64, vs(0))

    def subm(x, name, s, relu=True, res=None):
        W, sc, sh = P64[name]
        y = _bn(dense_ref.dense_conv_subm(coords[s], x, W), sc, sh)
        if res is not None:
            y = y + res
        return np.maximum(y, 0.0) if relu else y

    def resblock(x, name, s):
        h = subm(x, name + ".a", s)
        if name + ".sc" in P64:
            W, sc, sh = P64[name + ".sc"]
            r = _bn(x @ W, sc, sh)
        else:
            r = x
        return subm(h, name + ".b", s, res=r)

    def fuse(vfeat, s, z, name):
        d, _ = dense_ref.dense_trilinear(coords[s], vfeat, xyz, v, s, mode)
        W, sc, sh = P64[name]
        return d + np.maximum(_bn(z @ W, sc, sh), 0.0)

    def vox(z, s):
        _, f, _ = dense_ref.eq2_literal(xyz, z, vs(s))
        return f

    x = subm(x, "stem.0", 0)
    x = subm(x, "stem.1", 0)
    skips = [x]
    z = fuse(x, 0, feat64, "point.0")
    x = vox(z, 0)
    for s in range(1, 5):
        W, sc, sh = P64[f"down.{s}"]
        x = np.maximum(_bn(dense_ref.dense_conv_down(coords[s - 1], x, W, coords[s])[0], sc, sh), 0.0)
        x = resblock(x, f"enc.{s}.0", s)
        x = resblock(x, f"enc.{s}.1", s)
        skips.append(x)
    z = fuse(x, 4, z, "point.1")

    def up(y, u):
        W, sc, sh = P64[f"up.{u}"]
        t = np.maximum(_bn(dense_ref.dense_conv_transposed(coords[5 - u], y, W, coords[4 - u]), sc, sh), 0.0)
        y = np.concatenate([t, skips[4 - u]], axis=1)
        y = resblock(y, f"dec.{u}.0", 4 - u)
        return resblock(y, f"dec.{u}.1", 4 - u)

    y = vox(z, 4)
    y = up(up(y, 1), 2)
    z = fuse(y, 2, z, "point.2")
    y = vox(z, 2)
    y = up(up(y, 3), 4)
    z = fuse(y, 0, z, "point.3")
    W, _, bias = P64["head"]
    return z @ W + np.asarray(bias, np.float64), [len(c) for c in coords]
