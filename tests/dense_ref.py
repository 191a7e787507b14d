"""Independent dense / brute-force formulations used to pin the oracle.

Nothing here calls the oracle or the HIP library.  Each function is a textbook
formulation of what the SPVConv path computes, evaluated the slow, dense way:

* ``quantize``           Eq. 1 with numpy float32 division and floor.
* ``eq2_literal``        Eq. 2 exactly as printed: an m x n indicator matrix.
* ``kmap_allpairs``      every (input, output) pair tested against every offset.
* ``dense_conv*``        torch.nn.functional.conv3d / conv_transpose3d in float64
                         on the zero-filled dense grid.
* ``dense_trilinear``    torch.nn.functional.grid_sample (trilinear,
                         align_corners=True) in float64 on the zero-filled grid;
                         renormalization over present corners is the ratio of the
                         sampled features to the sampled occupancy mask.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def quantize(xyz, v):
    a = np.asarray(xyz, np.float32) / np.float32(v)
    return np.floor(a.astype(np.float64)).astype(np.int64)


def eq2_literal(xyz, feat64, v, batch=None):
    """Returns (coords sorted [m,4], mean features [m,C] in float64) by Eq. 1-2 as written."""
    q = quantize(xyz, v)
    b = np.zeros(len(q), np.int64) if batch is None else np.asarray(batch, np.int64)
    keys = sorted({(int(b[k]), int(q[k, 0]), int(q[k, 1]), int(q[k, 2])) for k in range(len(q))})
    coords = np.array(keys, np.int64).reshape(-1, 4)
    pk = np.concatenate([b[:, None], q], axis=1)
    # indicator I[m, k] = [p_hat_k == p_m]
    ind = np.all(coords[:, None, :] == pk[None, :, :], axis=2).astype(np.float64)
    N = ind.sum(axis=1)
    return coords, (ind @ feat64) / N[:, None], N


def kmap_allpairs(in_coords, K, stride):
    """Brute-force kernel map: returns (out_coords, sorted list of (k, out, in))."""
    c = np.asarray(in_coords, np.int64)
    if stride == 1:
        oc = c
        deltas = [(dx, dy, dz) for dx in (-1, 0, 1) for dy in (-1, 0, 1) for dz in (-1, 0, 1)]
    else:
        oc = np.array(sorted({(int(r[0]), int(r[1]) // 2, int(r[2]) // 2, int(r[3]) // 2) for r in c}),
                      np.int64).reshape(-1, 4)
        deltas = [(dx, dy, dz) for dx in (0, 1) for dy in (0, 1) for dz in (0, 1)]
    trip = []
    for j in range(len(oc)):
        for i in range(len(c)):
            if c[i, 0] != oc[j, 0]:
                continue
            d = tuple(int(x) for x in (c[i, 1:] - stride * oc[j, 1:]))
            if d in deltas:
                trip.append((deltas.index(d), j, i))
    return oc, sorted(trip)


def _grid(coords, feat64, pad=1, origin=None, shape=None):
    """Zero-filled dense grid [C, X, Y, Z] (single batch) holding feat at coords."""
    xyz = np.asarray(coords, np.int64)[:, 1:]
    if origin is None:
        origin = xyz.min(axis=0) - pad
    if shape is None:
        shape = xyz.max(axis=0) - origin + 1 + pad
    C = feat64.shape[1]
    g = np.zeros((C,) + tuple(int(s) for s in shape), np.float64)
    idx = xyz - origin
    g[:, idx[:, 0], idx[:, 1], idx[:, 2]] = feat64.T
    return g, origin


def _w_subm_torch(W64):
    """[27][Cin][Cout] with k = 9(dx+1)+3(dy+1)+(dz+1) -> Conv3d weight [Cout][Cin][3][3][3]."""
    K3, Cin, Cout = W64.shape
    return torch.from_numpy(np.ascontiguousarray(W64.reshape(3, 3, 3, Cin, Cout).transpose(4, 3, 0, 1, 2)))


def dense_conv_subm(coords, feat64, W64):
    """Submanifold conv = dense conv3d(padding=1) on the zero-filled grid read at the active sites."""
    g, o = _grid(coords, feat64, pad=1)
    y = F.conv3d(torch.from_numpy(g)[None], _w_subm_torch(W64), padding=1)[0].numpy()
    idx = np.asarray(coords, np.int64)[:, 1:] - o
    return y[:, idx[:, 0], idx[:, 1], idx[:, 2]].T


def dense_conv_down(coords, feat64, W64, out_coords):
    """k=2 s=2 conv = dense conv3d(kernel 2, stride 2) on a grid whose origin is even."""
    xyz = np.asarray(coords, np.int64)[:, 1:]
    o = xyz.min(axis=0)
    o = o - (o % 2)  # even origin keeps floor(c/2) aligned with the stride-2 windows
    g, _ = _grid(coords, feat64, pad=0, origin=o, shape=xyz.max(axis=0) - o + 2)
    K3, Cin, Cout = W64.shape
    w = torch.from_numpy(np.ascontiguousarray(W64.reshape(2, 2, 2, Cin, Cout).transpose(4, 3, 0, 1, 2)))
    y = F.conv3d(torch.from_numpy(g)[None], w, stride=2)[0].numpy()
    idx = np.asarray(out_coords, np.int64)[:, 1:] - o // 2
    return y[:, idx[:, 0], idx[:, 1], idx[:, 2]].T, y


def dense_conv_transposed(coarse_coords, feat64, W64, fine_coords):
    """Transposed k=2 s=2 conv = dense conv_transpose3d read at the fine active sites."""
    cxyz = np.asarray(coarse_coords, np.int64)[:, 1:]
    o = cxyz.min(axis=0)
    g, _ = _grid(coarse_coords, feat64, pad=0, origin=o, shape=cxyz.max(axis=0) - o + 1)
    K3, Cin, Cout = W64.shape
    w = torch.from_numpy(np.ascontiguousarray(W64.reshape(2, 2, 2, Cin, Cout).transpose(3, 4, 0, 1, 2)))
    y = F.conv_transpose3d(torch.from_numpy(g)[None], w, stride=2)[0].numpy()
    idx = np.asarray(fine_coords, np.int64)[:, 1:] - 2 * o
    return y[:, idx[:, 0], idx[:, 1], idx[:, 2]].T


def dense_trilinear(coords, vfeat64, xyz, v, stride_log2=0, mode="center"):
    """Renormalized trilinear devoxelization via grid_sample on the dense grid."""
    g, o = _grid(coords, vfeat64, pad=2)
    mask, _ = _grid(coords, np.ones((len(coords), 1)), pad=2, origin=o, shape=g.shape[1:])
    a = (np.asarray(xyz, np.float32) / np.float32(v)).astype(np.float64) * 2.0 ** (-stride_log2)
    u = a - 0.5 if mode == "center" else a
    pos = u - o  # continuous index into the grid
    size = np.array(g.shape[1:], np.float64)
    gn = 2.0 * pos / (size - 1.0) - 1.0
    grid = torch.from_numpy(gn[:, ::-1].copy()).reshape(1, 1, 1, -1, 3)  # (z, y, x) -> (W, H, D)
    num = F.grid_sample(torch.from_numpy(g)[None], grid, mode="bilinear", align_corners=True)[0, :, 0, 0].numpy()
    den = F.grid_sample(torch.from_numpy(mask)[None], grid, mode="bilinear", align_corners=True)[0, 0, 0, 0].numpy()
    out = np.where(den[None, :] > 0, num / np.where(den > 0, den, 1.0)[None, :], 0.0)
    return out.T, den
