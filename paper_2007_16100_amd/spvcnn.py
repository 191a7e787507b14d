"""SPVCNN-style encoder-decoder forward on the libspv C ABI.

The backbone of the paper's appendix A.1: MinkowskiNet-style residual sparse-conv
blocks (a U-Net with four stride-2 stages and four transposed stages with skip
connections) wrapped by four SPVConv point branches (Sec. 3.3).  The first
module voxelizes the points and devoxelizes after the stem; the second
voxelizes again and devoxelizes after the four downsampling stages; the last two
each wrap two upsampling stages.  Every devoxelization is fused with the point
branch's MLP by addition; a linear head gives per-point class scores.

Every step runs in libspv's kernels; this module only sequences the calls and
holds the device buffers:

* plan: voxelization at stride 1, the four stride-2 maps (which give the
  coordinate sets of strides 2..16) and a submanifold neighbour table per stride,
  one synchronization per stride to size what follows exactly; every 3x3x3 conv
  the neighbour-table kernel takes runs on that table (no per-call plan), the
  others on the stride's pairs, built on first use;
* the later modules' voxelizations scatter the point features onto the voxel set the
  plan holds for their stride (no sort);
* the transposed stride-2 convs run on the stride-2 maps' child tables: every
  fine voxel has its parent, so each output row is one product row, stored once;
* a conv over a skip concatenation [t; x] runs as two sliced convs,
  W_t t (scaled, unshifted) handed as the residual input of W_x x + shift;
  the 1x1 shortcut over it likewise as two linear layers;
* the stride-1 fusions read each point's corners from the stride-1 neighbour table (the grid
  is the points' own voxelization), without a hash table;
* the weights of the neighbour-table, upsampling and linear layers are packed into
  matrix-core fragments once, on first use, and read packed by every later forward;
* a devoxelization whose point MLP the fused kernel does not take on matrix
  cores (C_p above 128) runs as a devoxelization plus a linear layer that adds
  it after the activation.
Layer names and widths follow ``synth.spvcnn_params``.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np
import torch

from . import spv

_TORCH = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}


def voxel_size_at(v: float, s: int) -> float:
    """Voxel size of stride 2^s: the float32 voxel size scaled by 2^s (exact in float32), so
    that voxelizing at stride 2^s gives the cascaded stride-2 coordinates."""
    return float(np.float32(v) * np.float32(2.0 ** s))


@dataclass
class Plan:
    coords: List[torch.Tensor]      # [m_s][4] per stride 2^s, s = 0..4
    m: List[int]
    down: List[Optional[spv.KernelMap]]   # down[s]: stride 2^(s-1) -> 2^s (s = 1..4)
    nbr: List[torch.Tensor]         # submanifold neighbour table [m_s][27] per stride
    subm: List[Optional[spv.KernelMap]]   # submanifold pairs, built on first use
    children: List[Optional[torch.Tensor]]  # children[s]: child table [m_s][8] of down[s]
    pt2vox0: torch.Tensor           # every point's stride-1 voxel


class SPVCNN:
    def __init__(self, params: Dict[str, tuple], dtype: str = "bf16", voxel_size: float = 0.05,
                 mode: int = spv.SPV_DEVOX_CENTER, device: str = "cuda"):
        self.dt = _TORCH[dtype]
        self.v = voxel_size
        self.mode = mode
        self.device = device
        # the input channels are padded with zeros to 32, the narrowest width of the
        # neighbour-table conv kernel (whose matrix-core K step is 32 channels), so that the stem
        # runs on the stride's neighbour table like every other 3x3x3 conv: the stem conv and the
        # first point MLP get zero weight rows for them, which adds exact zeros
        self.c_in = params["stem.0"][0].shape[1]
        self.c_pad = self.c_in if self.dt == torch.float32 else (self.c_in + 31) // 32 * 32
        self.P = {}
        for name, (W, sc, sh) in params.items():
            if name in ("stem.0", "point.0") and self.c_pad != self.c_in:
                W = np.asarray(W)
                pad = [(0, 0)] * W.ndim
                pad[-2] = (0, self.c_pad - self.c_in)
                W = np.pad(W, pad)
            self.P[name] = (self._dev(W), None if sc is None else torch.from_numpy(np.asarray(sc)).to(device),
                            None if sh is None else torch.from_numpy(np.asarray(sh)).to(device))
        self.ws = None
        # matrix-core fragments of every (layer, input-channel slice) that a kernel reading packed
        # weights runs, packed on first use: the weights stay fixed across forwards
        self._pk: Dict[tuple, Optional[torch.Tensor]] = {}

    def _dev(self, a):
        a = np.ascontiguousarray(a)
        if self.dt == torch.float32:
            return torch.from_numpy(a.astype(np.float32)).to(self.device)
        return torch.from_numpy(a.view(np.int16)).view(self.dt).to(self.device)

    def _workspace(self, n):
        need = spv.spv_workspace_bytes(max(n, 1), 256)
        if self.ws is None or self.ws.nbytes < need:
            self.ws = spv.Workspace(need, self.device)
        return self.ws

    # -- plan ----------------------------------------------------------------
    def plan(self, xyz: torch.Tensor, batch: Optional[torch.Tensor] = None, feat: Optional[torch.Tensor] = None):
        ws = self._workspace(xyz.shape[0])
        vox = spv.spv_voxelize(ws, xyz, self.v, feat, batch)
        m = [vox.m]
        coords = [vox.coords[: vox.m]]
        down: List[Optional[spv.KernelMap]] = [None]
        for s in range(1, 5):
            km = spv.spv_kernel_map(ws, coords[s - 1], K=2, stride=2)
            ms = int(km.m_out_dev.item())
            down.append(km)
            m.append(ms)
            coords.append(km.out_coords[:ms])
        nbr = [spv.spv_kernel_map_nbr(ws, c) for c in coords]
        children = [None] + [spv.spv_map_children(ws, down[s].off, down[s].pairs, m[s - 1], m[s]) for s in range(1, 5)]
        return Plan(coords, m, down, nbr, [None] * 5, children, vox.pt2vox), vox

    # -- layers --------------------------------------------------------------
    def clear_packed(self):
        """Drop the packed weights: call after changing any weight in ``self.P`` in place, so that
        the next forward packs the new values."""
        self._pk.clear()

    def _packed(self, name, cin_offset, Cin, Cout):
        key = (name, cin_offset, Cin, Cout)
        if key not in self._pk:
            self._pk[key] = spv.spv_pack_weights(self.P[name][0], Cin, Cout, cin_offset)
        return self._pk[key]

    def _conv(self, x, name, km, m_out, relu=True, transposed=False, res=None, cin_offset=0, shift=True):
        W, sc, sh = self.P[name]
        return spv.spv_sparse_conv_sliced(self.ws, x, km.off, km.pairs, W, x.shape[1], W.shape[2], m_out, scale=sc,
                                          shift=sh if shift else None, relu=relu, transposed=transposed, res=res,
                                          cin_offset=cin_offset)

    def _subm(self, plan, x, name, s, relu=True, res=None, cin_offset=0, shift=True):
        """A submanifold 3x3x3 conv at stride 2^s: on the stride's neighbour table where the
        neighbour-table kernel takes the shape, else on the pairs (built once per stride)."""
        W, sc, sh = self.P[name]
        Cin, Cout = x.shape[1], W.shape[2]
        widths = (32, 64, 96, 128, 256)
        if self.dt != torch.float32 and Cin in widths and Cout in widths:
            return spv.spv_sparse_conv_nbr_packed(self.ws, x, plan.nbr[s], self._packed(name, cin_offset, Cin, Cout),
                                                  Cout, plan.m[s], scale=sc, shift=sh if shift else None, relu=relu,
                                                  res=res)
        if plan.subm[s] is None:
            plan.subm[s] = spv.spv_kernel_map(self.ws, plan.coords[s], sync=False)
        return self._conv(x, name, plan.subm[s], plan.m[s], relu=relu, res=res, cin_offset=cin_offset, shift=shift)

    def _lin(self, x, name, relu=False, res=None, res_after=False, cin_offset=0, shift=True):
        W, sc, sh = self.P[name]
        Cin, Cout = x.shape[1], W.shape[1]
        key = (name, cin_offset, Cin, Cout)
        wp = self._packed(name, cin_offset, Cin, Cout)
        if wp is not None:
            try:
                return spv.spv_linear_packed(self.ws, x, wp, Cout, scale=sc, shift=sh if shift else None,
                                             relu=relu, res=res, res_after_act=res_after)
            except spv.SpvError as e:
                # a shape only the vector-ALU kernel takes: that kernel reads W itself
                if e.status != spv.SPV_ERR_UNSUPPORTED:
                    raise
                self._pk[key] = None
        return spv.spv_linear(self.ws, x, W, scale=sc, shift=sh if shift else None, relu=relu, res=res,
                              res_after_act=res_after, cin_offset=cin_offset)

    def _resblock(self, plan, parts, name, s):
        """Residual block at stride 2^s over the concatenation of `parts` (one tensor: no
        concatenation).  Each layer over the concatenation runs part by part: every part but
        the last gives a scaled, unshifted, unactivated partial sum, the residual input of the
        next part's layer."""
        offs = np.cumsum([0] + [p.shape[1] for p in parts[:-1]])

        def over_parts(layer):
            r = None
            for i, (p, o) in enumerate(zip(parts, offs)):
                r = layer(p, int(o), r, i == len(parts) - 1)
            return r

        h = over_parts(lambda p, o, r, final: self._subm(plan, p, name + ".a", s, relu=final, res=r, cin_offset=o,
                                                          shift=final))
        if name + ".sc" in self.P:
            sc = over_parts(lambda p, o, r, final: self._lin(p, name + ".sc", res=r, cin_offset=o, shift=final))
        else:
            sc = parts[0]
        return self._subm(plan, h, name + ".b", s, res=sc)

    def _fuse(self, plan, vfeat, s, z, name, xyz, batch):
        W, sc, sh = self.P[name]
        C, Cp = vfeat.shape[1], z.shape[1]
        fused = self.dt != torch.float32 and C % 16 == 0 and C // 16 in (1, 2, 4, 6, 8, 16) and Cp % 8 == 0 and \
            Cp <= 128
        if fused and s == 0:
            # the grid is the points' own voxelization: corners from the stride's neighbour table
            return spv.spv_devoxelize_nbr(self.ws, plan.coords[0], vfeat, plan.nbr[0], plan.pt2vox0, xyz, self.v, 0,
                                          self.mode, batch, pfeat=z, Wp=W, scale_p=sc, shift_p=sh, relu_p=True)
        if fused:
            return spv.spv_devoxelize(self.ws, plan.coords[s], vfeat, xyz, self.v, s, self.mode, batch, pfeat=z, Wp=W,
                                      scale_p=sc, shift_p=sh, relu_p=True)
        d = spv.spv_devoxelize(self.ws, plan.coords[s], vfeat, xyz, self.v, s, self.mode, batch)
        return self._lin(z, name, relu=True, res=d, res_after=True)

    def _revoxelize(self, plan, xyz, z, s, batch):
        """Scatter-mean of the point features at stride 2^s onto that stride's voxels, which the
        plan already holds (the points quantized at voxel_size_at(v, s) land exactly on them):
        no insert and no sort, one table probe per point."""
        vox = spv.spv_voxelize_onto(self.ws, plan.coords[s], xyz, voxel_size_at(self.v, s), z, batch)
        return vox.vfeat[: plan.m[s]], vox

    # -- forward -------------------------------------------------------------
    def forward(self, xyz: torch.Tensor, feat: torch.Tensor, batch: Optional[torch.Tensor] = None,
                trace: Optional[dict] = None) -> torch.Tensor:
        if feat.shape[1] != self.c_pad:
            f = torch.zeros((feat.shape[0], self.c_pad), dtype=feat.dtype, device=feat.device)
            f[:, : feat.shape[1]] = feat
            feat = f
        plan, vox = self.plan(xyz, batch, feat)
        m = plan.m
        x = vox.vfeat[: m[0]]
        x = self._subm(plan, x, "stem.0", 0)
        x = self._subm(plan, x, "stem.1", 0)
        skips = [x]
        z = self._fuse(plan, x, 0, feat, "point.0", xyz, batch)

        x, _ = self._revoxelize(plan, xyz, z, 0, batch)
        for s in range(1, 5):
            x = self._conv(x, f"down.{s}", plan.down[s], m[s])
            x = self._resblock(plan, [x], f"enc.{s}.0", s)
            x = self._resblock(plan, [x], f"enc.{s}.1", s)
            skips.append(x)
        z = self._fuse(plan, x, 4, z, "point.1", xyz, batch)

        def up(y, u):
            W, sc, sh = self.P[f"up.{u}"]
            widths = (32, 64, 96, 128, 256)
            if self.dt != torch.float32 and y.shape[1] in widths and W.shape[2] in widths:
                # every fine voxel has its parent: the child-table kernel writes each output row once
                t = spv.spv_sparse_conv_up_packed(self.ws, y, plan.children[5 - u],
                                                  self._packed(f"up.{u}", 0, y.shape[1], W.shape[2]), W.shape[2],
                                                  m[4 - u], scale=sc, shift=sh, relu=True)
            else:
                t = self._conv(y, f"up.{u}", plan.down[5 - u], m[4 - u], transposed=True)
            y = self._resblock(plan, [t, skips[4 - u]], f"dec.{u}.0", 4 - u)
            return self._resblock(plan, [y], f"dec.{u}.1", 4 - u)

        y, vox4 = self._revoxelize(plan, xyz, z, 4, batch)
        y = up(up(y, 1), 2)
        z = self._fuse(plan, y, 2, z, "point.2", xyz, batch)
        y, vox2 = self._revoxelize(plan, xyz, z, 2, batch)
        y = up(up(y, 3), 4)
        z = self._fuse(plan, y, 0, z, "point.3", xyz, batch)
        out = self._lin(z, "head")
        if trace is not None:
            trace.update(plan=plan, revox=[vox4, vox2], z3=z, y4=y, skips=skips)
        return out
