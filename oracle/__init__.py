"""CPU oracle for the SPVConv hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and its
binding in ``paper_2007_16100_amd``) never touches it.

This module is a numpy/ctypes wrapper over ``libspv_oracle.so`` (plain C, fp64
accumulation, single-threaded), built from ``spv_oracle.c`` by ``build()``.
Arrays are host numpy arrays; 16-bit storage dtypes travel as uint16 bit patterns.
"""
from __future__ import annotations

import ctypes as ct
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spv_oracle.c")
_LIB = os.path.join(_HERE, "libspv_oracle.so")

OK, ERR_INVALID_ARG, ERR_CAPACITY, ERR_RANGE, ERR_NONFINITE, ERR_UNSUPPORTED = 0, 1, 2, 3, 4, 5
DT = {"f32": 0, "bf16": 1, "f16": 2}
MODE = {"center": 0, "corner": 1, "nearest": 2}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                               "-shared", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ct.CDLL(_LIB)
        vp, i64, i32, f32 = ct.c_void_p, ct.c_int64, ct.c_int32, ct.c_float
        L.spvo_voxelize.argtypes = [vp, vp, i64, f32, vp, i32, i32, vp, vp, vp, vp, vp]
        L.spvo_voxelize_onto.argtypes = [vp, i64, vp, vp, i64, f32, vp, i32, i32, vp, vp, vp]
        L.spvo_kernel_map.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, i64, vp]
        L.spvo_sparse_conv.argtypes = [vp, i64, i32, vp, vp, i32, i32, vp, vp, vp, i32, vp, i64, i32, i32]
        L.spvo_sparse_conv_res.argtypes = [vp, i64, i32, vp, vp, i32, i32, vp, vp, vp, vp, i32, vp, i64, i32, i32]
        L.spvo_devoxelize.argtypes = [vp, i64, i32, vp, vp, i64, f32, i32, vp, i32, vp, i32, vp, vp, vp, i32,
                                      vp, i32, vp, vp]
        L.spvo_block.argtypes = [vp, vp, vp, i64, vp, vp, vp]
        L.spvo_linear.argtypes = [vp, i64, i32, vp, vp, vp, vp, i32, i32, vp, i32, i32]
        L.spvo_sparse_conv_wgrad.argtypes = [vp, i64, i32, vp, i64, i32, vp, vp, i32, i32, vp, i32]
        L.spvo_voxelize_backward.argtypes = [vp, i64, i32, vp, vp, i64, vp, i32]
        L.spvo_devoxelize_backward.argtypes = [vp, vp, vp, i64, i32, vp, i64, i32]
        L.spvo_epilogue_backward.argtypes = [vp, vp, vp, vp, i32, vp, i32, i64, i32, vp, vp, vp, vp, i32]
        L.spvo_linear_backward.argtypes = [vp, i64, i32, vp, i32, vp, vp, vp, i32]
        L.spvo_decode.argtypes = [vp, i64, i32]
        L.spvo_decode.restype = ct.c_double
        L.spvo_round_store.argtypes = [ct.c_double, vp, i64, i32]
        for f in ("spvo_voxelize", "spvo_kernel_map", "spvo_sparse_conv", "spvo_sparse_conv_res", "spvo_devoxelize",
                  "spvo_block", "spvo_linear", "spvo_sparse_conv_wgrad", "spvo_voxelize_backward",
                  "spvo_devoxelize_backward", "spvo_epilogue_backward", "spvo_linear_backward"):
            getattr(L, f).restype = ct.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: oracle status {status}")
        self.status = status


def _p(a):
    return None if a is None else a.ctypes.data_as(ct.c_void_p)


def _chk(st, what):
    if st != OK:
        raise OracleError(st, what)


def _sdt(dtype):
    return np.float32 if dtype == "f32" else np.uint16


def voxelize(xyz, voxel_size, feat=None, dtype="f32", batch=None):
    """Eq. 1 + Eq. 2.  Returns (coords [m,4], vfeat [m,C] or None, counts [m], pt2vox [n])."""
    xyz = np.ascontiguousarray(xyz, dtype=np.float32)
    n = xyz.shape[0]
    batch = None if batch is None else np.ascontiguousarray(batch, dtype=np.int32)
    C = 0 if feat is None else feat.shape[1]
    feat = None if feat is None else np.ascontiguousarray(feat, dtype=_sdt(dtype))
    nn = max(n, 1)
    coords = np.zeros((nn, 4), np.int32)
    counts = np.zeros(nn, np.int32)
    pt2vox = np.zeros(nn, np.int32)
    vfeat = None if feat is None else np.zeros((nn, C), _sdt(dtype))
    m = ct.c_int64(0)
    st = lib().spvo_voxelize(_p(xyz), _p(batch), n, ct.c_float(voxel_size), _p(feat), C, DT[dtype], _p(coords),
                             _p(vfeat), _p(counts), _p(pt2vox), ct.byref(m))
    _chk(st, "voxelize")
    m = m.value
    return coords[:m], (None if vfeat is None else vfeat[:m]), counts[:m], pt2vox[:n]


def voxelize_onto(coords, xyz, voxel_size, feat=None, dtype="f32", batch=None):
    """Eq. 2 onto a given voxel set.  Returns (vfeat [m,C] or None, counts [m], pt2vox [n])."""
    coords = np.ascontiguousarray(coords, dtype=np.int32).reshape(-1, 4)
    xyz = np.ascontiguousarray(xyz, dtype=np.float32)
    m, n = coords.shape[0], xyz.shape[0]
    batch = None if batch is None else np.ascontiguousarray(batch, dtype=np.int32)
    C = 0 if feat is None else feat.shape[1]
    feat = None if feat is None else np.ascontiguousarray(feat, dtype=_sdt(dtype))
    counts = np.zeros(max(m, 1), np.int32)
    pt2vox = np.zeros(max(n, 1), np.int32)
    vfeat = None if feat is None else np.zeros((max(m, 1), C), _sdt(dtype))
    st = lib().spvo_voxelize_onto(_p(coords), m, _p(xyz), _p(batch), n, ct.c_float(voxel_size), _p(feat), C,
                                  DT[dtype], _p(vfeat), _p(counts), _p(pt2vox))
    _chk(st, "voxelize_onto")
    return (None if vfeat is None else vfeat[:m]), counts[:m], pt2vox[:n]


def kernel_map(in_coords, K=3, stride=1, pair_cap=None):
    """Returns (out_coords [m_out,4], off [K^3+1], pairs [total,2] as (in, out))."""
    in_coords = np.ascontiguousarray(in_coords, dtype=np.int32).reshape(-1, 4)
    m_in = in_coords.shape[0]
    K3 = K ** 3
    cap = (K3 * max(m_in, 1)) if pair_cap is None else pair_cap
    off = np.zeros(max(K3, 1) + 1, np.int32)
    pairs = np.zeros((max(cap, 1), 2), np.int32)
    out_coords = np.zeros((max(m_in, 1), 4), np.int32)
    m_out = ct.c_int64(0)
    total = ct.c_int64(0)
    st = lib().spvo_kernel_map(_p(in_coords), m_in, K, stride, _p(out_coords), ct.byref(m_out), _p(off),
                               _p(pairs), cap, ct.byref(total))
    _chk(st, "kernel_map")
    oc = out_coords[:m_out.value] if stride == 2 else in_coords
    return oc, off[:K3 + 1], pairs[:total.value]


def sparse_conv(x, off, pairs, W, m_out, dtype="f32", scale=None, shift=None, relu=False, transposed=False,
                res=None):
    x = np.ascontiguousarray(x, dtype=_sdt(dtype))
    W = np.ascontiguousarray(W, dtype=_sdt(dtype))
    K3, Cin, Cout = W.shape
    off = np.ascontiguousarray(off, dtype=np.int32)
    pairs = np.ascontiguousarray(pairs, dtype=np.int32).reshape(-1, 2)
    scale = None if scale is None else np.ascontiguousarray(scale, dtype=np.float32)
    shift = None if shift is None else np.ascontiguousarray(shift, dtype=np.float32)
    out = np.zeros((max(m_out, 1), Cout), _sdt(dtype))
    res = None if res is None else np.ascontiguousarray(res, dtype=_sdt(dtype)).reshape(m_out, Cout)
    st = lib().spvo_sparse_conv_res(_p(x), x.shape[0], Cin, _p(off), _p(pairs), K3, int(transposed), _p(W),
                                    _p(scale), _p(shift), _p(res), int(relu), _p(out), m_out, Cout, DT[dtype])
    _chk(st, "sparse_conv")
    return out[:m_out]


def sparse_conv_sliced(x, off, pairs, W_full, m_out, Cout, dtype="f32", scale=None, shift=None, relu=False,
                       transposed=False):
    """Weight sharing in the super network (Sec. 4.2): a layer run at C_in input and
    Cout output channels (C_in = x's width) uses the first C_in and the first Cout
    channels of the full weight tensor W_full [K3][Cin_full][Cout_full], and the
    first Cout entries of the full normalization scale / shift."""
    W_full = np.asarray(W_full)
    Cin = np.asarray(x).shape[1]
    if Cin > W_full.shape[1] or Cout > W_full.shape[2]:
        raise OracleError(ERR_INVALID_ARG, "sparse_conv_sliced")
    return sparse_conv(x, off, pairs, W_full[:, :Cin, :Cout], m_out, dtype,
                       None if scale is None else np.asarray(scale)[:Cout],
                       None if shift is None else np.asarray(shift)[:Cout], relu, transposed)


def conv_dgrad(dy, off, pairs, W, m_in, dtype="f32", transposed=False):
    """Input gradient of a sparse conv: dx[i] = sum over the pairs (i, j, k) of dy[j] @ W[k]^T --
    the same map with the roles of each pair swapped and every W[k] transposed."""
    WT = np.ascontiguousarray(np.asarray(W).transpose(0, 2, 1))
    return sparse_conv(dy, off, pairs, WT, m_in, dtype, transposed=not transposed)


def conv_wgrad(x, dy, off, pairs, K3, dtype="f32", transposed=False):
    """Weight gradient of a sparse conv: dW[k] = sum over the pairs (i, j) of offset k of
    x[i]^T dy[j]; float32 [K3][Cin][Cout]."""
    x = np.ascontiguousarray(x, dtype=_sdt(dtype))
    dy = np.ascontiguousarray(dy, dtype=_sdt(dtype))
    off = np.ascontiguousarray(off, dtype=np.int32)
    pairs = np.ascontiguousarray(pairs, dtype=np.int32).reshape(-1, 2)
    dW = np.zeros((K3, x.shape[1], dy.shape[1]), np.float32)
    st = lib().spvo_sparse_conv_wgrad(_p(x), x.shape[0], x.shape[1], _p(dy), dy.shape[0], dy.shape[1], _p(off),
                                      _p(pairs), K3, int(transposed), _p(dW), DT[dtype])
    _chk(st, "conv_wgrad")
    return dW


def voxelize_backward(dv, counts, pt2vox, dtype="f32"):
    """Backward of the scatter-mean (Eq. 2): dfeat[k] = dv[pt2vox[k]] / N_{pt2vox[k]}."""
    dv = np.ascontiguousarray(dv, dtype=_sdt(dtype))
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    pt2vox = np.ascontiguousarray(pt2vox, dtype=np.int32)
    m, C = dv.shape
    n = len(pt2vox)
    out = np.zeros((max(n, 1), C), _sdt(dtype))
    st = lib().spvo_voxelize_backward(_p(dv), m, C, _p(counts), _p(pt2vox), n, _p(out), DT[dtype])
    _chk(st, "voxelize_backward")
    return out[:n]


def devoxelize_backward(corner_idx, corner_w, dout, m, dtype="f32"):
    """Backward of the renormalized trilinear devoxelization w.r.t. the voxel features
    (float32 [m][C]), from devoxelize's corner indices and raw weights."""
    ci = np.ascontiguousarray(corner_idx, dtype=np.int32)
    cw = np.ascontiguousarray(corner_w, dtype=np.float32)
    dout = np.ascontiguousarray(dout, dtype=_sdt(dtype))
    n, C = dout.shape
    dv = np.zeros((max(m, 1), C), np.float32)
    st = lib().spvo_devoxelize_backward(_p(ci), _p(cw), _p(dout), n, C, _p(dv), m, DT[dtype])
    _chk(st, "devoxelize_backward")
    return dv[:m]


def linear(x, W, dtype="f32", scale=None, shift=None, relu=False, res=None, res_after_act=False):
    """Pointwise linear layer (the point MLP of Sec. 3.3, a 1x1 shortcut, a classifier):
    act(scale * (x @ W) + shift + res), or act(...) + res with res_after_act."""
    x = np.ascontiguousarray(x, dtype=_sdt(dtype))
    W = np.ascontiguousarray(W, dtype=_sdt(dtype))
    m, Cin = x.shape
    Cout = W.shape[1]
    if W.shape[0] != Cin:
        raise OracleError(ERR_INVALID_ARG, "linear")
    scale = None if scale is None else np.ascontiguousarray(scale, dtype=np.float32)
    shift = None if shift is None else np.ascontiguousarray(shift, dtype=np.float32)
    res = None if res is None else np.ascontiguousarray(res, dtype=_sdt(dtype)).reshape(m, Cout)
    out = np.zeros((max(m, 1), Cout), _sdt(dtype))
    st = lib().spvo_linear(_p(x), m, Cin, _p(W), _p(scale), _p(shift), _p(res), int(res_after_act), int(relu), _p(out),
                           Cout, DT[dtype])
    _chk(st, "linear")
    return out[:m]


def epilogue_backward(dy, a, scale=None, shift=None, relu=False, res=None, res_after_act=False, dtype="f32"):
    """Backward of act(scale * a + shift + res) (or act(...) + res with res_after_act) w.r.t.
    a, res, scale and shift, given the raw product a: (da, dres, dscale, dshift)."""
    dy = np.ascontiguousarray(dy, dtype=_sdt(dtype))
    m, C = dy.shape
    a = np.ascontiguousarray(a, dtype=_sdt(dtype)).reshape(m, C)
    scale = None if scale is None else np.ascontiguousarray(scale, dtype=np.float32)
    shift = None if shift is None else np.ascontiguousarray(shift, dtype=np.float32)
    res = None if res is None else np.ascontiguousarray(res, dtype=_sdt(dtype)).reshape(m, C)
    da = np.zeros((max(m, 1), C), _sdt(dtype))
    dres = np.zeros((max(m, 1), C), _sdt(dtype))
    dscale = np.zeros(C, np.float32)
    dshift = np.zeros(C, np.float32)
    st = lib().spvo_epilogue_backward(_p(dy), _p(a), _p(scale), _p(shift), int(relu), _p(res), int(res_after_act), m,
                                      C, _p(da), _p(dres), _p(dscale), _p(dshift), DT[dtype])
    _chk(st, "epilogue_backward")
    return da[:m], dres[:m], dscale, dshift


def linear_backward(x, W, da, dtype="f32"):
    """Gradients of x @ W: (dx = da @ W^T in dtype, dW = x^T @ da in float32)."""
    x = np.ascontiguousarray(x, dtype=_sdt(dtype))
    W = np.ascontiguousarray(W, dtype=_sdt(dtype))
    m, Cin = x.shape
    Cout = W.shape[1]
    da = np.ascontiguousarray(da, dtype=_sdt(dtype)).reshape(m, Cout)
    dx = np.zeros((max(m, 1), Cin), _sdt(dtype))
    dW = np.zeros((Cin, Cout), np.float32)
    st = lib().spvo_linear_backward(_p(x), m, Cin, _p(W), Cout, _p(da), _p(dx), _p(dW), DT[dtype])
    _chk(st, "linear_backward")
    return dx[:m], dW


def devoxelize(grid_coords, vfeat, xyz, voxel_size, stride_log2=0, mode="center", batch=None, pfeat=None,
               Wp=None, scale_p=None, shift_p=None, relu_p=False, dtype="f32", want_corners=False):
    grid_coords = np.ascontiguousarray(grid_coords, dtype=np.int32).reshape(-1, 4)
    vfeat = np.ascontiguousarray(vfeat, dtype=_sdt(dtype))
    xyz = np.ascontiguousarray(xyz, dtype=np.float32)
    n = xyz.shape[0]
    C = vfeat.shape[1]
    batch = None if batch is None else np.ascontiguousarray(batch, dtype=np.int32)
    Cp = 0
    if pfeat is not None:
        pfeat = np.ascontiguousarray(pfeat, dtype=_sdt(dtype))
        Wp = np.ascontiguousarray(Wp, dtype=_sdt(dtype))
        Cp = pfeat.shape[1]
    scale_p = None if scale_p is None else np.ascontiguousarray(scale_p, dtype=np.float32)
    shift_p = None if shift_p is None else np.ascontiguousarray(shift_p, dtype=np.float32)
    out = np.zeros((max(n, 1), C), _sdt(dtype))
    ci = np.zeros((max(n, 1), 8), np.int32) if want_corners else None
    cw = np.zeros((max(n, 1), 8), np.float32) if want_corners else None
    st = lib().spvo_devoxelize(_p(grid_coords), grid_coords.shape[0], stride_log2, _p(xyz), _p(batch), n,
                               ct.c_float(voxel_size), MODE[mode], _p(vfeat), C, _p(pfeat), Cp, _p(Wp),
                               _p(scale_p), _p(shift_p), int(relu_p), _p(out), DT[dtype], _p(ci), _p(cw))
    _chk(st, "devoxelize")
    if want_corners:
        return out[:n], ci[:n], cw[:n]
    return out[:n]


class _BlockParams(ct.Structure):
    _fields_ = [("C", ct.c_int32), ("dtype", ct.c_int32), ("voxel_size", ct.c_float), ("n_convs", ct.c_int32),
                ("W", ct.c_void_p * 2), ("scale", ct.c_void_p * 2), ("shift", ct.c_void_p * 2),
                ("relu", ct.c_int32 * 2), ("Wp", ct.c_void_p), ("scale_p", ct.c_void_p), ("shift_p", ct.c_void_p),
                ("relu_p", ct.c_int32), ("devox_mode", ct.c_int32), ("residual", ct.c_int32)]


def block(xyz, feat, voxel_size, convs, Wp, scale_p=None, shift_p=None, relu_p=True, dtype="f32", batch=None,
          mode="center", residual=False):
    """SPVConv block.  convs: list of (W [27,C,C], scale|None, shift|None, relu).  residual: the last
    conv adds the block's voxel input before its activation (a residual block, Sec. 3.3)."""
    xyz = np.ascontiguousarray(xyz, dtype=np.float32)
    feat = np.ascontiguousarray(feat, dtype=_sdt(dtype))
    n, C = feat.shape
    keep = []

    def arr(a, t):
        if a is None:
            return None
        a = np.ascontiguousarray(a, dtype=t)
        keep.append(a)
        return a.ctypes.data

    p = _BlockParams()
    p.C, p.dtype, p.voxel_size, p.n_convs = C, DT[dtype], voxel_size, len(convs)
    for l, (W, sc, sh, r) in enumerate(convs):
        p.W[l] = arr(W, _sdt(dtype))
        p.scale[l] = arr(sc, np.float32)
        p.shift[l] = arr(sh, np.float32)
        p.relu[l] = int(r)
    p.Wp = arr(Wp, _sdt(dtype))
    p.scale_p = arr(scale_p, np.float32)
    p.shift_p = arr(shift_p, np.float32)
    p.relu_p = int(relu_p)
    p.devox_mode = MODE[mode]
    p.residual = int(residual)
    batch = None if batch is None else np.ascontiguousarray(batch, dtype=np.int32)
    out = np.zeros((max(n, 1), C), _sdt(dtype))
    m = ct.c_int64(0)
    st = lib().spvo_block(ct.byref(p), _p(xyz), _p(batch), n, _p(feat), _p(out), ct.byref(m))
    _chk(st, "block")
    return out[:n], m.value


def raw_status(fn: str, *args) -> int:
    """Call an oracle entry point with raw ctypes arguments; return its status (error-path tests)."""
    return getattr(lib(), fn)(*args)
