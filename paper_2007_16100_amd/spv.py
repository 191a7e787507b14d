"""Python binding of libspv.so (ctypes): argument marshalling only.

Every function below forwards to the C entry point of the same name in
``include/spv.h``; all computation happens in the library's HIP kernels.
torch supplies device memory (tensor ``data_ptr``) and the stream
(``torch.cuda.current_stream().cuda_stream``).  Output tensors are allocated
here with torch when the caller does not pass them.

There is no fallback: if ``libspv.so`` is missing, or the tensors are not on a
GPU, the call raises.
"""
from __future__ import annotations

import ctypes as ct
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspv.so")

SPV_OK, SPV_ERR_INVALID_ARG, SPV_ERR_CAPACITY, SPV_ERR_RANGE, SPV_ERR_NONFINITE, SPV_ERR_UNSUPPORTED, SPV_ERR_HIP = \
    range(7)
SPV_F32, SPV_BF16, SPV_F16 = 0, 1, 2
SPV_DEVOX_CENTER, SPV_DEVOX_CORNER, SPV_DEVOX_NEAREST = 0, 1, 2

_DT = {torch.float32: SPV_F32, torch.bfloat16: SPV_BF16, torch.float16: SPV_F16}

# every symbol include/spv.h declares
EXPORTS = ("spv_workspace_bytes", "spv_voxelize", "spv_voxelize_onto", "spv_packed_weights_bytes",
           "spv_pack_weights", "spv_devoxelize_nbr", "spv_sparse_conv_nbr_packed", "spv_sparse_conv_up_packed", "spv_linear_packed",
           "spv_kernel_map", "spv_sparse_conv", "spv_sparse_conv_sliced",
           "spv_linear", "spv_kernel_map_nbr", "spv_sparse_conv_nbr", "spv_map_children", "spv_sparse_conv_up",
           "spv_sparse_conv_dgrad", "spv_sparse_conv_dgrad_nbr", "spv_wgrad_workspace_bytes", "spv_sparse_conv_wgrad",
           "spv_voxelize_backward",
           "spv_devoxelize_backward_workspace_bytes", "spv_devoxelize_backward", "spv_devoxelize",
           "spv_epilogue_backward_workspace_bytes", "spv_epilogue_backward",
           "spv_linear_backward_workspace_bytes", "spv_linear_backward",
           "spv_block_workspace_bytes", "spv_block", "spv_lookup", "spv_voxel_lookup", "spv_conv_kernel",
           "spv_sparse_conv_nbr_noalloc",
           "spv_block_conv_kernel", "spv_status_check", "spv_status_string", "spv_last_hip_error")


class SpvError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        msg = lib().spv_status_string(status).decode() if _lib is not None else str(status)
        super().__init__(f"{what}: {msg} (status {status})")


class BlockParams(ct.Structure):
    _fields_ = [("C", ct.c_int32), ("dtype", ct.c_int32), ("voxel_size", ct.c_float), ("n_convs", ct.c_int32),
                ("W", ct.c_void_p * 2), ("scale", ct.c_void_p * 2), ("shift", ct.c_void_p * 2),
                ("relu", ct.c_int32 * 2), ("Wp", ct.c_void_p), ("scale_p", ct.c_void_p), ("shift_p", ct.c_void_p),
                ("relu_p", ct.c_int32), ("devox_mode", ct.c_int32), ("residual", ct.c_int32),
                ("events", ct.POINTER(ct.c_void_p)),
                ("n_events", ct.c_int32)]


_lib = None


def lib():
    """Load libspv.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2007_16100_amd.build`")
        L = ct.CDLL(LIB_PATH)
        vp, i64, i32, f32, sz = ct.c_void_p, ct.c_int64, ct.c_int32, ct.c_float, ct.c_size_t
        L.spv_workspace_bytes.argtypes = [i64, i32]
        L.spv_workspace_bytes.restype = sz
        L.spv_block_workspace_bytes.argtypes = [i64, i32]
        L.spv_block_workspace_bytes.restype = sz
        L.spv_voxelize.argtypes = [vp, vp, sz, vp, vp, i64, f32, vp, i32, i32, vp, vp, vp, vp, vp, vp]
        L.spv_packed_weights_bytes.argtypes = [i32, i32, i32]
        L.spv_packed_weights_bytes.restype = sz
        L.spv_pack_weights.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, vp, sz]
        L.spv_sparse_conv_nbr_packed.argtypes = [vp, vp, sz, vp, i64, i32, vp, vp, vp, vp, vp, i32, vp, vp, i64, i32,
                                                 i32]
        L.spv_sparse_conv_up_packed.argtypes = [vp, vp, sz, vp, vp, i64, i32, vp, vp, vp, vp, vp, i32, vp, i64, i32,
                                                i32]
        L.spv_linear_packed.argtypes = [vp, vp, sz, vp, vp, i64, i32, vp, vp, vp, i32, vp, i32, vp, i32, i32]
        L.spv_voxelize_onto.argtypes = [vp, vp, sz, vp, vp, i64, vp, vp, i64, f32, vp, i32, i32, vp, vp, vp]
        L.spv_kernel_map.argtypes = [vp, vp, sz, vp, vp, i64, i32, i32, vp, vp, vp, vp, i64, vp]
        L.spv_sparse_conv.argtypes = [vp, vp, sz, vp, i64, i32, vp, vp, i64, i32, i32, vp, vp, vp, i32, vp, vp, i64,
                                      i32, i32]
        L.spv_sparse_conv_sliced.argtypes = [vp, vp, sz, vp, i64, i32, vp, vp, i64, i32, i32, vp, i32, i32, vp, vp,
                                             vp, i32, vp, vp, i64, i32, i32]
        L.spv_linear.argtypes = [vp, vp, sz, vp, vp, i64, i32, vp, i32, i32, vp, vp, i32, vp, i32, vp, i32, i32]
        L.spv_kernel_map_nbr.argtypes = [vp, vp, sz, vp, vp, i64, vp]
        L.spv_sparse_conv_nbr.argtypes = [vp, vp, sz, vp, i64, i32, vp, vp, i32, i32, vp, vp, vp, i32, vp, vp, i64, i32,
                                          i32]
        L.spv_map_children.argtypes = [vp, vp, sz, vp, vp, i64, i64, vp, i64, vp]
        L.spv_sparse_conv_up.argtypes = [vp, vp, sz, vp, vp, i64, i32, vp, vp, i32, i32, vp, vp, vp, i32, vp, i64, i32,
                                         i32]
        L.spv_sparse_conv_dgrad.argtypes = [vp, vp, sz, vp, i64, i32, vp, vp, i64, i32, i32, vp, vp, vp, i64, i32, i32]
        L.spv_sparse_conv_dgrad_nbr.argtypes = [vp, vp, sz, vp, i32, vp, vp, vp, vp, i64, i32, i32]
        L.spv_sparse_conv_wgrad.argtypes = [vp, vp, sz, vp, i64, i32, vp, i64, i32, vp, vp, i64, i32, i32, vp, i32]
        L.spv_wgrad_workspace_bytes.argtypes = [i32, i32, i32]
        L.spv_wgrad_workspace_bytes.restype = sz
        L.spv_voxelize_backward.argtypes = [vp, vp, i64, i32, vp, vp, i64, vp, i32]
        L.spv_devoxelize_backward.argtypes = [vp, vp, sz, vp, vp, vp, i64, i32, vp, i64, i32]
        L.spv_devoxelize_backward_workspace_bytes.argtypes = [i64, i64]
        L.spv_epilogue_backward_workspace_bytes.argtypes = [i64, i32]
        L.spv_epilogue_backward_workspace_bytes.restype = sz
        L.spv_epilogue_backward.argtypes = [vp, vp, sz, vp, vp, vp, vp, i32, vp, i32, i64, i32, vp, vp, vp, vp, i32]
        L.spv_linear_backward_workspace_bytes.argtypes = [i32, i32]
        L.spv_linear_backward_workspace_bytes.restype = sz
        L.spv_linear_backward.argtypes = [vp, vp, sz, vp, i64, i32, vp, i32, vp, vp, vp, i32]
        L.spv_devoxelize_backward_workspace_bytes.restype = sz
        L.spv_devoxelize.argtypes = [vp, vp, sz, vp, vp, i64, i32, vp, vp, i64, f32, i32, vp, i32, vp, i32, vp, vp,
                                     vp, i32, vp, i32, vp, vp]
        L.spv_devoxelize_nbr.argtypes = [vp, vp, sz, vp, vp, i64, vp, vp, i32, vp, vp, i64, f32, i32, vp, i32, vp,
                                         i32, vp, vp, vp, i32, vp, i32]
        L.spv_block.argtypes = [vp, vp, sz, ct.POINTER(BlockParams), vp, vp, i64, vp, vp, vp]
        L.spv_lookup.argtypes = [vp, vp, sz, vp, vp, i64, vp, i64, vp]
        L.spv_voxel_lookup.argtypes = [vp, vp, sz, i64, vp, i64, vp]
        L.spv_sparse_conv_nbr_noalloc.argtypes = [vp, vp, i64, i32, vp, vp, i32, i32, vp, vp, vp, i32, vp, vp, i64,
                                                  i32, i32]
        L.spv_conv_kernel.argtypes = [i32, i32, i32, i32, i64, i64, i64, i32]
        L.spv_conv_kernel.restype = i32
        L.spv_block_conv_kernel.argtypes = [i64, i32, i32]
        L.spv_block_conv_kernel.restype = i32
        L.spv_status_check.argtypes = [vp, vp]
        L.spv_status_string.argtypes = [i32]
        L.spv_status_string.restype = ct.c_char_p
        L.spv_last_hip_error.argtypes = []
        for f in ("spv_voxelize", "spv_voxelize_onto", "spv_pack_weights", "spv_devoxelize_nbr", "spv_sparse_conv_nbr_packed",
                  "spv_sparse_conv_up_packed", "spv_linear_packed", "spv_kernel_map", "spv_sparse_conv", "spv_sparse_conv_sliced", "spv_linear",
                  "spv_kernel_map_nbr", "spv_sparse_conv_nbr", "spv_map_children", "spv_sparse_conv_up",
                  "spv_sparse_conv_dgrad", "spv_sparse_conv_dgrad_nbr", "spv_sparse_conv_wgrad",
                  "spv_voxelize_backward",
                  "spv_devoxelize_backward", "spv_epilogue_backward", "spv_linear_backward", "spv_devoxelize",
                  "spv_block", "spv_lookup", "spv_voxel_lookup",
                  "spv_sparse_conv_nbr_noalloc", "spv_status_check"):
            getattr(L, f).restype = ct.c_int
        _lib = L
    return _lib


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libspv takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libspv takes contiguous tensors")
    return ct.c_void_p(t.data_ptr())


def _stream():
    return ct.c_void_p(torch.cuda.current_stream().cuda_stream)


def _chk(st: int, what: str):
    if st != SPV_OK:
        raise SpvError(st, what)


class Workspace:
    """A caller-owned device workspace (a torch uint8 buffer, 256-byte aligned)."""

    def __init__(self, nbytes: int, device="cuda"):
        self.nbytes = int(nbytes)
        self.buf = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
        off = (-self.buf.data_ptr()) % 256
        self.ptr = ct.c_void_p(self.buf.data_ptr() + off)

    @classmethod
    def for_ops(cls, max_points: int, max_C: int, device="cuda"):
        return cls(lib().spv_workspace_bytes(max_points, max_C), device)

    @classmethod
    def for_wgrad(cls, K3: int, Cin: int, Cout: int, device="cuda"):
        return cls(lib().spv_wgrad_workspace_bytes(K3, Cin, Cout), device)

    @classmethod
    def for_devox_backward(cls, n: int, m: int, device="cuda"):
        return cls(lib().spv_devoxelize_backward_workspace_bytes(n, m), device)

    @classmethod
    def for_epilogue_backward(cls, m: int, C: int, device="cuda"):
        return cls(max(lib().spv_epilogue_backward_workspace_bytes(m, C), 256), device)

    @classmethod
    def for_linear_backward(cls, Cin: int, Cout: int, device="cuda"):
        return cls(lib().spv_linear_backward_workspace_bytes(Cin, Cout), device)

    @classmethod
    def for_block(cls, max_points: int, C: int, device="cuda"):
        return cls(lib().spv_block_workspace_bytes(max_points, C), device)


def spv_workspace_bytes(max_points: int, max_C: int) -> int:
    return lib().spv_workspace_bytes(max_points, max_C)


def spv_block_workspace_bytes(max_points: int, C: int) -> int:
    return lib().spv_block_workspace_bytes(max_points, C)


def spv_status_check(ws: Workspace) -> int:
    return lib().spv_status_check(ws.ptr, _stream())


@dataclass
class Voxelized:
    coords: torch.Tensor    # [cap, 4] int32
    vfeat: Optional[torch.Tensor]
    counts: torch.Tensor    # [cap] int32
    pt2vox: torch.Tensor    # [n] int32
    m_dev: torch.Tensor     # [1] int64 on device
    m: Optional[int]        # host copy when synchronized


def spv_voxelize(ws: Workspace, xyz: torch.Tensor, voxel_size: float, feat: Optional[torch.Tensor] = None,
                 batch: Optional[torch.Tensor] = None, sync: bool = True, out: Optional[Voxelized] = None
                 ) -> Voxelized:
    n = xyz.shape[0]
    dev = xyz.device
    C = feat.shape[1] if feat is not None else 0
    dt = _DT[feat.dtype] if feat is not None else SPV_F32
    cap = max(n, 1)
    if out is None:
        out = Voxelized(torch.empty((cap, 4), dtype=torch.int32, device=dev),
                        torch.empty((cap, C), dtype=feat.dtype, device=dev) if feat is not None else None,
                        torch.empty(cap, dtype=torch.int32, device=dev),
                        torch.empty(cap, dtype=torch.int32, device=dev),
                        torch.zeros(1, dtype=torch.int64, device=dev), None)
    m_host = ct.c_int64(0)
    st = lib().spv_voxelize(_stream(), ws.ptr, ws.nbytes, _ptr(xyz), _ptr(batch), n, ct.c_float(voxel_size),
                            _ptr(feat), C, dt, _ptr(out.coords), _ptr(out.vfeat), _ptr(out.counts), _ptr(out.pt2vox),
                            _ptr(out.m_dev), ct.byref(m_host) if sync else None)
    _chk(st, "spv_voxelize")
    out.m = m_host.value if sync else None
    return out


def spv_voxelize_onto(ws: Workspace, coords: torch.Tensor, xyz: torch.Tensor, voxel_size: float,
                      feat: Optional[torch.Tensor] = None, batch: Optional[torch.Tensor] = None,
                      m_dev: Optional[torch.Tensor] = None, out: Optional[Voxelized] = None) -> Voxelized:
    """Scatter-mean of the points onto the given voxel set (row j of the outputs is coords row j);
    points whose voxel is not in the set get pt2vox -1.  Returns a Voxelized whose coords are
    the given ones."""
    n = xyz.shape[0]
    m_cap = coords.shape[0]
    dev = xyz.device
    C = feat.shape[1] if feat is not None else 0
    dt = _DT[feat.dtype] if feat is not None else SPV_F32
    if out is None:
        out = Voxelized(coords, torch.empty((max(m_cap, 1), C), dtype=feat.dtype, device=dev)
                        if feat is not None else None,
                        torch.empty(max(m_cap, 1), dtype=torch.int32, device=dev),
                        torch.empty(max(n, 1), dtype=torch.int32, device=dev), m_dev,
                        m_cap if m_dev is None else None)
    st = lib().spv_voxelize_onto(_stream(), ws.ptr, ws.nbytes, _ptr(coords), _ptr(m_dev), m_cap, _ptr(xyz),
                                 _ptr(batch), n, ct.c_float(voxel_size), _ptr(feat), C, dt, _ptr(out.vfeat),
                                 _ptr(out.counts), _ptr(out.pt2vox))
    _chk(st, "spv_voxelize_onto")
    return out


@dataclass
class KernelMap:
    out_coords: Optional[torch.Tensor]
    m_out_dev: torch.Tensor
    off: torch.Tensor       # [K^3 + 1] int32
    pairs: torch.Tensor     # [pair_cap, 2] int32 (in, out)
    total: Optional[int]


def spv_kernel_map(ws: Workspace, in_coords: torch.Tensor, K: int = 3, stride: int = 1,
                   m_in_dev: Optional[torch.Tensor] = None, m_cap: Optional[int] = None,
                   pair_cap: Optional[int] = None, sync: bool = True) -> KernelMap:
    dev = in_coords.device
    m_cap = in_coords.shape[0] if m_cap is None else m_cap
    K3 = K ** 3
    if pair_cap is None:
        # K=2 s2: each input in one pair; K=3 s2: at most 2 outputs per odd axis
        pair_cap = max(1, m_cap if K == 2 else (8 * m_cap if stride == 2 else K3 * m_cap))
    oc = torch.empty((max(m_cap, 1), 4), dtype=torch.int32, device=dev) if stride == 2 else None
    km = KernelMap(oc, torch.zeros(1, dtype=torch.int64, device=dev), torch.empty(K3 + 1, dtype=torch.int32, device=dev),
                   torch.empty((pair_cap, 2), dtype=torch.int32, device=dev), None)
    tot = ct.c_int64(0)
    st = lib().spv_kernel_map(_stream(), ws.ptr, ws.nbytes, _ptr(in_coords), _ptr(m_in_dev), m_cap, K, stride,
                              _ptr(oc), _ptr(km.m_out_dev), _ptr(km.off), _ptr(km.pairs), pair_cap,
                              ct.byref(tot) if sync else None)
    if sync:
        km.total = tot.value
    _chk(st, "spv_kernel_map")
    return km


def spv_sparse_conv(ws: Workspace, x: torch.Tensor, off: torch.Tensor, pairs: torch.Tensor, W: torch.Tensor,
                    m_out_cap: int, m_out_dev: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                    shift: Optional[torch.Tensor] = None, relu: bool = False, transposed: bool = False,
                    out: Optional[torch.Tensor] = None) -> torch.Tensor:
    K3, Cin, Cout = W.shape
    if out is None:
        out = torch.empty((max(m_out_cap, 1), Cout), dtype=x.dtype, device=x.device)
    st = lib().spv_sparse_conv(_stream(), ws.ptr, ws.nbytes, _ptr(x), x.shape[0], Cin, _ptr(off), _ptr(pairs),
                               pairs.shape[0], K3, int(transposed), _ptr(W), _ptr(scale), _ptr(shift), int(relu),
                               _ptr(out), _ptr(m_out_dev), m_out_cap, Cout, _DT[x.dtype])
    _chk(st, "spv_sparse_conv")
    return out


def spv_sparse_conv_sliced(ws: Workspace, x: torch.Tensor, off: torch.Tensor, pairs: torch.Tensor,
                           W_full: torch.Tensor, Cin: int, Cout: int, m_out_cap: int,
                           m_out_dev: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                           shift: Optional[torch.Tensor] = None, relu: bool = False, transposed: bool = False,
                           out: Optional[torch.Tensor] = None, res: Optional[torch.Tensor] = None,
                           cin_offset: int = 0, in_rows: Optional[int] = None) -> torch.Tensor:
    """The conv with input channels cin_offset .. cin_offset+Cin and the first Cout output
    channels of the full weight W_full [K3][Cin_full][Cout_full] (and the first Cout entries of
    the full scale / shift); res: a residual input added before the activation."""
    K3, Cin_full, Cout_full = W_full.shape
    if x.shape[1] != Cin:
        raise ValueError(f"x has {x.shape[1]} channels, the slice takes {Cin}")
    if cin_offset < 0 or cin_offset + Cin > Cin_full:
        raise ValueError("input-channel slice outside the weight")
    if out is None:
        out = torch.empty((max(m_out_cap, 1), Cout), dtype=x.dtype, device=x.device)
    wp = ct.c_void_p(_ptr(W_full).value + cin_offset * Cout_full * W_full.element_size())
    st = lib().spv_sparse_conv_sliced(_stream(), ws.ptr, ws.nbytes, _ptr(x), x.shape[0] if in_rows is None else in_rows,
                                      Cin, _ptr(off), _ptr(pairs), pairs.shape[0], K3, int(transposed), wp,
                                      Cin_full, Cout_full, _ptr(scale),
                                      _ptr(shift), _ptr(res), int(relu), _ptr(out), _ptr(m_out_dev), m_out_cap, Cout,
                                      _DT[x.dtype])
    _chk(st, "spv_sparse_conv_sliced")
    return out


def spv_linear(ws: Workspace, x: torch.Tensor, W: torch.Tensor, Cout: Optional[int] = None,
               m_dev: Optional[torch.Tensor] = None, m_cap: Optional[int] = None,
               scale: Optional[torch.Tensor] = None, shift: Optional[torch.Tensor] = None, relu: bool = False,
               res: Optional[torch.Tensor] = None, res_after_act: bool = False, cin_offset: int = 0,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """act(scale * (x @ W[cin_offset : cin_offset + Cin, :Cout]) + shift [+ res]) [+ res]."""
    Cin = x.shape[1]
    Cin_full, Cout_full = W.shape
    Cout = Cout_full if Cout is None else Cout
    if cin_offset < 0 or cin_offset + Cin > Cin_full:
        raise ValueError("input-channel slice outside the weight")
    m_cap = x.shape[0] if m_cap is None else m_cap
    if out is None:
        out = torch.empty((max(m_cap, 1), Cout), dtype=x.dtype, device=x.device)
    wp = ct.c_void_p(_ptr(W).value + cin_offset * Cout_full * W.element_size())
    st = lib().spv_linear(_stream(), ws.ptr, ws.nbytes, _ptr(x), _ptr(m_dev), m_cap, Cin, wp, Cin_full - cin_offset,
                          Cout_full, _ptr(scale), _ptr(shift), int(relu), _ptr(res), int(res_after_act), _ptr(out),
                          Cout, _DT[x.dtype])
    _chk(st, "spv_linear")
    return out


def spv_pack_weights(W: torch.Tensor, Cin: Optional[int] = None, Cout: Optional[int] = None,
                     cin_offset: int = 0) -> Optional[torch.Tensor]:
    """The matrix-core fragments of W[:, cin_offset : cin_offset + Cin, :Cout] (W [K3][Cin_full][Cout_full],
    or [Cin_full][Cout_full] for a linear layer) as a uint8 device tensor, or None where no kernel
    reads that shape (and for float32)."""
    W3 = W if W.dim() == 3 else W.unsqueeze(0)
    K3, Cin_full, Cout_full = W3.shape
    Cin = Cin_full - cin_offset if Cin is None else Cin
    Cout = Cout_full if Cout is None else Cout
    if cin_offset < 0 or cin_offset + Cin > Cin_full:
        raise ValueError("input-channel slice outside the weight")
    nbytes = lib().spv_packed_weights_bytes(K3, Cin, Cout)
    if nbytes == 0 or W.dtype == torch.float32:
        return None
    out = torch.empty(nbytes, dtype=torch.uint8, device=W.device)
    wp = ct.c_void_p(_ptr(W3).value + cin_offset * Cout_full * W3.element_size())
    st = lib().spv_pack_weights(_stream(), wp, K3, Cin_full, Cout_full, Cin, Cout, _DT[W.dtype], _ptr(out), nbytes)
    _chk(st, "spv_pack_weights")
    return out


def spv_sparse_conv_nbr_packed(ws: Workspace, x: torch.Tensor, nbr: torch.Tensor, Wp: torch.Tensor, Cout: int,
                               m_out_cap: int, m_out_dev: Optional[torch.Tensor] = None,
                               scale: Optional[torch.Tensor] = None, shift: Optional[torch.Tensor] = None,
                               relu: bool = False, res: Optional[torch.Tensor] = None,
                               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """spv_sparse_conv_nbr with weights from spv_pack_weights (K3 = 27, x's width, Cout)."""
    if out is None:
        out = torch.empty((max(m_out_cap, 1), Cout), dtype=x.dtype, device=x.device)
    st = lib().spv_sparse_conv_nbr_packed(_stream(), ws.ptr, ws.nbytes, _ptr(x), x.shape[0], x.shape[1], _ptr(nbr),
                                          _ptr(Wp), _ptr(scale), _ptr(shift), _ptr(res), int(relu), _ptr(out),
                                          _ptr(m_out_dev), m_out_cap, Cout, _DT[x.dtype])
    _chk(st, "spv_sparse_conv_nbr_packed")
    return out


def spv_sparse_conv_up_packed(ws: Workspace, x: torch.Tensor, children: torch.Tensor, Wp: torch.Tensor, Cout: int,
                              out_rows: int, m_in_dev: Optional[torch.Tensor] = None,
                              scale: Optional[torch.Tensor] = None, shift: Optional[torch.Tensor] = None,
                              relu: bool = False, res: Optional[torch.Tensor] = None,
                              out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """spv_sparse_conv_up with weights from spv_pack_weights (K3 = 8, x's width, Cout)."""
    if out is None:
        out = torch.empty((max(out_rows, 1), Cout), dtype=x.dtype, device=x.device)
    st = lib().spv_sparse_conv_up_packed(_stream(), ws.ptr, ws.nbytes, _ptr(x), _ptr(m_in_dev), x.shape[0],
                                         x.shape[1], _ptr(children), _ptr(Wp), _ptr(scale), _ptr(shift), _ptr(res),
                                         int(relu), _ptr(out), out_rows, Cout, _DT[x.dtype])
    _chk(st, "spv_sparse_conv_up_packed")
    return out


def spv_linear_packed(ws: Workspace, x: torch.Tensor, Wp: torch.Tensor, Cout: int,
                      m_dev: Optional[torch.Tensor] = None, m_cap: Optional[int] = None,
                      scale: Optional[torch.Tensor] = None, shift: Optional[torch.Tensor] = None, relu: bool = False,
                      res: Optional[torch.Tensor] = None, res_after_act: bool = False,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """spv_linear with weights from spv_pack_weights (K3 = 1, x's width, Cout)."""
    m_cap = x.shape[0] if m_cap is None else m_cap
    if out is None:
        out = torch.empty((max(m_cap, 1), Cout), dtype=x.dtype, device=x.device)
    st = lib().spv_linear_packed(_stream(), ws.ptr, ws.nbytes, _ptr(x), _ptr(m_dev), m_cap, x.shape[1], _ptr(Wp),
                                 _ptr(scale), _ptr(shift), int(relu), _ptr(res), int(res_after_act), _ptr(out), Cout,
                                 _DT[x.dtype])
    _chk(st, "spv_linear_packed")
    return out


def spv_kernel_map_nbr(ws: Workspace, coords: torch.Tensor, m_dev: Optional[torch.Tensor] = None,
                       out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """nbr [m][27] int32: entry k of row j is i + 1 for the voxel i at c_j + delta_k, else 0."""
    m_cap = coords.shape[0]
    if out is None:
        out = torch.empty((max(m_cap, 1), 27), dtype=torch.int32, device=coords.device)
    st = lib().spv_kernel_map_nbr(_stream(), ws.ptr, ws.nbytes, _ptr(coords), _ptr(m_dev), m_cap, _ptr(out))
    _chk(st, "spv_kernel_map_nbr")
    return out


def spv_sparse_conv_nbr(ws: Workspace, x: torch.Tensor, nbr: torch.Tensor, W_full: torch.Tensor, Cout: int,
                        m_out_cap: int, m_out_dev: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                        shift: Optional[torch.Tensor] = None, relu: bool = False,
                        res: Optional[torch.Tensor] = None, cin_offset: int = 0,
                        out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The sliced conv (input channels cin_offset .. + x's width, first Cout outputs) on a
    neighbour table from spv_kernel_map_nbr."""
    K3, Cin_full, Cout_full = W_full.shape
    Cin = x.shape[1]
    if cin_offset < 0 or cin_offset + Cin > Cin_full:
        raise ValueError("input-channel slice outside the weight")
    if out is None:
        out = torch.empty((max(m_out_cap, 1), Cout), dtype=x.dtype, device=x.device)
    wp = ct.c_void_p(_ptr(W_full).value + cin_offset * Cout_full * W_full.element_size())
    st = lib().spv_sparse_conv_nbr(_stream(), ws.ptr, ws.nbytes, _ptr(x), x.shape[0], Cin, _ptr(nbr), wp, Cin_full,
                                   Cout_full, _ptr(scale), _ptr(shift), _ptr(res), int(relu), _ptr(out),
                                   _ptr(m_out_dev), m_out_cap, Cout, _DT[x.dtype])
    _chk(st, "spv_sparse_conv_nbr")
    return out


def spv_sparse_conv_nbr_noalloc(x: torch.Tensor, nbr: torch.Tensor, W_full: torch.Tensor, Cout: int,
                                m_out_cap: int, m_out_dev: Optional[torch.Tensor] = None,
                                scale: Optional[torch.Tensor] = None, shift: Optional[torch.Tensor] = None,
                                relu: bool = False, res: Optional[torch.Tensor] = None, cin_offset: int = 0,
                                out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """spv_sparse_conv_nbr with no workspace (the library's device-resident scratch holds the
    packed weights); out must be given by callers that cannot allocate."""
    K3, Cin_full, Cout_full = W_full.shape
    Cin = x.shape[1]
    if cin_offset < 0 or cin_offset + Cin > Cin_full:
        raise ValueError("input-channel slice outside the weight")
    if out is None:
        out = torch.empty((max(m_out_cap, 1), Cout), dtype=x.dtype, device=x.device)
    wp = ct.c_void_p(_ptr(W_full).value + cin_offset * Cout_full * W_full.element_size())
    st = lib().spv_sparse_conv_nbr_noalloc(_stream(), _ptr(x), x.shape[0], Cin, _ptr(nbr), wp, Cin_full, Cout_full,
                                           _ptr(scale), _ptr(shift), _ptr(res), int(relu), _ptr(out),
                                           _ptr(m_out_dev), m_out_cap, Cout, _DT[x.dtype])
    _chk(st, "spv_sparse_conv_nbr_noalloc")
    return out


def spv_map_children(ws: Workspace, off: torch.Tensor, pairs: torch.Tensor, fine_rows: int, m_coarse: int,
                     m_coarse_dev: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """children [m_coarse][8] int32 of a K=2 stride-2 map: fine row + 1 per offset, 0 = none."""
    if out is None:
        out = torch.empty((max(m_coarse, 1), 8), dtype=torch.int32, device=off.device)
    st = lib().spv_map_children(_stream(), ws.ptr, ws.nbytes, _ptr(off), _ptr(pairs), pairs.shape[0], fine_rows,
                                _ptr(m_coarse_dev), m_coarse, _ptr(out))
    _chk(st, "spv_map_children")
    return out


def spv_sparse_conv_up(ws: Workspace, x: torch.Tensor, children: torch.Tensor, W_full: torch.Tensor, Cout: int,
                       out_rows: int, m_in_dev: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                       shift: Optional[torch.Tensor] = None, relu: bool = False, res: Optional[torch.Tensor] = None,
                       cin_offset: int = 0, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The transposed k=2 s=2 conv of the coarse rows x onto the fine rows, from the child table."""
    K3, Cin_full, Cout_full = W_full.shape
    Cin = x.shape[1]
    if K3 != 8 or cin_offset < 0 or cin_offset + Cin > Cin_full:
        raise ValueError("W_full must be [8][Cin_full][Cout_full] holding the input-channel slice")
    if out is None:
        out = torch.empty((max(out_rows, 1), Cout), dtype=x.dtype, device=x.device)
    wp = ct.c_void_p(_ptr(W_full).value + cin_offset * Cout_full * W_full.element_size())
    st = lib().spv_sparse_conv_up(_stream(), ws.ptr, ws.nbytes, _ptr(x), _ptr(m_in_dev), x.shape[0], Cin,
                                  _ptr(children), wp, Cin_full, Cout_full, _ptr(scale), _ptr(shift), _ptr(res),
                                  int(relu), _ptr(out), out_rows, Cout, _DT[x.dtype])
    _chk(st, "spv_sparse_conv_up")
    return out


def spv_sparse_conv_dgrad(ws: Workspace, dy: torch.Tensor, off: torch.Tensor, pairs: torch.Tensor, W: torch.Tensor,
                          m_in_cap: int, m_in_dev: Optional[torch.Tensor] = None, transposed: bool = False,
                          out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """dx[i] = sum over the pairs (i, j, k) of dy[j] @ W[k]^T (W: the forward weights [K3][Cin][Cout])."""
    K3, Cin, Cout = W.shape
    if out is None:
        out = torch.empty((max(m_in_cap, 1), Cin), dtype=dy.dtype, device=dy.device)
    st = lib().spv_sparse_conv_dgrad(_stream(), ws.ptr, ws.nbytes, _ptr(dy), dy.shape[0], Cout, _ptr(off), _ptr(pairs),
                                     pairs.shape[0], K3, int(transposed), _ptr(W), _ptr(out), _ptr(m_in_dev), m_in_cap,
                                     Cin, _DT[dy.dtype])
    _chk(st, "spv_sparse_conv_dgrad")
    return out


def spv_sparse_conv_wgrad(ws: Workspace, x: torch.Tensor, dy: torch.Tensor, off: torch.Tensor, pairs: torch.Tensor,
                          K3: int, transposed: bool = False, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """dW[k] = sum over the pairs (i, j) of offset k of x[i]^T dy[j], float32 [K3][Cin][Cout]."""
    Cin, Cout = x.shape[1], dy.shape[1]
    if out is None:
        out = torch.empty((K3, Cin, Cout), dtype=torch.float32, device=x.device)
    st = lib().spv_sparse_conv_wgrad(_stream(), ws.ptr, ws.nbytes, _ptr(x), x.shape[0], Cin, _ptr(dy), dy.shape[0],
                                     Cout, _ptr(off), _ptr(pairs), pairs.shape[0], K3, int(transposed), _ptr(out),
                                     _DT[x.dtype])
    _chk(st, "spv_sparse_conv_wgrad")
    return out


def spv_sparse_conv_dgrad_nbr(ws: Workspace, dy: torch.Tensor, nbr: torch.Tensor, W: torch.Tensor,
                              m_dev: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Input gradient of the 3x3x3 submanifold conv with weights W [27][Cin][Cout] on the neighbour table."""
    m_cap, Cout = dy.shape
    Cin = W.shape[1]
    if out is None:
        out = torch.empty((max(m_cap, 1), Cin), dtype=dy.dtype, device=dy.device)
    st = lib().spv_sparse_conv_dgrad_nbr(_stream(), ws.ptr, ws.nbytes, _ptr(dy), Cout, _ptr(nbr), _ptr(W), _ptr(out),
                                         _ptr(m_dev), m_cap, Cin, _DT[dy.dtype])
    _chk(st, "spv_sparse_conv_dgrad_nbr")
    return out


def spv_voxelize_backward(dvfeat: torch.Tensor, counts: torch.Tensor, pt2vox: torch.Tensor, m: int,
                          out: Optional[torch.Tensor] = None) -> torch.Tensor:
    n, C = pt2vox.shape[0], dvfeat.shape[1]
    if out is None:
        out = torch.empty((max(n, 1), C), dtype=dvfeat.dtype, device=dvfeat.device)
    st = lib().spv_voxelize_backward(_stream(), _ptr(dvfeat), m, C, _ptr(counts), _ptr(pt2vox), n, _ptr(out),
                                     _DT[dvfeat.dtype])
    _chk(st, "spv_voxelize_backward")
    return out


def spv_devoxelize_backward(ws: Workspace, corner_idx: torch.Tensor, corner_w: torch.Tensor, dout: torch.Tensor,
                            m: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    n, C = dout.shape
    if out is None:
        out = torch.empty((max(m, 1), C), dtype=torch.float32, device=dout.device)
    st = lib().spv_devoxelize_backward(_stream(), ws.ptr, ws.nbytes, _ptr(corner_idx), _ptr(corner_w), _ptr(dout), n,
                                       C, _ptr(out), m, _DT[dout.dtype])
    _chk(st, "spv_devoxelize_backward")
    return out


def spv_epilogue_backward(ws: Workspace, dy: torch.Tensor, a: torch.Tensor, scale: Optional[torch.Tensor] = None,
                          shift: Optional[torch.Tensor] = None, relu: bool = False,
                          res: Optional[torch.Tensor] = None, res_after_act: bool = False):
    """(da, dres, dscale, dshift) of the epilogue act(scale * a + shift (+ res)) (+ res)."""
    m, C = dy.shape
    d = dy.device
    da = torch.empty((max(m, 1), C), dtype=dy.dtype, device=d)
    dres = torch.empty((max(m, 1), C), dtype=dy.dtype, device=d) if res is not None else None
    dscale = torch.empty(C, dtype=torch.float32, device=d)
    dshift = torch.empty(C, dtype=torch.float32, device=d)
    st = lib().spv_epilogue_backward(_stream(), ws.ptr, ws.nbytes, _ptr(dy), _ptr(a), _ptr(scale), _ptr(shift),
                                     int(relu), _ptr(res), int(res_after_act), m, C, _ptr(da), _ptr(dres),
                                     _ptr(dscale), _ptr(dshift), _DT[dy.dtype])
    _chk(st, "spv_epilogue_backward")
    return da, dres, dscale, dshift


def spv_linear_backward(ws: Workspace, x: torch.Tensor, W: torch.Tensor, da: torch.Tensor):
    """(dx, dW) of the product x @ W, given its gradient da."""
    m, Cin = x.shape
    Cout = W.shape[1]
    dx = torch.empty((max(m, 1), Cin), dtype=x.dtype, device=x.device)
    dW = torch.empty((Cin, Cout), dtype=torch.float32, device=x.device)
    st = lib().spv_linear_backward(_stream(), ws.ptr, ws.nbytes, _ptr(x), m, Cin, _ptr(W), Cout, _ptr(da), _ptr(dx),
                                   _ptr(dW), _DT[x.dtype])
    _chk(st, "spv_linear_backward")
    return dx, dW


def spv_devoxelize(ws: Workspace, grid_coords: torch.Tensor, vfeat: torch.Tensor, xyz: torch.Tensor,
                   voxel_size: float, stride_log2: int = 0, mode: int = SPV_DEVOX_CENTER,
                   batch: Optional[torch.Tensor] = None, m_dev: Optional[torch.Tensor] = None,
                   m_cap: Optional[int] = None, pfeat: Optional[torch.Tensor] = None, Wp: Optional[torch.Tensor] = None,
                   scale_p: Optional[torch.Tensor] = None, shift_p: Optional[torch.Tensor] = None,
                   relu_p: bool = False, want_corners: bool = False, out: Optional[torch.Tensor] = None):
    n = xyz.shape[0]
    C = vfeat.shape[1]
    m_cap = grid_coords.shape[0] if m_cap is None else m_cap
    Cp = pfeat.shape[1] if pfeat is not None else 0
    if out is None:
        out = torch.empty((max(n, 1), C), dtype=vfeat.dtype, device=xyz.device)
    ci = torch.empty((max(n, 1), 8), dtype=torch.int32, device=xyz.device) if want_corners else None
    cw = torch.empty((max(n, 1), 8), dtype=torch.float32, device=xyz.device) if want_corners else None
    st = lib().spv_devoxelize(_stream(), ws.ptr, ws.nbytes, _ptr(grid_coords), _ptr(m_dev), m_cap, stride_log2,
                              _ptr(xyz), _ptr(batch), n, ct.c_float(voxel_size), mode, _ptr(vfeat), C, _ptr(pfeat),
                              Cp, _ptr(Wp), _ptr(scale_p), _ptr(shift_p), int(relu_p), _ptr(out), _DT[vfeat.dtype],
                              _ptr(ci), _ptr(cw))
    _chk(st, "spv_devoxelize")
    return (out, ci, cw) if want_corners else out


def spv_devoxelize_nbr(ws: Workspace, grid_coords: torch.Tensor, vfeat: torch.Tensor, nbr: torch.Tensor,
                       pt2vox: torch.Tensor, xyz: torch.Tensor, voxel_size: float, stride_log2: int = 0,
                       mode: int = SPV_DEVOX_CENTER, batch: Optional[torch.Tensor] = None,
                       m_dev: Optional[torch.Tensor] = None, m_cap: Optional[int] = None,
                       pfeat: Optional[torch.Tensor] = None, Wp: Optional[torch.Tensor] = None,
                       scale_p: Optional[torch.Tensor] = None, shift_p: Optional[torch.Tensor] = None,
                       relu_p: bool = False, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """spv_devoxelize on the points' own voxelization at that stride: corners from the neighbour table."""
    n = xyz.shape[0]
    C = vfeat.shape[1]
    m_cap = grid_coords.shape[0] if m_cap is None else m_cap
    Cp = pfeat.shape[1] if pfeat is not None else 0
    if out is None:
        out = torch.empty((max(n, 1), C), dtype=vfeat.dtype, device=xyz.device)
    st = lib().spv_devoxelize_nbr(_stream(), ws.ptr, ws.nbytes, _ptr(grid_coords), _ptr(m_dev), m_cap, _ptr(nbr),
                                  _ptr(pt2vox), stride_log2, _ptr(xyz), _ptr(batch), n, ct.c_float(voxel_size), mode,
                                  _ptr(vfeat), C, _ptr(pfeat), Cp, _ptr(Wp), _ptr(scale_p), _ptr(shift_p), int(relu_p),
                                  _ptr(out), _DT[vfeat.dtype])
    _chk(st, "spv_devoxelize_nbr")
    return out


def make_block_params(C: int, dtype: torch.dtype, voxel_size: float, convs: Sequence, Wp: torch.Tensor,
                      scale_p=None, shift_p=None, relu_p: bool = True, mode: int = SPV_DEVOX_CENTER,
                      residual: bool = False) -> BlockParams:
    """convs: list of (W [27,C,C], scale|None, shift|None, relu) device tensors.

    The struct holds raw device pointers; it also keeps references to every
    tensor it points into, so they stay allocated as long as the struct lives."""
    def ptr(t):
        return None if t is None else _ptr(t).value
    p = BlockParams()
    p.C, p.dtype, p.voxel_size, p.n_convs = C, _DT[dtype], voxel_size, len(convs)
    keep = [Wp, scale_p, shift_p]
    for l, (W, sc, sh, r) in enumerate(convs):
        p.W[l] = ptr(W)
        p.scale[l] = ptr(sc)
        p.shift[l] = ptr(sh)
        p.relu[l] = int(r)
        keep += [W, sc, sh]
    p.Wp = ptr(Wp)
    p.scale_p = ptr(scale_p)
    p.shift_p = ptr(shift_p)
    p.relu_p = int(relu_p)
    p.devox_mode = mode
    p.residual = int(residual)
    p._keep = keep
    return p


def spv_block(ws: Workspace, params: BlockParams, xyz: torch.Tensor, feat: torch.Tensor,
              batch: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None, sync: bool = False):
    n, C = feat.shape
    if out is None:
        out = torch.empty((max(n, 1), C), dtype=feat.dtype, device=feat.device)
    m = ct.c_int64(0)
    st = lib().spv_block(_stream(), ws.ptr, ws.nbytes, ct.byref(params), _ptr(xyz), _ptr(batch), n, _ptr(feat),
                         _ptr(out), ct.byref(m) if sync else None)
    _chk(st, "spv_block")
    return (out, m.value) if sync else out


def spv_lookup(ws: Workspace, table_coords: torch.Tensor, qcoords: torch.Tensor,
               m_dev: Optional[torch.Tensor] = None) -> torch.Tensor:
    q = qcoords.shape[0]
    idx = torch.empty(max(q, 1), dtype=torch.int32, device=qcoords.device)
    st = lib().spv_lookup(_stream(), ws.ptr, ws.nbytes, _ptr(table_coords), _ptr(m_dev), table_coords.shape[0],
                          _ptr(qcoords), q, _ptr(idx))
    _chk(st, "spv_lookup")
    return idx[:q]


def spv_voxel_lookup(ws: Workspace, n: int, qcoords: torch.Tensor) -> torch.Tensor:
    """Lookups in the table the last spv_voxelize(ws, ..., n points) built."""
    q = qcoords.shape[0]
    idx = torch.empty(max(q, 1), dtype=torch.int32, device=qcoords.device)
    st = lib().spv_voxel_lookup(_stream(), ws.ptr, ws.nbytes, n, _ptr(qcoords), q, _ptr(idx))
    _chk(st, "spv_voxel_lookup")
    return idx[:q]


def spv_conv_kernel(K3: int, Cin: int, Cout: int, dtype: torch.dtype, in_rows: int, m_out_cap: int,
                    pair_cap: int, transposed: bool = False) -> int:
    """Host query: 0 neighbour-table MFMA, 1 tile MFMA, 2 vector ALU, -1 rejected."""
    return lib().spv_conv_kernel(K3, Cin, Cout, _DT[dtype], in_rows, m_out_cap, pair_cap, int(transposed))


def spv_block_conv_kernel(n: int, C: int, dtype: torch.dtype) -> int:
    return lib().spv_block_conv_kernel(n, C, _DT[dtype])
