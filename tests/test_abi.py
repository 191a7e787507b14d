"""The C-ABI library loads and exports every symbol include/spv.h declares (no GPU calls)."""
import ctypes as ct
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spv.h")
LIB = os.path.join(ROOT, "paper_2007_16100_amd", "libspv.so")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_][a-z0-9_]*\s*\**\s+(spv_[a-z_0-9]+)\s*\(", src, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for required in ("spv_voxelize", "spv_kernel_map", "spv_sparse_conv", "spv_devoxelize", "spv_block"):
        assert required in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libspv.so not built")
def test_library_exports_every_declared_symbol():
    lib = ct.CDLL(LIB)
    missing = [f for f in declared_functions() if not hasattr(lib, f)]
    assert not missing, missing
    from paper_2007_16100_amd import spv
    assert sorted(spv.EXPORTS) == declared_functions()


@pytest.mark.skipif(not os.path.exists(LIB), reason="libspv.so not built")
def test_host_side_validation_without_gpu():
    """Host-detectable errors return before any HIP call, so they are testable on a CPU-only host."""
    from paper_2007_16100_amd import spv
    L = spv.lib()
    ws = ct.c_void_p(256)  # never dereferenced: validation fails first
    # non-positive / NaN voxel size
    for v in (0.0, -1.0, float("nan")):
        st = L.spv_voxelize(None, ws, 1 << 30, ct.c_void_p(16), None, 4, ct.c_float(v), None, 0, 0,
                            ct.c_void_p(16), None, ct.c_void_p(16), ct.c_void_p(16), None, None)
        assert st == spv.SPV_ERR_INVALID_ARG
    # workspace too small -> capacity
    st = L.spv_voxelize(None, ws, 16, ct.c_void_p(16), None, 4, ct.c_float(0.1), None, 0, 0, ct.c_void_p(16), None,
                        ct.c_void_p(16), ct.c_void_p(16), None, None)
    assert st == spv.SPV_ERR_CAPACITY
    # scatter-mean onto a given set: bad voxel size, a missing coordinate list, negative
    # capacity, features without an output, a workspace too small
    P = ct.c_void_p(16)
    for v in (0.0, float("inf")):
        assert L.spv_voxelize_onto(None, ws, 1 << 30, P, None, 4, P, None, 4, ct.c_float(v), None, 0, 0, None, P,
                                   P) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_voxelize_onto(None, ws, 1 << 30, None, None, 4, P, None, 4, ct.c_float(0.1), None, 0, 0, None, P,
                               P) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_voxelize_onto(None, ws, 1 << 30, P, None, -1, P, None, 4, ct.c_float(0.1), None, 0, 0, None, P,
                               P) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_voxelize_onto(None, ws, 1 << 30, P, None, 4, P, None, 4, ct.c_float(0.1), P, 8, 1, None, P,
                               P) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_voxelize_onto(None, ws, 16, P, None, 4, P, None, 4, ct.c_float(0.1), None, 0, 0, None, P,
                               P) == spv.SPV_ERR_CAPACITY
    # pre-packed weights: sizes, and the host-side rejections
    frag = 64 * 16
    assert L.spv_packed_weights_bytes(27, 96, 96) == 27 * 3 * 6 * frag
    assert L.spv_packed_weights_bytes(1, 96, 19) == 3 * 2 * frag
    assert L.spv_packed_weights_bytes(8, 256, 256) == 8 * 8 * 16 * frag
    assert L.spv_packed_weights_bytes(27, 160, 96) == 0 and L.spv_packed_weights_bytes(27, 96, 272) == 0
    big = ct.c_size_t(1 << 30)
    assert L.spv_pack_weights(None, None, 27, 96, 96, 96, 96, 1, P, big) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_pack_weights(None, P, 27, 64, 96, 96, 96, 1, P, big) == spv.SPV_ERR_INVALID_ARG  # slice too wide
    assert L.spv_pack_weights(None, P, 27, 96, 96, 96, 96, 0, P, big) == spv.SPV_ERR_UNSUPPORTED  # float32
    assert L.spv_pack_weights(None, P, 27, 160, 96, 160, 96, 1, P, big) == spv.SPV_ERR_UNSUPPORTED
    assert L.spv_pack_weights(None, P, 27, 96, 96, 96, 96, 1, P, 1000) == spv.SPV_ERR_CAPACITY
    assert L.spv_linear_packed(None, ws, 1 << 30, P, None, 4, 96, P, None, None, 0, None, 0, P, 96,
                               0) == spv.SPV_ERR_UNSUPPORTED  # float32: no matrix-core linear
    assert L.spv_sparse_conv_nbr_packed(None, ws, 1 << 30, P, 4, 96, P, None, None, None, None, 0, P, None, 4, 96,
                                        1) == spv.SPV_ERR_INVALID_ARG  # no packed weights
    # unsupported kernel-map geometry
    st = L.spv_kernel_map(None, ws, 1 << 30, ct.c_void_p(16), None, 4, 2, 1, ct.c_void_p(16), None, ct.c_void_p(16),
                          ct.c_void_p(16), 100, None)
    assert st == spv.SPV_ERR_UNSUPPORTED
    # unsupported conv K3, bad dtype
    st = L.spv_sparse_conv(None, ws, 1 << 30, ct.c_void_p(16), 4, 8, ct.c_void_p(16), ct.c_void_p(16), 4, 9, 0,
                           ct.c_void_p(16), None, None, 0, ct.c_void_p(16), None, 4, 16, 1)
    assert st == spv.SPV_ERR_UNSUPPORTED
    st = L.spv_sparse_conv(None, ws, 1 << 30, ct.c_void_p(16), 4, 8, ct.c_void_p(16), ct.c_void_p(16), 4, 27, 0,
                           ct.c_void_p(16), None, None, 0, ct.c_void_p(16), None, 4, 16, 7)
    assert st == spv.SPV_ERR_INVALID_ARG
    # a weight slice wider than the stored tensor; a residual that is the output
    st = L.spv_sparse_conv_sliced(None, ws, 1 << 30, ct.c_void_p(16), 4, 64, ct.c_void_p(16), ct.c_void_p(16), 4, 27,
                                  0, ct.c_void_p(16), 32, 64, None, None, None, 0, ct.c_void_p(16), None, 4, 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    st = L.spv_sparse_conv_sliced(None, ws, 1 << 30, ct.c_void_p(16), 4, 32, ct.c_void_p(16), ct.c_void_p(16), 4, 27,
                                  0, ct.c_void_p(16), 32, 32, None, None, None, 0, ct.c_void_p(16), None, 4, 48, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    st = L.spv_sparse_conv_sliced(None, ws, 1 << 30, ct.c_void_p(16), 4, 32, ct.c_void_p(16), ct.c_void_p(16), 4, 27,
                                  0, ct.c_void_p(16), 32, 32, None, None, ct.c_void_p(32), 0, ct.c_void_p(32), None, 4,
                                  32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    # linear: slice wider than W, misaligned rows, output aliasing the input
    st = L.spv_linear(None, ws, 1 << 30, ct.c_void_p(16), None, 4, 64, ct.c_void_p(16), 32, 32, None, None, 0, None,
                      0, ct.c_void_p(48), 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    st = L.spv_linear(None, ws, 1 << 30, ct.c_void_p(18), None, 4, 32, ct.c_void_p(16), 32, 32, None, None, 0, None,
                      0, ct.c_void_p(48), 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    st = L.spv_linear(None, ws, 1 << 30, ct.c_void_p(16), None, 4, 32, ct.c_void_p(16), 32, 32, None, None, 0, None,
                      0, ct.c_void_p(16), 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    st = L.spv_linear(None, ws, 16, ct.c_void_p(16), None, 4, 32, ct.c_void_p(16), 32, 32, None, None, 0, None,
                      0, ct.c_void_p(48), 32, 1)
    assert st == spv.SPV_ERR_CAPACITY
    # neighbour-table conv: a width the kernel does not take; a missing table
    st = L.spv_sparse_conv_nbr(None, ws, 1 << 30, ct.c_void_p(16), 4, 48, ct.c_void_p(16), ct.c_void_p(16), 48, 48,
                               None, None, None, 0, ct.c_void_p(32), None, 4, 48, 1)
    assert st == spv.SPV_ERR_UNSUPPORTED
    st = L.spv_sparse_conv_nbr(None, ws, 1 << 30, ct.c_void_p(16), 4, 32, None, ct.c_void_p(16), 32, 32,
                               None, None, None, 0, ct.c_void_p(32), None, 4, 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    # child-table upsampling: f32 is not taken; children misaligned
    st = L.spv_sparse_conv_up(None, ws, 1 << 30, ct.c_void_p(16), None, 4, 32, ct.c_void_p(16), ct.c_void_p(16), 32,
                              32, None, None, None, 0, ct.c_void_p(32), 8, 32, 0)
    assert st == spv.SPV_ERR_UNSUPPORTED
    st = L.spv_map_children(None, ws, 1 << 30, ct.c_void_p(16), ct.c_void_p(16), 4, 8, None, 4, ct.c_void_p(20))
    assert st == spv.SPV_ERR_INVALID_ARG
    # weight gradient: Cin * Cout too large; workspace too small
    st = L.spv_sparse_conv_wgrad(None, ws, 1 << 30, ct.c_void_p(16), 4, 512, ct.c_void_p(16), 4, 256,
                                 ct.c_void_p(16), ct.c_void_p(16), 4, 27, 0, ct.c_void_p(16), 1)
    assert st == spv.SPV_ERR_UNSUPPORTED
    st = L.spv_sparse_conv_wgrad(None, ws, 1024, ct.c_void_p(16), 4, 32, ct.c_void_p(16), 4, 32,
                                 ct.c_void_p(16), ct.c_void_p(16), 4, 27, 0, ct.c_void_p(16), 1)
    assert st == spv.SPV_ERR_CAPACITY
    assert L.spv_wgrad_workspace_bytes(27, 32, 32) >= 27 * 32 * 32 * 4
    assert L.spv_wgrad_workspace_bytes(27, 0, 32) == 0
    # backward of the scatter-mean / devox: negative sizes
    assert L.spv_voxelize_backward(None, None, -1, 4, None, None, 0, None, 1) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_devoxelize_backward(None, ws, 1 << 30, None, None, None, 4, 8, None, 4, 1) == spv.SPV_ERR_INVALID_ARG
    # devox backward: no workspace; a small one; sizes past the int32 entry numbers
    dvb = (ct.c_void_p(16), ct.c_void_p(16), ct.c_void_p(16), 4, 8, ct.c_void_p(64), 4, 1)
    assert L.spv_devoxelize_backward(None, None, 1 << 30, *dvb) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_devoxelize_backward(None, ws, 64, *dvb) == spv.SPV_ERR_CAPACITY
    # the output aliasing the gradient
    assert L.spv_devoxelize_backward(None, ws, 1 << 40, ct.c_void_p(16), ct.c_void_p(16), ct.c_void_p(48), 4, 8,
                                     ct.c_void_p(48), 4, 1) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_devoxelize_backward(None, ws, 1 << 40, ct.c_void_p(16), ct.c_void_p(16), ct.c_void_p(16), 1 << 28, 8,
                                     ct.c_void_p(64), 4, 1) == spv.SPV_ERR_INVALID_ARG
    need = L.spv_devoxelize_backward_workspace_bytes(1000, 700)
    assert need >= 1000 * 8 * 20 + 700 * 8
    assert L.spv_devoxelize_backward_workspace_bytes(-1, 700) == 0
    # epilogue backward: sums without a workspace; a small one; negative sizes
    epi = (ct.c_void_p(16), ct.c_void_p(16), None, None, 1, None, 0, 4, 8, ct.c_void_p(16), None, ct.c_void_p(16),
           None, 1)
    assert L.spv_epilogue_backward(None, None, 0, *epi) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_epilogue_backward(None, ws, 8, *epi) == spv.SPV_ERR_CAPACITY
    assert L.spv_epilogue_backward(None, ws, 1 << 30, ct.c_void_p(16), ct.c_void_p(16), None, None, 1, None, 0, -1, 8,
                                   None, None, None, None, 1) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_epilogue_backward_workspace_bytes(1000, 96) >= 4 * 2 * 96 * 8
    # linear backward: misaligned rows, output aliasing the gradient, too wide for dW, small workspace
    lin = lambda ws_, nb, x_, da_, din_, cin=32, cout=32: L.spv_linear_backward(
        None, ws_, nb, x_, 4, cin, ct.c_void_p(16), cout, da_, din_, ct.c_void_p(16), 1)
    assert lin(ws, 1 << 30, ct.c_void_p(18), ct.c_void_p(16), ct.c_void_p(32)) == spv.SPV_ERR_INVALID_ARG
    assert lin(ws, 1 << 30, ct.c_void_p(16), ct.c_void_p(32), ct.c_void_p(32)) == spv.SPV_ERR_INVALID_ARG
    assert lin(ws, 1 << 30, ct.c_void_p(16), ct.c_void_p(32), ct.c_void_p(48), 512, 256) == spv.SPV_ERR_UNSUPPORTED
    assert lin(ws, 1024, ct.c_void_p(16), ct.c_void_p(32), ct.c_void_p(48)) == spv.SPV_ERR_CAPACITY
    assert L.spv_linear_backward_workspace_bytes(32, 32) >= 27 * 32 * 32 * 4
    # input gradient on the neighbour table: a width the kernel does not take; dx aliasing dy
    st = L.spv_sparse_conv_dgrad_nbr(None, ws, 1 << 30, ct.c_void_p(16), 48, ct.c_void_p(16), ct.c_void_p(16),
                                     ct.c_void_p(32), None, 4, 48, 1)
    assert st == spv.SPV_ERR_UNSUPPORTED
    st = L.spv_sparse_conv_dgrad_nbr(None, ws, 1 << 30, ct.c_void_p(16), 32, ct.c_void_p(16), ct.c_void_p(16),
                                     ct.c_void_p(16), None, 4, 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    # misaligned feature pointer
    st = L.spv_sparse_conv(None, ws, 1 << 30, ct.c_void_p(18), 4, 8, ct.c_void_p(16), ct.c_void_p(16), 4, 27, 0,
                           ct.c_void_p(16), None, None, 0, ct.c_void_p(16), None, 4, 16, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
    # devox: bad mode, stride out of range
    st = L.spv_devoxelize(None, ws, 1 << 30, ct.c_void_p(16), None, 4, 0, ct.c_void_p(16), None, 4, ct.c_float(0.1),
                          7, ct.c_void_p(16), 16, None, 0, None, None, None, 0, ct.c_void_p(16), 1, None, None)
    assert st == spv.SPV_ERR_INVALID_ARG
    st = L.spv_devoxelize(None, ws, 1 << 30, ct.c_void_p(16), None, 4, 16, ct.c_void_p(16), None, 4,
                          ct.c_float(0.1), 0, ct.c_void_p(16), 16, None, 0, None, None, None, 0, ct.c_void_p(16), 1,
                          None, None)
    assert st == spv.SPV_ERR_INVALID_ARG
    # block: n_convs out of range
    p = spv.BlockParams()
    p.C, p.dtype, p.voxel_size, p.n_convs = 16, 1, 0.1, 3
    st = L.spv_block(None, ws, 1 << 30, ct.byref(p), ct.c_void_p(16), None, 4, ct.c_void_p(16), ct.c_void_p(16), None)
    assert st == spv.SPV_ERR_INVALID_ARG
    assert spv.lib().spv_status_string(3) == b"coordinate out of range"
    # workspace sizing is monotone and covers the block
    assert spv.spv_workspace_bytes(1000, 96) < spv.spv_workspace_bytes(100000, 96)
    assert spv.spv_block_workspace_bytes(121180, 96) > 100 * 1024 * 1024


@pytest.mark.skipif(not os.path.exists(LIB), reason="libspv.so not built")
def test_conv_kernel_choice_at_the_32bit_offset_bound():
    """The conv's kernel is chosen once on the host: the neighbour-table kernel
    only while its 32-bit buffer offsets cover the input rows (n * C * 2 bytes),
    else the pairs path, whose plan builds the tile bounds it reads."""
    import torch
    from paper_2007_16100_amd import spv
    bound = 0xFFFFE000
    for C in (96, 256):
        n_max = bound // (2 * C)  # largest row count the neighbour-table kernel addresses
        assert spv.spv_block_conv_kernel(n_max, C, torch.bfloat16) == 0
        assert spv.spv_block_conv_kernel(n_max + 1, C, torch.bfloat16) == 2  # 27 n pairs exceed 32 bits too
        assert spv.spv_conv_kernel(27, C, C, torch.bfloat16, n_max, n_max, 27 * n_max) == 0
        # too many input rows for either matrix-core kernel's 32-bit offsets: the vector-ALU kernel
        assert spv.spv_conv_kernel(27, C, C, torch.bfloat16, n_max + 1, 1000, 27 * 1000) == 2
    # the neighbour table itself: m_out * 27 * 4 bytes
    m_max = bound // (27 * 4)
    assert spv.spv_conv_kernel(27, 32, 32, torch.bfloat16, 1000, m_max, 0) == 0
    assert spv.spv_conv_kernel(27, 32, 32, torch.bfloat16, 1000, m_max + 1, 0) == 1
    # fp32 and K = 2 never take the table kernel; a sparse transposed map takes the tile kernel
    assert spv.spv_conv_kernel(27, 32, 32, torch.float32, 1000, 1000, 27000) == 2
    assert spv.spv_conv_kernel(8, 64, 128, torch.bfloat16, 1000, 600, 1000) == 1
    assert spv.spv_conv_kernel(8, 128, 64, torch.bfloat16, 600, 1000, 1000, True) == 1
    assert spv.spv_conv_kernel(27, 96, 96, torch.bfloat16, 1000, 1000, 27000, True) == 0  # dgrad of a submanifold map
    assert spv.spv_conv_kernel(5, 32, 32, torch.bfloat16, 10, 10, 10) == -1


@pytest.mark.skipif(not os.path.exists(LIB), reason="libspv.so not built")
def test_workspace_alignment_and_voxel_lookup_validation():
    from paper_2007_16100_amd import spv
    L = spv.lib()
    P = ct.c_void_p(16)
    for ws in (ct.c_void_p(16), ct.c_void_p(256 + 64), None):  # misaligned or null: rejected before any launch
        assert L.spv_voxel_lookup(None, ws, 1 << 30, 4, P, 4, P) == spv.SPV_ERR_INVALID_ARG
        assert L.spv_kernel_map_nbr(None, ws, 1 << 30, P, None, 4, P) == spv.SPV_ERR_INVALID_ARG
        assert L.spv_devoxelize_nbr(None, ws, 1 << 30, P, None, 4, P, P, 0, P, None, 4, ct.c_float(0.1), 0, P, 32,
                                    None, 0, None, None, None, 0, P, 1) == spv.SPV_ERR_INVALID_ARG
        assert L.spv_status_check(ws, None) == spv.SPV_ERR_INVALID_ARG
    ws = ct.c_void_p(512)
    assert L.spv_voxel_lookup(None, ws, 16, 4, P, 4, P) == spv.SPV_ERR_CAPACITY
    assert L.spv_voxel_lookup(None, ws, 1 << 30, -1, P, 4, P) == spv.SPV_ERR_INVALID_ARG
    assert L.spv_voxel_lookup(None, ws, 1 << 30, 4, None, 4, P) == spv.SPV_ERR_INVALID_ARG
