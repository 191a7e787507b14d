"""The allocation-free neighbour-table conv (spv_sparse_conv_nbr_noalloc), through the C ABI,
against the workspace entry point it varies: the same kernels on the same inputs give the
same bits.  Two calls in a row share the library's device scratch, the second with a
smaller input (fewer voxels, narrower channels), and both must match."""
import ctypes as ct

import numpy as np
import pytest
import torch

from paper_2007_16100_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def spv():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2007_16100_amd import spv as s
    s.lib()
    return s


def _bf(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def _case(spv, step, cin, cout, seed):
    xyz = synth.lidar_sweep(1002)[::step]
    ws = spv.Workspace.for_ops(len(xyz), 256)
    vox = spv.spv_voxelize(ws, torch.from_numpy(xyz).cuda(), 0.05)
    m = vox.m
    nbr = spv.spv_kernel_map_nbr(ws, vox.coords[:m].contiguous())
    x = _bf(synth.normal((m, cin), seed, dtype="bf16"))
    W = _bf(synth.conv_weight(27, cin, cout, seed + 1, "bf16"))
    sc, sh = (torch.from_numpy(a).cuda() for a in synth.folded_bn(cout, seed + 2))
    return ws, m, nbr, x, W, sc, sh


def test_noalloc_matches_workspace_call_twice(spv):
    big = _case(spv, 1, 96, 96, 31)
    small = _case(spv, 3, 32, 64, 41)
    outs = []
    for ws, m, nbr, x, W, sc, sh in (big, small):
        print(f"noalloc conv m={m} {x.shape[1]}->{W.shape[2]}", flush=True)
        cout = W.shape[2]
        ref = spv.spv_sparse_conv_nbr(ws, x, nbr, W, cout, m, scale=sc, shift=sh, relu=True)
        got = spv.spv_sparse_conv_nbr_noalloc(x, nbr, W, cout, m, scale=sc, shift=sh, relu=True)
        torch.cuda.synchronize()
        assert torch.equal(got[:m].view(torch.int16), ref[:m].view(torch.int16))
        outs.append(got[:m].clone())
    # the first result was not disturbed by the second call's use of the shared scratch
    assert outs[0].shape[1] == 96 and outs[1].shape[1] == 64


def test_noalloc_rejects_before_any_launch(spv):
    L = spv.lib()
    P = ct.c_void_p(16)
    # Cout 512: no packing of that size fits (and the kernel does not take it)
    st = L.spv_sparse_conv_nbr_noalloc(None, P, 4, 256, P, P, 256, 512, None, None, None, 0, P, None, 4, 512, 1)
    assert st == spv.SPV_ERR_UNSUPPORTED
    st = L.spv_sparse_conv_nbr_noalloc(None, P, -1, 32, P, P, 32, 32, None, None, None, 0, P, None, 4, 32, 1)
    assert st == spv.SPV_ERR_INVALID_ARG
