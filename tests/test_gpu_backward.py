"""GPU parity of the backward passes (through the C ABI) against the oracle's.

* conv input gradient: the conv kernels over the swapped map with W read
  transposed -- normwise bound of the forward conv;
* conv weight gradient: fp32 result, sums over up to ~10^5 pairs per offset in
  fp32 -- normwise 1e-3 -- and bit-identical across runs (fixed slices, added in
  order);
* scatter-mean backward: bit-exact (fp64 quotient, one rounding on both sides);
* devoxelization backward: fp32 atomics -- normwise 1e-5.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2007_16100_amd import synth
from tests import parity

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-2}
TD = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


@pytest.fixture(scope="module")
def spv():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2007_16100_amd import spv as s
    s.lib()
    return s


@pytest.fixture(scope="module")
def sweep():
    return synth.lidar_sweep(1002)


def dev(a, dtype=None):
    if dtype in ("bf16", "f16"):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(TD[dtype]).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t, dtype=None):
    t = t.detach().cpu()
    if dtype in ("bf16", "f16"):
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def normwise(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def _map(rc, kind):
    if kind == "subm":
        oc, off, pairs = oracle.kernel_map(rc)
        return len(rc), len(rc), 27, False, off, pairs
    if kind == "k2s2":
        oc, off, pairs = oracle.kernel_map(rc, 2, 2)
        return len(rc), len(oc), 8, False, off, pairs
    if kind == "k3s2":
        oc, off, pairs = oracle.kernel_map(rc, 3, 2)
        return len(rc), len(oc), 27, False, off, pairs
    oc, off, pairs = oracle.kernel_map(rc, 2, 2)  # transposed k2s2: coarse -> fine
    return len(oc), len(rc), 8, True, off, pairs


@pytest.mark.parametrize("kind,cin,cout,dtype,step", [
    ("subm", 32, 32, "bf16", 2), ("subm", 96, 96, "bf16", 2), ("subm", 64, 128, "f16", 2), ("subm", 16, 16, "f32", 6),
    ("subm", 256, 256, "bf16", 8), ("k2s2", 64, 128, "bf16", 2), ("k3s2", 32, 64, "bf16", 2),
    ("transposed", 128, 64, "bf16", 2)])
def test_conv_dgrad(spv, sweep, kind, cin, cout, dtype, step):
    rc, _, _, _ = oracle.voxelize(sweep[::step], 0.05)
    m_in, m_out, K3, tr, off, pairs = _map(rc, kind)
    W = synth.conv_weight(K3, cin, cout, 1101, dtype)
    dy = synth.normal((m_out, cout), 1102, dtype=dtype)
    ws = spv.Workspace.for_ops(max(m_in, m_out), max(cin, cout))
    got = spv.spv_sparse_conv_dgrad(ws, dev(dy, dtype), dev(off), dev(pairs), dev(W, dtype), m_in, transposed=tr)
    ref = oracle.conv_dgrad(dy, off, pairs, W, m_in, dtype, transposed=tr)
    g = synth.from_storage(host(got, dtype)[:m_in], dtype)
    parity.check(g, synth.from_storage(ref, dtype), dtype)


@pytest.mark.parametrize("cin,cout,dtype,step", [(96, 96, "bf16", 2), (32, 64, "f16", 2), (128, 32, "bf16", 3),
                                                 (256, 256, "bf16", 8)])
def test_conv_dgrad_nbr(spv, sweep, cin, cout, dtype, step):
    """The input gradient on the neighbour table (mirrored, transposed weights, no plan) against the oracle's
    dgrad over the CSR map; the table has a live row count below its capacity."""
    rc, _, _, _ = oracle.voxelize(sweep[::step], 0.05)
    m = len(rc)
    _, off, pairs = oracle.kernel_map(rc)
    W = synth.conv_weight(27, cin, cout, 1111, dtype)
    dy = synth.normal((m, cout), 1112, dtype=dtype)
    cap = m + 37
    ws = spv.Workspace.for_ops(cap, max(cin, cout))
    coords = torch.zeros((cap, 4), dtype=torch.int32, device="cuda")
    coords[:m] = dev(rc)
    m_dev = torch.tensor([m], dtype=torch.int64, device="cuda")
    nbr = spv.spv_kernel_map_nbr(ws, coords, m_dev=m_dev)
    dyp = torch.zeros((cap, cout), dtype=TD[dtype], device="cuda")
    dyp[:m] = dev(dy, dtype)
    got = spv.spv_sparse_conv_dgrad_nbr(ws, dyp, nbr, dev(W, dtype), m_dev=m_dev)
    ref = oracle.conv_dgrad(dy, off, pairs, W, m, dtype)
    parity.check(synth.from_storage(host(got, dtype)[:m], dtype), synth.from_storage(ref, dtype), dtype)


@pytest.mark.parametrize("kind,cin,cout,dtype,step", [
    ("subm", 32, 32, "bf16", 2), ("subm", 96, 96, "bf16", 4), ("subm", 64, 128, "f16", 4), ("subm", 16, 16, "f32", 8),
    ("subm", 256, 256, "bf16", 16), ("subm", 24, 40, "bf16", 8), ("k2s2", 64, 128, "bf16", 2),
    ("k3s2", 32, 64, "bf16", 4), ("transposed", 128, 64, "bf16", 2),
    # pairs wider than 512 channels: past what the MFMA kernel gathers per pair
    ("subm", 128, 512, "bf16", 16)])
def test_conv_wgrad(spv, sweep, kind, cin, cout, dtype, step):
    rc, _, _, _ = oracle.voxelize(sweep[::step], 0.05)
    m_in, m_out, K3, tr, off, pairs = _map(rc, kind)
    x = synth.normal((m_in, cin), 1103, dtype=dtype)
    dy = synth.normal((m_out, cout), 1104, dtype=dtype)
    print(f"wgrad {kind} {cin}->{cout} {dtype} pairs={len(pairs)}", flush=True)
    ws = spv.Workspace.for_wgrad(K3, cin, cout)
    args = (ws, dev(x, dtype), dev(dy, dtype), dev(off), dev(pairs), K3)
    got = host(spv.spv_sparse_conv_wgrad(*args, transposed=tr))
    again = host(spv.spv_sparse_conv_wgrad(*args, transposed=tr))
    np.testing.assert_array_equal(got, again)  # deterministic
    ref = oracle.conv_wgrad(x, dy, off, pairs, K3, dtype, transposed=tr)
    # fp32 results of up to ~10^5-term sums: 1e-3 normwise and elementwise
    parity.check(got, ref, "f32", normwise_tol=1e-3, elemwise_tol=1e-3)


@pytest.mark.parametrize("dtype,C", [("bf16", 96), ("f32", 8), ("f16", 5)])
def test_voxelize_backward(spv, sweep, dtype, C):
    coords, vf, counts, p2v = oracle.voxelize(sweep, 0.2)
    dv = synth.normal((len(coords), C), 1105, dtype=dtype)
    got = spv.spv_voxelize_backward(dev(dv, dtype), dev(counts), dev(p2v), len(coords))
    ref = oracle.voxelize_backward(dv, counts, p2v, dtype)
    np.testing.assert_array_equal(host(got, dtype)[: len(sweep)], ref)


@pytest.mark.parametrize("mode,stride_log2,C,dtype", [("center", 0, 96, "bf16"), ("corner", 0, 32, "f32"),
                                                      ("center", 2, 64, "bf16")])
def test_devoxelize_backward(spv, sweep, mode, stride_log2, C, dtype):
    pts = sweep[::2]
    rc, _, _, _ = oracle.voxelize(pts, 0.05)
    for _ in range(stride_log2):
        rc, _, _ = oracle.kernel_map(rc, 2, 2)
    vf = synth.normal((len(rc), C), 1106, dtype=dtype)
    _, ci, cw = oracle.devoxelize(rc, vf, pts, 0.05, stride_log2, mode, dtype=dtype, want_corners=True)
    dout = synth.normal((len(pts), C), 1107, dtype=dtype)
    ws = spv.Workspace.for_devox_backward(len(pts), len(rc))
    args = (ws, dev(ci), dev(cw), dev(dout, dtype), len(rc))
    got = host(spv.spv_devoxelize_backward(*args))[: len(rc)]
    again = host(spv.spv_devoxelize_backward(*args))[: len(rc)]
    np.testing.assert_array_equal(got, again)  # deterministic
    assert spv.spv_status_check(ws) == spv.SPV_OK
    ref = oracle.devoxelize_backward(ci, cw, dout, len(rc), dtype)
    parity.check(got, ref, "f32")


def test_devoxelize_backward_edges(spv):
    """Voxels with 0 to ~80 terms, and of 300 to 1500 (several chunks of 256: the merge by binary search), three
    voxels with none, absent corners, weights summing to 0, odd C (one channel per thread), a misaligned gradient
    (no vector loads) and a corner index past m."""
    rng = np.random.default_rng(1108)
    lengths = np.concatenate([np.arange(71), [256, 257, 300, 777, 1500]])
    m = len(lengths) + 3  # the last three voxels get no terms: their rows must be zeros
    # point k has corner 0 on voxel owner[k]; each other corner on a random voxel below len(lengths) with
    # probability 1/20, else absent
    owner = np.repeat(np.arange(len(lengths)), lengths)
    n = len(owner)
    ci = rng.integers(0, len(lengths), size=(n, 8)).astype(np.int32)
    ci[rng.random((n, 8)) >= 0.05] = -1
    ci[:, 0] = owner
    cw = rng.random((n, 8)).astype(np.float32)
    cw[::7] = 0.0  # present weights summing to 0: the point adds nothing
    for C, dtype in ((5, "f32"), (16, "bf16")):
        dout = synth.normal((n, C), 1109, dtype=dtype)
        ref = oracle.devoxelize_backward(ci, cw, dout, m, dtype)
        ws = spv.Workspace.for_devox_backward(n, m)
        got = host(spv.spv_devoxelize_backward(ws, dev(ci), dev(cw), dev(dout, dtype), m))[:m]
        assert spv.spv_status_check(ws) == spv.SPV_OK
        assert not got[len(lengths):].any()
        parity.check(got, ref, "f32")
        if dtype == "bf16":  # a gradient 2 bytes off a 16-byte boundary
            buf = torch.empty(n * C + 1, dtype=torch.bfloat16, device="cuda")
            shifted = buf[1:].view(n, C)
            shifted.copy_(dev(dout, dtype))
            got2 = host(spv.spv_devoxelize_backward(ws, dev(ci), dev(cw), shifted, m))[:m]
            parity.check(got2, ref, "f32")
    # a corner index past m: skipped, reported as a range error
    bad = ci.copy()
    bad[3, 5] = m + 2
    ws = spv.Workspace.for_devox_backward(n, m)
    spv.spv_devoxelize_backward(ws, dev(bad), dev(cw), dev(synth.normal((n, 8), 1110, dtype="f32"), "f32"), m)
    assert spv.spv_status_check(ws) == spv.SPV_ERR_RANGE


def _epi_inputs(m, C, dtype, seed):
    rng = np.random.default_rng(seed)
    a = synth.normal((m, C), seed, dtype=dtype)
    dy = synth.normal((m, C), seed + 1, dtype=dtype)
    res = synth.normal((m, C), seed + 2, dtype=dtype)
    s = (0.5 + rng.random(C)).astype(np.float32)
    s[1] = -s[1]
    b = (0.3 * rng.standard_normal(C)).astype(np.float32)
    b[0] = 0.0  # rows 0..3 of channel 0: the activation's input is exactly 0
    zero = synth.to_storage(np.zeros(4, np.float32), dtype)
    a[:4, 0] = zero
    res[:4, 0] = zero
    return a, dy, res, s, b


@pytest.mark.parametrize("dtype,C,m", [("bf16", 96, 20000), ("f32", 19, 3001), ("f16", 64, 777)])
@pytest.mark.parametrize("relu,res_after_act", [(True, False), (True, True), (False, False)])
def test_epilogue_backward(spv, dtype, C, m, relu, res_after_act):
    a, dy, res, s, b = _epi_inputs(m, C, dtype, 1210)
    ref = oracle.epilogue_backward(dy, a, s, b, relu, res, res_after_act, dtype)
    ws = spv.Workspace.for_epilogue_backward(m, C)
    args = (ws, dev(dy, dtype), dev(a, dtype), dev(s), dev(b), relu, dev(res, dtype), res_after_act)
    got = spv.spv_epilogue_backward(*args)
    again = spv.spv_epilogue_backward(*args)
    da, dres, dscale, dshift = (host(got[0], dtype)[:m], host(got[1], dtype)[:m], host(got[2]), host(got[3]))
    np.testing.assert_array_equal(da, ref[0])      # one rounding of an exact product: bit-exact
    np.testing.assert_array_equal(dres, ref[1])    # dy or 0, unchanged
    np.testing.assert_array_equal(host(again[2]), dscale)  # deterministic sums
    np.testing.assert_array_equal(host(again[3]), dshift)
    # fp64 sums in another order, one rounding to float32
    np.testing.assert_allclose(dscale, ref[2], rtol=1e-6, atol=1e-6)
    np.testing.assert_allclose(dshift, ref[3], rtol=1e-6, atol=1e-6)


def test_epilogue_backward_empty_and_partial_outputs(spv):
    d = "cuda"
    ws = spv.Workspace.for_epilogue_backward(0, 8)
    e = torch.zeros((0, 8), dtype=torch.bfloat16, device=d)
    da, _, dscale, dshift = spv.spv_epilogue_backward(ws, e, e)
    assert not dscale.any() and not dshift.any()
    # no sums asked for: no workspace needed
    L = spv.lib()
    m, C = 100, 16
    a, dy, _, s, b = _epi_inputs(m, C, "bf16", 1211)
    out = torch.empty((m, C), dtype=torch.bfloat16, device=d)
    dyt, at, st_, bt = dev(dy, "bf16"), dev(a, "bf16"), dev(s), dev(b)  # held until the call has run
    st = L.spv_epilogue_backward(None, None, 0, spv._ptr(dyt), spv._ptr(at), spv._ptr(st_), spv._ptr(bt), 1, None, 0,
                                 m, C, spv._ptr(out), None, None, None, spv.SPV_BF16)
    assert st == spv.SPV_OK
    torch.cuda.synchronize()
    ref = oracle.epilogue_backward(dy, a, s, b, True, dtype="bf16")
    np.testing.assert_array_equal(host(out, "bf16"), ref[0])


@pytest.mark.parametrize("dtype,cin,cout,m", [("bf16", 96, 96, 30011), ("f16", 32, 64, 5000), ("f32", 24, 40, 2003),
                                              ("bf16", 256, 19, 1500), ("bf16", 40, 24, 999)])
def test_linear_backward(spv, dtype, cin, cout, m):
    x = synth.normal((m, cin), 1212, dtype=dtype)
    W = synth.linear_weight(cin, cout, 1213, dtype)
    da = synth.normal((m, cout), 1214, dtype=dtype)
    ws = spv.Workspace.for_linear_backward(cin, cout)
    args = (ws, dev(x, dtype), dev(W, dtype), dev(da, dtype))
    dx, dW = spv.spv_linear_backward(*args)
    _, dW2 = spv.spv_linear_backward(*args)
    np.testing.assert_array_equal(host(dW2), host(dW))  # deterministic
    rdx, rdW = oracle.linear_backward(x, W, da, dtype)
    parity.check(host(dx, dtype)[:m], rdx, dtype)
    # fp32 sums of m terms: 1e-3 normwise and elementwise, as the conv weight gradient
    parity.check(host(dW), rdW, "f32", normwise_tol=1e-3, elemwise_tol=1e-3)


def test_point_branch_layer_backward_chain(spv):
    """out = ReLU(scale * (x @ W) + shift) + res on the GPU: the raw product by spv_linear without
    its epilogue, spv_epilogue_backward, spv_linear_backward, against the oracle's same chain."""
    m, cin, cout, dtype = 12000, 64, 96, "bf16"
    x = synth.normal((m, cin), 1215, dtype=dtype)
    W = synth.linear_weight(cin, cout, 1216, dtype)
    _, dy, res, s, b = _epi_inputs(m, cout, dtype, 1217)
    wsl = spv.Workspace.for_ops(m, max(cin, cout))
    a = spv.spv_linear(wsl, dev(x, dtype), dev(W, dtype))
    a_ref = host(a, dtype)[:m]  # both chains start from the same raw product
    parity.check(a_ref, oracle.linear(x, W, dtype), dtype)
    wse = spv.Workspace.for_epilogue_backward(m, cout)
    da, dres, dscale, dshift = spv.spv_epilogue_backward(wse, dev(dy, dtype), a, dev(s), dev(b), True,
                                                         dev(res, dtype), True)
    dx, dW = spv.spv_linear_backward(spv.Workspace.for_linear_backward(cin, cout), dev(x, dtype), dev(W, dtype), da)
    rda, rdres, rdscale, rdshift = oracle.epilogue_backward(dy, a_ref, s, b, True, res, True, dtype)
    rdx, rdW = oracle.linear_backward(x, W, rda, dtype)
    np.testing.assert_array_equal(host(da, dtype)[:m], rda)
    np.testing.assert_array_equal(host(dres, dtype)[:m], rdres)
    np.testing.assert_allclose(host(dscale), rdscale, rtol=1e-6, atol=1e-6)
    np.testing.assert_allclose(host(dshift), rdshift, rtol=1e-6, atol=1e-6)
    parity.check(host(dx, dtype)[:m], rdx, dtype)
    parity.check(host(dW), rdW, "f32", normwise_tol=1e-3, elemwise_tol=1e-3)
