"""GPU parity: every HIP entry point (through the C ABI) against the CPU oracle.

Integers (voxel coordinates, counts, point->voxel indices, hash lookups, kernel
maps, devoxelization corner indices) must match bit for bit.  Floats must
satisfy the normwise bound max|gpu - oracle| / max|oracle| <= 1e-5 (fp32) or
2e-2 (bf16 / fp16 storage with fp32 accumulation).
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
    """numpy (float32 / int32 / uint16 bit patterns) -> device tensor."""
    if dtype in ("bf16", "f16"):
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(TD[dtype])
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.cuda()


def host(t, dtype=None):
    t = t.detach().cpu()
    if dtype in ("bf16", "f16"):
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def normwise(g, r, dtype):
    return parity.errors(synth.from_storage(g, dtype), synth.from_storage(r, dtype))[0]


def check_close(g, r, dtype, kind="op"):
    """Normwise and elementwise (99.9th percentile) bounds, both logged (tests/parity.py)."""
    return parity.check(synth.from_storage(g, dtype), synth.from_storage(r, dtype), dtype, kind)


# ---------------------------------------------------------------------------
# voxelization
# ---------------------------------------------------------------------------
def run_voxelize(spv, xyz, v, feat=None, dtype="f32", batch=None):
    ws = spv.Workspace.for_ops(max(len(xyz), 1), feat.shape[1] if feat is not None else 16)
    out = spv.spv_voxelize(ws, dev(xyz), v, None if feat is None else dev(feat, dtype),
                           None if batch is None else dev(batch))
    m = out.m
    return (host(out.coords)[:m], None if feat is None else host(out.vfeat, dtype)[:m], host(out.counts)[:m],
            host(out.pt2vox)[:len(xyz)], out)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_voxelize_tiny_cube(spv, dtype):
    xyz = synth.uniform_cube(2000, 1.6, 1001)
    feat = synth.normal((2000, 16), 1002, dtype=dtype)
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, 0.1, feat, dtype)
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, 0.1, feat, dtype)
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    check_close(vf, rvf, dtype)


def test_voxelize_sweep_c96(spv, sweep):
    feat = synth.normal((len(sweep), 96), 1005, dtype="bf16")
    c, vf, cnt, p2v, _ = run_voxelize(spv, sweep, 0.05, feat, "bf16")
    rc, rvf, rcnt, rp2v = oracle.voxelize(sweep, 0.05, feat, "bf16")
    assert len(rc) > 80000
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    check_close(vf, rvf, "bf16")


@pytest.mark.parametrize("case", ["empty", "one", "one_voxel", "faces", "negative_batch", "odd_c"])
def test_voxelize_edge_cases(spv, case):
    rng = np.random.default_rng(77)
    batch = None
    C, dtype, v = 8, "bf16", 0.1
    if case == "empty":
        xyz = np.zeros((0, 3), np.float32)
    elif case == "one":
        xyz = np.array([[0.123, -4.5, 7.0]], np.float32)
    elif case == "one_voxel":
        xyz = rng.uniform(0.001, 0.099, size=(20000, 3)).astype(np.float32)
    elif case == "faces":
        k = np.arange(-50, 50, dtype=np.float32) * np.float32(v)
        xyz = np.stack([np.concatenate([k, np.nextafter(k, np.float32(1e9)), np.nextafter(k, np.float32(-1e9))])] * 3,
                       1).astype(np.float32)
        xyz[:, 1] = xyz[::-1, 1]
    elif case == "negative_batch":
        xyz = rng.uniform(-3000.0, -2990.0, size=(5000, 3)).astype(np.float32)
        batch = rng.integers(0, 3, size=5000).astype(np.int32)
    else:  # channel count not a multiple of 8 -> scalar path
        xyz = rng.uniform(-1, 1, size=(3000, 3)).astype(np.float32)
        C, dtype = 5, "f32"
    feat = synth.normal((len(xyz), C), 5, dtype=dtype)
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, v, feat, dtype, batch)
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, v, feat, dtype, batch)
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    check_close(vf, rvf, dtype)


def test_voxelize_many_tiles(spv):
    """Over 524k distinct voxels: the sort's offsets come from a multi-tile scan
    of digit-major histograms instead of the scatter's own."""
    rng = np.random.default_rng(4242)
    xyz = rng.uniform(-60.0, 60.0, size=(700_000, 3)).astype(np.float32)
    xyz[::7] = xyz[1::7][: len(xyz[::7])]  # some shared voxels
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, 0.05, synth.normal((len(xyz), 8), 9, dtype="bf16"), "bf16")
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, 0.05, synth.normal((len(xyz), 8), 9, dtype="bf16"), "bf16")
    assert len(rc) > 524288
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    check_close(vf, rvf, "bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_voxelize_mean_bit_exact(spv, sweep, dtype):
    """The scatter-mean sums in fp64 (exact for these features) and rounds once,
    as the oracle does, so voxel features agree bit for bit."""
    feat = synth.normal((len(sweep), 32), 1011, dtype=dtype)
    _, vf, _, _, _ = run_voxelize(spv, sweep, 0.05, feat, dtype)
    _, rvf, _, _ = oracle.voxelize(sweep, 0.05, feat, dtype)
    np.testing.assert_array_equal(vf, rvf)


@pytest.mark.parametrize("dtype,C", [("bf16", 256), ("bf16", 8), ("f16", 96), ("f32", 12), ("bf16", 5)])
def test_voxelize_coarse_long_runs(spv, sweep, dtype, C):
    """At 0.8 m voxels a sweep's voxels hold up to ~10^3 points; those over 32 are summed
    by a whole workgroup (point slices, then the slices in order).  The fp64 sums are
    exact for these features, so the means still match the oracle bit for bit."""
    feat = synth.normal((len(sweep), C), 1012, dtype=dtype)
    _, vf, cnt, _, _ = run_voxelize(spv, sweep, 0.8, feat, dtype)
    assert cnt.max() > 500 and (cnt > 32).sum() > 100
    _, rvf, _, _ = oracle.voxelize(sweep, 0.8, feat, dtype)
    np.testing.assert_array_equal(vf, rvf)


# ---------------------------------------------------------------------------
# scatter-mean onto a given voxel set
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,C,v", [("bf16", 96, 0.05), ("bf16", 256, 0.8), ("f32", 12, 0.8), ("f16", 5, 0.1)])
def test_voxelize_onto_own_set(spv, sweep, dtype, C, v):
    """Onto the set spv_voxelize finds (its device count), the outputs are spv_voxelize's and
    the oracle's bit for bit -- voxels of over 32 points included at 0.8 m."""
    feat = synth.normal((len(sweep), C), 1013, dtype=dtype)
    c, vf, cnt, p2v, out = run_voxelize(spv, sweep, v, feat, dtype)
    ws = spv.Workspace.for_ops(len(sweep), C)
    o = spv.spv_voxelize_onto(ws, out.coords, dev(sweep), v, dev(feat, dtype), m_dev=out.m_dev)
    assert spv.spv_status_check(ws) == 0
    m = len(c)
    np.testing.assert_array_equal(host(o.counts)[:m], cnt)
    np.testing.assert_array_equal(host(o.pt2vox)[:len(sweep)], p2v)
    np.testing.assert_array_equal(host(o.vfeat, dtype)[:m], vf)
    rvf, rcnt, rp2v = oracle.voxelize_onto(c, sweep, v, feat, dtype)
    np.testing.assert_array_equal(host(o.vfeat, dtype)[:m], rvf)
    np.testing.assert_array_equal(rcnt, cnt)


@pytest.mark.parametrize("dtype,C", [("bf16", 32), ("f32", 8)])
def test_voxelize_onto_subset(spv, sweep, dtype, C):
    """A shuffled two-thirds of the occupied voxels plus voxels no point falls into: the
    points of the dropped voxels get -1, the empty voxels count 0 with zero features."""
    rng = np.random.default_rng(1014)
    v = 0.1
    batch = (np.arange(len(sweep)) * 3 // len(sweep)).astype(np.int32)
    feat = synth.normal((len(sweep), C), 1015, dtype=dtype)
    rc, _, _, _ = oracle.voxelize(sweep, v, batch=batch)
    keep = rng.permutation(len(rc))[: 2 * len(rc) // 3]
    empty = np.array([[0, 30000, 0, 0], [2, -5, 7, 9], [5, 0, 0, 0]], np.int32)
    gset = np.concatenate([rc[keep], empty])
    gset = np.ascontiguousarray(gset[rng.permutation(len(gset))])
    ws = spv.Workspace.for_ops(len(sweep), C)
    o = spv.spv_voxelize_onto(ws, dev(gset), dev(sweep), v, dev(feat, dtype), dev(batch))
    assert spv.spv_status_check(ws) == 0
    rvf, rcnt, rp2v = oracle.voxelize_onto(gset, sweep, v, feat, dtype, batch)
    assert (rp2v < 0).sum() > 1000 and (rcnt == 0).sum() == len(empty)
    np.testing.assert_array_equal(host(o.counts), rcnt)
    np.testing.assert_array_equal(host(o.pt2vox), rp2v)
    np.testing.assert_array_equal(host(o.vfeat, dtype), rvf)


def test_voxelize_onto_edge_cases(spv):
    xyz = np.array([[0.05, 0.05, 0.05], [0.15, 0.05, 0.05], [0.16, 0.07, 0.01]], np.float32)
    feat = synth.normal((3, 8), 3, dtype="bf16")
    ws = spv.Workspace.for_ops(16, 8)
    # empty set: every point outside it
    o = spv.spv_voxelize_onto(ws, torch.zeros((0, 4), dtype=torch.int32, device="cuda"), dev(xyz), 0.1,
                              dev(feat, "bf16"))
    np.testing.assert_array_equal(host(o.pt2vox), [-1, -1, -1])
    # no features: counts and pt2vox only
    gset = np.array([[0, 1, 0, 0], [0, 0, 0, 0], [0, 9, 9, 9]], np.int32)
    o = spv.spv_voxelize_onto(ws, dev(gset), dev(xyz), 0.1)
    np.testing.assert_array_equal(host(o.counts), [2, 1, 0])
    np.testing.assert_array_equal(host(o.pt2vox), [1, 0, 0])
    # no points: every voxel of the set counts 0
    o = spv.spv_voxelize_onto(ws, dev(gset), dev(np.zeros((0, 3), np.float32)), 0.1)
    np.testing.assert_array_equal(host(o.counts), [0, 0, 0])
    # a repeated set coordinate is a device-detected invalid argument
    spv.spv_voxelize_onto(ws, dev(np.array([[0, 1, 0, 0], [0, 1, 0, 0]], np.int32)), dev(xyz), 0.1)
    assert spv.spv_status_check(ws) == spv.SPV_ERR_INVALID_ARG


def test_voxelize_wide_keys(spv):
    """Coordinates spanning nearly the whole key range (48 significant bits once
    compacted): the sort's passes past 32 bits run."""
    rng = np.random.default_rng(4343)
    xyz = rng.uniform(-1600.0, 1600.0, size=(20_000, 3)).astype(np.float32)
    batch = rng.integers(0, 4, size=len(xyz)).astype(np.int32)
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, 0.05, synth.normal((len(xyz), 8), 3, dtype="bf16"), "bf16", batch)
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, 0.05, synth.normal((len(xyz), 8), 3, dtype="bf16"), "bf16", batch)
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    np.testing.assert_array_equal(vf, rvf)


def test_voxelize_wide_keys_many_tiles(spv):
    """Keys past 32 significant bits (4 batches over +-1600 m) and over 524k of
    them: every pass of the sort runs over more than 256 tiles, with scanned offsets."""
    rng = np.random.default_rng(4444)
    xyz = rng.uniform(-1600.0, 1600.0, size=(600_000, 3)).astype(np.float32)
    xyz[::5] = xyz[1::5][: len(xyz[::5])]  # some shared voxels
    batch = rng.integers(0, 4, size=len(xyz)).astype(np.int32)
    batch[::5] = batch[1::5][: len(batch[::5])]
    feat = synth.normal((len(xyz), 8), 5, dtype="bf16")
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, 0.05, feat, "bf16", batch)
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, 0.05, feat, "bf16", batch)
    assert len(xyz) > 256 * 2048 and len(rc) > 400_000  # more than 256 sort tiles
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    np.testing.assert_array_equal(vf, rvf)


def _bucket_case(case):
    """Points on a 1 m grid (v = 1): x spans 0..4095 voxels, y 0..63, z 0..31, so
    the compacted key has 12 + 6 + 5 bits and its top 12 bits (the sort's fine
    bin) are x.  The buckets group consecutive fine bins by count, so fine bin 0
    with k points is a bucket of its own (the next bin's running count already
    maps past bucket 0) of exactly k items."""
    rng = np.random.default_rng(6161)
    if case == "narrow":  # 6 significant bits: every key its own fine bin
        vox = rng.integers(0, 3, size=(9000, 3))
    elif case == "most_blocks":  # 256 histogram blocks of 1024 keys exactly
        vox = np.stack([rng.integers(0, 4096, 262_144), rng.integers(0, 64, 262_144),
                        rng.integers(0, 32, 262_144)], 1)
    else:  # one bucket of 8192 items (the bucket sort's capacity) or one more
        k = 8_192 if case == "cap" else 8_193
        a = np.stack([np.zeros(k, np.int64), rng.integers(0, 64, k), rng.integers(0, 32, k)], 1)
        b = np.stack([rng.integers(1, 4096, 30_000), rng.integers(0, 64, 30_000), rng.integers(0, 32, 30_000)], 1)
        a[0] = (0, 0, 0)
        b[0] = (4095, 63, 31)
        vox = np.concatenate([b[: 20_000], a, b[20_000:]])
    return (vox + rng.uniform(0.1, 0.9, size=vox.shape)).astype(np.float32)


@pytest.mark.parametrize("case", ["narrow", "cap", "over", "most_blocks"])
def test_voxelize_bucket_sort_bounds(spv, case):
    """The sort's bucket path at its limits: keys of 6 bits, a bucket at the
    in-LDS capacity, one item over it (the passes run instead), and the most
    histogram blocks the bucket path takes."""
    xyz = _bucket_case(case)
    feat = synth.normal((len(xyz), 8), 6162, dtype="bf16")
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, 1.0, feat, "bf16")
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, 1.0, feat, "bf16")
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    np.testing.assert_array_equal(vf, rvf)


def test_voxelize_over_a_million_points(spv):
    """2.2M points (a sixth of them sharing voxels) over +-900 m: the quantize and histogram
    kernels stride with their largest grids (1024 blocks), the sort launches every pass
    (over 256 tiles), and the scatter-mean interleaves its insert blocks."""
    rng = np.random.default_rng(5555)
    xyz = rng.uniform(-900.0, 900.0, size=(2_200_000, 3)).astype(np.float32)
    xyz[::6] = xyz[1::6][: len(xyz[::6])]
    feat = synth.normal((len(xyz), 8), 5556, dtype="bf16")
    c, vf, cnt, p2v, _ = run_voxelize(spv, xyz, 0.05, feat, "bf16")
    rc, rvf, rcnt, rp2v = oracle.voxelize(xyz, 0.05, feat, "bf16")
    assert len(xyz) > 1024 * 1024  # beyond 1024 histogram blocks of 1024 keys: they stride
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(cnt, rcnt)
    np.testing.assert_array_equal(p2v, rp2v)
    np.testing.assert_array_equal(vf, rvf)


def test_voxelize_device_errors(spv):
    xyz = np.zeros((100, 3), np.float32)
    xyz[17, 1] = np.nan
    with pytest.raises(spv.SpvError) as e:
        run_voxelize(spv, xyz, 0.1)
    assert e.value.status == spv.SPV_ERR_NONFINITE
    xyz[17, 1] = 5000.0  # floor(5000 / 0.1) = 50000 > 32766
    with pytest.raises(spv.SpvError) as e:
        run_voxelize(spv, xyz, 0.1)
    assert e.value.status == spv.SPV_ERR_RANGE
    xyz[17, 1] = 0.0
    with pytest.raises(spv.SpvError) as e:
        run_voxelize(spv, xyz, 0.1, batch=np.full(100, 65535, np.int32))
    assert e.value.status == spv.SPV_ERR_RANGE


def test_voxelize_deterministic_integers(spv, sweep):
    a = run_voxelize(spv, sweep, 0.05)
    b = run_voxelize(spv, sweep, 0.05)
    for x, y in zip(a[:4], b[:4]):
        if x is not None:
            np.testing.assert_array_equal(x, y)


def test_lookup(spv, sweep):
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    rng = np.random.default_rng(3)
    q = rc[rng.integers(0, len(rc), 20000)].copy()
    q[::2, 1:] += rng.integers(-1, 2, size=(10000, 3)).astype(np.int32)  # neighbours, present or absent
    ws = spv.Workspace.for_ops(len(rc), 16)
    idx = host(spv.spv_lookup(ws, dev(rc), dev(q)))
    table = {tuple(r): i for i, r in enumerate(rc)}
    expect = np.array([table.get(tuple(r), -1) for r in q], np.int32)
    np.testing.assert_array_equal(idx, expect)


def test_voxel_lookup_on_the_voxelization_table(spv, sweep):
    """The table spv_voxelize itself built, queried in place (no rebuild): every voxel,
    neighbours present or absent, points of another batch and far-away coordinates."""
    batch = (np.arange(len(sweep)) % 3 == 0).astype(np.int32)
    rc, _, _, _ = oracle.voxelize(sweep, 0.05, batch=batch)
    ws = spv.Workspace.for_ops(len(sweep), 16)
    vox = spv.spv_voxelize(ws, dev(sweep), 0.05, None, dev(batch))
    assert vox.m == len(rc)
    rng = np.random.default_rng(5)
    q = np.concatenate([rc, rc[rng.integers(0, len(rc), 30000)]]).copy()
    q[len(rc)::2, 1:] += rng.integers(-1, 2, size=(15000, 3)).astype(np.int32)
    q[len(rc) + 1::4, 0] = 2  # a batch with no points
    q[-5:] = [[0, 32766, 0, 0], [0, -32767, 0, 0], [65534, 0, 0, 0], [0, 40000, 0, 0], [-1, 0, 0, 0]]
    idx = host(spv.spv_voxel_lookup(ws, len(sweep), dev(q)))
    table = {tuple(r): i for i, r in enumerate(rc)}
    expect = np.array([table.get(tuple(r), -1) for r in q], np.int32)
    np.testing.assert_array_equal(idx, expect)
    np.testing.assert_array_equal(idx[: len(rc)], np.arange(len(rc), dtype=np.int32))


# ---------------------------------------------------------------------------
# kernel maps
# ---------------------------------------------------------------------------
def run_kmap(spv, coords, K, stride):
    ws = spv.Workspace.for_ops(len(coords), 16)
    km = spv.spv_kernel_map(ws, dev(coords), K, stride)
    oc = host(km.out_coords)[:int(host(km.m_out_dev)[0])] if stride == 2 else None
    return oc, host(km.off), host(km.pairs)[:km.total], km


@pytest.mark.parametrize("K,stride", [(3, 1), (2, 2), (3, 2)])
def test_kmap_sweep_bitexact(spv, sweep, K, stride):
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    oc, off, pairs, _ = run_kmap(spv, rc, K, stride)
    roc, roff, rpairs = oracle.kernel_map(rc, K, stride)
    np.testing.assert_array_equal(off, roff)
    np.testing.assert_array_equal(pairs, rpairs)
    if stride == 2:
        np.testing.assert_array_equal(oc, roc)


@pytest.mark.parametrize("seed", range(6))
def test_kmap_random_small(spv, seed):
    rng = np.random.default_rng(500 + seed)
    m = int(rng.integers(1, 3000))
    pts = np.unique(np.concatenate([rng.integers(0, 2, (m, 1)), rng.integers(-12, 12, (m, 3))], 1), axis=0)
    pts = pts.astype(np.int32)
    for K, stride in [(3, 1), (2, 2), (3, 2)]:
        oc, off, pairs, _ = run_kmap(spv, pts, K, stride)
        roc, roff, rpairs = oracle.kernel_map(pts, K, stride)
        np.testing.assert_array_equal(off, roff)
        np.testing.assert_array_equal(pairs, rpairs)
        if stride == 2:
            np.testing.assert_array_equal(oc, roc)


@pytest.mark.parametrize("K,stride", [(3, 1), (2, 2), (3, 2)])
def test_kmap_large_batched(spv, K, stride):
    """~400k voxels in 4 batches over a wide range (coarse keys past 32 bits):
    the stride-2 parity partition and the submanifold map over more than 256
    count tiles, against the oracle exactly."""
    rng = np.random.default_rng(4545)
    c = rng.integers(-1500, 1500, size=(420_000, 3))
    c[1::3] = c[::3][: len(c[1::3])] + rng.integers(-1, 2, size=(len(c[1::3]), 3))  # local clusters
    b = rng.integers(0, 4, size=(len(c), 1))
    pts = np.unique(np.concatenate([b, c], 1), axis=0).astype(np.int32)
    assert len(pts) > 256 * 256
    oc, off, pairs, _ = run_kmap(spv, pts, K, stride)
    roc, roff, rpairs = oracle.kernel_map(pts, K, stride)
    np.testing.assert_array_equal(off, roff)
    np.testing.assert_array_equal(pairs, rpairs)
    if stride == 2:
        np.testing.assert_array_equal(oc, roc)


def test_kmap_k3_stride2_key_range_edges(spv):
    """3x3x3 stride-2 probes 2C + delta reach one step past the coordinate range
    at both ends (2 * -16384 - 1 and 2 * 16383 + 1): they must find nothing
    rather than wrap onto a stored key."""
    e = []
    for b in (0, 3):
        for x in (-32767, -32766, -32765, 32764, 32765, 32766):
            for y in (-32767, 0, 1, 32766):
                for z in (-32767, -1, 32765, 32766):
                    e.append((b, x, y, z))
    pts = np.array(sorted(set(e)), np.int32)
    oc, off, pairs, _ = run_kmap(spv, pts, 3, 2)
    roc, roff, rpairs = oracle.kernel_map(pts, 3, 2)
    np.testing.assert_array_equal(oc, roc)
    np.testing.assert_array_equal(off, roff)
    np.testing.assert_array_equal(pairs, rpairs)


def test_kmap_duplicate_coords_rejected(spv):
    pts = np.array([[0, 1, 2, 3], [0, 1, 2, 3]], np.int32)
    with pytest.raises(spv.SpvError) as e:
        run_kmap(spv, pts, 3, 1)
    assert e.value.status == spv.SPV_ERR_INVALID_ARG


# ---------------------------------------------------------------------------
# sparse convolution
# ---------------------------------------------------------------------------
def run_conv(spv, x, off, pairs, W, m_out, dtype, scale=None, shift=None, relu=False, transposed=False):
    ws = spv.Workspace.for_ops(max(m_out, len(x), 1), max(W.shape[1], W.shape[2]))
    out = spv.spv_sparse_conv(ws, dev(x, dtype), dev(off), dev(pairs), dev(W, dtype), m_out,
                              scale=None if scale is None else dev(scale), shift=None if shift is None else dev(shift),
                              relu=relu, transposed=transposed)
    return host(out, dtype)[:m_out]


@pytest.mark.parametrize("cin,cout,dtype,bn", [(32, 32, "bf16", False), (96, 96, "bf16", True),
                                               (96, 96, "f16", True), (16, 16, "f32", False), (4, 32, "bf16", True),
                                               (24, 48, "bf16", False), (128, 256, "bf16", True),
                                               (32, 64, "bf16", True), (64, 128, "f16", False),
                                               (128, 64, "bf16", True), (96, 32, "bf16", False),
                                               (128, 128, "bf16", True), (64, 96, "f16", True),
                                               (256, 256, "bf16", True), (192, 256, "f16", False),
                                               (128, 256, "f16", True), (256, 64, "bf16", False),
                                               (32, 256, "bf16", True)])
def test_conv_submanifold_sweep(spv, sweep, cin, cout, dtype, bn):
    rc, _, _, _ = oracle.voxelize(sweep[::3] if cout >= 256 else sweep, 0.05)
    _, off, pairs = oracle.kernel_map(rc)
    x = synth.normal((len(rc), cin), 1003, dtype=dtype)
    W = synth.conv_weight(27, cin, cout, 1004, dtype)
    sc, sh = synth.folded_bn(cout, 1005) if bn else (None, None)
    got = run_conv(spv, x, off, pairs, W, len(rc), dtype, sc, sh, bn)
    ref = oracle.sparse_conv(x, off, pairs, W, len(rc), dtype, sc, sh, bn)
    check_close(got, ref, dtype)


@pytest.mark.parametrize("c0,c1", [(64, 128), (256, 256)])
def test_conv_strided_and_transposed_sweep(spv, sweep, c0, c1):
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    oc, off, pairs = oracle.kernel_map(rc, 2, 2)
    x = synth.normal((len(rc), c0), 1006, dtype="bf16")
    W = synth.conv_weight(8, c0, c1, 1007, "bf16")
    got = run_conv(spv, x, off, pairs, W, len(oc), "bf16")
    ref = oracle.sparse_conv(x, off, pairs, W, len(oc), "bf16")
    check_close(got, ref, "bf16")
    WT = synth.conv_weight(8, c1, c0, 1008, "bf16")
    gotT = run_conv(spv, ref, off, pairs, WT, len(rc), "bf16", transposed=True)
    refT = oracle.sparse_conv(ref, off, pairs, WT, len(rc), "bf16", transposed=True)
    check_close(gotT, refT, "bf16")


@pytest.mark.parametrize("cin,cout,dtype", [(32, 64, "bf16"), (64, 128, "bf16"), (16, 16, "f32"), (96, 96, "f16")])
def test_conv_k3_stride2_and_transposed_sweep(spv, sweep, cin, cout, dtype):
    """Strided 3x3x3 conv on the K=3 stride-2 map (GPU-built, bit-exact against the
    oracle's map) and the transposed conv back onto the fine voxels."""
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    oc, off, pairs, _ = run_kmap(spv, rc, 3, 2)
    x = synth.normal((len(rc), cin), 1016, dtype=dtype)
    W = synth.conv_weight(27, cin, cout, 1017, dtype)
    sc, sh = synth.folded_bn(cout, 1018)
    got = run_conv(spv, x, off, pairs, W, len(oc), dtype, sc, sh, True)
    ref = oracle.sparse_conv(x, off, pairs, W, len(oc), dtype, sc, sh, True)
    check_close(got, ref, dtype)
    WT = synth.conv_weight(27, cout, cin, 1019, dtype)
    gotT = run_conv(spv, ref, off, pairs, WT, len(rc), dtype, transposed=True)
    refT = oracle.sparse_conv(ref, off, pairs, WT, len(rc), dtype, transposed=True)
    check_close(gotT, refT, dtype)


@pytest.mark.parametrize("K,full,cin,cout,dtype,transposed", [
    (3, (128, 128), 96, 64, "bf16", False),   # neighbour-table kernel
    (3, (128, 128), 64, 96, "f16", False),
    (3, (128, 128), 32, 32, "bf16", False),
    (3, (128, 128), 48, 80, "bf16", False),   # tile kernel (80 outputs)
    (3, (40, 24), 16, 24, "f32", False),      # vector ALU
    (2, (128, 128), 64, 96, "bf16", False),   # stride-2 tile kernel
    (2, (128, 96), 96, 48, "bf16", True),     # transposed
])
def test_conv_sliced_weights(spv, sweep, K, full, cin, cout, dtype, transposed):
    """Channel-sliced weight sharing (Sec. 4.2): a (cin, cout) candidate reads the first
    channels of the full weight tensor and BN vectors in place."""
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    if K == 3:
        _, off, pairs = oracle.kernel_map(rc)
        m_in = m_out = len(rc)
    else:
        oc, off, pairs = oracle.kernel_map(rc, 2, 2)
        m_in, m_out = (len(oc), len(rc)) if transposed else (len(rc), len(oc))
    Wf = synth.conv_weight(K ** 3, full[0], full[1], 1030, dtype)
    sc, sh = synth.folded_bn(full[1], 1031)
    x = synth.normal((m_in, cin), 1032, dtype=dtype)
    ws = spv.Workspace.for_ops(max(m_in, m_out), 128)
    got = spv.spv_sparse_conv_sliced(ws, dev(x, dtype), dev(off), dev(pairs), dev(Wf, dtype), cin, cout, m_out,
                                     scale=dev(sc), shift=dev(sh), relu=True, transposed=transposed)
    got = host(got, dtype)[:m_out]
    ref = oracle.sparse_conv_sliced(x, off, pairs, Wf, m_out, cout, dtype, sc, sh, True, transposed)
    check_close(got, ref, dtype)
    # the same layer from a dense copy of the slice, through spv_sparse_conv: identical bits
    Ws = np.ascontiguousarray(Wf[:, :cin, :cout])
    dense = spv.spv_sparse_conv(ws, dev(x, dtype), dev(off), dev(pairs), dev(Ws, dtype), m_out,
                                scale=dev(np.ascontiguousarray(sc[:cout])), shift=dev(np.ascontiguousarray(sh[:cout])),
                                relu=True, transposed=transposed)
    np.testing.assert_array_equal(got, host(dense, dtype)[:m_out])


def test_conv_sliced_rejects_wider_slice(spv):
    ws = spv.Workspace.for_ops(16, 32)
    c = np.array([[0, 0, 0, 0], [0, 0, 0, 1]], np.int32)
    _, off, pairs = oracle.kernel_map(c)
    Wf = np.zeros((27, 32, 32), np.float32)
    with pytest.raises(spv.SpvError) as e:
        spv.spv_sparse_conv_sliced(ws, dev(np.zeros((2, 32), np.float32)), dev(off), dev(pairs), dev(Wf), 32, 48, 2)
    assert e.value.status == spv.SPV_ERR_INVALID_ARG


@pytest.mark.parametrize("K,cin,cout,dtype", [(3, 32, 32, "bf16"), (3, 16, 16, "f32"), (2, 64, 128, "bf16")])
@pytest.mark.parametrize("defect", ["none", "swapped", "repeated"])
def test_conv_rejects_malformed_map(spv, K, cin, cout, dtype, defect):
    """A map whose offset group is out of output order, or holds one (output,
    offset) twice, is not a kernel map: the conv reports SPV_ERR_INVALID_ARG."""
    rng = np.random.default_rng(77)
    c = np.unique(rng.integers(-6, 6, size=(900, 3)), axis=0).astype(np.int32)
    rc = np.concatenate([np.zeros((len(c), 1), np.int32), c], axis=1)
    if K == 3:
        _, off, pairs = oracle.kernel_map(rc)
        m_out = len(rc)
    else:
        oc, off, pairs = oracle.kernel_map(rc, 2, 2)
        m_out = len(oc)
    pairs = pairs.copy()
    g = int(np.argmax(np.diff(off)))  # the largest offset group
    p = int(off[g]) + 5
    assert off[g + 1] - off[g] > 10
    if defect == "swapped":
        pairs[[p, p + 1]] = pairs[[p + 1, p]]
    elif defect == "repeated":
        pairs[p] = pairs[p - 1]
    x = synth.normal((len(rc), cin), 5, dtype=dtype)
    W = synth.conv_weight(K ** 3, cin, cout, 6, dtype)
    ws = spv.Workspace.for_ops(max(m_out, len(rc)), max(cin, cout))
    spv.spv_sparse_conv(ws, dev(x, dtype), dev(off), dev(pairs), dev(W, dtype), m_out)
    st = spv.spv_status_check(ws)
    assert st == (spv.SPV_OK if defect == "none" else spv.SPV_ERR_INVALID_ARG)


def test_conv_deterministic(spv, sweep):
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    _, off, pairs = oracle.kernel_map(rc)
    x = synth.normal((len(rc), 32), 11, dtype="bf16")
    W = synth.conv_weight(27, 32, 32, 12, "bf16")
    a = run_conv(spv, x, off, pairs, W, len(rc), "bf16")
    b = run_conv(spv, x, off, pairs, W, len(rc), "bf16")
    np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------------------
# devoxelization + point MLP + fusion
# ---------------------------------------------------------------------------
MODE_CODE = {"center": 0, "corner": 1, "nearest": 2}  # spv_devox_mode


@pytest.mark.parametrize("mode", ["center", "corner", "nearest"])
@pytest.mark.parametrize("dtype,C", [("bf16", 96), ("f32", 16), ("f16", 32)])
def test_devox_sweep(spv, sweep, mode, dtype, C):
    pts = sweep[::2]
    rc, _, _, _ = oracle.voxelize(pts, 0.05)
    vf = synth.normal((len(rc), C), 21, dtype=dtype)
    pf = synth.normal((len(pts), C), 22, dtype=dtype)
    Wp = synth.linear_weight(C, C, 23, dtype)
    sc, sh = synth.folded_bn(C, 24)
    ws = spv.Workspace.for_ops(len(pts), C)
    m = MODE_CODE[mode]
    out, ci, cw = spv.spv_devoxelize(ws, dev(rc), dev(vf, dtype), dev(pts), 0.05, mode=m, pfeat=dev(pf, dtype),
                                     Wp=dev(Wp, dtype), scale_p=dev(sc), shift_p=dev(sh), relu_p=True,
                                     want_corners=True)
    rout, rci, rcw = oracle.devoxelize(rc, vf, pts, 0.05, mode=mode, pfeat=pf, Wp=Wp, scale_p=sc, shift_p=sh,
                                       relu_p=True, dtype=dtype, want_corners=True)
    np.testing.assert_array_equal(host(ci)[:len(pts)], rci)
    np.testing.assert_array_equal(host(cw)[:len(pts)], rcw)
    check_close(host(out, dtype)[:len(pts)], rout, dtype)


@pytest.mark.parametrize("C,Cp,n", [(16, 0, 1000), (64, 24, 3001), (128, 128, 2047), (256, 96, 1500), (32, 8, 1),
                                    (256, 0, 5000), (256, 32, 4097), (256, 128, 3000), (256, 200, 999)])
def test_devox_shapes(spv, C, Cp, n):
    """Channel widths with and without a point branch, partial 32-channel slabs
    of the point MLP, widths past the matrix-core kernel and ragged point counts."""
    rng = np.random.default_rng(C + Cp + n)
    pts = rng.uniform(-1.0, 1.0, size=(n, 3)).astype(np.float32)
    rc, _, _, _ = oracle.voxelize(pts, 0.1)
    vf = synth.normal((len(rc), C), 31, dtype="bf16")
    pf = synth.normal((n, Cp), 32, dtype="bf16") if Cp else None
    Wp = synth.linear_weight(Cp, C, 33, "bf16") if Cp else None
    sc, sh = synth.folded_bn(C, 34)
    ws = spv.Workspace.for_ops(n, max(C, Cp))
    out = spv.spv_devoxelize(ws, dev(rc), dev(vf, "bf16"), dev(pts), 0.1,
                             pfeat=None if pf is None else dev(pf, "bf16"), Wp=None if Wp is None else dev(Wp, "bf16"),
                             scale_p=dev(sc) if Cp else None, shift_p=dev(sh) if Cp else None, relu_p=bool(Cp))
    ref = oracle.devoxelize(rc, vf, pts, 0.1, pfeat=pf, Wp=Wp, scale_p=sc if Cp else None,
                            shift_p=sh if Cp else None, relu_p=bool(Cp), dtype="bf16")
    check_close(host(out, "bf16")[:n], ref, "bf16")


@pytest.mark.parametrize("C", [32, 256])
def test_devox_coarse_grid(spv, sweep, C):
    pts = sweep[::4]
    rc, _, _, _ = oracle.voxelize(pts, 0.05)
    c1, _, _ = oracle.kernel_map(rc, 2, 2)
    c2, _, _ = oracle.kernel_map(c1, 2, 2)
    vf = synth.normal((len(c2), C), 31, dtype="bf16")
    ws = spv.Workspace.for_ops(len(pts), C)
    out = spv.spv_devoxelize(ws, dev(c2), dev(vf, "bf16"), dev(pts), 0.05, stride_log2=2)
    rout = oracle.devoxelize(c2, vf, pts, 0.05, stride_log2=2, dtype="bf16")
    check_close(host(out, "bf16")[:len(pts)], rout, "bf16")


# ---------------------------------------------------------------------------
# the SPVConv block
# ---------------------------------------------------------------------------
def block_inputs(cfg):
    if cfg == "tiny":
        xyz = synth.uniform_cube(2000, 1.6, 1001)
        C, dtype, v = 16, "f32", 0.1
        feat = synth.normal((2000, C), 1002, dtype=dtype)
        convs = [(synth.conv_weight(27, C, C, 1003, dtype), None, None, False)]
        Wp = synth.linear_weight(C, C, 1004, dtype)
        return xyz, feat, v, convs, Wp, None, None, dtype
    xyz = synth.lidar_sweep(1004)
    C, dtype, v = 96, "bf16", 0.05
    feat = synth.normal((len(xyz), C), 1005, dtype=dtype)
    convs = []
    for l in range(2):
        sc, sh = synth.folded_bn(C, 1010 + l)
        convs.append((synth.conv_weight(27, C, C, 1006 + l, dtype), sc, sh, True))
    Wp = synth.linear_weight(C, C, 1008, dtype)
    scp, shp = synth.folded_bn(C, 1009)
    return xyz, feat, v, convs, Wp, scp, shp, dtype


@pytest.mark.parametrize("cfg", ["tiny", "sweep_c96"])
def test_block(spv, cfg):
    xyz, feat, v, convs, Wp, scp, shp, dtype = block_inputs(cfg)
    C = feat.shape[1]
    dconvs = [(dev(W, dtype), None if sc is None else dev(sc), None if sh is None else dev(sh), r)
              for W, sc, sh, r in convs]
    dWp = dev(Wp, dtype)
    dscp = None if scp is None else dev(scp)
    dshp = None if shp is None else dev(shp)
    params = spv.make_block_params(C, TD[dtype], v, dconvs, dWp, dscp, dshp, relu_p=True)
    ws = spv.Workspace.for_block(len(xyz), C)
    out, m = spv.spv_block(ws, params, dev(xyz), dev(feat, dtype), sync=True)
    rout, rm = oracle.block(xyz, feat, v, convs, Wp, scp, shp, relu_p=True, dtype=dtype)
    assert m == rm
    check_close(host(out, dtype)[:len(xyz)], rout, dtype, kind="block")


@pytest.mark.parametrize("mode", ["center", "corner", "nearest"])
@pytest.mark.parametrize("C", [32, 96])
def test_block_equals_stand_alone_ops(spv, sweep, mode, C):
    """The block reads every point's interpolation corners from the kernel map's
    neighbour table; the stand-alone devoxelization probes the hash for them.
    Everything else runs the same kernels, so the block's output equals the
    stand-alone chain (voxelize, map, 2 convs, devoxelize + MLP) bit for bit;
    both agree with the oracle's block."""
    dt = "bf16"
    xyz = sweep
    feat = synth.normal((len(xyz), C), 71, dtype=dt)
    convs = []
    for l in range(2):
        sc, sh = synth.folded_bn(C, 72 + l)
        convs.append((synth.conv_weight(27, C, C, 74 + l, dt), sc, sh, True))
    Wp = synth.linear_weight(C, C, 76, dt)
    scp, shp = synth.folded_bn(C, 77)
    m_code = MODE_CODE[mode]
    dconvs = [(dev(W, dt), dev(sc), dev(sh), r) for W, sc, sh, r in convs]
    d_xyz, d_feat, d_Wp, d_scp, d_shp = dev(xyz), dev(feat, dt), dev(Wp, dt), dev(scp), dev(shp)
    params = spv.make_block_params(C, torch.bfloat16, 0.05, dconvs, d_Wp, d_scp, d_shp, relu_p=True, mode=m_code)
    out, m = spv.spv_block(spv.Workspace.for_block(len(xyz), C), params, d_xyz, d_feat, sync=True)
    # the same pipeline through the stand-alone entry points
    ws = spv.Workspace.for_ops(len(xyz), C)
    vox = spv.spv_voxelize(ws, d_xyz, 0.05, d_feat)
    assert vox.m == m
    coords = vox.coords[:m].contiguous()
    km = spv.spv_kernel_map(spv.Workspace.for_ops(len(xyz), C), coords)
    x = vox.vfeat[:m].contiguous()
    for W, sc, sh, r in dconvs:
        x = spv.spv_sparse_conv(spv.Workspace.for_ops(len(xyz), C), x, km.off, km.pairs, W, m, scale=sc, shift=sh,
                                relu=r)[:m].contiguous()
    ref = spv.spv_devoxelize(spv.Workspace.for_ops(len(xyz), C), coords, x, d_xyz, 0.05, mode=m_code, pfeat=d_feat,
                             Wp=d_Wp, scale_p=d_scp, shift_p=d_shp, relu_p=True)
    ref = ref[0] if isinstance(ref, tuple) else ref
    torch.cuda.synchronize()
    assert torch.equal(out[:len(xyz)].view(torch.int16), ref[:len(xyz)].view(torch.int16))
    rout, rm = oracle.block(xyz, feat, 0.05, convs, Wp, scp, shp, relu_p=True, dtype=dt, mode=mode)
    assert rm == m
    check_close(host(out, dt)[:len(xyz)], rout, dt, kind="block")


@pytest.mark.parametrize("C,dtype,nconv", [(16, "f32", 1), (16, "f32", 2), (48, "bf16", 2), (96, "bf16", 2)])
def test_block_residual(spv, sweep, C, dtype, nconv):
    """Residual blocks (Sec. 3.3): the last conv adds the block's voxel input
    before its ReLU -- through the vector-ALU (f32), tile (C = 48) and
    neighbour-table (C = 96) conv kernels -- against the oracle's residual block."""
    xyz = sweep[::2] if C != 96 else sweep
    v = 0.05
    feat = synth.normal((len(xyz), C), 81, dtype=dtype)
    convs = []
    for l in range(nconv):
        sc, sh = synth.folded_bn(C, 82 + l)
        convs.append((synth.conv_weight(27, C, C, 84 + l, dtype), sc, sh, True))
    Wp = synth.linear_weight(C, C, 86, dtype)
    dconvs = [(dev(W, dtype), dev(sc), dev(sh), r) for W, sc, sh, r in convs]
    params = spv.make_block_params(C, TD[dtype], v, dconvs, dev(Wp, dtype), None, None, relu_p=True, residual=True)
    ws = spv.Workspace.for_block(len(xyz), C)
    out, m = spv.spv_block(ws, params, dev(xyz), dev(feat, dtype), sync=True)
    rout, rm = oracle.block(xyz, feat, v, convs, Wp, relu_p=True, dtype=dtype, residual=True)
    assert m == rm
    got = host(out, dtype)[:len(xyz)]
    check_close(got, rout, dtype, kind="block")
    plain, _ = oracle.block(xyz, feat, v, convs, Wp, relu_p=True, dtype=dtype)
    diff = np.abs(synth.from_storage(rout, dtype) - synth.from_storage(plain, dtype)).max()
    assert diff > 0.05  # the identity branch matters here


def test_block_graph_replay(spv, sweep):
    """spv_block captured into a graph: every replay, with eager work and
    synchronization between them, reproduces the eager result bit for bit."""
    C = 32
    xyz = sweep
    feat = synth.normal((len(xyz), C), 61, dtype="bf16")
    convs = []
    for l in range(2):
        sc, sh = synth.folded_bn(C, 62 + l)
        convs.append((dev(synth.conv_weight(27, C, C, 64 + l, "bf16"), "bf16"), dev(sc), dev(sh), True))
    scp, shp = synth.folded_bn(C, 66)
    params = spv.make_block_params(C, torch.bfloat16, 0.05, convs, dev(synth.linear_weight(C, C, 67, "bf16"), "bf16"),
                                   dev(scp), dev(shp), relu_p=True)
    d_xyz, d_feat = dev(xyz), dev(feat, "bf16")
    ws = spv.Workspace.for_block(len(xyz), C)
    out = torch.empty((len(xyz), C), dtype=torch.bfloat16, device="cuda")
    spv.spv_block(ws, params, d_xyz, d_feat, out=out)
    torch.cuda.synchronize()
    ref = out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        spv.spv_block(ws, params, d_xyz, d_feat, out=out)
    torch.cuda.synchronize()
    scratch = torch.empty_like(out)
    for i in range(3):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"replay {i}"
        spv.spv_block(ws, params, d_xyz, d_feat, out=scratch)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(scratch.view(torch.int16), ref.view(torch.int16)), f"eager after replay {i}"


# ---------------------------------------------------------------------------
# pointwise linear layer and the split of a conv over concatenated inputs
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("cin,cout,dtype", [(32, 64, "bf16"), (96, 256, "bf16"), (256, 128, "f16"),
                                            (128, 96, "bf16"), (8, 16, "bf16"), (96, 19, "bf16"), (32, 7, "f16"),
                                            (96, 40, "bf16"), (12, 16, "bf16"), (40, 24, "f32")])
@pytest.mark.parametrize("mode", ["plain", "res_before", "res_after"])
def test_linear(spv, cin, cout, dtype, mode):
    """Rows past the live count (m_dev < m_cap) are left alone; 16-row blocks with a ragged tail."""
    m_cap, m = 20011, 19997
    x = synth.normal((m_cap, cin), 1040, dtype=dtype)
    W = synth.linear_weight(cin, cout, 1041, dtype)
    sc, sh = synth.folded_bn(cout, 1042)
    res = synth.normal((m_cap, cout), 1043, dtype=dtype) if mode != "plain" else None
    after = mode == "res_after"
    ws = spv.Workspace.for_ops(16, max(cin, cout))
    out = torch.full((m_cap, cout), 7.0, dtype=TD[dtype], device="cuda")
    spv.spv_linear(ws, dev(x, dtype), dev(W, dtype), m_dev=torch.tensor([m], dtype=torch.int64, device="cuda"),
                   scale=dev(sc), shift=dev(sh), relu=True, res=None if res is None else dev(res, dtype),
                   res_after_act=after, out=out)
    got = host(out, dtype)
    ref = oracle.linear(x[:m], W, dtype, sc, sh, True, None if res is None else res[:m], after)
    check_close(got[:m], ref, dtype)
    assert np.all(synth.from_storage(got[m:], dtype) == 7.0)


def test_linear_input_channel_offset(spv):
    """The rows cin_offset .. of a wider weight (one part of a concatenated input)."""
    x = synth.normal((5000, 64), 1044, dtype="bf16")
    W = synth.linear_weight(192, 128, 1045, "bf16")
    ws = spv.Workspace.for_ops(16, 192)
    got = host(spv.spv_linear(ws, dev(x, "bf16"), dev(W, "bf16"), cin_offset=128), "bf16")
    ref = oracle.linear(x, np.ascontiguousarray(W[128:]), "bf16")
    check_close(got, ref, "bf16")


@pytest.mark.parametrize("ca,cb,cout,transposed", [(96, 32, 96, False), (128, 64, 128, False),
                                                   (256, 128, 256, False), (64, 32, 64, True)])
def test_conv_concat_split(spv, sweep, ca, cb, cout, transposed):
    """A conv over the concatenation [a; b] (a decoder's skip connection) as two sliced convs,
    W_a a scaled into a residual and W_b b + shift + that residual, against the oracle's conv on
    the concatenated features with the full weight."""
    rc, _, _, _ = oracle.voxelize(sweep[::2], 0.05)
    if transposed:
        oc, off, pairs = oracle.kernel_map(rc, 2, 2)
        m_in, m_out, K3 = len(oc), len(rc), 8
    else:
        _, off, pairs = oracle.kernel_map(rc)
        m_in = m_out = len(rc)
        K3 = 27
    a = synth.normal((m_in, ca), 1046, dtype="bf16")
    b = synth.normal((m_in, cb), 1047, dtype="bf16")
    W = synth.conv_weight(K3, ca + cb, cout, 1048, "bf16")
    sc, sh = synth.folded_bn(cout, 1049)
    ref = oracle.sparse_conv(np.concatenate([a, b], 1), off, pairs, W, m_out, "bf16", sc, sh, True, transposed)
    ws = spv.Workspace.for_ops(max(m_in, m_out), 256)
    d_off, d_pairs, d_W = dev(off), dev(pairs), dev(W, "bf16")
    part = spv.spv_sparse_conv_sliced(ws, dev(a, "bf16"), d_off, d_pairs, d_W, ca, cout, m_out, scale=dev(sc),
                                      transposed=transposed)
    got = spv.spv_sparse_conv_sliced(ws, dev(b, "bf16"), d_off, d_pairs, d_W, cb, cout, m_out, scale=dev(sc),
                                     shift=dev(sh), relu=True, transposed=transposed, res=part, cin_offset=ca)
    check_close(host(got, "bf16")[:m_out], ref, "bf16")


# ---------------------------------------------------------------------------
# neighbour tables shared by several convs
# ---------------------------------------------------------------------------
def test_kernel_map_nbr_matches_pairs(spv, sweep):
    """nbr[j][k] = i + 1 exactly for the pairs (i, j, k) of the oracle's submanifold map."""
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    _, off, pairs = oracle.kernel_map(rc)
    ws = spv.Workspace.for_ops(len(rc), 16)
    got = host(spv.spv_kernel_map_nbr(ws, dev(rc)))[: len(rc)]
    want = np.zeros((len(rc), 27), np.int32)
    for k in range(27):
        p = pairs[off[k]:off[k + 1]]
        want[p[:, 1], k] = p[:, 0] + 1
    np.testing.assert_array_equal(got, want)


def test_kernel_map_nbr_shuffled_into_a_dirty_buffer(spv, sweep):
    """The table from half the probes (each pair found fills both rows) on coordinates in a
    shuffled order, a device count below the capacity, and an output buffer full of garbage:
    every entry of the live rows is written, rows past the count are left alone."""
    rc, _, _, _ = oracle.voxelize(sweep[::3], 0.05)
    perm = np.random.default_rng(77).permutation(len(rc))
    sc = np.ascontiguousarray(rc[perm])
    m = len(sc) - 123
    _, off, pairs = oracle.kernel_map(sc[:m])
    want = np.zeros((m, 27), np.int32)
    for k in range(27):
        p = pairs[off[k]:off[k + 1]]
        want[p[:, 1], k] = p[:, 0] + 1
    ws = spv.Workspace.for_ops(len(sc), 16)
    out = torch.full((len(sc), 27), -5, dtype=torch.int32, device="cuda")
    spv.spv_kernel_map_nbr(ws, dev(sc), m_dev=torch.tensor([m], dtype=torch.int64, device="cuda"), out=out)
    got = host(out)
    np.testing.assert_array_equal(got[:m], want)
    assert (got[m:] == -5).all()


@pytest.mark.parametrize("cin,cout,dtype,res", [(32, 32, "bf16", False), (96, 96, "bf16", True),
                                                (64, 128, "f16", True), (256, 256, "bf16", False)])
def test_conv_on_neighbour_table(spv, sweep, cin, cout, dtype, res):
    """The conv on a prebuilt table gives the bits of the conv planned from the pairs."""
    rc, _, _, _ = oracle.voxelize(sweep[::2] if cin == 256 else sweep, 0.05)
    _, off, pairs = oracle.kernel_map(rc)
    x = synth.normal((len(rc), cin), 1201, dtype=dtype)
    W = synth.conv_weight(27, cin, cout, 1202, dtype)
    sc, sh = synth.folded_bn(cout, 1203)
    r = synth.normal((len(rc), cout), 1204, dtype=dtype) if res else None
    ws = spv.Workspace.for_ops(len(rc), max(cin, cout))
    nbr = spv.spv_kernel_map_nbr(ws, dev(rc))
    got = spv.spv_sparse_conv_nbr(ws, dev(x, dtype), nbr, dev(W, dtype), cout, len(rc), scale=dev(sc),
                                  shift=dev(sh), relu=True, res=None if r is None else dev(r, dtype))
    want = spv.spv_sparse_conv_sliced(ws, dev(x, dtype), dev(off), dev(pairs), dev(W, dtype), cin, cout, len(rc),
                                      scale=dev(sc), shift=dev(sh), relu=True, res=None if r is None else dev(r, dtype))
    np.testing.assert_array_equal(host(got, dtype)[: len(rc)], host(want, dtype)[: len(rc)])
    ref = oracle.sparse_conv(x, off, pairs, W, len(rc), dtype, sc, sh, True, res=r)
    check_close(host(got, dtype)[: len(rc)], ref, dtype)


def test_conv_on_neighbour_table_rejects_other_shapes(spv):
    ws = spv.Workspace.for_ops(16, 48)
    x = torch.zeros((4, 48), dtype=torch.bfloat16, device="cuda")
    nbr = torch.zeros((4, 27), dtype=torch.int32, device="cuda")
    W = torch.zeros((27, 48, 48), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(spv.SpvError) as e:
        spv.spv_sparse_conv_nbr(ws, x, nbr, W, 48, 4)
    assert e.value.status == spv.SPV_ERR_UNSUPPORTED


# ---------------------------------------------------------------------------
# the transposed k=2 s=2 conv on the child table
# ---------------------------------------------------------------------------
def test_map_children_matches_pairs(spv, sweep):
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    oc, off, pairs = oracle.kernel_map(rc, 2, 2)
    ws = spv.Workspace.for_ops(len(rc), 16)
    got = host(spv.spv_map_children(ws, dev(off), dev(pairs), len(rc), len(oc)))[: len(oc)]
    want = np.zeros((len(oc), 8), np.int32)
    for k in range(8):
        p = pairs[off[k]:off[k + 1]]
        want[p[:, 1], k] = p[:, 0] + 1
    np.testing.assert_array_equal(got, want)
    assert spv.spv_status_check(ws) == spv.SPV_OK


@pytest.mark.parametrize("cin,cout,dtype,res", [(128, 64, "bf16", False), (96, 96, "bf16", True),
                                                (256, 128, "f16", False), (256, 256, "bf16", True),
                                                (32, 96, "bf16", False)])
def test_conv_up(spv, sweep, cin, cout, dtype, res):
    """The child-table upsampling conv equals the transposed conv on the pairs (every fine
    voxel has its parent), against the oracle."""
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    oc, off, pairs = oracle.kernel_map(rc, 2, 2)
    x = synth.normal((len(oc), cin), 1301, dtype=dtype)
    W = synth.conv_weight(8, cin, cout, 1302, dtype)
    sc, sh = synth.folded_bn(cout, 1303)
    r = synth.normal((len(rc), cout), 1304, dtype=dtype) if res else None
    ws = spv.Workspace.for_ops(len(rc), max(cin, cout))
    ch = spv.spv_map_children(ws, dev(off), dev(pairs), len(rc), len(oc))
    out = torch.full((len(rc), cout), 7.0, dtype=TD[dtype], device="cuda")
    spv.spv_sparse_conv_up(ws, dev(x, dtype), ch, dev(W, dtype), cout, len(rc), scale=dev(sc), shift=dev(sh),
                           relu=True, res=None if r is None else dev(r, dtype), out=out)
    got = host(out, dtype)
    ref = oracle.sparse_conv(x, off, pairs, W, len(rc), dtype, sc, sh, True, transposed=True, res=r)
    check_close(got, ref, dtype)


def test_conv_up_rejects_other_shapes(spv):
    ws = spv.Workspace.for_ops(16, 48)
    x = torch.zeros((4, 48), dtype=torch.bfloat16, device="cuda")
    ch = torch.zeros((4, 8), dtype=torch.int32, device="cuda")
    W = torch.zeros((8, 48, 48), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(spv.SpvError) as e:
        spv.spv_sparse_conv_up(ws, x, ch, W, 48, 4)
    assert e.value.status == spv.SPV_ERR_UNSUPPORTED


# ---------------------------------------------------------------------------
# devoxelization with corners from the neighbour table
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("C,Cp,s,mode", [(96, 96, 0, "center"), (96, 0, 0, "corner"), (256, 32, 0, "center"),
                                         (64, 64, 2, "center"), (32, 32, 2, "nearest")])
def test_devoxelize_nbr_matches_hash(spv, sweep, C, Cp, s, mode):
    """On the points' own voxelization at stride 2^s, corners read from the neighbour table give
    the hash-table devoxelization's outputs bit for bit; against the oracle as well."""
    from paper_2007_16100_amd.spvcnn import voxel_size_at
    dt, v = "bf16", 0.05
    md = {"center": spv.SPV_DEVOX_CENTER, "corner": spv.SPV_DEVOX_CORNER, "nearest": spv.SPV_DEVOX_NEAREST}[mode]
    ws = spv.Workspace.for_ops(len(sweep), 256)
    xyz = dev(sweep)
    vox = spv.spv_voxelize(ws, xyz, voxel_size_at(v, s))
    m = vox.m
    coords = vox.coords[:m]
    nbr = spv.spv_kernel_map_nbr(ws, coords)
    vf = synth.normal((m, C), 1501, dtype=dt)
    kw = {}
    if Cp:
        kw = dict(pfeat=dev(synth.normal((len(sweep), Cp), 1502, dtype=dt), dt),
                  Wp=dev(synth.linear_weight(Cp, C, 1503, dt), dt), relu_p=True)
        kw["scale_p"], kw["shift_p"] = (dev(a) for a in synth.folded_bn(C, 1504))
    a = spv.spv_devoxelize(ws, coords, dev(vf, dt), xyz, v, s, md, **kw)
    b = spv.spv_devoxelize_nbr(ws, coords, dev(vf, dt), nbr, vox.pt2vox, xyz, v, s, md, **kw)
    torch.cuda.synchronize()
    assert spv.spv_status_check(ws) == spv.SPV_OK
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    if not Cp:
        ref = oracle.devoxelize(host(coords), vf, sweep, v, s, mode, dtype=dt)
        check_close(host(b, dt)[: len(sweep)], ref, dt)


def test_devoxelize_nbr_bad_voxel_index(spv):
    """A pt2vox entry outside the grid gives the point no corners (no read outside the table)."""
    d = "cuda"
    xyz = torch.tensor([[0.01, 0.01, 0.01], [0.06, 0.01, 0.01]], dtype=torch.float32, device=d)
    ws = spv.Workspace.for_ops(16, 32)
    vox = spv.spv_voxelize(ws, xyz, 0.05)
    coords = vox.coords[: vox.m]
    nbr = spv.spv_kernel_map_nbr(ws, coords)
    vf = torch.ones((vox.m, 32), dtype=torch.bfloat16, device=d)
    p2v = vox.pt2vox.clone()
    p2v[0] = 1000
    out = spv.spv_devoxelize_nbr(ws, coords, vf, nbr, p2v, xyz, 0.05)
    torch.cuda.synchronize()
    assert float(out[0].float().abs().max()) == 0.0 and float(out[1, 0]) == 1.0
    # a live row count below the capacity: an entry past it (a row the map did not
    # write) gives no corners either
    assert vox.m == 2
    p2v = vox.pt2vox.clone()
    m_dev = torch.tensor([1], dtype=torch.int64, device=d)
    coords_cap = torch.cat([coords, torch.zeros((6, 4), dtype=torch.int32, device=d)]).contiguous()
    nbr_cap = torch.cat([nbr[: vox.m], torch.full((6, 27), 7, dtype=torch.int32, device=d)]).contiguous()
    vf_cap = torch.ones((8, 32), dtype=torch.bfloat16, device=d)
    out = spv.spv_devoxelize_nbr(ws, coords_cap, vf_cap, nbr_cap, p2v, xyz, 0.05, m_dev=m_dev, m_cap=8)
    torch.cuda.synchronize()
    row = int(p2v[1])
    assert row >= 1  # the second point's voxel is past the live count
    assert float(out[1].float().abs().max()) == 0.0


# ---------------------------------------------------------------------------
# pre-packed weights
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("cin,cout,coff", [(96, 96, 0), (256, 256, 0), (32, 64, 32), (128, 96, 64), (64, 256, 0)])
def test_packed_weights_match_unpacked(spv, sweep, cin, cout, coff):
    """Weights packed once give the unpacked calls' outputs bit for bit: the neighbour-table
    conv and the upsampling conv (on an input-channel slice at offset coff), and the linear layer."""
    dt = "bf16"
    rc, _, _, _ = oracle.voxelize(sweep, 0.05)
    oc, off, pairs = oracle.kernel_map(rc, 2, 2)
    ws = spv.Workspace.for_ops(len(rc), 256)
    sc, sh = (dev(a) for a in synth.folded_bn(cout, 1403))
    r = dev(synth.normal((len(rc), cout), 1404, dtype=dt), dt)
    # neighbour-table conv
    nbr = spv.spv_kernel_map_nbr(ws, dev(rc))
    x = dev(synth.normal((len(rc), cin), 1401, dtype=dt), dt)
    W = dev(synth.conv_weight(27, cin + coff, cout, 1402, dt), dt)
    a = spv.spv_sparse_conv_nbr(ws, x, nbr, W, cout, len(rc), scale=sc, shift=sh, relu=True, res=r, cin_offset=coff)
    wp = spv.spv_pack_weights(W, cin, cout, coff)
    assert wp.numel() == spv.lib().spv_packed_weights_bytes(27, cin, cout)
    b = spv.spv_sparse_conv_nbr_packed(ws, x, nbr, wp, cout, len(rc), scale=sc, shift=sh, relu=True, res=r)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # upsampling conv on the stride-2 map's child table
    ch = spv.spv_map_children(ws, dev(off), dev(pairs), len(rc), len(oc))
    x2 = dev(synth.normal((len(oc), cin), 1405, dtype=dt), dt)
    W8 = dev(synth.conv_weight(8, cin + coff, cout, 1406, dt), dt)
    a = spv.spv_sparse_conv_up(ws, x2, ch, W8, cout, len(rc), scale=sc, shift=sh, relu=True, res=r, cin_offset=coff)
    b = spv.spv_sparse_conv_up_packed(ws, x2, ch, spv.spv_pack_weights(W8, cin, cout, coff), cout, len(rc), scale=sc,
                                      shift=sh, relu=True, res=r)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # linear layer, and the ragged classifier width
    for co in (cout, 19):
        W1 = dev(synth.linear_weight(cin + coff, co, 1407, dt), dt)
        sc1, sh1 = (dev(v) for v in synth.folded_bn(co, 1408))
        a = spv.spv_linear(ws, x, W1, scale=sc1, shift=sh1, relu=True, cin_offset=coff)
        b = spv.spv_linear_packed(ws, x, spv.spv_pack_weights(W1, cin, co, coff), co, scale=sc1, shift=sh1, relu=True)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    torch.cuda.synchronize()
    assert spv.spv_status_check(ws) == spv.SPV_OK


def test_calls_without_device_errors_keep_the_status_word(spv):
    """The linear layer, the upsampling conv (plain and packed) and the weight gradient record
    no device errors and keep their weights and partial sums clear of the status word: a
    pending error of an earlier call on the same workspace survives them."""
    d, bf = "cuda", torch.bfloat16
    ws = spv.Workspace.for_ops(64, 64)
    spv.spv_voxelize(ws, torch.tensor([[1e6, 0.0, 0.0]], dtype=torch.float32, device=d), 0.05, sync=False)
    x = torch.ones((16, 32), dtype=bf, device=d)
    W = torch.ones((32, 32), dtype=bf, device=d)
    W8 = torch.ones((8, 32, 32), dtype=bf, device=d)
    ch = torch.zeros((16, 8), dtype=torch.int32, device=d)
    spv.spv_linear(ws, x, W)
    spv.spv_linear_packed(ws, x, spv.spv_pack_weights(W), 32)
    spv.spv_sparse_conv_up(ws, x, ch, W8, 32, 16)
    spv.spv_sparse_conv_up_packed(ws, x, ch, spv.spv_pack_weights(W8), 32, 16)
    torch.cuda.synchronize()
    assert spv.spv_status_check(ws) == spv.SPV_ERR_RANGE
    wsw = spv.Workspace.for_wgrad(27, 32, 32)
    wsw.buf.zero_()
    off = torch.ones(28, dtype=torch.int32, device=d)
    off[0] = 0
    pairs = torch.zeros((1, 2), dtype=torch.int32, device=d)
    dW = spv.spv_sparse_conv_wgrad(wsw, x, x, off, pairs, 27)
    assert float(dW[0, 0, 0]) == 1.0
    assert spv.spv_status_check(wsw) == spv.SPV_OK


# ---------------------------------------------------------------------------
# empty inputs of the later entry points
# ---------------------------------------------------------------------------
def test_empty_inputs_of_network_entry_points(spv):
    """Zero rows: every entry point returns SPV_OK and writes nothing it should not; the
    weight gradient of an empty map is zero, the devox gradient of no points is zero."""
    d = "cuda"
    ws = spv.Workspace.for_ops(16, 64)
    ws.buf.fill_(3)  # a stale status word: the calls that record device errors clear it
    e32 = torch.zeros((0, 32), dtype=torch.bfloat16, device=d)
    W = torch.ones((32, 32), dtype=torch.bfloat16, device=d)
    out = spv.spv_linear(ws, e32, W)
    assert out.shape[0] == 1  # capacity floor of the binding; nothing to compute
    nbr = spv.spv_kernel_map_nbr(ws, torch.zeros((0, 4), dtype=torch.int32, device=d))
    assert nbr.shape == (1, 27)
    W27 = torch.ones((27, 32, 32), dtype=torch.bfloat16, device=d)
    spv.spv_sparse_conv_nbr(ws, e32, nbr, W27, 32, 0)
    W8 = torch.ones((8, 32, 32), dtype=torch.bfloat16, device=d)
    ch = torch.zeros((1, 8), dtype=torch.int32, device=d)
    spv.spv_sparse_conv_up(ws, e32, ch, W8, 32, 0)
    off = torch.zeros(28, dtype=torch.int32, device=d)
    pairs = torch.zeros((1, 2), dtype=torch.int32, device=d)
    wsw = spv.Workspace.for_wgrad(27, 32, 32)
    dW = spv.spv_sparse_conv_wgrad(wsw, torch.zeros((4, 32), dtype=torch.bfloat16, device=d),
                                   torch.zeros((4, 32), dtype=torch.bfloat16, device=d), off, pairs, 27)
    assert torch.count_nonzero(dW).item() == 0
    dv = spv.spv_devoxelize_backward(spv.Workspace.for_devox_backward(0, 5),
                                     torch.zeros((0, 8), dtype=torch.int32, device=d),
                                     torch.zeros((0, 8), dtype=torch.float32, device=d),
                                     torch.zeros((0, 16), dtype=torch.bfloat16, device=d), 5,
                                     out=torch.full((5, 16), 3.0, dtype=torch.float32, device=d))
    assert torch.count_nonzero(dv).item() == 0
    spv.spv_voxelize_backward(torch.zeros((3, 16), dtype=torch.bfloat16, device=d),
                              torch.ones(3, dtype=torch.int32, device=d), torch.zeros(0, dtype=torch.int32, device=d),
                              3)
    torch.cuda.synchronize()
    assert spv.spv_status_check(ws) == spv.SPV_OK
    # the other empty calls that record device errors clear a stale status word too
    off9 = torch.zeros(9, dtype=torch.int32, device=d)
    for call in (lambda: spv.spv_map_children(ws, off9, pairs, 0, 0),
                 lambda: spv.spv_sparse_conv(ws, e32, off, pairs, W27, 0),
                 lambda: spv.spv_voxelize_onto(ws, torch.zeros((0, 4), dtype=torch.int32, device=d),
                                               torch.zeros((0, 3), dtype=torch.float32, device=d), 0.1)):
        ws.buf.fill_(3)
        call()
        assert spv.spv_status_check(ws) == spv.SPV_OK
