"""Kernel-map statistics and the MAC model of Sec. 4.3 (host-side bookkeeping).

Pins: a fully occupied L^3 block has |map_k| = prod over axes of (L - |delta|)
(closed form); a submanifold map's centre offset holds every voxel and
mirrored offsets have equal sizes; the per-offset sizes sum to the pair count;
the MAC sum equals pairs * C_in * C_out counted pair by pair."""
import numpy as np
import pytest

import oracle
from paper_2007_16100_amd import mapstats, synth


def _block_coords(L):
    g = np.stack(np.meshgrid(np.arange(L), np.arange(L), np.arange(L), indexing="ij"), -1).reshape(-1, 3)
    return np.concatenate([np.zeros((len(g), 1), np.int32), g.astype(np.int32)], 1)


@pytest.mark.parametrize("L", [2, 3, 5])
def test_dense_block_closed_form(oracle_lib, L):
    _, off, _ = oracle.kernel_map(_block_coords(L))
    got = mapstats.map_sizes(off)
    want = []
    for k in range(27):
        d = (k // 9 - 1, (k // 3) % 3 - 1, k % 3 - 1)
        want.append(np.prod([max(L - abs(x), 0) for x in d]))
    np.testing.assert_array_equal(got, want)


def test_submanifold_invariants_and_average(oracle_lib):
    stats = mapstats.MapStats()
    per_scan = []
    for seed in (3, 4, 5):
        rng = np.random.default_rng(seed)
        pts = np.unique(np.concatenate([np.zeros((900, 1)), rng.integers(-7, 7, (900, 3))], 1), axis=0).astype(np.int32)
        _, off, pairs = oracle.kernel_map(pts)
        s = stats.add("s1k3", off)
        per_scan.append(s)
        assert s[13] == len(pts)                      # centre: every voxel with itself
        np.testing.assert_array_equal(s, s[::-1])     # offset k and its mirror 26 - k
        assert s.sum() == len(pairs)
    np.testing.assert_allclose(stats.mean("s1k3"), np.mean(per_scan, axis=0))


def test_strided_map_sizes(oracle_lib):
    rng = np.random.default_rng(9)
    pts = np.unique(np.concatenate([rng.integers(0, 2, (1500, 1)), rng.integers(-9, 9, (1500, 3))], 1),
                    axis=0).astype(np.int32)
    _, off, pairs = oracle.kernel_map(pts, 2, 2)
    s = mapstats.map_sizes(off)
    assert s.size == 8 and s.sum() == len(pts) == len(pairs)  # every input in exactly one pair
    parity = ((pts[:, 1] & 1) << 2) | ((pts[:, 2] & 1) << 1) | (pts[:, 3] & 1)
    np.testing.assert_array_equal(s, np.bincount(parity, minlength=8))


def test_conv_macs_counts_pairs(oracle_lib):
    xyz = synth.uniform_cube(2500, 1.6, 21)
    rc, _, _, _ = oracle.voxelize(xyz, 0.1)
    _, off1, pairs1 = oracle.kernel_map(rc)
    _, off2, pairs2 = oracle.kernel_map(rc, 2, 2)
    stats = mapstats.MapStats()
    stats.add("s1k3", off1)
    stats.add("s2k2", off2)
    layers = [("s1k3", 4, 32), ("s1k3", 32, 32), ("s2k2", 32, 64)]
    total, per = mapstats.conv_macs(layers, stats)
    brute = [len(pairs1) * 4 * 32, len(pairs1) * 32 * 32, len(pairs2) * 32 * 64]
    assert per == [float(b) for b in brute]
    assert total == float(sum(brute))
    assert mapstats.flops_of_map(off1, 32, 32) == 2.0 * 32 * 32 * len(pairs1)


def test_rejects_bad_offsets():
    with pytest.raises(ValueError):
        mapstats.map_sizes(np.array([0, 5, 3], np.int32))
    with pytest.raises(ValueError):
        mapstats.map_sizes(np.array([0], np.int32))
    st = mapstats.MapStats()
    st.add("a", np.array([0, 1, 2]))
    with pytest.raises(ValueError):
        st.add("a", np.array([0, 1, 2, 3]))
    with pytest.raises(KeyError):
        st.mean("b")
