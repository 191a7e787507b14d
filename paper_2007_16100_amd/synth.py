"""Seeded synthetic inputs shared by the HIP path, the oracle, the tests and the bench.

This module holds no arithmetic of the SPVConv method itself (no voxelization,
no kernel map, no convolution, no interpolation).  It only draws inputs:

* ``uniform_cube``   -- points uniform in an axis-aligned cube (the tiny block).
* ``lidar_sweep``    -- a 64-beam spinning-LiDAR sweep over a ground plane with
  40 boxes / vertical cylinders, the stand-in for a SemanticKITTI scan
  (roughly 1e5 returns per scan, Sec. 3.3 "Sparse Voxelization" and Sec. 5.1).
* ``normal_bf16`` / ``weights`` -- features and layer parameters.

Every generator takes an explicit seed and uses ``numpy.random.default_rng``.
Low-precision storage values are produced as raw 16-bit patterns so both sides
read exactly the same bits.
"""
from __future__ import annotations

import math

import numpy as np

# ---------------------------------------------------------------------------
# 16-bit storage helpers (input preparation only)
# ---------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def f16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(b, dtype=np.uint16).view(np.float16).astype(np.float32)


DTYPES = ("f32", "bf16", "f16")


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """float32 array -> storage array (float32 or uint16 bit patterns)."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f16":
        return f32_to_f16_bits(x)
    raise ValueError(dtype)


def from_storage(b: np.ndarray, dtype: str) -> np.ndarray:
    """storage array -> float32 values (exact)."""
    if dtype == "f32":
        return np.ascontiguousarray(b, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_to_f32(b)
    if dtype == "f16":
        return f16_bits_to_f32(b)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# point clouds
# ---------------------------------------------------------------------------


def uniform_cube(n: int, half: float, seed: int) -> np.ndarray:
    """n points uniform in [-half, half)^3, float32 [n][3]."""
    rng = np.random.default_rng(seed)
    return rng.uniform(-half, half, size=(n, 3)).astype(np.float32)


def _ray_box(d, c, L, W, H, yaw, z0):
    """Distance along unit rays d[N,3] (origin at 0) to a yawed box; inf where missed."""
    cy, sy = math.cos(yaw), math.sin(yaw)
    # box frame: rotate by -yaw about z, translate by -centre
    ox, oy = -c[0], -c[1]
    o = np.array([cy * ox + sy * oy, -sy * ox + cy * oy, -(z0 + H / 2.0)])
    dl = np.stack([cy * d[:, 0] + sy * d[:, 1], -sy * d[:, 0] + cy * d[:, 1], d[:, 2]], axis=1)
    half = np.array([L / 2.0, W / 2.0, H / 2.0])
    with np.errstate(divide="ignore", invalid="ignore"):
        inv = 1.0 / dl
        t1 = (-half - o) * inv
        t2 = (half - o) * inv
    tmin = np.nanmax(np.minimum(t1, t2), axis=1)
    tmax = np.nanmin(np.maximum(t1, t2), axis=1)
    hit = (tmax >= tmin) & (tmax > 0)
    t = np.where(tmin > 0, tmin, np.inf)
    return np.where(hit, t, np.inf)


def _ray_cyl(d, c, r, H, z0):
    """Distance along unit rays to a vertical solid cylinder (side + top cap)."""
    ox, oy = -c[0], -c[1]
    a = d[:, 0] ** 2 + d[:, 1] ** 2
    b = 2.0 * (ox * d[:, 0] + oy * d[:, 1])
    cc = ox * ox + oy * oy - r * r
    disc = b * b - 4 * a * cc
    with np.errstate(invalid="ignore", divide="ignore"):
        sq = np.sqrt(np.maximum(disc, 0.0))
        t_side = (-b - sq) / (2 * a)
    z = t_side * d[:, 2]
    side_ok = (disc >= 0) & (t_side > 0) & (z >= z0) & (z <= z0 + H)
    t = np.where(side_ok, t_side, np.inf)
    with np.errstate(invalid="ignore", divide="ignore"):
        t_top = (z0 + H) / d[:, 2]
    px = t_top * d[:, 0] - c[0]
    py = t_top * d[:, 1] - c[1]
    top_ok = (t_top > 0) & (px * px + py * py <= r * r)
    return np.minimum(t, np.where(top_ok, t_top, np.inf))


def lidar_sweep(seed: int, n_beams: int = 64, n_azimuth: int = 2048,
                elev_lo_deg: float = -25.0, elev_hi_deg: float = 3.0,
                ground_z: float = -1.7, n_objects: int = 40,
                max_range: float = 100.0, range_noise: float = 0.02) -> np.ndarray:
    """A synthetic spinning-LiDAR sweep, float32 [n][3] (sensor at the origin).

    64 elevations evenly spaced in [-25, +3] degrees x 2048 azimuths; the scene is
    a ground plane at z = -1.7 m plus 40 objects (half yawed boxes with sides
    U(1,5) m, half vertical cylinders with radius U(0.5,2.5) m, height U(1,5) m)
    standing on the ground with centres at radius U(5,50) m.  Each ray returns its
    nearest hit within 100 m, with N(0, 2 cm) range noise.
    """
    rng = np.random.default_rng(seed)
    el = np.deg2rad(elev_lo_deg + np.arange(n_beams) * (elev_hi_deg - elev_lo_deg) / (n_beams - 1))
    az = np.deg2rad(np.arange(n_azimuth) * 360.0 / n_azimuth)
    E, A = np.meshgrid(el, az, indexing="ij")
    d = np.stack([np.cos(E) * np.cos(A), np.cos(E) * np.sin(A), np.sin(E)], axis=-1).reshape(-1, 3)
    t = np.full(d.shape[0], np.inf)
    down = d[:, 2] < 0
    t[down] = ground_z / d[down, 2]
    for i in range(n_objects):
        rad = rng.uniform(5.0, 50.0)
        phi = rng.uniform(0.0, 2 * math.pi)
        c = (rad * math.cos(phi), rad * math.sin(phi))
        if i % 2 == 0:
            L, W, H = rng.uniform(1.0, 5.0, size=3)
            yaw = rng.uniform(0.0, math.pi)
            t = np.minimum(t, _ray_box(d, c, L, W, H, yaw, ground_z))
        else:
            r = rng.uniform(0.5, 2.5)
            H = rng.uniform(1.0, 5.0)
            t = np.minimum(t, _ray_cyl(d, c, r, H, ground_z))
    keep = t <= max_range
    t = t[keep] + rng.normal(0.0, range_noise, size=int(keep.sum()))
    return (d[keep] * t[:, None]).astype(np.float32)


# ---------------------------------------------------------------------------
# features and parameters
# ---------------------------------------------------------------------------


def normal(shape, seed: int, std: float = 1.0, dtype: str = "f32") -> np.ndarray:
    """N(0, std^2) values in the given storage dtype (float32 or uint16 bits)."""
    rng = np.random.default_rng(seed)
    return to_storage(rng.normal(0.0, std, size=shape).astype(np.float32), dtype)


def conv_weight(K3: int, cin: int, cout: int, seed: int, dtype: str) -> np.ndarray:
    """Conv weights [K3][cin][cout] ~ N(0, std 1/sqrt(K3*cin)) (fan-in scaling)."""
    return normal((K3, cin, cout), seed, std=1.0 / math.sqrt(K3 * cin), dtype=dtype)


def linear_weight(cin: int, cout: int, seed: int, dtype: str) -> np.ndarray:
    """Point-MLP weights [cin][cout] ~ N(0, std 1/sqrt(cin))."""
    return normal((cin, cout), seed, std=1.0 / math.sqrt(cin), dtype=dtype)


def folded_bn(c: int, seed: int):
    """Inference-form BatchNorm as per-channel (scale, shift), float32: U(0.5,1.5), N(0,0.1)."""
    rng = np.random.default_rng(seed)
    scale = rng.uniform(0.5, 1.5, size=c).astype(np.float32)
    shift = rng.normal(0.0, 0.1, size=c).astype(np.float32)
    return scale, shift


# ---------------------------------------------------------------------------
# an SPVCNN-style network: point features and random-init parameters
# ---------------------------------------------------------------------------
# channel widths: stem, four encoder stages, four decoder stages
SPVCNN_WIDTHS = (32, 32, 64, 128, 256, 256, 128, 96, 96)
SPVCNN_IN = 4        # x, y, z, intensity
SPVCNN_CLASSES = 19


def point_features(xyz: np.ndarray, seed: int, dtype: str = "f32") -> np.ndarray:
    """Per-point input features [n][4]: the coordinates and an intensity ~ U(0, 1)."""
    rng = np.random.default_rng(seed)
    f = np.concatenate([np.asarray(xyz, np.float32), rng.uniform(0.0, 1.0, (len(xyz), 1)).astype(np.float32)], 1)
    return to_storage(f, dtype)


def spvcnn_params(seed: int, dtype: str, widths=SPVCNN_WIDTHS, c_in: int = SPVCNN_IN,
                  classes: int = SPVCNN_CLASSES) -> dict:
    """Random-init parameters by layer name; each entry is (W, scale, shift), scale / shift the
    folded BatchNorm of that layer (the classifier's scale is None and its shift is the bias).

    stem.0 / stem.1      3x3x3 convs c_in -> w0 -> w0
    down.s               2x2x2 stride-2 conv w[s-1] -> w[s-1]               (s = 1..4)
    enc.s.r.{a,b,sc}     residual block r of stage s (r = 0: w[s-1] -> w[s], r = 1: w[s] -> w[s]);
                         a, b: 3x3x3 convs; sc: 1x1 shortcut when the width changes
    up.u                 2x2x2 transposed conv w[3+u] -> w[4+u]             (u = 1..4)
    dec.u.r.{a,b,sc}     residual blocks after the skip concatenation [up output; encoder x_{4-u}]
                         (r = 0: w[4+u] + w[4-u] -> w[4+u], r = 1: w[4+u] -> w[4+u])
    point.0 .. point.3   point-branch MLPs c_in -> w0, w0 -> w4, w4 -> w6, w6 -> w8
    head                 linear w8 -> classes with a bias
    """
    w = widths
    P = {}
    sd = [seed]

    def nxt():
        sd[0] += 1
        return sd[0]

    def conv(name, K3, cin, cout):
        P[name] = (conv_weight(K3, cin, cout, nxt(), dtype),) + folded_bn(cout, nxt())

    def lin(name, cin, cout):
        P[name] = (linear_weight(cin, cout, nxt(), dtype),) + folded_bn(cout, nxt())

    def res(name, cin, cout):
        conv(name + ".a", 27, cin, cout)
        conv(name + ".b", 27, cout, cout)
        if cin != cout:
            lin(name + ".sc", cin, cout)

    conv("stem.0", 27, c_in, w[0])
    conv("stem.1", 27, w[0], w[0])
    for s in range(1, 5):
        conv(f"down.{s}", 8, w[s - 1], w[s - 1])
        res(f"enc.{s}.0", w[s - 1], w[s])
        res(f"enc.{s}.1", w[s], w[s])
    for u in range(1, 5):
        conv(f"up.{u}", 8, w[3 + u], w[4 + u])
        res(f"dec.{u}.0", w[4 + u] + w[4 - u], w[4 + u])
        res(f"dec.{u}.1", w[4 + u], w[4 + u])
    for i, (cin, cout) in enumerate([(c_in, w[0]), (w[0], w[4]), (w[4], w[6]), (w[6], w[8])]):
        lin(f"point.{i}", cin, cout)
    rng = np.random.default_rng(nxt())
    P["head"] = (linear_weight(w[8], classes, nxt(), dtype), None,
                 rng.normal(0.0, 0.1, size=classes).astype(np.float32))
    return P
