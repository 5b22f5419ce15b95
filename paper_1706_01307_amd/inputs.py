"""Seeded synthetic inputs: active-site sets, features, weights and biases.

This module produces inputs only.  It holds none of the convolution's
arithmetic (no rulebook, no neighbour search, no multiply-add), so both the
HIP path and the CPU oracle can be fed from it without sharing any of the
method.

Two families of site sets stand in for the paper's two datasets (neither is
available here; no item of either dataset is reproduced):

* pen strokes on a 2-D grid, standing in for the online handwriting dataset of
  the experiments section (64x64 grids, "about 8% of the pixels are active");
* thin voxelised surfaces in a 3-D grid, standing in for the rendered CAD
  surfaces of the same section (a 1-voxel-thick surface, 1.3% active at 32^3
  in the related-work example).

Every generator is deterministic in its seed.  Rows come out in lexicographic
order of (sample, x1, ..., xd), i.e. ``numpy.argwhere`` order.

Site-count variants
-------------------
``literal``   draws the stated number of components (8 strokes; U{1,2,3}
              shells) and takes whatever site count results.
``matched``   draws components one at a time from the same distribution
              until the per-sample site count reaches the stated target
              (for example ~100k sites on a 128^3 grid).
"""
from __future__ import annotations

import dataclasses
import numpy as np

__all__ = [
    "pen_strokes", "surfaces", "normal_f32", "to_bf16_bits", "bf16_bits_to_f32",
    "WORKLOADS", "Workload", "make_workload",
]


# ----------------------------------------------------------------------------
# Pen strokes (2-D)
# ----------------------------------------------------------------------------

def _raster_segment(p, q):
    """Integer points of the segment p->q, one per step of the major axis.

    x_t = p_x + floor((2 t dx + n) / (2 n)) for t = 0..n, n = max(|dx|, |dy|),
    i.e. round-half-up of the exact line; a zero-length segment is one point.
    """
    dx, dy = int(q[0] - p[0]), int(q[1] - p[1])
    n = max(abs(dx), abs(dy))
    if n == 0:
        return np.array([[p[0], p[1]]], dtype=np.int64)
    t = np.arange(n + 1, dtype=np.int64)
    x = p[0] + (2 * t * dx + n) // (2 * n)
    y = p[1] + (2 * t * dy + n) // (2 * n)
    return np.stack([x, y], axis=1)


def _one_stroke(rng, size):
    nseg = int(rng.integers(3, 7))                 # U{3..6} segments
    verts = rng.integers(0, size, size=(nseg + 1, 2))
    pts = [_raster_segment(verts[k], verts[k + 1]) for k in range(nseg)]
    return np.concatenate(pts, axis=0)


def pen_strokes(n_grids, size=64, n_strokes=8, seed=0, variant="matched",
                target=400):
    """Coordinates int32[N, 3] = (grid, x, y) of rasterised random polylines.

    Each stroke is a polyline of U{3..6} segments whose vertices are uniform on
    the grid, drawn 1 px wide.  ``literal`` draws ``n_strokes`` strokes per
    grid; ``matched`` draws strokes (at most ``n_strokes``) until the grid has
    at least ``target`` active pixels.
    """
    out = []
    for g in range(n_grids):
        rng = np.random.default_rng(np.random.SeedSequence([seed, g]))
        grid = np.zeros((size, size), dtype=bool)
        for _ in range(n_strokes):
            p = _one_stroke(rng, size)
            grid[p[:, 0], p[:, 1]] = True
            if variant == "matched" and grid.sum() >= target:
                break
        xy = np.argwhere(grid)
        out.append(np.concatenate(
            [np.full((len(xy), 1), g, dtype=np.int64), xy], axis=1))
    if not out:
        return np.zeros((0, 3), dtype=np.int32)
    return np.ascontiguousarray(np.concatenate(out, axis=0), dtype=np.int32)


# ----------------------------------------------------------------------------
# Voxelised surfaces (3-D)
# ----------------------------------------------------------------------------

def _random_rotation(rng):
    q, r = np.linalg.qr(rng.standard_normal((3, 3)))
    q = q * np.sign(np.diag(r))[None, :]
    return q


def _shell_mask(rng, size, r_lo, r_hi):
    """Boolean grid of one 1-voxel-thick shell: sphere, ellipsoid or plane.

    A voxel v is on the shell when |phi(v + 1/2)| <= 1/2, phi being the signed
    distance (sphere, plane) or the scaled radial distance
    (||R^T (p - c) / a|| - 1) * min(a) (ellipsoid).
    """
    kind = int(rng.integers(0, 3))
    grid = np.zeros((size,) * 3, dtype=bool)
    if kind in (0, 1):
        c = rng.uniform(0, size, size=3)
        if kind == 0:
            a = np.full(3, rng.uniform(r_lo, r_hi))
            rot = np.eye(3)
        else:
            a = rng.uniform(r_lo, r_hi, size=3)
            rot = _random_rotation(rng)
        ext = float(a.max()) + 2.0
        lo = np.clip(np.floor(c - ext).astype(int), 0, size)
        hi = np.clip(np.ceil(c + ext).astype(int) + 1, 0, size)
        if np.any(hi <= lo):
            return grid
        ax = [np.arange(lo[k], hi[k], dtype=np.float64) + 0.5 - c[k]
              for k in range(3)]
        px, py, pz = np.meshgrid(*ax, indexing="ij")
        # local coordinates u = R^T (p - c)
        u0 = rot[0, 0] * px + rot[1, 0] * py + rot[2, 0] * pz
        u1 = rot[0, 1] * px + rot[1, 1] * py + rot[2, 1] * pz
        u2 = rot[0, 2] * px + rot[1, 2] * py + rot[2, 2] * pz
        rad = np.sqrt((u0 / a[0]) ** 2 + (u1 / a[1]) ** 2 + (u2 / a[2]) ** 2)
        phi = (rad - 1.0) * a.min()
        grid[lo[0]:hi[0], lo[1]:hi[1], lo[2]:hi[2]] = np.abs(phi) <= 0.5
    else:
        nrm = rng.standard_normal(3)
        nrm /= np.linalg.norm(nrm)
        q = rng.uniform(0, size, size=3)
        off = float(nrm @ q)
        ax = np.arange(size, dtype=np.float64) + 0.5
        for x0 in range(0, size, 32):
            xs = ax[x0:x0 + 32]
            phi = (nrm[0] * xs[:, None, None] + nrm[1] * ax[None, :, None]
                   + nrm[2] * ax[None, None, :] - off)
            grid[x0:x0 + 32] = np.abs(phi) <= 0.5
    return grid


def surfaces(n_samples, size, r_lo, r_hi, seed=0, variant="matched",
             target=None, max_components=256):
    """Coordinates int32[N, 4] = (sample, x, y, z) of unions of thin shells.

    ``literal`` draws U{1,2,3} shells per sample; ``matched`` draws shells
    until the sample has at least ``target`` active voxels.
    """
    out = []
    for s in range(n_samples):
        rng = np.random.default_rng(np.random.SeedSequence([seed, s]))
        grid = np.zeros((size,) * 3, dtype=bool)
        if variant == "literal" or target is None:
            for _ in range(int(rng.integers(1, 4))):
                grid |= _shell_mask(rng, size, r_lo, r_hi)
        else:
            count = 0
            for _ in range(max_components):
                grid |= _shell_mask(rng, size, r_lo, r_hi)
                count = int(grid.sum())
                if count >= target:
                    break
        xyz = np.argwhere(grid)
        out.append(np.concatenate(
            [np.full((len(xyz), 1), s, dtype=np.int64), xyz], axis=1))
    if not out:
        return np.zeros((0, 4), dtype=np.int32)
    return np.ascontiguousarray(np.concatenate(out, axis=0), dtype=np.int32)


# ----------------------------------------------------------------------------
# Dense tensors
# ----------------------------------------------------------------------------

def normal_f32(shape, std=1.0, seed=0):
    """float32 samples of N(0, std^2), deterministic in ``seed``."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 7919]))
    return (rng.standard_normal(shape) * std).astype(np.float32)


def to_bf16_bits(a):
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.

    NaN inputs map to a quiet NaN.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b):
    """bfloat16 bit patterns (uint16) -> float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------
# Named workloads
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Layer:
    kind: str            # "vsc" or "sc"
    f: int
    s: int
    c_in: int
    c_out: int


@dataclasses.dataclass
class Workload:
    name: str
    d: int                       # spatial dimensions
    size: int                    # grid side
    batch: int
    layers: list
    dtype: str                   # "f32" or "bf16" for features and weights
    coords: np.ndarray = None    # int32[N, 1+d]

    @property
    def spatial_size(self):
        return [self.batch] + [self.size] * self.d


def _layer_list(spec):
    return [Layer(*t) for t in spec]


_SITE_SETS = {}


def _site_set(name, variant, seed):
    """Coordinates of a named workload, generated once per process (the
    256^3 surfaces take tens of seconds); callers get their own copy."""
    key = (name, variant, seed)
    if key not in _SITE_SETS:
        spec = WORKLOADS[name]
        if spec["family"] == "pen":
            coords = pen_strokes(spec["batch"], spec["size"], seed=seed,
                                 variant=variant, target=spec["target"])
        else:
            coords = surfaces(spec["batch"], spec["size"], spec["r_lo"],
                              spec["r_hi"], seed=seed, variant=variant,
                              target=spec["target"])
        _SITE_SETS[key] = coords
    return _SITE_SETS[key].copy()


def make_workload(name, variant="matched", seed=None):
    """Build one named workload (site set plus layer list)."""
    spec = WORKLOADS[name]
    seed = spec["seed"] if seed is None else seed
    coords = _site_set(name, variant, seed)
    return Workload(name=name, d=spec["d"], size=spec["size"],
                    batch=spec["batch"], layers=_layer_list(spec["layers"]),
                    dtype=spec["dtype"], coords=coords)


# The five workloads.  Channel widths, kernel sizes, strides and dtypes are
# those of the benchmark configurations; site counts follow the targets above.
WORKLOADS = {
    # one 64x64 grid of pen strokes, VSC 3x3, 1 -> 16 features, fp32
    "pen64_vsc3_c1x16": dict(
        family="pen", d=2, size=64, batch=1, target=400, seed=0,
        dtype="f32", layers=[("vsc", 3, 1, 1, 16)]),
    # 64 grids, three VSC 3x3 (1->32->32->32) then SC 2x2 stride 2, fp32
    "pen64x64_vsc3x3_sc2": dict(
        family="pen", d=2, size=64, batch=64, target=400, seed=1,
        dtype="f32", layers=[("vsc", 3, 1, 1, 32), ("vsc", 3, 1, 32, 32),
                             ("vsc", 3, 1, 32, 32), ("sc", 2, 2, 32, 32)]),
    # 16 surfaces at 64^3, VSC 3^3, 32 -> 32, fp32
    "surf64x16_vsc3_c32": dict(
        family="surf", d=3, size=64, batch=16, r_lo=8.0, r_hi=28.0,
        target=20000, seed=2, dtype="f32", layers=[("vsc", 3, 1, 32, 32)]),
    # 8 surfaces at 128^3, VSC 3^3, 64 -> 64, bf16 in, fp32 accumulate
    "surf128x8_vsc3_c64_bf16": dict(
        family="surf", d=3, size=128, batch=8, r_lo=16.0, r_hi=60.0,
        target=100000, seed=3, dtype="bf16", layers=[("vsc", 3, 1, 64, 64)]),
    # 4 surfaces at 256^3, four-level encoder: per level two VSC 3^3 at
    # C = 32/64/96/128, levels joined by SC 2^3 stride 2, bf16
    "surf256x4_unet_enc_bf16": dict(
        family="surf", d=3, size=256, batch=4, r_lo=32.0, r_hi=120.0,
        target=400000, seed=4, dtype="bf16",
        layers=[("vsc", 3, 1, 32, 32), ("vsc", 3, 1, 32, 32),
                ("sc", 2, 2, 32, 64),
                ("vsc", 3, 1, 64, 64), ("vsc", 3, 1, 64, 64),
                ("sc", 2, 2, 64, 96),
                ("vsc", 3, 1, 96, 96), ("vsc", 3, 1, 96, 96),
                ("sc", 2, 2, 96, 128),
                ("vsc", 3, 1, 128, 128), ("vsc", 3, 1, 128, 128)]),
}
