"""Brute-force dense statements of SC and VSC for tiny grids (test pins).

These never touch the oracle's map or rule book.  They build a zero-filled
dense grid (inactive sites are exactly zero, Section 3: the ground state is
discarded) and evaluate the convolution at every grid site with array
slicing, then read off the active outputs:

* VSC: pad by (f-1)/2 on each side, output active iff the centre input is
  active (Section 3, VSC definition);
* SC: no padding, stride s, output active iff some input in the f^d field is
  active; extent floor((l - f)/s) + 1 (Section 3, SC definition).
"""
from __future__ import annotations

import itertools

import numpy as np


def offsets(f):
    """All filter offsets in flattened order (last dimension fastest)."""
    return list(itertools.product(*[range(k) for k in f]))


def dense_grid(coords, size, feats):
    """Zero-filled dense array [size..., C] holding feats at coords."""
    C = feats.shape[1]
    g = np.zeros(tuple(size) + (C,), np.float64)
    g[tuple(coords.T)] = feats
    return g


def occupancy(coords, size):
    g = np.zeros(tuple(size), bool)
    g[tuple(coords.T)] = True
    return g


def row_grid(coords, size):
    g = np.full(tuple(size), -1, np.int64)
    g[tuple(coords.T)] = np.arange(len(coords))
    return g


def vsc_dense(coords, size, f, x, w, bias=None):
    """VSC output rows (same order as coords), float64."""
    size = list(size)
    D = len(size)
    pad = [(k - 1) // 2 for k in f]
    X = dense_grid(coords, size, x.astype(np.float64))
    Xp = np.pad(X, [(p, p) for p in pad] + [(0, 0)])
    C_out = w.shape[2]
    out = np.zeros(tuple(size) + (C_out,), np.float64)
    for i, o in enumerate(offsets(f)):
        sl = tuple(slice(o[j], o[j] + size[j]) for j in range(D))
        out += Xp[sl] @ w[i].astype(np.float64)
    if bias is not None:
        out += bias.astype(np.float64)
    return out[tuple(coords.T)]


def sc_extent(size, f, s):
    return [(l - k) // t + 1 if l >= k else 0 for l, k, t in zip(size, f, s)]


def sc_dense(coords, size, f, s, x, w, bias=None):
    """SC output: (active output coords in lexicographic order, features)."""
    size = list(size)
    D = len(size)
    E = sc_extent(size, f, s)
    X = dense_grid(coords, size, x.astype(np.float64))
    occ = occupancy(coords, size)
    C_out = w.shape[2]
    out = np.zeros(tuple(E) + (C_out,), np.float64)
    act = np.zeros(tuple(E), bool)
    if min(E) > 0:
        for i, o in enumerate(offsets(f)):
            sl = tuple(slice(o[j], o[j] + s[j] * (E[j] - 1) + 1, s[j])
                       for j in range(D))
            out += X[sl] @ w[i].astype(np.float64)
            act |= occ[sl]
    if bias is not None:
        out += bias.astype(np.float64)
    oc = np.argwhere(act)
    return oc.astype(np.int32), out[tuple(oc.T)]


def zorder(sites):
    """Permutation visiting sites along the Z-order curve: sample first, then
    bit planes from bit 15 down, dimension 1 first inside a plane (a plain
    lexicographic sort of the bit columns)."""
    sites = np.asarray(sites, np.int64)
    cols = [sites[:, 0]]
    for L in range(15, -1, -1):
        for j in range(1, sites.shape[1]):
            cols.append((sites[:, j] >> L) & 1)
    return np.lexsort(cols[::-1])


def rulebook_dense(kind, coords, size, f, s, out_coords):
    """Per-offset (input row, output row) lists from a dense row grid, each
    list ordered by ascending output row."""
    size = list(size)
    D = len(size)
    rg = row_grid(coords, size)
    R = []
    for o in offsets(f):
        if kind == "vsc":
            x = out_coords + np.array([o[j] - (f[j] - 1) // 2 for j in range(D)])
        else:
            x = out_coords * np.array(s) + np.array(o)
        inb = np.all((x >= 0) & (x < np.array(size)), axis=1)
        rows = np.full(len(out_coords), -1, np.int64)
        rows[inb] = rg[tuple(x[inb].T)]
        y = np.nonzero(rows >= 0)[0]
        R.append(np.stack([rows[y], y], axis=1).astype(np.int32))
    return R


def random_sites(rng, size, density, batch=None):
    """Random distinct active sites of a grid, lexicographic order."""
    occ = rng.random(tuple(size)) < density
    return np.argwhere(occ).astype(np.int32)
