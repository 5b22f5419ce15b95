"""Comparison of a GPU rule book with the oracle's.

The oracle lists the pairs of every R_i by ascending output row (Section 4
leaves the order inside R_i open; each output row has at most one input per
offset, so the output row orders R_i totally).  The library promises a
different order, the Z-order (Morton) curve of the output site, which its
forward walks.  So the comparison is in two parts:
  * the GPU's R_i, sorted by output row, equals the oracle's R_i, pair for
    pair (and the pair offsets match exactly);
  * the GPU's R_i is in Z-order of the output site, checked against
    ``dense_ref.zorder`` (pinned separately against the textbook curve).
"""
import numpy as np

from tests import dense_ref


def offset_index(pair_off):
    """Offset i of every pair, from the prefix sums pair_off [K+1]."""
    pair_off = np.asarray(pair_off, np.int64)
    return np.repeat(np.arange(len(pair_off) - 1), np.diff(pair_off))


def canonical_pairs(pairs, pair_off):
    """Pairs with every R_i sorted by ascending output row."""
    pairs = np.asarray(pairs)
    idx = offset_index(pair_off)
    order = np.lexsort((pairs[:, 1], idx))
    return pairs[order]


def assert_zorder_within_offsets(pairs, pair_off, out_coords):
    """Inside every R_i the output sites strictly follow the Z-order curve."""
    pairs = np.asarray(pairs)
    if len(pairs) < 2:
        return
    rank = np.empty(len(out_coords), np.int64)
    rank[dense_ref.zorder(out_coords)] = np.arange(len(out_coords))
    r = rank[pairs[:, 1]]
    idx = offset_index(pair_off)
    same = idx[1:] == idx[:-1]
    bad = same & (np.diff(r) <= 0)
    assert not bad.any(), f"{int(bad.sum())} pairs out of Z-order (first at {int(np.argmax(bad))})"


def check_rulebook(out_coords, pairs, pair_off, ref):
    """GPU (out_coords, pairs, pair_off) against an oracle.Rulebook."""
    np.testing.assert_array_equal(out_coords, ref.out_coords)
    np.testing.assert_array_equal(np.asarray(pair_off), ref.pair_off)
    assert len(pairs) == len(ref.pairs)
    np.testing.assert_array_equal(canonical_pairs(pairs, pair_off), ref.pairs)
    assert_zorder_within_offsets(pairs, pair_off, out_coords)
