"""The near-tie rule of tests/parity.py on constructed inputs (CPU): a pair
of scores that rounding swaps across a rank-bin edge is excused, a token
moved away from any edge is not."""

import numpy as np

from parity import near_tie_bin_moves


def test_rounding_swap_at_a_bin_edge_is_excused():
    r = np.random.default_rng(0)
    v = r.random(1000)
    order = np.argsort(v)
    e = v[order[125]]                     # first score of bin 1 at K = 8
    v[order[124]] = e * (1 - 1e-7)        # an oracle near tie at the edge
    w = v.copy()
    w[order[124]] = e * (1 + 1e-7)        # rounding swaps the pair
    assert near_tie_bin_moves(v, w, 8) == 2
    assert near_tie_bin_moves(v, v.astype(np.float32), 8) == 0


def test_moves_off_an_edge_are_not_excused():
    r = np.random.default_rng(1)
    v = r.random(1000)
    order = np.argsort(v)
    w = v.copy()
    w[order[10]] = v[order[900]]          # a low score jumps seven bins
    assert near_tie_bin_moves(v, w, 8) is None
    w = v.copy()
    w[order[100]] = v[order[130]] * 1.0001    # one bin up, but not a near tie
    assert near_tie_bin_moves(v, w, 8) is None
