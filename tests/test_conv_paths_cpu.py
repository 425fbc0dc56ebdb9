"""Random canonical split strings (the inputs of the convolution path
tests): canonical form, and that they put split neighbours in every
direction of both edge-8 and edge-4 cells."""
import itertools

import numpy as np

import octref as O
from paper_1611_05009_amd import synth


def split_neighbour_directions(words, n, gd, gh, gw):
    """Directions (of 26) in which some edge-8 cell has a split neighbour
    tree, and in which some edge-4 cell has a split neighbouring depth-1
    node, counted from the bits alone."""
    w0 = words[:, 0].reshape(n, gd, gh, gw).astype(np.int64)
    root = (w0 & 1).astype(bool)
    d8, d4 = set(), set()
    for s, td, th, tw in itertools.product(range(n), range(gd), range(gh), range(gw)):
        cells = []
        if not root[s, td, th, tw]:
            cells.append((8, 8 * td, 8 * th, 8 * tw))
        else:
            for o1 in range(8):
                if not (w0[s, td, th, tw] >> (1 + o1)) & 1:
                    cells.append((4, 8 * td + 4 * (o1 >> 2 & 1), 8 * th + 4 * (o1 >> 1 & 1), 8 * tw + 4 * (o1 & 1)))
        for sz, od, oh, ow in cells:
            for dv in itertools.product((-1, 0, 1), repeat=3):
                if dv == (0, 0, 0):
                    continue
                vd, vh, vw = od + sz * dv[0], oh + sz * dv[1], ow + sz * dv[2]
                if not (0 <= vd < 8 * gd and 0 <= vh < 8 * gh and 0 <= vw < 8 * gw):
                    continue
                q = w0[s, vd // 8, vh // 8, vw // 8]
                if not q & 1:
                    continue
                if sz == 8:
                    d8.add(dv)
                else:
                    o1 = 4 * (vd % 8 >> 2) + 2 * (vh % 8 >> 2) + (vw % 8 >> 2)
                    if (q >> (1 + o1)) & 1:
                        d4.add(dv)
    return d8, d4


CASES = [
    # (seed, n, gd, gh, gw, p_root, p_d1, p_d2)
    (11, 2, 4, 4, 4, 0.5, 0.5, 0.5),
    (12, 1, 5, 3, 4, 0.35, 0.6, 0.3),
    (13, 2, 3, 4, 3, 0.7, 0.4, 0.7),
]



def test_random_split_strings_are_canonical():
    for seed, n, gd, gh, gw, p0, p1, p2 in CASES:
        words = synth.random_trees(np.random.default_rng(seed), n, gd, gh, gw, p0, p1, p2)
        assert all(O.tree_valid(t) for t in words)


def test_random_split_strings_cover_every_direction():
    """The first case puts split neighbours in all 26 directions of both
    edge-8 and edge-4 cells."""
    seed, n, gd, gh, gw, p0, p1, p2 = CASES[0]
    words = synth.random_trees(np.random.default_rng(seed), n, gd, gh, gw, p0, p1, p2)
    d8, d4 = split_neighbour_directions(words, n, gd, gh, gw)
    assert len(d8) == 26 and len(d4) == 26, (len(d8), len(d4))
